// Burst-Gap model of the post-issue stage (Sec. 3.3-3.5), host side.
//   per burst n:  P_n = T0_n + G_n, rho_n = V_n / (R P_n)              (Eq. 3)
//                 delta_b_n = V_n - R P_n                               (Eq. 4)
//                 b_iso_n = [V_n - R T0_n]_+, guard q_n + b_iso_n <= Q  (Eq. 6)
//   issue time:   T0_n while the guard holds, else (q_n + V_n - Q) / R: a fluid queue capped
//                 at Q and drained at R stretches issue until enough volume has drained
//   backlog:      q_{n+1} = [q_n + V_n - R (T_iss_n + G_n)]_+, which is the recurrence of
//                 Eq. 5 whenever the guard holds.
//   MMA side:     dt_n = [T_iss_n - T_cover_n]_+ (App. A.2, the remote-store span taken as
//                 the predicted issue time).
// Pacing audit (Sec. 4.1, 4.2; App. A.1): the burst sequence of a tile order of the
// persistent EP kernel, rebuilt from the schedule, run through the same recurrence.
// Calibration: T0(V) least squares, R = sum V^2 / sum V T over zero-gap periods (T = V / R),
// Q = median of V - R T_iss over isolated bursts past the knee.
#include <algorithm>
#include <cmath>
#include <limits>
#include <vector>

#include "xstage.h"

extern "C" int xs_model_predict(const xs_model* m, const xs_burst* bursts, int32_t n, double q0,
                                xs_burst_pred* out) {
  if (!m || n < 0 || (n > 0 && (!bursts || !out)) || !(m->R_bytes_per_us > 0) || q0 < 0)
    return XS_EINVAL;
  const double R = m->R_bytes_per_us, Q = m->Q_bytes;
  double q = q0;
  for (int32_t i = 0; i < n; ++i) {
    const double V = bursts[i].V_bytes, T0 = bursts[i].T0_us, G = bursts[i].G_us;
    const double cover = bursts[i].cover_us;
    const double P = T0 + G;
    const double biso = std::max(0.0, V - R * T0);
    const bool ok = q + biso <= Q;
    const double tiss = ok ? T0 : std::max(T0, (q + V - Q) / R);
    xs_burst_pred& o = out[i];
    o.rho = P > 0 ? V / (R * P) : std::numeric_limits<double>::infinity();
    o.delta_b = V - R * P;
    o.q_before = q;
    o.b_iso = biso;
    o.T_iss_us = tiss;
    o.stall_us = tiss - T0;
    o.mma_stall_us = std::max(0.0, tiss - cover);   // App. A.2 with T_RS = T_iss
    o.guard_ok = ok ? 1 : 0;
    o._pad = 0;
    q = std::max(0.0, q + V - R * (tiss + G));
  }
  return XS_OK;
}

extern "C" int xs_model_fit(const xs_calib* c, xs_model* out) {
  if (!c || !out || c->n_rec < 1 || c->n_zg < 1 || c->n_iso < 0 || !c->rec_V || !c->rec_T ||
      !c->zg_V || !c->zg_T || (c->n_iso > 0 && (!c->iso_V || !c->iso_T)))
    return XS_EINVAL;
  // T0(V) = a + b V, ordinary least squares (a constant if all V are equal)
  double mv = 0, mt = 0;
  for (int i = 0; i < c->n_rec; ++i) {
    mv += c->rec_V[i];
    mt += c->rec_T[i];
  }
  mv /= c->n_rec;
  mt /= c->n_rec;
  double sxx = 0, sxy = 0;
  for (int i = 0; i < c->n_rec; ++i) {
    sxx += (c->rec_V[i] - mv) * (c->rec_V[i] - mv);
    sxy += (c->rec_V[i] - mv) * (c->rec_T[i] - mt);
  }
  const double b = sxx > 0 ? sxy / sxx : 0.0;
  const double a = mt - b * mv;
  double svv = 0, svt = 0;
  for (int i = 0; i < c->n_zg; ++i) {
    svv += c->zg_V[i] * c->zg_V[i];
    svt += c->zg_V[i] * c->zg_T[i];
  }
  if (!(svt > 0)) return XS_EINVAL;
  const double R = svv / svt;
  std::vector<double> qs;
  for (int i = 0; i < c->n_iso; ++i) {
    const double V = c->iso_V[i], T = c->iso_T[i];
    if (T > (a + b * V) * (1.0 + c->knee_excess)) qs.push_back(V - R * T);
  }
  double Q = std::numeric_limits<double>::infinity();
  if (!qs.empty()) {
    std::sort(qs.begin(), qs.end());
    const size_t n = qs.size();
    Q = n % 2 ? qs[n / 2] : 0.5 * (qs[n / 2 - 1] + qs[n / 2]);
  }
  out->t0_a_us = a;
  out->t0_b_us_per_byte = b;
  out->R_bytes_per_us = R;
  out->Q_bytes = Q;
  out->K = c->K;
  out->_pad = 0;
  return XS_OK;
}

// ------------------------------------------------------------------------------ pacing audit
namespace xs_host {
int persistent_grid(int max_producers);
double wall_rate_hz();
}

namespace {

constexpr int kTile = 256;          // rows / columns of an EP GEMM tile
constexpr int kL1Cols = 128;        // h columns per Linear-1 tile (gate + up = 256 wide)

struct Order {                       // producer 0's tiles: kind 1 / 2 and row
  std::vector<int> kind, row;
};

// Scheduler rows (expert row blocks) in expert-major order and the rows of each block, as
// the plan kernel forms them: m rows -> ceil(m / 256) blocks; bf16 blocks are equal (the
// rows divided evenly, rounded up to 32, at most 256), MX blocks 256 with a ragged tail.
void row_blocks(const std::vector<int>& m, bool equal, std::vector<int>& block_rows,
                std::vector<int>& block_expert) {
  for (size_t x = 0; x < m.size(); ++x) {
    const int mt = (m[x] + kTile - 1) / kTile;
    const int bm = equal ? std::min(kTile, ((m[x] + mt - 1) / std::max(mt, 1) + 31) & ~31) : kTile;
    for (int b = 0; b < mt; ++b) {
      block_rows.push_back(std::min(bm, m[x] - b * bm));
      block_expert.push_back(static_cast<int>(x));
    }
  }
}

// The interleave rule on producer 0's own entries (0, G, 2G, ... of each stream): a Linear-2
// entry runs when the next own Linear-1 entry is D rows past it (or none is left) and the
// chunk cap allows.
Order own_interleave(int P, int P1, int P2, int G, int D, int chunk) {
  Order o;
  const long n1 = static_cast<long>(P) * P1, n2 = static_cast<long>(P) * P2;
  long e1 = 0, e2 = 0;
  int run = 0;
  for (;;) {
    const bool l1_left = e1 < n1;
    const bool may2 = e2 < n2 && !(chunk > 0 && run >= chunk && l1_left) &&
                      (!l1_left || e2 / P2 + D <= e1 / P1);
    if (may2) {
      o.kind.push_back(2);
      o.row.push_back(static_cast<int>(e2 / P2));
      e2 += G;
      ++run;
    } else if (l1_left) {
      o.kind.push_back(1);
      o.row.push_back(static_cast<int>(e1 / P1));
      e1 += G;
      run = 0;
    } else {
      break;
    }
  }
  return o;
}

// Expert-Wave: the wave list [L1 of wave 0, L2 of wave 0, ...], producer 0's entries 0, G, ...
Order own_wave(const std::vector<int>& block_expert, int P1, int P2, int G, int wave_tiles) {
  std::vector<int> bounds{0};
  int wl1 = 0;
  const int P = static_cast<int>(block_expert.size());
  for (int p = 0; p < P; ++p) {
    wl1 += P1;
    const bool last_of_expert = p + 1 == P || block_expert[p + 1] != block_expert[p];
    if (last_of_expert && wl1 >= wave_tiles) {
      bounds.push_back(p + 1);
      wl1 = 0;
    }
  }
  if (bounds.back() != P) bounds.push_back(P);
  Order o;
  long pos = 0;
  for (size_t w = 0; w + 1 < bounds.size(); ++w) {
    const int r0 = bounds[w], r1 = bounds[w + 1];
    const long n1 = static_cast<long>(r1 - r0) * P1, n2 = static_cast<long>(r1 - r0) * P2;
    for (long i = 0; i < n1 + n2; ++i, ++pos) {
      if (pos % G) continue;
      if (i < n1) {
        o.kind.push_back(1);
        o.row.push_back(static_cast<int>(r0 + i / P1));
      } else {
        o.kind.push_back(2);
        o.row.push_back(static_cast<int>(r0 + (i - n1) / P2));
      }
    }
  }
  return o;
}

struct Eval {
  int bursts = 0, guard_fail = 0;
  double stall = 0, mma = 0, compute = 0;
};

// Aligned burst volumes: the n-th burst is every producer's n-th Linear-2 tile issued together
// (full alignment, Sec. 4.2), V_n = the sum of those tiles' stored bytes; a producer with fewer
// Linear-2 tiles does not take part in the later bursts (K_act < G).
std::vector<double> aligned_volumes(bool wave, const std::vector<int>& block_rows,
                                    const std::vector<int>& block_expert, int P1, int P2, int G,
                                    int wave_tiles, double share) {
  const int P = static_cast<int>(block_rows.size());
  std::vector<double> V;
  auto add = [&](size_t n, int row) {
    if (V.size() <= n) V.resize(n + 1, 0.0);
    V[n] += static_cast<double>(block_rows[row]) * kTile * 2.0 * share;
  };
  if (!wave) {
    // producer g's Linear-2 tiles are its own entries g, g + G, ... in order
    const long n2 = static_cast<long>(P) * P2;
    for (long e = 0; e < n2; ++e) add(static_cast<size_t>(e / G), static_cast<int>(e / P2));
    return V;
  }
  std::vector<int> bounds{0};
  int wl1 = 0;
  for (int p = 0; p < P; ++p) {
    wl1 += P1;
    const bool last_of_expert = p + 1 == P || block_expert[p + 1] != block_expert[p];
    if (last_of_expert && wl1 >= wave_tiles) {
      bounds.push_back(p + 1);
      wl1 = 0;
    }
  }
  if (bounds.back() != P) bounds.push_back(P);
  std::vector<int> count(G, 0);   // Linear-2 tiles each producer has taken so far
  long pos = 0;
  for (size_t w = 0; w + 1 < bounds.size(); ++w) {
    const int r0 = bounds[w], r1 = bounds[w + 1];
    const long n1 = static_cast<long>(r1 - r0) * P1, n2 = static_cast<long>(r1 - r0) * P2;
    for (long i = 0; i < n1 + n2; ++i, ++pos) {
      if (i < n1) continue;
      const int g = static_cast<int>(pos % G);
      add(static_cast<size_t>(count[g]++), static_cast<int>(r0 + (i - n1) / P2));
    }
  }
  return V;
}

Eval evaluate(const Order& o, const std::vector<double>& Vn, const xs_model& m, double tl1, double tl2) {
  Eval ev;
  std::vector<xs_burst> b;
  const size_t n = o.kind.size();
  for (size_t i = 0; i < n; ++i) ev.compute += o.kind[i] == 1 ? tl1 : tl2;
  for (size_t i = 0; i < n; ++i) {
    if (o.kind[i] != 2) continue;
    const double V = b.size() < Vn.size() ? Vn[b.size()] : 0.0;
    const double T0 = m.t0_a_us + m.t0_b_us_per_byte * V;
    double gap = 0;
    for (size_t j = i + 1; j < n; ++j) {
      gap += o.kind[j] == 1 ? tl1 : tl2;
      if (o.kind[j] == 2) break;
    }
    b.push_back(xs_burst{V, T0, gap, T0});
  }
  if (b.empty()) return ev;
  std::vector<xs_burst_pred> pr(b.size());
  if (xs_model_predict(&m, b.data(), static_cast<int32_t>(b.size()), 0.0, pr.data()) != XS_OK) return ev;
  ev.bursts = static_cast<int>(b.size());
  for (const auto& p : pr) {
    ev.stall += p.stall_us;
    ev.mma += p.mma_stall_us;
    ev.guard_fail += p.guard_ok ? 0 : 1;
  }
  return ev;
}

}  // namespace

extern "C" int xs_pacing_audit_run(const xs_ep_layer* L, const xs_pacing* pc, xs_pacing_audit* out) {
  if (!L || !pc || !out || !pc->model || L->W < 1 || L->E % L->W || L->n_experts < 1 ||
      L->n_experts > 1024 || L->H % kTile || L->I % kL1Cols || L->n_src < 1 || L->T < 0 || L->k < 1 ||
      pc->lead_rows < 0 || pc->chunk_tiles < 0 || pc->max_producers < 0 || pc->wave_tiles < 0 ||
      !(pc->sink_share >= 0 && pc->sink_share <= 1) || !(pc->model->R_bytes_per_us > 0) ||
      pc->policy < XS_POLICY_BURST || pc->policy > XS_POLICY_AUTO)
    return XS_EINVAL;
  const xs_model& m = *pc->model;
  const int G = xs_host::persistent_grid(pc->max_producers);
  const int P1 = L->I / kL1Cols, P2 = L->H / kTile;
  std::vector<int> rows(L->n_experts);
  for (int x = 0; x < L->n_experts; ++x) {
    if (pc->expert_rows) {
      if (pc->expert_rows[x] < 0) return XS_EINVAL;
      rows[x] = pc->expert_rows[x];
    } else {
      rows[x] = static_cast<int>(static_cast<int64_t>(L->n_src) * L->T * L->k / L->E);
    }
  }
  std::vector<int> block_rows, block_expert;
  row_blocks(rows, L->precision == XS_PREC_BF16, block_rows, block_expert);
  const int P = static_cast<int>(block_rows.size());
  // mainloop times: given, else the tile FLOPs at 40 % of one CU's share of the dense peak
  const double peak = L->precision == XS_PREC_BF16 ? 2.5e15 : 5.0e15;
  const double cu_flops_us = peak / 256.0 * 0.4 * 1e-6;
  const double tl1 = pc->t_l1_us > 0 ? pc->t_l1_us : 2.0 * kTile * kTile * L->H / cu_flops_us;
  const double tl2 = pc->t_l2_us > 0 ? pc->t_l2_us : 2.0 * kTile * kTile * L->I / cu_flops_us;
  const double share = pc->sink_share > 0 ? pc->sink_share : 1.0;
  const int D = pc->lead_rows > 0 ? pc->lead_rows : (G + P1 - 1) / P1;
  const int wave_tiles = pc->wave_tiles > 0 ? pc->wave_tiles : G;
  *out = xs_pacing_audit{};
  out->producers = G;
  out->rows = P;
  out->lead_rows = D;
  out->t_l1_us = tl1;
  out->t_l2_us = tl2;
  out->V_full_bytes = static_cast<double>(G) * kTile * kTile * 2.0 * share;
  {  // Eq. 9 at the share's mix: per producer n1 = P P1 / G Linear-1 and n2 = P P2 / G Linear-2
    const double n1 = static_cast<double>(P) * P1 / G, n2 = static_cast<double>(P) * P2 / G;
    const double V = out->V_full_bytes, T0 = m.t0_a_us + m.t0_b_us_per_byte * V;
    const double den = n2 * (T0 + tl2) + n1 * tl1;
    out->rate_feasible = den > 0 && n2 * V / den <= m.R_bytes_per_us ? 1 : 0;
  }
  std::vector<std::pair<int, int>> cands;    // (policy, chunk)
  if (pc->policy == XS_POLICY_AUTO) {
    cands.push_back({XS_POLICY_BURST, 0});
    cands.push_back({XS_POLICY_INTERLEAVE, 0});
    for (int c = 1; c <= 32; c *= 2) cands.push_back({XS_POLICY_CHUNK, c});
  } else {
    cands.push_back({pc->policy, pc->policy == XS_POLICY_CHUNK ? pc->chunk_tiles : 0});
  }
  out->n_cand = static_cast<int>(cands.size());
  for (size_t i = 0; i < cands.size(); ++i) {
    const bool wave = cands[i].first == XS_POLICY_BURST;
    const Order o = wave ? own_wave(block_expert, P1, P2, G, wave_tiles)
                         : own_interleave(P, P1, P2, G, D, cands[i].second);
    const Eval ev = evaluate(o, aligned_volumes(wave, block_rows, block_expert, P1, P2, G, wave_tiles, share),
                             m, tl1, tl2);
    out->cand_policy[i] = cands[i].first;
    out->cand_chunk[i] = cands[i].second;
    out->cand_bursts[i] = ev.bursts;
    out->cand_guard_fail[i] = ev.guard_fail;
    out->cand_stall_us[i] = ev.stall;
    out->cand_mma_stall_us[i] = ev.mma;
    out->cand_compute_us[i] = ev.compute;
  }
  int pick = 0;
  if (pc->policy == XS_POLICY_AUTO) {
    // the least predicted stall; among the candidates within 1 % of BURST's mainloop time of
    // it, the plain interleave first, then the largest chunk, then BURST (Expert-Wave's
    // Linear-2 tiles wait for their whole wave's Linear-1 tiles, a cost outside the audit
    // that made it the slower order on HBM windows in every layer measured)
    double best = out->cand_stall_us[0];
    for (int i = 1; i < out->n_cand; ++i) best = std::min(best, out->cand_stall_us[i]);
    const double tol = 0.01 * out->cand_compute_us[0];
    pick = -1;
    if (out->cand_stall_us[1] <= best + tol) pick = 1;
    for (int i = out->n_cand - 1; i >= 2 && pick < 0; --i)
      if (out->cand_stall_us[i] <= best + tol) pick = i;
    if (pick < 0) pick = 0;
  }
  out->policy = out->cand_policy[pick];
  out->chunk = out->cand_chunk[pick];
  return XS_OK;
}

extern "C" int xs_trace_tile_times(const uint64_t* recs, const uint64_t* ext, int64_t n, int32_t min_rows,
                                   double* t_l1_us, double* t_l2_us, double* l2_issue_us) {
  if (!recs || n < 0 || !t_l1_us || !t_l2_us || !l2_issue_us) return XS_EINVAL;
  const double hz = xs_host::wall_rate_hz();
  const double us = 1e6 / (hz > 0 ? hz : 1e8);
  std::vector<double> a, b, c;
  for (int64_t i = 0; i < n; ++i) {
    const uint64_t* r = recs + 4 * i;
    const int kind = static_cast<int>(r[0] >> 56);
    if (ext && static_cast<int64_t>(ext[4 * i + 3]) < min_rows) continue;
    if (kind == 1) {
      a.push_back(static_cast<double>(r[2] - r[1]) * us);
    } else if (kind == 2) {
      const uint64_t start = ext ? ext[4 * i] : r[1];
      b.push_back(static_cast<double>(r[2] - start) * us);
      c.push_back(static_cast<double>(r[3] - r[2]) * us);
    }
  }
  auto median = [](std::vector<double>& v) {
    if (v.empty()) return 0.0;
    std::sort(v.begin(), v.end());
    const size_t k = v.size();
    return k % 2 ? v[k / 2] : 0.5 * (v[k / 2 - 1] + v[k / 2]);
  };
  *t_l1_us = median(a);
  *t_l2_us = median(b);
  *l2_issue_us = median(c);
  return XS_OK;
}

// ------------------------------------------------------------------------------ calibration
extern "C" int xs_drain_rate(const double* zg_V, const double* zg_T, int32_t n, double* R) {
  if (!zg_V || !zg_T || n < 1 || !R) return XS_EINVAL;
  double svv = 0, svt = 0;
  for (int i = 0; i < n; ++i) {
    svv += zg_V[i] * zg_V[i];
    svt += zg_V[i] * zg_T[i];
  }
  if (!(svt > 0)) return XS_EINVAL;
  *R = svv / svt;
  return XS_OK;
}

extern "C" int xs_calib_knee(const double* iso_V, const double* iso_T, int32_t n, double excess,
                             int32_t* knee) {
  if (n < 0 || !knee || (n > 0 && (!iso_V || !iso_T)) || excess < 0) return XS_EINVAL;
  *knee = n;
  for (int i = 2; i < n; ++i) {
    const double v0 = iso_V[0], t0 = iso_T[0], v1 = iso_V[i - 1], t1 = iso_T[i - 1];
    const double slope = v1 > v0 ? (t1 - t0) / (v1 - v0) : 0.0;
    const double line = t0 + slope * (iso_V[i] - v0);
    if (iso_T[i] > (1.0 + excess) * line) {
      *knee = i;
      break;
    }
  }
  return XS_OK;
}

extern "C" int xs_model_calibrate(const xs_calib* c, xs_calib_summary* out) {
  if (!c || !out) return XS_EINVAL;
  xs_model m;
  int rc = xs_model_fit(c, &m);
  if (rc) return rc;
  int32_t knee = c->n_iso;
  rc = xs_calib_knee(c->iso_V, c->iso_T, c->n_iso, c->knee_excess, &knee);
  if (rc) return rc;
  out->model = m;
  out->knee = knee;
  out->_pad = 0;
  const double inf = std::numeric_limits<double>::infinity();
  out->Q_bracket_lo = out->Q_bracket_hi = inf;
  if (knee > 0 && knee < c->n_iso) {
    auto q_at = [&](double V) { return V - m.R_bytes_per_us * (m.t0_a_us + m.t0_b_us_per_byte * V); };
    out->Q_bracket_lo = q_at(c->iso_V[knee - 1]);
    out->Q_bracket_hi = q_at(c->iso_V[knee]);
  }
  return XS_OK;
}

extern "C" int xs_burst_gap(const xs_model* m, double V, double G, double* T_period, double* T_iss) {
  if (!m || !T_period || !T_iss || !(m->R_bytes_per_us > 0) || V < 0 || G < 0) return XS_EINVAL;
  const double T0 = m->t0_a_us + m->t0_b_us_per_byte * V, drain = V / m->R_bytes_per_us;
  *T_period = std::max(T0 + G, drain);
  *T_iss = std::max(T0, drain - G);
  return XS_OK;
}

extern "C" int xs_recovery_audit(const xs_model* m, double V, int32_t n_bursts, double G, double sigma,
                                 int32_t b_n, xs_recovery* out) {
  if (!m || !out || n_bursts < 1 || V < 0 || G < 0 || b_n < 1 || !(m->R_bytes_per_us > 0)) return XS_EINVAL;
  const double R = m->R_bytes_per_us, T0 = m->t0_a_us + m->t0_b_us_per_byte * V;
  std::vector<xs_burst> b(n_bursts, xs_burst{V, T0, G, T0});
  std::vector<xs_burst_pred> pr(n_bursts);
  int rc = xs_model_predict(m, b.data(), n_bursts, 0.0, pr.data());
  if (rc) return rc;
  out->T0_us = T0;
  out->G_star_us = std::max(0.0, V / R - T0);
  out->rho = pr[0].rho;
  out->delta_b = pr[0].delta_b;
  out->b_iso = pr[0].b_iso;
  out->stall_us = 0;
  out->guard_ok = 1;
  for (const auto& p : pr) {
    out->stall_us += p.stall_us;
    if (!p.guard_ok) out->guard_ok = 0;
  }
  out->tail_us = std::max(0.0, (pr[n_bursts - 1].q_before + V) / R - T0);
  out->coupled_us = n_bursts * std::max(T0, V / R);
  out->M_ub_star = sigma > 0 ? static_cast<int32_t>(b_n * std::ceil(out->G_star_us / sigma)) : 0;
  return XS_OK;
}
