// Burst-Gap model of the post-issue stage (Sec. 3.3-3.5), host side.
//   per burst n:  P_n = T0_n + G_n, rho_n = V_n / (R P_n)              (Eq. 3)
//                 delta_b_n = V_n - R P_n                               (Eq. 4)
//                 b_iso_n = [V_n - R T0_n]_+, guard q_n + b_iso_n <= Q  (Eq. 6)
//   issue time:   T0_n while the guard holds, else (q_n + V_n - Q) / R: a fluid queue capped
//                 at Q and drained at R stretches issue until enough volume has drained
//   backlog:      q_{n+1} = [q_n + V_n - R (T_iss_n + G_n)]_+, which is the recurrence of
//                 Eq. 5 whenever the guard holds.
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
