// Expert-parallel routing, dispatch layout, dispatch stores and combine-reduce.
//
// Routing: top-k by repeated arg-max over the fp32 logits (ties to the lower expert index)
// and a softmax over all E experts; sixteen lanes per token with DPP reductions for
// E <= 256 and k <= 16, one wavefront per token otherwise.
// Layout: per 256-token chunk, every wave builds a 64-bit lane mask per expert in LDS
// (ds_or_b64), so a slot's rank among earlier tokens of the chunk routed to the same expert
// is a popcount: a deterministic, stable slot assignment. Chunk counts are scanned per
// source, then across sources and across the experts of each window.
// Dispatch: one wavefront per token row; every lane holds 16-byte pieces of the row in
// registers and stores them, 128-bit and coalesced, into the k destination rows. A row is
// contiguous on both sides, so no LDS staging is needed to coalesce.
#include <algorithm>

#include "xs_common.hpp"
#include "xs_plan.hpp"

namespace xs {

// ------------------------------------------------------------------------------ route
template <int EPL>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ logits, int T,
                                                         int E, int k, int renorm,
                                                         int* __restrict__ topk_idx,
                                                         float* __restrict__ topk_w) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* row = logits + static_cast<int64_t>(t) * E;
  float v[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    int e = i * 64 + lane;
    v[i] = e < E ? row[e] : -INFINITY;
  }
  // softmax denominator over all experts: lane partials in ascending i, then a butterfly
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < EPL; ++i) m = fmaxf(m, v[i]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < EPL; ++i)
    if (i * 64 + lane < E) s += expf(v[i] - m);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);

  uint32_t taken = 0;
  int my_idx = 0;
  float my_w = 0.f;
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      int e = i * 64 + lane;
      bool ok = e < E && !((taken >> i) & 1u);
      if (ok && (v[i] > bv || (v[i] == bv && e < bi))) {
        bv = v[i];
        bi = e;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      float ov = __shfl_xor(bv, off);
      int oi = __shfl_xor(bi, off);
      if (ov > bv || (ov == bv && oi < bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if ((bi & 63) == lane) taken |= 1u << (bi >> 6);
    if (lane == j) {
      my_idx = bi;
      my_w = expf(bv - m) / s;
    }
  }
  if (renorm) {
    float ws = lane < k ? my_w : 0.f;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) ws += __shfl_xor(ws, off);
    my_w = my_w / ws;
  }
  if (lane < k) {
    topk_idx[static_cast<int64_t>(t) * k + lane] = my_idx;
    topk_w[static_cast<int64_t>(t) * k + lane] = my_w;
  }
}

// Sixteen lanes per token (four tokens per wave), for E <= 16 * VPL and k <= 16. Lane s of
// a token holds the logits e = 64 q + 4 s + c (q < VPL / 4, c < 4): 16 contiguous bytes per
// lane and q, so a quarter-wave reads 256 contiguous bytes. The arg-max of each round and
// the softmax sum reduce over the 16 lanes with DPP row rotations (no LDS round trips).
template <int CTRL>
__device__ __forceinline__ void argmax_dpp(float& bv, int& bi) {
  const float ov = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(bv), CTRL, 0xF, 0xF, false));
  const int oi = __builtin_amdgcn_update_dpp(0, bi, CTRL, 0xF, 0xF, false);
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

template <int CTRL>
__device__ __forceinline__ float sum_dpp(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// all 16 lanes of a DPP row end with the reduction over the row: rotate by 8, 4, 2, 1
constexpr int kRor8 = 0x128, kRor4 = 0x124, kRor2 = 0x122, kRor1 = 0x121;

// Sixteen lanes per token, each holding VPL logits: lane sub has experts 64 q + 4 sub + c.
template <int VPL>
__device__ __forceinline__ void route16_load(const float* __restrict__ logits, int t, int T, int E, int sub,
                                             float (&v)[VPL]) {
  // tokens past T read the last row (every lane takes part in the row reductions) and store
  // nothing
  const float* row = logits + static_cast<int64_t>(t < T ? t : T - 1) * E;
  if ((E & 3) == 0) {
    // rows start 16-byte aligned: one 128-bit load per lane and q
#pragma unroll
    for (int q = 0; q < VPL / 4; ++q) {
      const int e = 64 * q + 4 * sub;
      const f32x4 x = e < E ? *reinterpret_cast<const f32x4*>(row + e)
                            : f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
      for (int c = 0; c < 4; ++c) v[4 * q + c] = x[c];
    }
  } else {
#pragma unroll
    for (int q = 0; q < VPL / 4; ++q)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int e = 64 * q + 4 * sub + c;
        v[4 * q + c] = e < E ? row[e] : -INFINITY;
      }
  }
}

template <int VPL>
__device__ __forceinline__ void route16_select(const float (&v)[VPL], int t, int T, int E, int k, int renorm,
                                               int sub, int* __restrict__ topk_idx, float* __restrict__ topk_w) {
  uint32_t taken = 0;
  float m = 0.f, my_v = -INFINITY;
  int my_idx = 0;
  for (int j = 0; j < k; ++j) {
    // a lane scans its experts in ascending index, so a strict > keeps the lowest index among
    // equal values; the first untaken expert is taken even at -inf. Padding slots (index >= E,
    // value -inf) come after every real expert of the lane and lose every tie to a real one.
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int q = 0; q < VPL / 4; ++q)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int s = 4 * q + c;
        if (!((taken >> s) & 1u) && (v[s] > bv || bi == 0x7fffffff)) {
          bv = v[s];
          bi = 64 * q + 4 * sub + c;
        }
      }
    // across the 16 lanes: ties (equal values, or only -inf left) go to the lower index
    argmax_dpp<kRor8>(bv, bi);
    argmax_dpp<kRor4>(bv, bi);
    argmax_dpp<kRor2>(bv, bi);
    argmax_dpp<kRor1>(bv, bi);
    if (j == 0) m = bv;   // the first winner is the row maximum
    if (((bi >> 2) & 15) == sub) taken |= 1u << ((bi >> 6) * 4 + (bi & 3));
    if (sub == j) {
      my_idx = bi;
      my_v = bv;
    }
  }
  // softmax denominator over all experts: lane partials in ascending e, then the row sum
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < VPL; ++i)
    if (64 * (i / 4) + 4 * sub + (i % 4) < E) s += expf(v[i] - m);
  s = sum_dpp<kRor8>(s);
  s = sum_dpp<kRor4>(s);
  s = sum_dpp<kRor2>(s);
  s = sum_dpp<kRor1>(s);
  float my_w = expf(my_v - m) / s;
  if (renorm) {
    float ws = sub < k ? my_w : 0.f;
    ws = sum_dpp<kRor8>(ws);
    ws = sum_dpp<kRor4>(ws);
    ws = sum_dpp<kRor2>(ws);
    ws = sum_dpp<kRor1>(ws);
    my_w = my_w / ws;
  }
  if (t < T && sub < k) {
    topk_idx[static_cast<int64_t>(t) * k + sub] = my_idx;
    topk_w[static_cast<int64_t>(t) * k + sub] = my_w;
  }
}

// Persistent: a workgroup (16 tokens at a time) walks the tokens with the grid's stride and
// loads the next group's logits while it selects the current group's experts, so the loads
// of a cold logits tensor overlap the selection instead of preceding it.
template <int VPL>
__global__ __launch_bounds__(256) void route_topk16_kernel(const float* __restrict__ logits, int T,
                                                           int E, int k, int renorm,
                                                           int* __restrict__ topk_idx,
                                                           float* __restrict__ topk_w) {
  const int sub = threadIdx.x & 15;
  const int stride = gridDim.x * 16;
  int t = blockIdx.x * 16 + (threadIdx.x >> 4);
  const int t_wave = blockIdx.x * 16 + (threadIdx.x >> 6) * 4;   // the wave's first token
  float v[VPL], nv[VPL];
  route16_load<VPL>(logits, t, T, E, sub, v);
  for (int tw = t_wave; tw < T; tw += stride, t += stride) {
    const bool more = tw + stride < T;
    if (more) route16_load<VPL>(logits, t + stride, T, E, sub, nv);
    route16_select<VPL>(v, t, T, E, k, renorm, sub, topk_idx, topk_w);
    if (more) {
#pragma unroll
      for (int i = 0; i < VPL; ++i) v[i] = nv[i];
    }
  }
}

// ------------------------------------------------------------------------------ layout
constexpr int kChunk = 256;   // tokens per layout chunk (4 waves)

// Per chunk: stable rank of each slot among the chunk's earlier slots of the same expert
// (written to slot_row as a partial value) and per-expert chunk counts.
__global__ __launch_bounds__(256) void layout_chunk_kernel(const int* __restrict__ idx, int T,
                                                           int k, int E, int n_chunks,
                                                           int* __restrict__ slot_row,
                                                           int* __restrict__ chunk_cnt,
                                                           int* status, int* scan_done) {
  extern __shared__ unsigned long long masks[];   // [4][E]
  const int s = blockIdx.y, c = blockIdx.x, tid = threadIdx.x;
  if (s == 0 && c == 0 && tid == 0) *scan_done = 0;   // the next kernel's completion count
  const int lane = tid & 63, w = tid >> 6;
  for (int i = tid; i < 4 * E; i += 256) masks[i] = 0ull;
  __syncthreads();
  const int t = c * kChunk + tid;
  const int64_t base = (static_cast<int64_t>(s) * T + t) * k;
  const unsigned long long bit = 1ull << lane;
  if (t < T) {
    for (int j = 0; j < k; ++j) {
      int e = idx[base + j];
      if (e >= 0 && e < E) atomicOr(&masks[w * E + e], bit);
      else set_status(status, XS_EBADINPUT);
      // a token that lists one expert twice would give both slots one row
      for (int j2 = 0; j2 < j; ++j2)
        if (idx[base + j2] == e) set_status(status, XS_EBADINPUT);
    }
  }
  __syncthreads();
  if (t < T) {
    const unsigned long long below = bit - 1ull;
    for (int j = 0; j < k; ++j) {
      int e = idx[base + j];
      if (e < 0 || e >= E) continue;
      int r = __popcll(masks[w * E + e] & below);
      for (int ww = 0; ww < w; ++ww) r += __popcll(masks[ww * E + e]);
      slot_row[base + j] = r;
    }
  }
  for (int e = tid; e < E; e += 256) {
    int n = 0;
    for (int ww = 0; ww < 4; ++ww) n += __popcll(masks[ww * E + e]);
    chunk_cnt[(static_cast<int64_t>(s) * n_chunks + c) * E + e] = n;
  }
}

// Per source (one block each): exclusive scan of the chunk counts of every expert, and the
// source's expert totals. The last block to finish then scans across sources and experts:
// src_base, expert_offsets (exclusive scan of expert totals within each window), dest_counts
// and the capacity check; with plan args (the fused layer) it also plans the expert FFN from
// the local experts' totals. Blocks release their counts with the counter increment (the
// block barrier orders every wave's stores before thread 0's agent-scope release); the last
// one acquires before it reads them.
__global__ __launch_bounds__(1024) void layout_scan_kernel(int* __restrict__ chunk_cnt, int n_chunks,
                                                           int n_src, int E, int W, int cap,
                                                           int* __restrict__ expert_counts,
                                                           int* __restrict__ src_base,
                                                           int* __restrict__ expert_offsets,
                                                           int* __restrict__ dest_counts, int* status,
                                                           int* done, PlanArgs pa) {
  __shared__ int tot[1024], s_m[1024], s_first[1024], s_rows, s_last;
  const int s = blockIdx.x;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int* col = chunk_cnt + static_cast<int64_t>(s) * n_chunks * E + e;
    int run = 0;
    int c = 0;
    for (; c + 8 <= n_chunks; c += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = col[static_cast<int64_t>(c + u) * E];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        col[static_cast<int64_t>(c + u) * E] = run;
        run += v[u];
      }
    }
    for (; c < n_chunks; ++c) {
      int v = col[static_cast<int64_t>(c) * E];
      col[static_cast<int64_t>(c) * E] = run;
      run += v;
    }
    expert_counts[static_cast<int64_t>(s) * E + e] = run;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    s_last = __hip_atomic_fetch_add(done, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) ==
             static_cast<int>(gridDim.x) - 1;
    if (s_last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
  if (!s_last) return;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int run = 0;
    // eight sources' counts in flight at a time (one dependent load per source took longer)
    for (int s0 = 0; s0 < n_src; s0 += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[u] = s0 + u < n_src ? expert_counts[static_cast<int64_t>(s0 + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (s0 + u < n_src) src_base[static_cast<int64_t>(s0 + u) * E + e] = run;
        run += v[u];
      }
    }
    tot[e] = run;
  }
  __syncthreads();
  const int epw = E / W;
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int d0 = (e / epw) * epw, off = 0;
    for (int x = d0; x < e; ++x) off += tot[x];
    expert_offsets[e] = off;
    if (pa.meta && e >= pa.e_begin && e < pa.e_begin + pa.n_experts)
      s_m[e - pa.e_begin] = max(0, min(tot[e], cap - off));
  }
  for (int d = threadIdx.x; d < W; d += blockDim.x) {
    int n = 0;
    for (int x = d * epw; x < (d + 1) * epw; ++x) n += tot[x];
    dest_counts[d] = n;
    if (n > cap) set_status(status, XS_ECAPACITY);
  }
  if (pa.meta) plan_rows(pa, 256, s_m, s_first, &s_rows);
}

// Every slot: final row = expert offset + source base + chunk base + rank in chunk;
// records the inverse map for rows inside the capacity.
__global__ __launch_bounds__(256) void layout_finalize_kernel(
    const int* __restrict__ idx, int n_src, int T, int k, int E, int W, int cap, int n_chunks,
    const int* __restrict__ chunk_base, const int* __restrict__ src_base,
    const int* __restrict__ expert_offsets, int* __restrict__ slot_row, int* __restrict__ row_src) {
  const int64_t n = static_cast<int64_t>(n_src) * T * k;
  const int epw = E / W;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    int e = idx[i];
    if (e < 0 || e >= E) continue;
    int64_t st = i / k;
    int j = static_cast<int>(i - st * k);
    int s = static_cast<int>(st / T);
    int t = static_cast<int>(st - static_cast<int64_t>(s) * T);
    int c = t / kChunk;
    int r = expert_offsets[e] + src_base[static_cast<int64_t>(s) * E + e] +
            chunk_base[(static_cast<int64_t>(s) * n_chunks + c) * E + e] + slot_row[i];
    slot_row[i] = r;
    if (r < cap) row_src[static_cast<int64_t>(e / epw) * cap + r] = (s << 24) | (t * k + j);
  }
}

// ------------------------------------------------------------------------------ dispatch
// The rest of the layout, done by the dispatch launch of the fused layer (FinArgs with idx_all
// set): the dispatch waves compute their own slots' final rows from the scan's bases (and
// record them with the inverse map), blocks past the dispatch ones finalize every other
// source's slots, and the last dispatch block to finish sets the windows' ready flags (done
// set; the plan zeroed it).

// Final row of slot (s, t, j) of expert e whose rank in its chunk is r.
__device__ __forceinline__ int final_row(const FinArgs& fa, int E, int s, int t, int e, int r) {
  return fa.expert_offsets[e] + fa.src_base[static_cast<int64_t>(s) * E + e] +
         fa.chunk_base[(static_cast<int64_t>(s) * fa.n_chunks + t / kChunk) * E + e] + r;
}

// One wave per token (measured: a quarter row per wave, four waves per token, is slower).
// Lanes hold up to 8 16-byte pieces of the row per round and store them into the k
// destination rows.
__global__ __launch_bounds__(256) void dispatch_kernel(const char* __restrict__ x, int64_t x_stride,
                                                       int nch, int T,
                                                       const int* __restrict__ idx,
                                                       int* __restrict__ slot_row, int k,
                                                       int E, WinSet win, int* status, FinArgs fa) {
  __shared__ int s_last;
  const int lane = threadIdx.x & 63;
  const int epw = E / win.n;
  if (fa.idx_all && static_cast<int>(blockIdx.x) >= fa.n_disp_blocks) {
    // finalize the other sources' slots
    const int64_t per = static_cast<int64_t>(T) * k;
    const int64_t n = static_cast<int64_t>(fa.n_src - 1) * per;
    const int64_t step = static_cast<int64_t>(gridDim.x - fa.n_disp_blocks) * blockDim.x;
    for (int64_t i0 = static_cast<int64_t>(blockIdx.x - fa.n_disp_blocks) * blockDim.x + threadIdx.x; i0 < n;
         i0 += step) {
      const int64_t i = i0 < fa.src * per ? i0 : i0 + per;
      const int e = fa.idx_all[i];
      if (e < 0 || e >= E) continue;
      const int64_t st = i / k;
      const int j = static_cast<int>(i - st * k);
      const int s = static_cast<int>(st / T);
      const int t = static_cast<int>(st - static_cast<int64_t>(s) * T);
      const int r = final_row(fa, E, s, t, e, fa.slot_row_all[i]);
      fa.slot_row_all[i] = r;
      if (r < fa.cap) fa.row_src[static_cast<int64_t>(e / epw) * fa.cap + r] = (s << 24) | (t * k + j);
    }
    return;
  }
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  // lane j < k resolves destination j; broadcast below with readlane
  char* my_dst = nullptr;
  if (t < T && lane < k) {
    const int64_t si = static_cast<int64_t>(t) * k + lane;
    int e = idx[si];
    int r = slot_row[si];
    if (e < 0 || e >= E) {
      set_status(status, XS_EBADINPUT);
    } else {
      if (fa.idx_all) {
        r = final_row(fa, E, fa.src, t, e, r);
        slot_row[si] = r;
        if (r < fa.cap) fa.row_src[static_cast<int64_t>(e / epw) * fa.cap + r] = (fa.src << 24) | (t * k + lane);
      }
      int d = e / epw;
      if (r < 0 || r >= win.cap[d]) set_status(status, XS_ECAPACITY);
      else my_dst = win.base[d] + static_cast<int64_t>(r) * win.stride[d];
    }
  }
  if (t < T) {
    const u32x4* src = reinterpret_cast<const u32x4*>(x + static_cast<int64_t>(t) * x_stride);
    for (int c0 = 0; c0 < nch; c0 += 64 * 8) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        int c = c0 + u * 64 + lane;
        if (c < nch) v[u] = src[c];
      }
      for (int j = 0; j < k; ++j) {
        uint64_t p = __shfl(reinterpret_cast<uint64_t>(my_dst), j);
        if (!p) continue;
        u32x4* dst = reinterpret_cast<u32x4*>(p);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          int c = c0 + u * 64 + lane;
          if (c < nch) dst[c] = v[u];   // (measured: nontemporal stores here are slower)
        }
      }
    }
  }
  if (!fa.done) return;
  // the window signal: every block's stores are released at system scope (host-coherent
  // windows included) before its count; the last block then sets the flags
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence_system();
    s_last = atomicAdd(fa.done, 1) == fa.n_disp_blocks - 1;
    if (s_last) {
      __threadfence_system();
      for (int d = 0; d < win.n; ++d)
        if (win.flag[d]) __hip_atomic_store(win.flag[d], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

// ------------------------------------------------------------------------------ combine
// out[t] = bf16(sum_j w[t][j] * C[t*k + j]); one wave per token, 8 values per lane-piece.
__global__ __launch_bounds__(256) void combine_reduce_kernel(const char* __restrict__ cbuf,
                                                             int64_t cstride,
                                                             const float* __restrict__ w, int T,
                                                             int k, int H,
                                                             uint16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  // four waves per token, each over a quarter of the row's 16-byte pieces (one wave per
  // token left 16 waves per CU at T = 4096, too few loads in flight to stream HBM)
  const int wv = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int t = wv >> 2;
  if (t >= T) return;
  const float wl = lane < k ? w[static_cast<int64_t>(t) * k + lane] : 0.f;
  const int nch = H >> 3;
  const int per = (nch + 3) >> 2;
  const int c_begin = (wv & 3) * per;
  const int c_end = min(nch, c_begin + per);
  u32x4* dst = reinterpret_cast<u32x4*>(out + static_cast<int64_t>(t) * H);
  const char* rows = cbuf + static_cast<int64_t>(t) * k * cstride;
  // two 16-byte pieces per lane per pass, the slots' loads issued in blocks of eight before
  // any sum (a loop over the runtime k kept only two loads in flight)
  for (int c0 = c_begin + lane; c0 < c_end; c0 += 128) {
    const int c1 = c0 + 64;
    const bool two = c1 < c_end;
    float acc[2][8];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[h][q] = 0.f;
    for (int j0 = 0; j0 < k; j0 += 8) {
      u32x4 p0[8], p1[8];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        p0[jj] = p1[jj] = u32x4{0u, 0u, 0u, 0u};
        if (j0 + jj < k) {
          const u32x4* r = reinterpret_cast<const u32x4*>(rows + static_cast<int64_t>(j0 + jj) * cstride);
          p0[jj] = __builtin_nontemporal_load(r + c0);   // each combine row is read once
          if (two) p1[jj] = __builtin_nontemporal_load(r + c1);
        }
      }
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if (j0 + jj >= k) break;
        const float wj = __shfl(wl, j0 + jj);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[0][2 * q] += wj * bf_lo(p0[jj][q]);
          acc[0][2 * q + 1] += wj * bf_hi(p0[jj][q]);
          acc[1][2 * q] += wj * bf_lo(p1[jj][q]);
          acc[1][2 * q + 1] += wj * bf_hi(p1[jj][q]);
        }
      }
    }
    u32x4 o0, o1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      o0[q] = pack_bf16x2(acc[0][2 * q], acc[0][2 * q + 1]);
      o1[q] = pack_bf16x2(acc[1][2 * q], acc[1][2 * q + 1]);
    }
    dst[c0] = o0;
    if (two) dst[c1] = o1;
  }
}

// Ready flags of windows written by the preceding kernels on the same stream: the kernel
// boundary orders those stores before these; the system-scope release makes them visible
// to host-coherent consumers before the flag.
__global__ void signal_windows_kernel(WinSet win) {
  int d = threadIdx.x;
  if (d < win.n && win.flag[d]) {
    __threadfence_system();
    __hip_atomic_store(win.flag[d], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

}  // namespace xs

// ------------------------------------------------------------------------------ C ABI
using namespace xs;

namespace xs_host {
int persistent_grid(int max_producers);
}  // namespace xs_host

namespace xs_host {
int signal_windows(const WinSet& ws, hipStream_t st) {
  bool any = false;
  for (int d = 0; d < ws.n; ++d) any |= ws.flag[d] != nullptr;
  if (!any) return XS_OK;
  hipLaunchKernelGGL(signal_windows_kernel, dim3(1), dim3(XS_MAX_WINDOWS), 0, st, ws);
  return launch_status();
}
}  // namespace xs_host

extern "C" int xs_route_topk_softmax(const float* logits, int32_t T, int32_t E, int32_t k,
                                     int32_t renormalize, int32_t* topk_idx, float* topk_w,
                                     void* stream) {
  if (!logits || !topk_idx || !topk_w || T < 0 || E < 1 || E > 1024 || k < 1 || k > E || k > 32)
    return XS_EINVAL;
  if (T == 0) return XS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (E <= 256 && k <= 16) {
    // up to eight workgroups per CU: the selection is a chain of dependent DPP steps, and with
    // two per CU it was exposed (32,768 tokens, top-8 of 256: 36.8 us against 30.6 us)
    const dim3 g16(std::min((T + 15) / 16, 8 * xs_host::persistent_grid(0))), b16(256);
    if (E <= 64)
      hipLaunchKernelGGL(route_topk16_kernel<4>, g16, b16, 0, st, logits, T, E, k, renormalize, topk_idx, topk_w);
    else if (E <= 128)
      hipLaunchKernelGGL(route_topk16_kernel<8>, g16, b16, 0, st, logits, T, E, k, renormalize, topk_idx, topk_w);
    else
      hipLaunchKernelGGL(route_topk16_kernel<16>, g16, b16, 0, st, logits, T, E, k, renormalize, topk_idx, topk_w);
    return xs_host::launch_status();
  }
  dim3 grid((T + 3) / 4), block(256);
  const int epl = (E + 63) / 64;
#define XS_ROUTE(N)                                                                        \
  case N:                                                                                  \
    hipLaunchKernelGGL(route_topk_kernel<N>, grid, block, 0, st, logits, T, E, k, renormalize, \
                       topk_idx, topk_w);                                                  \
    break;
  switch (epl) {
    XS_ROUTE(1) XS_ROUTE(2) XS_ROUTE(3) XS_ROUTE(4) XS_ROUTE(5) XS_ROUTE(6) XS_ROUTE(7) XS_ROUTE(8)
    XS_ROUTE(9) XS_ROUTE(10) XS_ROUTE(11) XS_ROUTE(12) XS_ROUTE(13) XS_ROUTE(14) XS_ROUTE(15)
    XS_ROUTE(16)
    default: return XS_EINVAL;
  }
#undef XS_ROUTE
  return xs_host::launch_status();
}

// The chunk counts, then 256 bytes holding the scan's completion count.
static int64_t layout_chunk_bytes(int32_t n_src, int32_t T, int32_t E) {
  int64_t n_chunks = (static_cast<int64_t>(T) + kChunk - 1) / kChunk;
  int64_t b = static_cast<int64_t>(n_src) * n_chunks * E * 4;
  return (b + 255) & ~int64_t(255);
}
static int64_t layout_ws_bytes(int32_t n_src, int32_t T, int32_t E) { return layout_chunk_bytes(n_src, T, E) + 256; }

__global__ void zero_int_kernel(int* p) { *p = 0; }

extern "C" int xs_dispatch_layout_workspace_bytes(int32_t n_src, int32_t T, int32_t E,
                                                  int64_t* bytes) {
  if (!bytes || n_src < 1 || T < 0 || E < 1) return XS_EINVAL;
  *bytes = layout_ws_bytes(n_src, T, E);
  return XS_OK;
}

namespace xs_host {
int dispatch_layout(const int32_t* topk_idx, int32_t n_src, int32_t T, int32_t k, int32_t E,
                    int32_t W, int32_t cap, int32_t* expert_counts, int32_t* src_base,
                    int32_t* expert_offsets, int32_t* dest_counts, int32_t* slot_row,
                    int32_t* row_src, void* workspace, int64_t workspace_bytes,
                    int32_t* dev_status, hipStream_t st, const PlanArgs* plan) {
  if (!topk_idx || !expert_counts || !src_base || !expert_offsets || !dest_counts || !slot_row ||
      !row_src)
    return XS_EINVAL;
  if (n_src < 1 || n_src > 127 || T < 0 || k < 1 || k > E || E < 1 || E > 1024 || W < 1 ||
      W > XS_MAX_WINDOWS || E % W || cap < 0 || static_cast<int64_t>(T) * k >= (1 << 24))
    return XS_EINVAL;
  if (!workspace || workspace_bytes < layout_ws_bytes(n_src, T, E)) return XS_EWORKSPACE;
  const int n_chunks = (T + kChunk - 1) / kChunk;
  int* chunk = static_cast<int*>(workspace);
  int* scan_done = reinterpret_cast<int*>(static_cast<char*>(workspace) + layout_chunk_bytes(n_src, T, E));
  if (n_chunks > 0) {
    hipLaunchKernelGGL(layout_chunk_kernel, dim3(n_chunks, n_src), dim3(256),
                       4 * E * sizeof(unsigned long long), st, topk_idx, T, k, E, n_chunks,
                       slot_row, chunk, dev_status, scan_done);
  } else {
    hipLaunchKernelGGL(zero_int_kernel, dim3(1), dim3(1), 0, st, scan_done);
  }
  if (launch_status()) return XS_EHIP;
  hipLaunchKernelGGL(layout_scan_kernel, dim3(n_src), dim3(1024), 0, st, chunk, n_chunks, n_src, E, W,
                     cap, expert_counts, src_base, expert_offsets, dest_counts, dev_status, scan_done,
                     plan ? *plan : PlanArgs{});
  if (launch_status()) return XS_EHIP;
  // with a plan (the fused layer), the dispatch launch finalizes the rows (FinArgs)
  const int64_t n = static_cast<int64_t>(n_src) * T * k;
  if (n > 0 && !plan) {
    int blocks = static_cast<int>(std::min<int64_t>((n + 255) / 256, 4096));
    hipLaunchKernelGGL(layout_finalize_kernel, dim3(blocks), dim3(256), 0, st, topk_idx, n_src, T,
                       k, E, W, cap, n_chunks, chunk, src_base, expert_offsets, slot_row, row_src);
    if (launch_status()) return XS_EHIP;
  }
  return XS_OK;
}

// Token rows of row_bytes bytes (a multiple of 16), x_stride apart, into the window rows of
// their slots.
// With fin (the fused layer), the same launch finishes the layout (FinArgs) and, when the
// windows have flags, signals them from its last dispatch block.
int dispatch_rows(const void* x, int64_t x_stride, int32_t row_bytes, int32_t T,
                  const int32_t* topk_idx, const int32_t* slot_row, int32_t k, int32_t E,
                  const WinSet& ws, int32_t* dev_status, hipStream_t st, const FinArgs* fin) {
  FinArgs fa{};
  const int nd = (T + 3) / 4;
  int nf = 0;
  if (fin) {
    fa = *fin;
    fa.n_disp_blocks = nd;
    const int64_t n_other = static_cast<int64_t>(fa.n_src - 1) * T * k;
    nf = static_cast<int>(std::min<int64_t>((n_other + 255) / 256, 4096));
    bool any = false;
    for (int d = 0; d < ws.n; ++d) any |= ws.flag[d] != nullptr;
    if (!any || nd == 0) fa.done = nullptr;
  }
  if (nd + nf > 0) {
    hipLaunchKernelGGL(dispatch_kernel, dim3(nd + nf), dim3(256), 0, st, static_cast<const char*>(x),
                       x_stride, row_bytes / 16, T, topk_idx, const_cast<int32_t*>(slot_row), k, E, ws,
                       dev_status, fa);
    if (launch_status()) return XS_EHIP;
  }
  return fa.done ? XS_OK : signal_windows(ws, st);
}

int dispatch(const void* x, int32_t T, int32_t H, const int32_t* topk_idx, const int32_t* slot_row,
             int32_t k, int32_t E, const WinSet& ws, int32_t* dev_status, hipStream_t st) {
  return dispatch_rows(x, static_cast<int64_t>(H) * 2, H * 2, T, topk_idx, slot_row, k, E, ws,
                       dev_status, st, nullptr);
}

int combine_reduce(const void* cbuf, int64_t cstride, const float* w, int32_t T, int32_t k,
                   int32_t H, void* out, hipStream_t st) {
  if (T == 0) return XS_OK;
  hipLaunchKernelGGL(combine_reduce_kernel, dim3(T), dim3(256), 0, st,
                     static_cast<const char*>(cbuf), cstride, w, T, k, H,
                     static_cast<uint16_t*>(out));
  return launch_status();
}
}  // namespace xs_host

extern "C" int xs_dispatch_layout(const int32_t* topk_idx, int32_t n_src, int32_t T, int32_t k,
                                  int32_t E, int32_t W, int32_t cap, int32_t* expert_counts,
                                  int32_t* src_base, int32_t* expert_offsets,
                                  int32_t* dest_counts, int32_t* slot_row, int32_t* row_src,
                                  void* workspace, int64_t workspace_bytes, int32_t* dev_status,
                                  void* stream) {
  return xs_host::dispatch_layout(topk_idx, n_src, T, k, E, W, cap, expert_counts, src_base,
                                  expert_offsets, dest_counts, slot_row, row_src, workspace,
                                  workspace_bytes, dev_status, static_cast<hipStream_t>(stream), nullptr);
}

extern "C" int xs_dispatch(const void* x, int32_t T, int32_t H, const int32_t* topk_idx,
                           const int32_t* slot_row, int32_t k, int32_t E, const xs_window* win,
                           int32_t W, int32_t* dev_status, void* stream) {
  if (!x || !topk_idx || !slot_row || T < 0 || H < 8 || k < 1 || k > 32 || k > E || E < 1 ||
      W < 1 || E % W)
    return XS_EINVAL;
  if (H % 8 || (reinterpret_cast<uintptr_t>(x) & 15)) return XS_EUNSUPPORTED;
  WinSet ws;
  int rc = xs_host::make_winset(win, W, static_cast<int64_t>(H) * 2, &ws);
  if (rc) return rc;
  return xs_host::dispatch(x, T, H, topk_idx, slot_row, k, E, ws, dev_status,
                           static_cast<hipStream_t>(stream));
}

extern "C" int xs_dispatch_rows(const void* rows, int64_t row_stride, int32_t row_bytes, int32_t T,
                                const int32_t* topk_idx, const int32_t* slot_row, int32_t k, int32_t E,
                                const xs_window* win, int32_t W, int32_t* dev_status, void* stream) {
  if (!rows || !topk_idx || !slot_row || T < 0 || row_bytes < 16 || k < 1 || k > 32 || k > E ||
      E < 1 || W < 1 || E % W || row_stride < row_bytes)
    return XS_EINVAL;
  if (row_bytes % 16 || row_stride % 16 || (reinterpret_cast<uintptr_t>(rows) & 15)) return XS_EUNSUPPORTED;
  WinSet ws;
  int rc = xs_host::make_winset(win, W, row_bytes, &ws);
  if (rc) return rc;
  return xs_host::dispatch_rows(rows, row_stride, row_bytes, T, topk_idx, slot_row, k, E, ws, dev_status,
                                static_cast<hipStream_t>(stream), nullptr);
}

extern "C" int xs_combine_reduce(const void* cbuf, int64_t cbuf_stride_bytes, const float* topk_w,
                                 int32_t T, int32_t k, int32_t H, void* out, void* stream) {
  if (!cbuf || !topk_w || !out || T < 0 || k < 1 || k > 32 || H < 8) return XS_EINVAL;
  if (H % 8 || (cbuf_stride_bytes & 15) || cbuf_stride_bytes < static_cast<int64_t>(H) * 2 ||
      (reinterpret_cast<uintptr_t>(cbuf) & 15) || (reinterpret_cast<uintptr_t>(out) & 15))
    return XS_EUNSUPPORTED;
  return xs_host::combine_reduce(cbuf, cbuf_stride_bytes, topk_w, T, k, H, out,
                                 static_cast<hipStream_t>(stream));
}
