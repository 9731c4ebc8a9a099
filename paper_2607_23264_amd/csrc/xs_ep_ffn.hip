// Persistent expert-FFN kernel of the EP layer (Sec. 4.3, App. A.2).
//
// Scheduler rows are (local expert, row block) pairs in expert-major order: an expert's m
// rows fall into ceil(m / 256) blocks (expert_block).
// Each row has P1 = I / 128 Linear-1 tiles (gate+up GEMM with the SwiGLU epilogue, 128
// columns of h each) and P2 = H / 256 Linear-2 tiles (down GEMM whose epilogue stores the
// output rows into the combine windows of their source ranks: the remote-store bursts of
// Sec. 4.3). A Linear-2 tile of row p reads the whole h row block, so it waits until all P1
// Linear-1 tiles of row p have released their stores (per-row counters, agent-scope
// release/acquire, bounded wait).
//
// Tile order per persistent workgroup ("scheduler instance" g of G):
//   BURST       Expert-Wave: global list [L1 of wave 0, L2 of wave 0, L1 of wave 1, ...],
//               instance g takes entries g, g + G, ...
//   INTERLEAVE  cross-wave interleaving (Alg. 1): a Linear-2 entry is taken only while the
//               first Linear-1 entry not yet taken is at least D rows ahead of it, otherwise
//               the next Linear-1 entry (l2_may_run).
//   CHUNK       the same with at most c consecutive Linear-2 tiles before a Linear-1 tile.
// The entries a workgroup sees are either its own share of each stream (static claiming:
// entries g, g + G, ...) or the next entries of two shared counters (dynamic claiming); the
// rule is the same.
// Deadlock freedom needs every workgroup resident (grid <= CUs, one workgroup per CU by
// LDS) and D >= 1: an instance only waits on a row strictly behind its own Linear-1 cursor,
// so the lowest row anyone waits on always has its Linear-1 owners running.
#include <algorithm>
#include <cmath>
#include <mutex>

#include "xs_gemm_mx.hpp"
#include "xs_plan.hpp"

namespace xs {

struct RowWin {
  char* base[XS_MAX_WINDOWS];
  int64_t stride[XS_MAX_WINDOWS];
};

struct EpArgs {
  int E, epw, H, I, e_begin, n_experts, cap, d_first;
  int n_src, tk;               // combine windows and rows per combine window (T * k)
  int P1, P2;
  RowWin dwin;                 // computed dispatch windows, index d - d_first
  RowWin cwin;                 // combine windows by source rank
  const int* expert_offsets;
  const int* row_src;          // [W][cap]
  const uint16_t* w1;
  const uint16_t* w2;
  uint16_t* h;
  uint16_t* y;
  const uint8_t* w1s;          // MX: weight scales in groups of 512 K elements (w1 / w2 then
  const uint8_t* w2s;          //     hold E4M3 or packed E2M1 codes)
  int64_t h_stride;            // MX: bytes per h code row (I)
  uint8_t* hs;                 // MX: h scales, groups [I / 512][h_rows][16 bytes]
  int64_t h_rows;
  const int* meta;             // [0] rows P, [1] waves, [2] wave-list length, [3] computed rows
  const int* row_expert;
  const int* exp_m;
  const int* exp_rowfirst;
  const int* exp_hrow;
  const int* wave_pos;
  const int* wave_row;
  int* l1_done;
  int* claim_ctr;              // [0] Linear-1 / wave-list entries taken, [1] Linear-2 entries taken
  int claim;                   // XS_CLAIM_STATIC / XS_CLAIM_DYNAMIC
  int l2_combine;              // Linear-2 epilogue: 1 = combine windows, 0 = y rows
  int policy, lead, chunk, withhold_row;
  int64_t gap_ticks, timeout_ticks;
  int* status;
  xs_trace tr;
};

// Per-expert row counts (clipped to the rows that fit in the window), then the plan. One block.
__global__ __launch_bounds__(1024) void ep_plan_kernel(const int* __restrict__ expert_counts,
                                                       int n_src, int E,
                                                       const int* __restrict__ expert_offsets,
                                                       PlanArgs pa) {
  __shared__ int s_m[1024], s_first[1024], s_rows;
  const int i = threadIdx.x;
  if (i < pa.n_experts) {
    const int e = pa.e_begin + i;
    const int off = expert_offsets[e];
    int m = 0;
    // eight sources' counts in flight at a time
    for (int s0 = 0; s0 < n_src; s0 += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = s0 + u < n_src ? expert_counts[static_cast<int64_t>(s0 + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) m += v[u];
    }
    s_m[i] = max(0, min(m, pa.cap - off));
  }
  plan_rows(pa, kBM, s_m, s_first, &s_rows);
}

// Rows [m0, m0 + rows) of local expert x covered by scheduler row p. The expert's m rows fall
// into mt = ceil(m / 256) blocks. With `equal` (the bf16 tiles) the blocks hold ceil(m / mt)
// rows rounded up to a whole 32-row MFMA block (at most 256, so mt blocks always cover m and
// the last one is never empty); otherwise 256 rows each, the last one ragged. A near-empty
// block still streams its full weight panel and waits out every K step's load latency with
// little MFMA work to hide it; in the bf16 core (two waves per SIMD, one per 128-row half)
// equal blocks shorten every tile in proportion to its 32-row blocks, while in the MX core
// (one wave per SIMD) a tile takes as long as its fuller half, so there 256-row blocks with
// a fast ragged tail are the cheaper split (measured: 1 % faster for bf16, 2 % slower for the
// MX layer). The blocking changes no result: every output element sums the same products in
// the same K order.
__device__ __forceinline__ void expert_block(const EpArgs& a, int x, int p, bool equal, int& m0,
                                             int& rows) {
  const int m = a.exp_m[x];
  const int mt = (m + kBM - 1) / kBM;
  const int bm = equal ? min(kBM, ((m + mt - 1) / mt + 31) & ~31) : kBM;
  m0 = (p - a.exp_rowfirst[x]) * bm;
  rows = min(bm, m - m0);
}

// Tracing with ext records only: the first wave waits until the stores of its previous
// epilogue have left it (vmcnt(0)), the point where this design reuses its local staging
// (App. A.2), and returns how many ticks that took. Without ext records nothing waits.
__device__ __forceinline__ uint64_t staging_wait(const EpArgs& a) {
  if (!a.tr.ext || threadIdx.x >= 64) return 0;
  __builtin_amdgcn_sched_barrier(0);
  const uint64_t t = wall_ticks();
  __builtin_amdgcn_sched_barrier(0);
  wait_vm0();
  __builtin_amdgcn_sched_barrier(0);
  const uint64_t d = wall_ticks() - t;
  __builtin_amdgcn_sched_barrier(0);
  return d;
}

// One trace record (thread 0): kind 1 / 2, tile index, start, mainloop end, issue end; with
// ext records also the dependency-wait end, the staging wait, the bytes stored and the rows.
__device__ __forceinline__ void trace_tile(const EpArgs& a, uint64_t kind, uint32_t tile, uint64_t t0,
                                           uint64_t t1, uint64_t t2, uint64_t t_dep, uint64_t stage,
                                           uint64_t bytes, int rows) {
  const uint32_t i = atomicAdd(a.tr.count, 1u);
  if (static_cast<int64_t>(i) >= a.tr.capacity) return;
  uint64_t* r = a.tr.buf + static_cast<int64_t>(i) * 4;
  r[0] = (kind << 56) | (static_cast<uint64_t>(blockIdx.x) << 32) | tile;
  r[1] = t0;
  r[2] = t1;
  r[3] = t2;
  if (a.tr.ext) {
    uint64_t* x = a.tr.ext + static_cast<int64_t>(i) * 4;
    x[0] = t_dep;
    x[1] = stage;
    x[2] = bytes;
    x[3] = static_cast<uint64_t>(rows);
  }
}

// The rule every claim mode applies (App. A.2): Linear-2 entry e2 may run next when the first
// Linear-1 entry not yet taken, e1, is at least the lead D rows past e2's row (or no Linear-1
// entry is left), and the chunk cap, if set, still allows another Linear-2 tile before a
// Linear-1 one ("run" Linear-2 tiles have run since the last Linear-1 tile).
__device__ __forceinline__ bool l2_may_run(const EpArgs& a, int e2, int e1, int n1, int run) {
  const bool l1_left = e1 < n1;
  if (a.chunk > 0 && run >= a.chunk && l1_left) return false;
  return !l1_left || e2 / a.P2 + a.lead <= e1 / a.P1;
}

// Thread 0's dynamic-claim state. The next tile is claimed ahead, during the current tile's
// epilogue: the counters are read right after the mainloop (claim_load), their values decide
// the next tile before the epilogue stores and at most one counter increment goes out there
// (claim_take), and the loop top only reads its result (claim_next). The round trips to the
// counters thus overlap the epilogue's staging and stores. The claim comes after the current
// tile's mainloop, so after any dependency wait of that tile: a workgroup never holds a
// claimed tile while it waits, and every Linear-1 tile a Linear-2 tile waits on still has an
// owner that reaches it without waiting. What the early read cannot settle (a ticket not yet
// eligible, a stream found exhausted) is left to ep_claim at the loop top. Counter values
// read early only lag, so their eligibility tests are conservative.
struct Claim {
  int on;            // claim ahead (fused interleave / chunk with dynamic claiming)
  int n1, n2;        // entries of the two streams
  int run, ticket;   // Linear-2 tiles since the last Linear-1 tile; held ticket, -1 none, -2 no more
  int c1, c2;        // counters as read after the mainloop
  int kind, k;       // 0 nothing taken, 1 Linear-1 increment (k its result), 2 ticket increment,
                     // 3 settled (k the claim value)
};

__device__ __forceinline__ void claim_load(const EpArgs& a, Claim* cl) {
  if (!cl || !cl->on || threadIdx.x != 0) return;
  cl->c1 = __hip_atomic_load(a.claim_ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  cl->c2 = __hip_atomic_load(a.claim_ctr + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  cl->kind = 0;
}

__device__ __forceinline__ void claim_take(const EpArgs& a, Claim* cl) {
  if (!cl || !cl->on || threadIdx.x != 0) return;
  if (cl->ticket >= 0 && l2_may_run(a, cl->ticket, cl->c1, cl->n1, cl->run)) {
    cl->k = -cl->ticket - 2;
    cl->ticket = -1;
    ++cl->run;
    cl->kind = 3;
  } else if (cl->ticket == -1 && cl->c2 < cl->n2 && l2_may_run(a, cl->c2, cl->c1, cl->n1, cl->run)) {
    cl->k = __hip_atomic_fetch_add(a.claim_ctr + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    cl->kind = 2;
  } else if (cl->c1 < cl->n1) {
    cl->k = __hip_atomic_fetch_add(a.claim_ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    cl->kind = 1;
  }
}

__device__ __forceinline__ void ep_l1_tile(const EpArgs& a, int p, int nt, bool fused,
                                           char* lds, char** rowptr, Claim* cl) {
  const int tid = threadIdx.x;
  const int x = a.row_expert[p];
  const int e = a.e_begin + x;
  const int dl = e / a.epw - a.d_first;
  int m0, rows;
  expert_block(a, x, p, true, m0, rows);
  const uint64_t t0 = a.tr.buf ? wall_ticks() : 0;
  const uint64_t stw = staging_wait(a);
  const int64_t lda = a.dwin.stride[dl] / 2;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(
      a.dwin.base[dl] + static_cast<int64_t>(a.expert_offsets[e] + m0) * a.dwin.stride[dl]);
  const uint16_t* B = a.w1 + static_cast<int64_t>(x) * 2 * a.I * a.H;
  Acc acc;
  gemm_mainloop<true>(A, lda, rows, B, a.H, nt * (kBN / 2), a.I, true, a.H, acc, lds);
  claim_load(a, cl);
  const uint64_t t1 = a.tr.buf ? wall_ticks() : 0;
  if (tid < rows)
    rowptr[tid] = reinterpret_cast<char*>(
        a.h + static_cast<int64_t>(a.exp_hrow[x] + m0 + tid) * a.I + nt * (kBN / 2));
  stage_swiglu(acc, lds);
  __syncthreads();
  claim_take(a, cl);
  store_rows(lds, kEpiPitchH, kBN / 2, rows, rowptr);
  if (fused) {
    // The workgroup barrier orders every wave's h stores before thread 0's agent-scope
    // release (one L2 writeback per tile instead of one per wave).
    __syncthreads();
    if (tid == 0 && p != a.withhold_row)
      __hip_atomic_fetch_add(&a.l1_done[p], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    lds_barrier();   // the unfused h rows are read by a later launch
  }
  if (a.tr.buf && tid == 0)
    trace_tile(a, 1, static_cast<uint32_t>(p * a.P1 + nt), t0, t1, wall_ticks(), t0, stw,
               static_cast<uint64_t>(rows) * (kBN / 2) * 2, rows);
}

// Returns false if the wait for row p's Linear-1 tiles expired (the tile is then skipped).
// Polls with relaxed agent-scope loads; one acquire fence once the row is complete (an
// acquire load per poll would invalidate the caches on every iteration).
__device__ __forceinline__ bool ep_wait_row(const EpArgs& a, int p, int* flag) {
  if (threadIdx.x == 0) {
    int ok = 1;
    if (__hip_atomic_load(&a.l1_done[p], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < a.P1) {
      const uint64_t t0 = wall_ticks();
      while (__hip_atomic_load(&a.l1_done[p], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
             a.P1) {
        if (wall_ticks() - t0 > static_cast<uint64_t>(a.timeout_ticks)) {
          ok = 0;
          set_status(a.status, XS_ETIMEOUT);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
    if (ok) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *flag = ok;
  }
  __syncthreads();
  const bool ok = *flag != 0;
  __syncthreads();
  return ok;
}

__device__ __forceinline__ void ep_l2_tile(const EpArgs& a, int p, int nt, bool fused,
                                           char* lds, char** rowptr, int* flag, Claim* cl) {
  const int tid = threadIdx.x;
  const uint64_t t0 = a.tr.buf ? wall_ticks() : 0;
  if (fused && !ep_wait_row(a, p, flag)) return;
  const uint64_t t_dep = a.tr.buf ? wall_ticks() : 0;
  const uint64_t stw = staging_wait(a);
  const int x = a.row_expert[p];
  const int e = a.e_begin + x;
  int m0, rows;
  expert_block(a, x, p, true, m0, rows);
  const uint16_t* A = a.h + static_cast<int64_t>(a.exp_hrow[x] + m0) * a.I;
  const uint16_t* B = a.w2 + static_cast<int64_t>(x) * a.H * a.I;
  const int n0 = nt * kBN;
  // the destination of this thread's output row, loaded before the mainloop so that its
  // latency is hidden behind the MFMAs
  int code = -1;
  if (a.l2_combine && tid < rows)
    code = a.row_src[static_cast<int64_t>(e / a.epw) * a.cap + a.expert_offsets[e] + m0 + tid];
  Acc acc;
  gemm_mainloop<true>(A, a.I, rows, B, a.I, n0, 0, false, a.I, acc, lds);
  claim_load(a, cl);
  const uint64_t t1 = a.tr.buf ? wall_ticks() : 0;
  if (tid < rows) {
    char* ptr;
    if (a.l2_combine) {
      const int src = code >> 24, slot = code & 0xffffff;
      if (code >= 0 && src < a.n_src && slot < a.tk) {
        ptr = a.cwin.base[src] + static_cast<int64_t>(slot) * a.cwin.stride[src] +
              static_cast<int64_t>(n0) * 2;
      } else {
        ptr = nullptr;   // a row the layout never assigned (bad routing input): not stored
        set_status(a.status, XS_EBADINPUT);
      }
    } else {
      ptr = reinterpret_cast<char*>(a.y + static_cast<int64_t>(a.exp_hrow[x] + m0 + tid) * a.H + n0);
    }
    rowptr[tid] = ptr;
  }
  stage_tile(acc, lds);
  __syncthreads();
  claim_take(a, cl);
  store_rows(lds, kEpiPitch, kBN, rows, rowptr);
  // The combine rows are read only after the kernel (window signal, combine-reduce): the
  // stores drain while the next tile runs.
  lds_barrier();
  if (tid == 0) {
    if (a.tr.buf)
      trace_tile(a, 2, static_cast<uint32_t>(p * a.P2 + nt), t0, t1, wall_ticks(), t_dep, stw,
                 static_cast<uint64_t>(rows) * kBN * 2, rows);
    spin_ticks(static_cast<uint64_t>(a.gap_ticks));   // non-injecting gap after the burst
  }
  if (a.gap_ticks) __syncthreads();
}

__device__ __forceinline__ int xcd_instance_ep(int b, int G) {
  return (G % 8) ? b : (b % 8) * (G / 8) + b / 8;
}

// MX tiles (256 threads, the MX core); BF4: the weights are packed E2M1 (W4A8), else E4M3.
// Weight scales are grouped by 512 K elements ([K / 512][n_experts * rows][16 bytes]), so a
// quarter of a scale group is one contiguous run of rows. Linear-1: the dispatch window rows
// hold H codes then H / 32 scales; the SwiGLU output is quantized in the epilogue into h code
// rows of I bytes (this tile's 128 columns at 128 nt) and one scale word per row into the h
// scale groups (group nt / 4, word nt % 4).
template <bool BF4>
__device__ __forceinline__ void ep_l1_tile_mx(const EpArgs& a, int p, int nt, bool fused, char* lds,
                                              char** rowptr, Claim* cl) {
  const int x = a.row_expert[p];
  const int e = a.e_begin + x;
  const int dl = e / a.epw - a.d_first;
  int m0, rows;
  expert_block(a, x, p, false, m0, rows);
  const uint64_t t0 = a.tr.buf ? wall_ticks() : 0;
  const uint64_t stw = staging_wait(a);
  const int64_t ws = a.dwin.stride[dl];
  const uint8_t* A = reinterpret_cast<const uint8_t*>(a.dwin.base[dl] +
                                                      static_cast<int64_t>(a.expert_offsets[e] + m0) * ws);
  const int64_t wrows = static_cast<int64_t>(x) * 2 * a.I;
  const int64_t ldb = BF4 ? a.H / 2 : a.H;
  const uint8_t* B = reinterpret_cast<const uint8_t*>(a.w1) + wrows * ldb;
  const uint8_t* Bs = a.w1s + wrows * 16;
  AccMx acc;
  gemm_mainloop_mx<BF4>(A, ws, A + a.H, ws, 16, rows, B, ldb, Bs, 16, static_cast<int64_t>(a.n_experts) * 2 * a.I * 16,
                        nt * (kBN / 2), a.I, true, a.H, acc, lds);
  claim_load(a, cl);
  const uint64_t t1 = a.tr.buf ? wall_ticks() : 0;
  const int tid = tid_here();   // not held across the mainloop
  const int64_t hrow0 = static_cast<int64_t>(a.exp_hrow[x] + m0);
  if (tid < rows) rowptr[tid] = reinterpret_cast<char*>(a.h) + (hrow0 + tid) * a.h_stride;
  stage_swiglu_mxq(acc, lds);
  __syncthreads();
  claim_take(a, cl);
  typedef __attribute__((address_space(1))) u32x4 global_u32x4;
  // four rows' LDS reads in flight before their stores
  constexpr int kRowsPerPass = kMxThreads / 8;
#pragma unroll 1
  for (int r = tid >> 3; r < rows; r += 4 * kRowsPerPass) {
    const int pc = tid & 7;
    char* dst[4];
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ru = r + u * kRowsPerPass;
      dst[u] = nullptr;
      if (ru < rows) {
        dst[u] = rowptr[ru];
        v[u] = *reinterpret_cast<const u32x4*>(lds + ru * kHqPitch + pc * 16);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (dst[u]) *(global_u32x4*)(dst[u] + nt * 128 + pc * 16) = v[u];
  }
  if (tid < rows)
    *(__attribute__((address_space(1))) uint32_t*)(a.hs + ((nt >> 2) * a.h_rows + hrow0 + tid) * 16 + (nt & 3) * 4) =
        *reinterpret_cast<const uint32_t*>(lds + kHqScaleOff + tid * 4);
  if (fused) {
    __syncthreads();
    if (tid == 0 && p != a.withhold_row)
      __hip_atomic_fetch_add(&a.l1_done[p], 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    lds_barrier();
  }
  if (a.tr.buf && tid == 0)
    trace_tile(a, 1, static_cast<uint32_t>(p * a.P1 + nt), t0, t1, wall_ticks(), t0, stw,
               static_cast<uint64_t>(rows) * (128 + 4), rows);
}

// Linear-2 on MXFP8 h rows; bf16 output rows into the combine windows as in the bf16 tile.
template <bool BF4>
__device__ __forceinline__ void ep_l2_tile_mx(const EpArgs& a, int p, int nt, bool fused, char* lds,
                                              char** rowptr, int* flag, Claim* cl) {
  const uint64_t t0 = a.tr.buf ? wall_ticks() : 0;
  if (fused && !ep_wait_row(a, p, flag)) return;
  const uint64_t t_dep = a.tr.buf ? wall_ticks() : 0;
  const uint64_t stw = staging_wait(a);
  const int x = a.row_expert[p];
  const int e = a.e_begin + x;
  int m0, rows;
  expert_block(a, x, p, false, m0, rows);
  const int64_t hrow0 = static_cast<int64_t>(a.exp_hrow[x] + m0);
  const uint8_t* A = reinterpret_cast<const uint8_t*>(a.h) + hrow0 * a.h_stride;
  const uint8_t* As = a.hs + hrow0 * 16;
  const int64_t wrows = static_cast<int64_t>(x) * a.H;
  const int64_t ldb = BF4 ? a.I / 2 : a.I;
  const uint8_t* B = reinterpret_cast<const uint8_t*>(a.w2) + wrows * ldb;
  const uint8_t* Bs = a.w2s + wrows * 16;
  const int n0 = nt * kBN;
  int code = -1;
  if (a.l2_combine && static_cast<int>(threadIdx.x) < rows)
    code = a.row_src[static_cast<int64_t>(e / a.epw) * a.cap + a.expert_offsets[e] + m0 + threadIdx.x];
  AccMx acc;
  gemm_mainloop_mx<BF4>(A, a.h_stride, As, 16, a.h_rows * 16, rows, B, ldb, Bs, 16,
                        static_cast<int64_t>(a.n_experts) * a.H * 16, n0, 0, false, a.I, acc, lds);
  claim_load(a, cl);
  const uint64_t t1 = a.tr.buf ? wall_ticks() : 0;
  const int tid = tid_here();   // not held across the mainloop
  if (tid < rows) {
    char* ptr = nullptr;
    const int src = code >> 24, slot = code & 0xffffff;
    if (code >= 0 && src < a.n_src && slot < a.tk)
      ptr = a.cwin.base[src] + static_cast<int64_t>(slot) * a.cwin.stride[src] + static_cast<int64_t>(n0) * 2;
    else
      set_status(a.status, XS_EBADINPUT);
    rowptr[tid] = ptr;
  }
  stage_tile_mx(acc, lds);
  __syncthreads();
  claim_take(a, cl);
  store_rows_n<kMxThreads>(lds, kEpiPitch * 2, kBN * 2 / 16, rows, rowptr);
  lds_barrier();
  if (tid == 0) {
    if (a.tr.buf)
      trace_tile(a, 2, static_cast<uint32_t>(p * a.P2 + nt), t0, t1, wall_ticks(), t_dep, stw,
                 static_cast<uint64_t>(rows) * kBN * 2, rows);
    spin_ticks(static_cast<uint64_t>(a.gap_ticks));
  }
  if (a.gap_ticks) __syncthreads();
}

// Tile dispatch by precision (PREC 0: bf16, 1: MXFP8, 2: W4A8).
template <int PREC>
__device__ __forceinline__ void l1_tile(const EpArgs& a, int p, int nt, bool fused, char* lds, char** rowptr,
                                        Claim* cl = nullptr) {
  if constexpr (PREC > 0) ep_l1_tile_mx<PREC == 2>(a, p, nt, fused, lds, rowptr, cl);
  else ep_l1_tile(a, p, nt, fused, lds, rowptr, cl);
}
template <int PREC>
__device__ __forceinline__ void l2_tile(const EpArgs& a, int p, int nt, bool fused, char* lds, char** rowptr,
                                        int* flag, Claim* cl = nullptr) {
  if constexpr (PREC > 0) ep_l2_tile_mx<PREC == 2>(a, p, nt, fused, lds, rowptr, flag, cl);
  else ep_l2_tile(a, p, nt, fused, lds, rowptr, flag, cl);
}

// Dynamic claiming. Thread 0 takes the next tile and broadcasts it through LDS:
//   > 0: Linear-1 entry (value - 1), < -1: Linear-2 entry (-value - 2), -1: no work left.
// Linear-2 entries are taken as tickets (one fetch_add, no retry loop): a producer holds at
// most one ticket and runs it only once its row p satisfies p + D <= (first untaken
// Linear-1 row); until then it keeps taking Linear-1 tiles itself. So every Linear-1 tile a
// Linear-2 tile waits on has an owner that runs it without waiting, and the holder of an
// early ticket advances the Linear-1 frontier it waits for. The ticket is taken when the
// shared Linear-2 counter's next entry is already eligible, so tickets are rarely held long.
__device__ __forceinline__ int ep_claim(const EpArgs& a, Claim& cl) {
  int* c1p = a.claim_ctr;
  int* c2p = a.claim_ctr + 1;
  const int n1 = cl.n1, n2 = cl.n2;
  int& run = cl.run;
  int& ticket = cl.ticket;
  for (;;) {
    const int c1 = __hip_atomic_load(c1p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (ticket == -1) {
      const int c2 = __hip_atomic_load(c2p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (c2 >= n2) {
        ticket = -2;   // Linear-2 entries exhausted
      } else if (l2_may_run(a, c2, c1, n1, run)) {
        const int k = __hip_atomic_fetch_add(c2p, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ticket = k < n2 ? k : -2;
      }
    }
    if (ticket >= 0 && l2_may_run(a, ticket, c1, n1, run)) {
      const int k = ticket;
      ticket = -1;
      ++run;
      return -k - 2;
    }
    if (c1 < n1) {
      const int k = __hip_atomic_fetch_add(c1p, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (k < n1) {
        run = 0;
        return k + 1;
      }
      continue;   // Linear-1 exhausted meanwhile: every held ticket is now eligible
    }
    if (ticket == -2) return -1;
    // Linear-1 exhausted, no ticket yet (chunk_ok holds): the loop takes one above
  }
}

// The next tile: what claim_take settled or started during the last epilogue, else ep_claim.
__device__ __forceinline__ int claim_next(const EpArgs& a, Claim& cl) {
  const int kind = cl.kind;
  cl.kind = 0;
  if (kind == 3) return cl.k;
  if (kind == 2) {
    if (cl.k < cl.n2 && l2_may_run(a, cl.k, cl.c1, cl.n1, cl.run)) {
      ++cl.run;
      return -cl.k - 2;
    }
    cl.ticket = cl.k < cl.n2 ? cl.k : -2;
  } else if (kind == 1 && cl.k < cl.n1) {
    cl.run = 0;
    return cl.k + 1;
  }
  return ep_claim(a, cl);
}

template <int MODE, int PREC>
__device__ __forceinline__ void ep_dynamic(const EpArgs& a, int n1, int n2, char* lds, char** rowptr,
                                           int* flag) {
  constexpr bool fused = MODE == 3;
  Claim cl{fused ? 1 : 0, n1, n2, 0, n2 > 0 ? -1 : -2, 0, 0, 0, 0};   // thread 0 only
  if (fused && a.policy == XS_POLICY_BURST) {
    const int nw = a.meta[1], total = a.meta[2];
    for (;;) {
      if (threadIdx.x == 0)
        flag[1] = __hip_atomic_fetch_add(a.claim_ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __syncthreads();
      const int pos = flag[1];
      __syncthreads();
      if (pos >= total) return;
      int w = 0;
      while (w + 1 < nw && a.wave_pos[w + 1] <= pos) ++w;
      const int off = pos - a.wave_pos[w];
      const int r0 = a.wave_row[w], nl1 = (a.wave_row[w + 1] - r0) * a.P1;
      if (off < nl1) {
        const int k1 = r0 * a.P1 + off;
        l1_tile<PREC>(a, k1 / a.P1, k1 % a.P1, true, lds, rowptr);
      } else {
        const int k2 = r0 * a.P2 + (off - nl1);
        l2_tile<PREC>(a, k2 / a.P2, k2 % a.P2, true, lds, rowptr, flag);
      }
    }
  }
  for (;;) {
    if (threadIdx.x == 0) flag[1] = claim_next(a, cl);
    __syncthreads();
    const int t = flag[1];
    __syncthreads();
    if (t == -1) return;
    if (t > 0) {
      const int k1 = t - 1;
      l1_tile<PREC>(a, k1 / a.P1, k1 % a.P1, fused, lds, rowptr, &cl);
    } else {
      const int k2 = -t - 2;
      l2_tile<PREC>(a, k2 / a.P2, k2 % a.P2, fused, lds, rowptr, flag, &cl);
    }
  }
}

// MODE 3: fused Linear-1 + Linear-2 (the EP layer); 1 / 2: one GEMM stream only (unfused
// expert FFN). A template parameter so each variant is its own kernel in a trace.
template <int MODE, int PREC>
__device__ __forceinline__ void ep_ffn_body(const EpArgs& a, char* smem) {
  char* lds = smem;
  char** rowptr = reinterpret_cast<char**>(smem + kLdsRowPtrOff);
  int* flag = reinterpret_cast<int*>(smem + kLdsMiscOff);
  const int P = a.meta[0];
  const int G = gridDim.x;
  const int g = xcd_instance_ep(blockIdx.x, G);
  constexpr bool fused = MODE == 3;
  const int n1 = (MODE & 1) ? P * a.P1 : 0;
  const int n2 = (MODE & 2) ? P * a.P2 : 0;
  if (fused && a.policy == XS_POLICY_BURST) {
    const int nw = a.meta[1], total = a.meta[2];
    int w = 0;
    for (int pos = g; pos < total; pos += G) {
      while (w + 1 < nw && a.wave_pos[w + 1] <= pos) ++w;
      const int off = pos - a.wave_pos[w];
      const int r0 = a.wave_row[w], nl1 = (a.wave_row[w + 1] - r0) * a.P1;
      if (off < nl1) {
        const int k1 = r0 * a.P1 + off;
        l1_tile<PREC>(a, k1 / a.P1, k1 % a.P1, true, lds, rowptr);
      } else {
        const int k2 = r0 * a.P2 + (off - nl1);
        l2_tile<PREC>(a, k2 / a.P2, k2 % a.P2, true, lds, rowptr, flag);
      }
    }
    return;
  }
  if (a.claim == XS_CLAIM_DYNAMIC) {
    ep_dynamic<MODE, PREC>(a, n1, n2, lds, rowptr, flag);
    return;
  }
  // Static claiming: this instance owns entries g, g + G, ... of each stream and applies the
  // claim rule to its own next entries (its own Linear-1 entries play the part of the shared
  // frontier). An owned Linear-2 entry then only waits on rows whose Linear-1 tiles every
  // instance has already passed, so with D >= 1 the lowest waited-on row always has running
  // owners.
  int e1 = g, e2 = g, run = 0;
  for (;;) {
    if (e2 < n2 && l2_may_run(a, e2, e1, n1, run)) {
      l2_tile<PREC>(a, e2 / a.P2, e2 % a.P2, fused, lds, rowptr, flag);
      e2 += G;
      ++run;
    } else if (e1 < n1) {
      l1_tile<PREC>(a, e1 / a.P1, e1 % a.P1, fused, lds, rowptr);
      e1 += G;
      run = 0;
    } else {
      break;
    }
  }
}

template <int MODE>
__global__ __launch_bounds__(kThreads, 1) void ep_ffn_kernel(EpArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBytes];
  ep_ffn_body<MODE, 0>(a, smem);
}

// The same schedule with MXFP8 tiles on the four-wave MX core.
template <int MODE>
__global__ __launch_bounds__(kMxThreads, 1) void ep_ffn_mx_kernel(EpArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBytes];
  ep_ffn_body<MODE, 1>(a, smem);
}

// The same with E2M1 weights (W4A8).
template <int MODE>
__global__ __launch_bounds__(kMxThreads, 1) void ep_ffn_w4a8_kernel(EpArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBytes];
  ep_ffn_body<MODE, 2>(a, smem);
}

// Prefix of the rows each computed window holds (rows past capacity were never stored).
__device__ __forceinline__ int window_prefix(const EpArgs& a, const int* dest_counts, int n_cwin,
                                             int* base) {
  if (threadIdx.x == 0) {
    base[0] = 0;
    for (int d = 0; d < n_cwin; ++d) base[d + 1] = base[d] + min(dest_counts[a.d_first + d], a.cap);
  }
  __syncthreads();
  return base[n_cwin];
}

__device__ __forceinline__ char* combine_row(const EpArgs& a, int dl, int r) {
  const int code = a.row_src[static_cast<int64_t>(a.d_first + dl) * a.cap + r];
  const int s = code >> 24, slot = code & 0xffffff;
  if (code < 0 || s >= a.n_src || slot >= a.tk) {
    set_status(a.status, XS_EBADINPUT);
    return nullptr;
  }
  return a.cwin.base[s] + static_cast<int64_t>(slot) * a.cwin.stride[s];
}

// Identity experts: y = x, i.e. the computed window rows are copied to y (unfused) or
// stored straight into the combine windows. One wave per computed row.
__global__ __launch_bounds__(256) void ep_identity_kernel(EpArgs a, const int* __restrict__ dest_counts,
                                                          int n_cwin, int to_combine) {
  __shared__ int base[XS_MAX_WINDOWS + 1];
  const int lane = threadIdx.x & 63;
  const int total = window_prefix(a, dest_counts, n_cwin, base);
  for (int gr = blockIdx.x * 4 + (threadIdx.x >> 6); gr < total; gr += gridDim.x * 4) {
    int dl = 0;
    while (base[dl + 1] <= gr) ++dl;
    const int r = gr - base[dl];
    const u32x4* src = reinterpret_cast<const u32x4*>(a.dwin.base[dl] + static_cast<int64_t>(r) * a.dwin.stride[dl]);
    u32x4* dst = reinterpret_cast<u32x4*>(to_combine ? combine_row(a, dl, r)
                                                     : reinterpret_cast<char*>(a.y + static_cast<int64_t>(gr) * a.H));
    if (!dst) continue;
    for (int pc = lane; pc < a.H / 8; pc += 64) dst[pc] = src[pc];
  }
}

// Unfused combine-send: computed row -> combine window of its source. Each workgroup is one
// producer issuing bursts of `burst_rows` consecutive computed rows (burst b of producer g is
// rows [(g + b G) burst_rows, ... + burst_rows)), optionally followed by a non-injecting gap.
// A wave copies two rows at a time, 8 16-byte pieces of each per lane in flight before their
// stores; the rows and their destinations are wave-uniform.
__global__ __launch_bounds__(256) void ep_combine_send_kernel(EpArgs a, const int* __restrict__ dest_counts,
                                                              int n_cwin, int burst_rows) {
  __shared__ int base[XS_MAX_WINDOWS + 1];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int total = window_prefix(a, dest_counts, n_cwin, base);
  const int npc = a.H / 8;   // 16-byte pieces per row
  for (int b0 = blockIdx.x * burst_rows; b0 < total; b0 += gridDim.x * burst_rows) {
    const int b1 = min(total, b0 + burst_rows);
    for (int gr = b0 + 2 * wv; gr < b1; gr += 8) {
      u32x4* dst[2];
      const u32x4* src[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int r = gr + q;
        dst[q] = nullptr;
        src[q] = nullptr;
        if (r < b1) {
          int dl = 0;
          while (base[dl + 1] <= r) ++dl;
          dst[q] = reinterpret_cast<u32x4*>(combine_row(a, dl, r - base[dl]));
          src[q] = reinterpret_cast<const u32x4*>(a.y + static_cast<int64_t>(r) * a.H);
        }
      }
      for (int p0 = 0; p0 < npc; p0 += 8 * 64) {
        u32x4 v[2][8];
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int pc = p0 + u * 64 + lane;
            if (dst[q] && pc < npc) v[q][u] = src[q][pc];
          }
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int pc = p0 + u * 64 + lane;
            if (dst[q] && pc < npc) dst[q][pc] = v[q][u];
          }
      }
    }
    if (a.gap_ticks) {
      __syncthreads();
      if (threadIdx.x == 0) spin_ticks(static_cast<uint64_t>(a.gap_ticks));
      __syncthreads();
    }
  }
}

}  // namespace xs

using namespace xs;

namespace xs_host {
int dispatch_layout(const int32_t*, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t*,
                    int32_t*, int32_t*, int32_t*, int32_t*, int32_t*, void*, int64_t, int32_t*,
                    hipStream_t, const PlanArgs*);
int dispatch_rows(const void*, int64_t, int32_t, int32_t, const int32_t*, const int32_t*, int32_t,
                  int32_t, const WinSet&, int32_t*, hipStream_t, const FinArgs*);
int dispatch(const void*, int32_t, int32_t, const int32_t*, const int32_t*, int32_t, int32_t,
             const WinSet&, int32_t*, hipStream_t);
int combine_reduce(const void*, int64_t, const float*, int32_t, int32_t, int32_t, void*,
                   hipStream_t);
int signal_windows(const WinSet&, hipStream_t);
int persistent_grid(int max_producers);
}  // namespace xs_host

namespace {

constexpr int64_t kAlign = 256;
int64_t align_up(int64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct EpWorkspace {
  int64_t layout_off, layout_bytes;
  int64_t meta_off, exp_off, rowexp_off, wave_pos_off, wave_row_off, l1_off;
  int64_t xq_off;              // MXFP8: quantized token rows of this source [T][H + H / 32]
  int64_t total;
  int64_t max_rows;
};

bool is_mx(const xs_ep_layer* L) { return L->precision == XS_PREC_MXFP8 || L->precision == XS_PREC_W4A8; }

// Bytes of one dispatched token row, and of one h code row. MX h holds I-byte code rows
// (whole 128-byte lines, as I is a multiple of 512) followed by the scale groups.
int64_t token_row_bytes(const xs_ep_layer* L) {
  return is_mx(L) ? static_cast<int64_t>(L->H) + L->H / 32 : static_cast<int64_t>(L->H) * 2;
}
int64_t h_row_bytes(const xs_ep_layer* L) {
  return is_mx(L) ? static_cast<int64_t>(L->I) : static_cast<int64_t>(L->I) * 2;
}

int n_cwin_of(const xs_ep_layer* L) { return L->n_experts / (L->E / L->W); }

EpWorkspace ep_workspace(const xs_ep_layer* L) {
  EpWorkspace w{};
  const int64_t n_chunks = (static_cast<int64_t>(L->T) + 255) / 256;
  w.layout_off = 0;
  // the chunk counts and the scan's completion count (xs_dispatch_layout_workspace_bytes)
  w.layout_bytes = align_up(static_cast<int64_t>(L->n_src) * n_chunks * L->E * 4) + 256;
  const int64_t max_rows = static_cast<int64_t>(n_cwin_of(L)) * L->cap / kBM + L->n_experts + 1;
  w.max_rows = max_rows;
  int64_t o = w.layout_bytes;
  w.meta_off = o;
  o += align_up(16 * 4);
  w.exp_off = o;
  o += align_up(4LL * L->n_experts * 4);
  w.rowexp_off = o;
  o += align_up(max_rows * 4);
  w.wave_pos_off = o;
  o += align_up((max_rows + 2) * 4);
  w.wave_row_off = o;
  o += align_up((max_rows + 2) * 4);
  w.l1_off = o;
  o += align_up(max_rows * 4);
  w.xq_off = o;
  if (is_mx(L)) o += align_up(static_cast<int64_t>(L->T) * token_row_bytes(L));
  w.total = o;
  return w;
}

int validate(const xs_ep_layer* L, bool need_out) {
  if (!L) return XS_EINVAL;
  if (L->n_src < 1 || L->n_src > 127 || L->T < 0 || L->H < 8 || L->E < 1 || L->E > 1024 ||
      L->k < 1 || L->k > L->E || L->k > 32 || L->W < 1 || L->W > XS_MAX_WINDOWS || L->E % L->W ||
      L->src < 0 || L->src >= L->n_src || L->cap < 0)
    return XS_EINVAL;
  const int epw = L->E / L->W;
  if (L->n_experts < 1 || L->e_begin < 0 || L->e_begin % epw || L->n_experts % epw ||
      L->e_begin + L->n_experts > L->E || L->n_experts > 1024)
    return XS_EINVAL;
  if (static_cast<int64_t>(L->T) * L->k >= (1 << 24)) return XS_EINVAL;
  if (!L->topk_idx || !L->topk_w || !L->expert_counts || !L->src_base || !L->expert_offsets ||
      !L->dest_counts || !L->slot_row || !L->row_src || !L->dispatch_win || !L->combine_win)
    return XS_EINVAL;
  if (need_out && (!L->x || !L->logits || !L->out)) return XS_EINVAL;
  if (L->expert_mode != XS_EXPERT_SWIGLU && L->expert_mode != XS_EXPERT_IDENTITY) return XS_EINVAL;
  if (L->precision != XS_PREC_BF16 && L->precision != XS_PREC_MXFP8 && L->precision != XS_PREC_W4A8)
    return XS_EINVAL;
  if (L->reserved != 0) return XS_EINVAL;
  if (is_mx(L)) {
    if (L->expert_mode != XS_EXPERT_SWIGLU) return XS_EUNSUPPORTED;
    if (!L->w1_scale || !L->w2_scale) return XS_EINVAL;
    // 16-byte code and scale rows (the GEMM core loads four K stages of scales at once), whole
    // 256 x 256 tiles along H, 128-column SwiGLU tiles and 512-deep scale groups along I
    if (L->H % 512 || L->I % 512) return XS_EUNSUPPORTED;
    if ((reinterpret_cast<uintptr_t>(L->w1) | reinterpret_cast<uintptr_t>(L->w2) |
         reinterpret_cast<uintptr_t>(L->h_ws) | reinterpret_cast<uintptr_t>(L->w1_scale) |
         reinterpret_cast<uintptr_t>(L->w2_scale)) & 15)
      return XS_EINVAL;
  }
  if (L->H % 8) return XS_EUNSUPPORTED;
  if (L->expert_mode == XS_EXPERT_SWIGLU) {
    if (!L->w1 || !L->w2 || !L->h_ws || L->I < 1) return XS_EINVAL;
    if (L->H % kBN || L->I % (kBN / 2) || L->I % kBK) return XS_EUNSUPPORTED;
    if (L->h_rows < static_cast<int64_t>(n_cwin_of(L)) * L->cap) return XS_EINVAL;
  }
  return XS_OK;
}

int fill_args(const xs_ep_layer* L, void* workspace, EpArgs* a, WinSet* dws, WinSet* cws) {
  int rc = xs_host::make_winset(L->dispatch_win, L->W, token_row_bytes(L), dws);
  if (rc) return rc;
  for (int d = 0; d < L->W; ++d)
    if (dws->cap[d] < L->cap) return XS_EINVAL;
  rc = xs_host::make_winset(L->combine_win, L->n_src, static_cast<int64_t>(L->H) * 2, cws);
  if (rc) return rc;
  for (int s = 0; s < L->n_src; ++s)
    if (cws->cap[s] < static_cast<int64_t>(L->T) * L->k) return XS_EINVAL;
  const EpWorkspace w = ep_workspace(L);
  char* ws = static_cast<char*>(workspace);
  *a = EpArgs{};
  a->E = L->E;
  a->epw = L->E / L->W;
  a->H = L->H;
  a->I = L->I;
  a->e_begin = L->e_begin;
  a->n_experts = L->n_experts;
  a->cap = L->cap;
  a->n_src = L->n_src;
  a->tk = L->T * L->k;
  a->d_first = L->e_begin / a->epw;
  a->P1 = L->I / (kBN / 2);
  a->P2 = L->H / kBN;
  for (int d = 0; d < n_cwin_of(L); ++d) {
    a->dwin.base[d] = dws->base[a->d_first + d];
    a->dwin.stride[d] = dws->stride[a->d_first + d];
  }
  for (int s = 0; s < L->n_src; ++s) {
    a->cwin.base[s] = cws->base[s];
    a->cwin.stride[s] = cws->stride[s];
  }
  a->expert_offsets = L->expert_offsets;
  a->row_src = L->row_src;
  a->w1 = static_cast<const uint16_t*>(L->w1);
  a->w2 = static_cast<const uint16_t*>(L->w2);
  a->h = static_cast<uint16_t*>(L->h_ws);
  a->y = static_cast<uint16_t*>(L->y_ws);
  a->w1s = static_cast<const uint8_t*>(L->w1_scale);
  a->w2s = static_cast<const uint8_t*>(L->w2_scale);
  a->h_stride = h_row_bytes(L);
  a->h_rows = L->h_rows;
  a->hs = is_mx(L) ? static_cast<uint8_t*>(L->h_ws) + L->h_rows * static_cast<int64_t>(L->I) : nullptr;
  int* meta = reinterpret_cast<int*>(ws + w.meta_off);
  int* exp = reinterpret_cast<int*>(ws + w.exp_off);
  a->meta = meta;
  a->exp_m = exp;
  a->exp_rowfirst = exp + L->n_experts;
  a->exp_hrow = exp + 2 * L->n_experts;
  a->row_expert = reinterpret_cast<int*>(ws + w.rowexp_off);
  a->wave_pos = reinterpret_cast<int*>(ws + w.wave_pos_off);
  a->wave_row = reinterpret_cast<int*>(ws + w.wave_row_off);
  a->l1_done = reinterpret_cast<int*>(ws + w.l1_off);
  a->claim_ctr = meta + 8;
  a->withhold_row = -1;
  a->lead = 1;
  return XS_OK;
}

PlanArgs plan_args(const xs_ep_layer* L, const EpArgs& a, int wave_tiles) {
  return PlanArgs{L->e_begin, L->n_experts, L->cap, a.P1, a.P2, wave_tiles,
                  const_cast<int*>(a.meta), const_cast<int*>(a.row_expert),
                  const_cast<int*>(a.exp_m), const_cast<int*>(a.exp_rowfirst),
                  const_cast<int*>(a.exp_hrow), const_cast<int*>(a.wave_pos),
                  const_cast<int*>(a.wave_row), a.l1_done};
}

int launch_plan(const xs_ep_layer* L, const EpArgs& a, int wave_tiles, hipStream_t st) {
  hipLaunchKernelGGL(ep_plan_kernel, dim3(1), dim3(1024), 0, st, L->expert_counts, L->n_src, L->E,
                     L->expert_offsets, plan_args(L, a, wave_tiles));
  return xs_host::launch_status();
}

}  // namespace

// Records the phase event `i` of the layer descriptor, if the caller set one.
static int record_event(const xs_ep_layer* L, int i, hipStream_t st) {
  if (!L->events[i]) return XS_OK;
  return hipEventRecord(static_cast<hipEvent_t>(L->events[i]), st) == hipSuccess ? XS_OK : XS_EHIP;
}

extern "C" int xs_ep_layer_workspace_bytes(const xs_ep_layer* L, int64_t* bytes) {
  if (!L || !bytes || L->n_src < 1 || L->T < 0 || L->E < 1 || L->W < 1 || L->E % L->W ||
      L->n_experts < 1 || L->cap < 0)
    return XS_EINVAL;
  *bytes = ep_workspace(L).total;
  return XS_OK;
}

static int run_ffn(const xs_ep_layer* L, const EpArgs& base, int mode, int l2_combine,
                   const xs_pacing* pc, const xs_trace* trace, int32_t* dev_status, hipStream_t st) {
  EpArgs a = base;
  a.l2_combine = l2_combine;
  a.status = dev_status;
  a.tr = xs_trace{nullptr, 0, nullptr};
  if (trace && trace->buf && trace->count) a.tr = *trace;
  int grid = xs_host::persistent_grid(pc ? pc->max_producers : 0);
  a.policy = pc ? pc->policy : XS_POLICY_INTERLEAVE;
  // lead 0 = the anti-starvation knee of App. A.2, ceil(b_n K / (2 I)) = ceil(G / P1) rows:
  // one round of Linear-1 tiles over all producers
  a.lead = pc && pc->lead_rows > 0 ? pc->lead_rows : (grid + a.P1 - 1) / a.P1;
  a.chunk = pc ? pc->chunk_tiles : 0;
  if (a.policy == XS_POLICY_INTERLEAVE) a.chunk = 0;
  if (a.policy == XS_POLICY_AUTO) {
    // the audited choice (xs_pacing_audit_run); plain interleave without a model
    xs_pacing_audit au;
    if (pc->model && xs_pacing_audit_run(L, pc, &au) == XS_OK) {
      a.policy = au.policy;
      a.chunk = au.chunk;
    } else {
      a.policy = XS_POLICY_INTERLEAVE;
      a.chunk = 0;
    }
  }
  a.withhold_row = pc ? pc->withhold_row : -1;
  a.claim = pc ? pc->claim : XS_CLAIM_STATIC;
  a.gap_ticks = pc ? xs_host::ns_to_ticks(pc->gap_ns) : 0;
  const int64_t tmo_us = pc && pc->spin_timeout_us > 0 ? pc->spin_timeout_us : 2000000;
  a.timeout_ticks = xs_host::ns_to_ticks(tmo_us * 1000);
  if (L->precision == XS_PREC_W4A8)
    hipLaunchKernelGGL(ep_ffn_w4a8_kernel<3>, dim3(grid), dim3(kMxThreads), 0, st, a);
  else if (is_mx(L))
    hipLaunchKernelGGL(ep_ffn_mx_kernel<3>, dim3(grid), dim3(kMxThreads), 0, st, a);
  else if (mode == 1)
    hipLaunchKernelGGL(ep_ffn_kernel<1>, dim3(grid), dim3(kThreads), 0, st, a);
  else if (mode == 2)
    hipLaunchKernelGGL(ep_ffn_kernel<2>, dim3(grid), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(ep_ffn_kernel<3>, dim3(grid), dim3(kThreads), 0, st, a);
  return xs_host::launch_status();
}

extern "C" int xs_expert_ffn(const xs_ep_layer* L, void* workspace, int64_t workspace_bytes,
                             int32_t* dev_status, void* stream) {
  int rc = validate(L, false);
  if (rc) return rc;
  if (is_mx(L)) return XS_EUNSUPPORTED;
  if (!L->y_ws) return XS_EINVAL;
  if (!workspace || workspace_bytes < ep_workspace(L).total) return XS_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  EpArgs a;
  WinSet dws, cws;
  rc = fill_args(L, workspace, &a, &dws, &cws);
  if (rc) return rc;
  a.status = dev_status;
  if (L->expert_mode == XS_EXPERT_IDENTITY) {
    hipLaunchKernelGGL(ep_identity_kernel, dim3(2048), dim3(256), 0, st, a, L->dest_counts,
                       n_cwin_of(L), 0);
    return xs_host::launch_status();
  }
  if ((rc = record_event(L, XS_EV_PLAN, st))) return rc;
  rc = launch_plan(L, a, 0, st);
  if (rc) return rc;
  if ((rc = record_event(L, XS_EV_FFN, st))) return rc;
  rc = run_ffn(L, a, 1, 0, nullptr, nullptr, dev_status, st);
  if (rc) return rc;
  rc = run_ffn(L, a, 2, 0, nullptr, nullptr, dev_status, st);
  if (rc) return rc;
  return record_event(L, XS_EV_FFN_END, st);
}

extern "C" int xs_combine_send(const xs_ep_layer* L, const xs_pacing* pacing, int32_t* dev_status,
                               void* stream) {
  int rc = validate(L, false);
  if (rc) return rc;
  if (is_mx(L)) return XS_EUNSUPPORTED;
  if (!L->y_ws) return XS_EINVAL;
  if (pacing && (pacing->max_producers < 0 || pacing->chunk_tiles < 0 || pacing->gap_ns < 0 ||
                 pacing->reserved != 0))
    return XS_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  EpArgs a;
  WinSet dws, cws;
  char dummy[256];
  rc = fill_args(L, dummy, &a, &dws, &cws);
  if (rc) return rc;
  a.status = dev_status;
  // producers: max_producers workgroups (default eight per CU); a burst is chunk_tiles blocks of
  // 256 rows, or by default 8 rows (one pass of the workgroup's four waves), so that the rows
  // spread over every wave of the grid rather than over a few workgroups' long row ranges
  const int grid = pacing && pacing->max_producers > 0 ? pacing->max_producers : 8 * xs_host::persistent_grid(0);
  const int burst_rows = pacing && pacing->chunk_tiles > 0 ? pacing->chunk_tiles * kBM : 8;
  a.gap_ticks = pacing ? xs_host::ns_to_ticks(pacing->gap_ns) : 0;
  hipLaunchKernelGGL(ep_combine_send_kernel, dim3(grid), dim3(256), 0, st, a, L->dest_counts,
                     n_cwin_of(L), burst_rows);
  if (xs_host::launch_status()) return XS_EHIP;
  return xs_host::signal_windows(cws, st);
}

static int fused_ep_layer(const xs_ep_layer* L, const xs_pacing* pacing, const xs_trace* trace,
                          void* workspace, int64_t workspace_bytes, int32_t* dev_status, void* stream);

extern "C" int xs_fused_ep_layer(const xs_ep_layer* L, const xs_pacing* pacing,
                                 const xs_trace* trace, void* workspace, int64_t workspace_bytes,
                                 int32_t* dev_status, void* stream) {
  return fused_ep_layer(L, pacing, trace, workspace, workspace_bytes, dev_status, stream);
}

// ------------------------------------------------------------------------------ no-alloc layer
// The layer's scratch for callers that cannot allocate: one library-owned array per GPU. Host
// code never uses the array's name as an address (on the host it names a stand-in, not device
// memory); it uses the device address hipGetSymbolAddress gives, taken once per device with
// that device current and kept in g_scratch.
static __device__ __align__(256) char scratch[XS_STATIC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch[256] = {};
}  // namespace

static int scratch_of_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 256) return XS_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return XS_EHIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return XS_OK;
}

extern "C" int xs_fused_ep_layer_noalloc(const xs_ep_layer* L, const xs_pacing* pacing,
                                         const xs_trace* trace, int32_t* dev_status, void* stream) {
  int64_t need = 0;
  int rc = xs_ep_layer_workspace_bytes(L, &need);
  if (rc) return rc;
  if (need > XS_STATIC_SCRATCH_BYTES) return XS_EWORKSPACE;
  void* ws = nullptr;
  if ((rc = scratch_of_current_device(&ws))) return rc;
  return fused_ep_layer(L, pacing, trace, ws, XS_STATIC_SCRATCH_BYTES, dev_status, stream);
}

static int fused_ep_layer(const xs_ep_layer* L, const xs_pacing* pacing, const xs_trace* trace,
                          void* workspace, int64_t workspace_bytes, int32_t* dev_status, void* stream) {
  int rc = validate(L, true);
  if (rc) return rc;
  if (pacing && (pacing->policy < XS_POLICY_BURST || pacing->policy > XS_POLICY_AUTO ||
                 pacing->lead_rows < 0 || pacing->chunk_tiles < 0 || pacing->max_producers < 0 ||
                 pacing->gap_ns < 0 || pacing->spin_timeout_us < 0 ||
                 (pacing->claim != XS_CLAIM_STATIC && pacing->claim != XS_CLAIM_DYNAMIC) ||
                 pacing->reserved != 0))
    return XS_EINVAL;
  const EpWorkspace w = ep_workspace(L);
  if (!workspace || workspace_bytes < w.total) return XS_EWORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  EpArgs a;
  WinSet dws, cws;
  rc = fill_args(L, workspace, &a, &dws, &cws);
  if (rc) return rc;
  const int64_t n_all = static_cast<int64_t>(L->n_src) * L->T;
  if (n_all > 0x7fffffff) return XS_EINVAL;
  if ((rc = record_event(L, XS_EV_ROUTE, st))) return rc;
  rc = xs_route_topk_softmax(L->logits, static_cast<int32_t>(n_all), L->E, L->k, L->renormalize,
                             L->topk_idx, L->topk_w, stream);
  if (rc) return rc;
  if ((rc = record_event(L, XS_EV_LAYOUT, st))) return rc;
  // The layout's scan launch also plans the expert FFN, and the dispatch launch finishes the
  // layout's rows and signals the dispatch windows (one launch each fewer than the
  // standalone calls, and no plan launch).
  const int grid = xs_host::persistent_grid(pacing ? pacing->max_producers : 0);
  const int wave_tiles = pacing && pacing->wave_tiles > 0 ? pacing->wave_tiles : grid;
  const PlanArgs pa = plan_args(L, a, wave_tiles);
  char* layout_ws = static_cast<char*>(workspace) + w.layout_off;
  rc = xs_host::dispatch_layout(L->topk_idx, L->n_src, L->T, L->k, L->E, L->W, L->cap,
                                L->expert_counts, L->src_base, L->expert_offsets, L->dest_counts,
                                L->slot_row, L->row_src, layout_ws, w.layout_bytes, dev_status, st, &pa);
  if (rc) return rc;
  const int64_t so = static_cast<int64_t>(L->src) * L->T * L->k;
  const FinArgs fin{L->src, L->n_src, L->cap, (L->T + 255) / 256, 0, L->topk_idx, L->slot_row,
                    reinterpret_cast<const int*>(layout_ws), L->src_base, L->expert_offsets, L->row_src,
                    const_cast<int*>(a.meta) + 11};
  if ((rc = record_event(L, XS_EV_DISPATCH, st))) return rc;
  if (is_mx(L)) {
    // quantize this source's token rows once (codes, then scales, in each staged row) and
    // dispatch the staged rows
    const int64_t rb = token_row_bytes(L);
    char* xq = static_cast<char*>(workspace) + w.xq_off;
    rc = xs_quantize_mx(L->x, L->T, L->H, L->H, XS_FMT_E4M3, xq, rb, xq + L->H, rb, stream);
    if (rc) return rc;
    rc = xs_host::dispatch_rows(xq, rb, static_cast<int32_t>(rb), L->T, L->topk_idx + so, L->slot_row + so,
                                L->k, L->E, dws, dev_status, st, &fin);
  } else {
    rc = xs_host::dispatch_rows(L->x, static_cast<int64_t>(L->H) * 2, L->H * 2, L->T, L->topk_idx + so,
                                L->slot_row + so, L->k, L->E, dws, dev_status, st, &fin);
  }
  if (rc) return rc;
  a.status = dev_status;
  if ((rc = record_event(L, XS_EV_PLAN, st))) return rc;
  if (L->expert_mode == XS_EXPERT_IDENTITY) {
    if ((rc = record_event(L, XS_EV_FFN, st))) return rc;
    hipLaunchKernelGGL(ep_identity_kernel, dim3(2048), dim3(256), 0, st, a, L->dest_counts,
                       n_cwin_of(L), 1);
    if (xs_host::launch_status()) return XS_EHIP;
  } else {
    if ((rc = record_event(L, XS_EV_FFN, st))) return rc;
    rc = run_ffn(L, a, 3, 1, pacing, trace, dev_status, st);
    if (rc) return rc;
  }
  if ((rc = record_event(L, XS_EV_FFN_END, st))) return rc;
  rc = xs_host::signal_windows(cws, st);
  if (rc) return rc;
  if ((rc = record_event(L, XS_EV_REDUCE, st))) return rc;
  const xs_window& cw = L->combine_win[L->src];
  rc = xs_host::combine_reduce(cw.base, cw.row_stride_bytes, L->topk_w + so, L->T, L->k, L->H,
                               L->out, st);
  if (rc) return rc;
  return record_event(L, XS_EV_END, st);
}
