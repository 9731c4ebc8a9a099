// Plain GEMM and GEMM with scatter epilogues (tensor-parallel row blocks, Ulysses head
// groups), persistent over 256 x 256 output tiles. The epilogue stores every finished tile
// straight into its destination windows with 128-bit stores; there is no separate
// permutation pass (the serial counterpart, xs_scatter_copy, exists for comparison).
#include <algorithm>

#include "xs_gemm.hpp"

namespace xs {

enum { KIND_PLAIN = 0, KIND_ROW_BLOCK = 1, KIND_HEAD_GROUP = 2 };

struct ScatterArgs {
  int rpd;
  int n_proj, n_heads, head_dim, hpg;
  int group_aligned;   // every 256-column tile lies inside one projection and one head group
  // store pacing: order 0 = the L2-grouped order; 1 = destination-major (Expert-Wave-like
  // bursts: every tile of window 0, then window 1, ...); 2 = `chunk` consecutive tiles of one
  // window, then the next window (chunk 1 = round robin over the windows)
  int order, chunk, n_dest;
  int64_t gap_ticks;   // non-injecting wait after every tile's stores
};

// Tile j of destination d's tiles: a row block's M-tiles walked down then across (ROW_BLOCK),
// or every M-tile of each of the group's column tiles, projection by projection (HEAD_GROUP).
__device__ __forceinline__ void dest_tile(const ScatterArgs& sa, int kind_head, int tm, int d, int j, int* mb,
                                          int* nb) {
  if (!kind_head) {
    const int mpd = sa.rpd / kBM;
    *mb = d * mpd + j % mpd;
    *nb = j / mpd;
  } else {
    const int cpg = sa.hpg * sa.head_dim / kBN;          // column tiles of one group per projection
    const int per_proj = sa.n_heads * sa.head_dim / kBN;
    *mb = j % tm;
    const int rest = j / tm;
    *nb = (rest / cpg) * per_proj + d * cpg + rest % cpg;
  }
}

// Work index -> tile under the pacing order (order 0 handled by grouped_tile).
__device__ __forceinline__ void paced_tile(const ScatterArgs& sa, int kind_head, int w, int tm, int ntiles,
                                           int* mb, int* nb) {
  const int W = sa.n_dest, td = ntiles / W;
  int d, j;
  if (sa.order == 1) {
    d = w / td;
    j = w - d * td;
  } else {
    const int c = sa.chunk, blk = w / (W * c), r = w - blk * W * c;
    d = r / c;
    j = blk * c + (r - d * c);
  }
  dest_tile(sa, kind_head, tm, d, j, mb, nb);
}

// Instance id with consecutive ids on one XCD: workgroups are dealt to the 8 XCDs round
// robin, so block b runs on XCD b % 8.
__device__ __forceinline__ int xcd_instance(int b, int G) {
  return (G % 8) ? b : (b % 8) * (G / 8) + b / 8;
}

// Work index -> output tile, grouped by kGroupM M-tiles: consecutive work indices walk down
// kGroupM tile rows, then across. With 32 instances per XCD taking 32 consecutive work
// indices per round, each XCD's L2 serves a 4 x 8 block of tiles: 4 A row-blocks and 8 B
// column-blocks instead of 1 and 32.
constexpr int kGroupM = 4;
__device__ __forceinline__ void grouped_tile(int w, int tm, int tn, int* mb, int* nb) {
  const int per_group = kGroupM * tn;
  const int g = w / per_group;
  const int first = g * kGroupM;
  const int gm = min(kGroupM, tm - first);
  const int local = w - g * per_group;
  *mb = first + local % gm;
  *nb = local / gm;
}

__device__ __forceinline__ void trace_tile(const xs_trace& tr, int kind, int tile, uint64_t t0,
                                           uint64_t t1, uint64_t t2) {
  uint32_t i = atomicAdd(tr.count, 1u);
  if (static_cast<int64_t>(i) < tr.capacity) {
    uint64_t* r = tr.buf + static_cast<int64_t>(i) * 4;
    r[0] = (static_cast<uint64_t>(kind) << 56) | (static_cast<uint64_t>(blockIdx.x) << 32) |
           static_cast<uint32_t>(tile);
    r[1] = t0;
    r[2] = t1;
    r[3] = t2;
  }
}

// Head-group destination of output element (m, col); col is a multiple of 8.
__device__ __forceinline__ char* head_group_dst(const WinSet& win, const ScatterArgs& sa, int M,
                                                int m, int col) {
  const int per_proj = sa.n_heads * sa.head_dim;
  const int p = col / per_proj;
  const int rem = col - p * per_proj;
  const int head = rem / sa.head_dim;
  const int dd = rem - head * sa.head_dim;
  const int g = head / sa.hpg, lh = head - g * sa.hpg;
  const int64_t row = (static_cast<int64_t>(p) * sa.hpg + lh) * M + m;
  return win.base[g] + row * win.stride[g] + dd * 2;
}

template <int KIND>
__global__ __launch_bounds__(kThreads, 1) void gemm_tiles_kernel(
    const uint16_t* __restrict__ A, int64_t lda, const uint16_t* __restrict__ B, int64_t ldb,
    char* __restrict__ C, int64_t ldc_bytes, int M, int N, int K, ScatterArgs sa, WinSet win,
    xs_trace tr) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBytes];
  char* lds = smem;
  char** rowptr = reinterpret_cast<char**>(smem + kLdsRowPtrOff);
  const int tid = threadIdx.x;
  const int tm = (M + kBM - 1) / kBM, tn = N / kBN, ntiles = tm * tn;
  const int G = gridDim.x;
  for (int t = xcd_instance(blockIdx.x, G); t < ntiles; t += G) {
    int mb, nb;
    if (KIND != KIND_PLAIN && sa.order)
      paced_tile(sa, KIND == KIND_HEAD_GROUP, t, tm, ntiles, &mb, &nb);
    else
      grouped_tile(t, tm, tn, &mb, &nb);
    const int m0 = mb * kBM, n0 = nb * kBN;
    const int rows = min(kBM, M - m0);
    const uint64_t t0 = tr.buf ? wall_ticks() : 0;
    Acc acc;
    gemm_mainloop(A + static_cast<int64_t>(m0) * lda, lda, rows, B, ldb, n0, 0, false, K, acc, lds);
    const uint64_t t1 = tr.buf ? wall_ticks() : 0;
    if (KIND != KIND_HEAD_GROUP && tid < rows) {
      const int m = m0 + tid;
      char* p;
      if (KIND == KIND_PLAIN) {
        p = C + static_cast<int64_t>(m) * ldc_bytes + static_cast<int64_t>(n0) * 2;
      } else {
        const int d = m / sa.rpd;
        p = win.base[d] + static_cast<int64_t>(m - d * sa.rpd) * win.stride[d] +
            static_cast<int64_t>(n0) * 2;
      }
      rowptr[tid] = p;
    }
    stage_tile(acc, lds);
    __syncthreads();
    if (KIND == KIND_HEAD_GROUP) {
      if (sa.group_aligned) {
        // The tile's columns are heads [head0, head0 + 256 / head_dim) of one projection and
        // one group: store head by head, consecutive lanes on consecutive 16-byte pieces of
        // consecutive rows, which are contiguous in a head plane (a wave stores 1 KiB runs).
        const int per_proj = sa.n_heads * sa.head_dim;
        const int p = n0 / per_proj;
        const int head0 = (n0 - p * per_proj) / sa.head_dim;
        const int g = head0 / sa.hpg;
        const int pph = sa.head_dim / 8;                 // 16-byte pieces per head row
        const int64_t stride = win.stride[g];
        char* plane0 = win.base[g] + (static_cast<int64_t>(p * sa.hpg + head0 - g * sa.hpg) * M + m0) * stride;
        const int64_t plane_bytes = static_cast<int64_t>(M) * stride;
        // head_dim divides 256, so pph divides the 512 threads: each thread keeps one piece
        // column and walks rows with a fixed step (no division inside the loop)
        const int rpp = kThreads / pph;
        const int piece = tid % pph, r0 = tid / pph;
        constexpr int U = 4;
        typedef __attribute__((address_space(1))) u32x4 global_u32x4;   // global, not flat, stores
        for (int hsel = 0; hsel < kBN / sa.head_dim; ++hsel) {
          const char* src = lds + (hsel * sa.head_dim + piece * 8) * 2;
          char* dst = plane0 + hsel * plane_bytes + piece * 16;
#pragma unroll 1
          for (int r = r0; r < rows; r += U * rpp) {
            u32x4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
              if (r + u * rpp < rows) v[u] = *reinterpret_cast<const u32x4*>(src + (r + u * rpp) * kEpiPitch * 2);
#pragma unroll
            for (int u = 0; u < U; ++u)
              if (r + u * rpp < rows)
                *(global_u32x4*)(dst + static_cast<int64_t>(r + u * rpp) * stride) = v[u];
          }
        }
      } else {
        const int pc = tid & 31;
        for (int r = tid >> 5; r < rows; r += kThreads / 32) {
          u32x4 v = *reinterpret_cast<const u32x4*>(lds + (r * kEpiPitch + pc * 8) * 2);
          *reinterpret_cast<u32x4*>(head_group_dst(win, sa, M, m0 + r, n0 + pc * 8)) = v;
        }
      }
    } else {
      store_rows(lds, kEpiPitch, kBN, rows, rowptr);
    }
    lds_barrier();   // output tiles are read only after the kernel
    if (tr.buf && tid == 0) trace_tile(tr, 3, t, t0, t1, wall_ticks());
    if (KIND != KIND_PLAIN && sa.gap_ticks) {
      if (tid == 0) spin_ticks(static_cast<uint64_t>(sa.gap_ticks));   // non-injecting gap
      __syncthreads();
    }
  }
}

// Grouped GEMM over row segments: segment s multiplies rows [seg_off[s], seg_off[s] + rows) of A
// by its own weight B_s ([N][K], K-contiguous) into the same rows of C. Tiles are numbered
// segment by segment (ceil(rows / 256) row blocks x nt column tiles each); a workgroup maps its
// tile number to (segment, block, column) with a wave scan over the segment counts, 64
// segments at a time, so no plan or workspace is needed. SWIGLU: B_s holds the gate rows
// [0, N / 2) and the up rows [N / 2, N); a column tile computes 128 gate and 128 up columns
// and stores 128 columns of silu(g) u.
__device__ __forceinline__ bool grouped_tile_of(int t, const int* __restrict__ seg_off,
                                                const int* __restrict__ seg_rows, int n_seg, int M,
                                                int nt, int* status, int* out) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    int base = 0, found = 0;
    for (int s0 = 0; s0 < n_seg; s0 += 64) {
      const int sg = s0 + lane;
      int tiles = 0;
      if (sg < n_seg) {
        int r = seg_rows[sg];
        const int o = seg_off[sg];
        if (r < 0 || o < 0 || static_cast<int64_t>(o) + r > M) {
          if (r != 0) set_status(status, XS_EBADINPUT);
          r = 0;
        }
        tiles = ((r + kBM - 1) / kBM) * nt;
      }
      int incl = tiles;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
      }
      const int total = __shfl(incl, 63);
      if (t < base + total) {
        const bool mine = t >= base + incl - tiles && t < base + incl;
        const unsigned long long m = __ballot(mine);
        if (lane == __ffsll(static_cast<long long>(m)) - 1) {
          out[0] = sg;
          out[1] = t - (base + incl - tiles);
        }
        found = 1;
        break;
      }
      base += total;
    }
    if (lane == 0 && !found) out[0] = -1;
  }
  __syncthreads();
  const bool ok = out[0] >= 0;
  return ok;
}

template <bool SWIGLU>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_kernel(
    const uint16_t* __restrict__ A, int64_t lda, int M, const int* __restrict__ seg_off,
    const int* __restrict__ seg_rows, int n_seg, const uint16_t* __restrict__ B, int N, int K,
    char* __restrict__ C, int64_t ldc_bytes, int* status) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBytes];
  char* lds = smem;
  char** rowptr = reinterpret_cast<char**>(smem + kLdsRowPtrOff);
  int* misc = reinterpret_cast<int*>(smem + kLdsMiscOff);
  const int tid = threadIdx.x;
  const int nt = SWIGLU ? (N / 2) / (kBN / 2) : N / kBN;
  for (int t = blockIdx.x;; t += gridDim.x) {
    const bool more = grouped_tile_of(t, seg_off, seg_rows, n_seg, M, nt, status, misc);
    const int sg = misc[0], local = misc[1];
    __syncthreads();   // every thread has read the mapping before the mainloop reuses the LDS
    if (!more) break;
    const int mb = local / nt, nb = local - mb * nt;
    const int m0 = seg_off[sg] + mb * kBM;
    const int rows = min(kBM, seg_rows[sg] - mb * kBM);
    const uint16_t* Bs = B + static_cast<int64_t>(sg) * N * K;
    Acc acc;
    if (SWIGLU) {
      gemm_mainloop<true>(A + static_cast<int64_t>(m0) * lda, lda, rows, Bs, K, nb * (kBN / 2), N / 2, true, K, acc, lds);
      if (tid < rows)
        rowptr[tid] = C + static_cast<int64_t>(m0 + tid) * ldc_bytes + static_cast<int64_t>(nb) * (kBN / 2) * 2;
      stage_swiglu(acc, lds);
      __syncthreads();
      store_rows(lds, kEpiPitchH, kBN / 2, rows, rowptr);
    } else {
      gemm_mainloop<true>(A + static_cast<int64_t>(m0) * lda, lda, rows, Bs, K, nb * kBN, 0, false, K, acc, lds);
      if (tid < rows)
        rowptr[tid] = C + static_cast<int64_t>(m0 + tid) * ldc_bytes + static_cast<int64_t>(nb) * kBN * 2;
      stage_tile(acc, lds);
      __syncthreads();
      store_rows(lds, kEpiPitch, kBN, rows, rowptr);
    }
    lds_barrier();   // the output rows are read only after the kernel
  }
}

// Serial permutation pass: plain output c -> windows (one wave per row).
template <int KIND>
__global__ __launch_bounds__(256) void scatter_copy_kernel(const char* __restrict__ c,
                                                           int64_t ldc_bytes, int M, int N,
                                                           ScatterArgs sa, WinSet win) {
  const int lane = threadIdx.x & 63;
  for (int m = blockIdx.x * 4 + (threadIdx.x >> 6); m < M; m += gridDim.x * 4) {
    const u32x4* src = reinterpret_cast<const u32x4*>(c + static_cast<int64_t>(m) * ldc_bytes);
    for (int pc = lane; pc < N / 8; pc += 64) {
      u32x4 v = src[pc];
      char* dst;
      if (KIND == KIND_ROW_BLOCK) {
        const int d = m / sa.rpd;
        dst = win.base[d] + static_cast<int64_t>(m - d * sa.rpd) * win.stride[d] + pc * 16;
      } else {
        dst = head_group_dst(win, sa, M, m, pc * 8);
      }
      *reinterpret_cast<u32x4*>(dst) = v;
    }
  }
}

}  // namespace xs

using namespace xs;

namespace xs_host {
int signal_windows(const WinSet& ws, hipStream_t st);

int persistent_grid(int max_producers) {
  int cus = num_cus();
  if (cus <= 0) cus = 256;
  if (max_producers > 0 && max_producers < cus) return max_producers;
  return cus;
}
}  // namespace xs_host

static bool gemm_shape_ok(int64_t lda, int64_t ldb, int32_t M, int32_t N, int32_t K) {
  return M >= 0 && N > 0 && K > 0 && N % kBN == 0 && K % kBK == 0 && lda >= K && ldb >= K &&
         lda % 8 == 0 && ldb % 8 == 0;
}

static xs_trace trace_or_empty(const xs_trace* t) {
  xs_trace e{nullptr, 0, nullptr};
  if (!t || !t->buf || !t->count) return e;
  return *t;
}

extern "C" int xs_gemm(const void* a, int64_t lda, const void* b, int64_t ldb, void* c,
                       int64_t ldc, int32_t M, int32_t N, int32_t K, const xs_trace* trace,
                       void* stream) {
  if (!a || !b || !c) return XS_EINVAL;
  if (!gemm_shape_ok(lda, ldb, M, N, K) || ldc < N || ldc % 8) return XS_EUNSUPPORTED;
  if (M == 0) return XS_OK;
  WinSet none{};
  none.n = 0;
  ScatterArgs sa{};
  const int tiles = ((M + kBM - 1) / kBM) * (N / kBN);
  const int grid = std::min(tiles, xs_host::persistent_grid(0));
  hipLaunchKernelGGL(gemm_tiles_kernel<KIND_PLAIN>, dim3(grid), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint16_t*>(a), lda,
                     static_cast<const uint16_t*>(b), ldb, static_cast<char*>(c), ldc * 2, M, N,
                     K, sa, none, trace_or_empty(trace));
  return xs_host::launch_status();
}

static int scatter_setup(const xs_scatter_desc* desc, int32_t M, int32_t N, const xs_window* win,
                         int32_t W, ScatterArgs* sa, WinSet* ws, int* kind) {
  if (!desc || !win) return XS_EINVAL;
  *sa = ScatterArgs{};
  if (desc->kind == XS_SCATTER_ROW_BLOCK) {
    const int rpd = desc->rows_per_dest;
    if (rpd <= 0 || M % rpd || M / rpd != W) return XS_EINVAL;
    if (rpd % kBM) return XS_EUNSUPPORTED;
    sa->rpd = rpd;
    int rc = xs_host::make_winset(win, W, static_cast<int64_t>(N) * 2, ws);
    if (rc) return rc;
    for (int d = 0; d < W; ++d)
      if (ws->cap[d] < rpd) return XS_EINVAL;
    *kind = KIND_ROW_BLOCK;
    return XS_OK;
  }
  if (desc->kind == XS_SCATTER_HEAD_GROUP) {
    const int np = desc->n_proj, nh = desc->n_heads, hd = desc->head_dim, hpg = desc->heads_per_group;
    if (np <= 0 || nh <= 0 || hd <= 0 || hpg <= 0 || nh % hpg || N != np * nh * hd ||
        nh / hpg != W)
      return XS_EINVAL;
    if (hd % 8) return XS_EUNSUPPORTED;
    sa->n_proj = np;
    sa->n_heads = nh;
    sa->head_dim = hd;
    sa->hpg = hpg;
    // tiles inside one projection and one head group, heads not straddling a tile
    sa->group_aligned = (nh * hd) % kBN == 0 && (hpg * hd) % kBN == 0 && kBN % hd == 0;
    int rc = xs_host::make_winset(win, W, static_cast<int64_t>(hd) * 2, ws);
    if (rc) return rc;
    for (int d = 0; d < W; ++d)
      if (ws->cap[d] < static_cast<int64_t>(np) * hpg * M) return XS_EINVAL;
    *kind = KIND_HEAD_GROUP;
    return XS_OK;
  }
  return XS_EINVAL;
}

extern "C" int xs_gemm_scatter(const void* a, int64_t lda, const void* b, int64_t ldb, int32_t M,
                               int32_t N, int32_t K, const xs_scatter_desc* desc,
                               const xs_window* win, int32_t W, const xs_pacing* pacing,
                               const xs_trace* trace, void* stream) {
  if (!a || !b) return XS_EINVAL;
  if (!gemm_shape_ok(lda, ldb, M, N, K)) return XS_EUNSUPPORTED;
  ScatterArgs sa;
  WinSet ws;
  int kind = 0;
  int rc = scatter_setup(desc, M, N, win, W, &sa, &ws, &kind);
  if (rc) return rc;
  int max_producers = 0;
  if (pacing) {
    if (pacing->max_producers < 0 || pacing->gap_ns < 0 || pacing->chunk_tiles < 0 || pacing->reserved != 0)
      return XS_EINVAL;
    max_producers = pacing->max_producers;
    sa.gap_ticks = xs_host::ns_to_ticks(pacing->gap_ns);
    sa.n_dest = W;
    const int ntiles = ((M + kBM - 1) / kBM) * (N / kBN);
    const int pol = pacing->policy;
    if (pol == XS_POLICY_BURST) {
      sa.order = 1;
    } else if (pol == XS_POLICY_INTERLEAVE || pol == XS_POLICY_CHUNK) {
      sa.order = 2;
      sa.chunk = pol == XS_POLICY_CHUNK && pacing->chunk_tiles > 0 ? pacing->chunk_tiles : 1;
      if ((ntiles / W) % sa.chunk) return XS_EINVAL;   // a chunk never spans two windows' lists
    } else {
      return XS_EINVAL;
    }
    // orders over destinations need each tile inside one window (head groups tile-aligned)
    if (kind == KIND_HEAD_GROUP && !sa.group_aligned) return XS_EUNSUPPORTED;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (M > 0) {
    const int tiles = ((M + kBM - 1) / kBM) * (N / kBN);
    const int grid = std::min(tiles, xs_host::persistent_grid(max_producers));
    if (kind == KIND_ROW_BLOCK)
      hipLaunchKernelGGL(gemm_tiles_kernel<KIND_ROW_BLOCK>, dim3(grid), dim3(kThreads), 0, st,
                         static_cast<const uint16_t*>(a), lda, static_cast<const uint16_t*>(b), ldb,
                         nullptr, 0, M, N, K, sa, ws, trace_or_empty(trace));
    else
      hipLaunchKernelGGL(gemm_tiles_kernel<KIND_HEAD_GROUP>, dim3(grid), dim3(kThreads), 0, st,
                         static_cast<const uint16_t*>(a), lda, static_cast<const uint16_t*>(b), ldb,
                         nullptr, 0, M, N, K, sa, ws, trace_or_empty(trace));
    if (xs_host::launch_status()) return XS_EHIP;
  }
  return xs_host::signal_windows(ws, st);
}

extern "C" int xs_grouped_gemm(const void* a, int64_t lda, int32_t M, const int32_t* seg_offsets,
                               const int32_t* seg_rows, int32_t n_seg, const void* b, int32_t N,
                               int32_t K, void* c, int64_t ldc, int32_t epilogue, int32_t* dev_status,
                               void* stream) {
  if (!a || !b || !c || !seg_offsets || !seg_rows || M < 0 || n_seg < 0 || n_seg > 1024) return XS_EINVAL;
  if (epilogue != XS_EPI_STORE && epilogue != XS_EPI_SWIGLU) return XS_EINVAL;
  const int n_out = epilogue == XS_EPI_SWIGLU ? N / 2 : N;
  if (N <= 0 || K <= 0 || K % kBK || lda < K || lda % 8 || ldc < n_out || ldc % 8) return XS_EUNSUPPORTED;
  if (epilogue == XS_EPI_STORE ? N % kBN : (N % 2 || (N / 2) % (kBN / 2))) return XS_EUNSUPPORTED;
  if (M == 0 || n_seg == 0) return XS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int grid = xs_host::persistent_grid(0);
  if (epilogue == XS_EPI_SWIGLU)
    hipLaunchKernelGGL(grouped_gemm_kernel<true>, dim3(grid), dim3(kThreads), 0, st,
                       static_cast<const uint16_t*>(a), lda, M, seg_offsets, seg_rows, n_seg,
                       static_cast<const uint16_t*>(b), N, K, static_cast<char*>(c), ldc * 2, dev_status);
  else
    hipLaunchKernelGGL(grouped_gemm_kernel<false>, dim3(grid), dim3(kThreads), 0, st,
                       static_cast<const uint16_t*>(a), lda, M, seg_offsets, seg_rows, n_seg,
                       static_cast<const uint16_t*>(b), N, K, static_cast<char*>(c), ldc * 2, dev_status);
  return xs_host::launch_status();
}

extern "C" int xs_scatter_copy(const void* c, int64_t ldc, int32_t M, int32_t N,
                               const xs_scatter_desc* desc, const xs_window* win, int32_t W,
                               void* stream) {
  if (!c || M < 0 || N <= 0 || N % 8 || ldc < N || ldc % 8) return XS_EINVAL;
  ScatterArgs sa;
  WinSet ws;
  int kind = 0;
  int rc = scatter_setup(desc, M, N, win, W, &sa, &ws, &kind);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (M > 0) {
    const int grid = std::min((M + 3) / 4, 8192);
    if (kind == KIND_ROW_BLOCK)
      hipLaunchKernelGGL(scatter_copy_kernel<KIND_ROW_BLOCK>, dim3(grid), dim3(256), 0, st,
                         static_cast<const char*>(c), ldc * 2, M, N, sa, ws);
    else
      hipLaunchKernelGGL(scatter_copy_kernel<KIND_HEAD_GROUP>, dim3(grid), dim3(256), 0, st,
                         static_cast<const char*>(c), ldc * 2, M, N, sa, ws);
    if (xs_host::launch_status()) return XS_EHIP;
  }
  return xs_host::signal_windows(ws, st);
}
