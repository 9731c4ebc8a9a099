// Attention with the post-attention Ulysses exchange fused into its output epilogue
// (Sec. 4.4, App. B; Table 4).
//
// A persistent workgroup (4 waves) takes 128-query output tiles of one head and streams the
// head's keys and values in 64-token tiles (the Q-loop). Each wave owns 32 queries and works
// in the transposed form
//   S' = K Q^T   (MFMA A operand: key rows from LDS, B operand: the wave's query rows, kept in
//                 registers for the whole tile)
//   O' = V^T P^T (A operand: value columns, B operand: the probabilities)
// so that every lane's accumulators belong to one query (lane % 32): the online softmax
// (running max and sum, in base 2) is lane-local apart from one exchange with lane ^ 32, which
// holds the other keys of the same query. The bf16 probabilities are already in registers
// in nearly the B-operand layout: per 16-key step, lanes l and l + 32 swap four of their
// eight values.
//
// The value columns for the A operand of O' come straight from the row-major V tile in LDS
// through gfx950's transposing LDS read (ds_read_b64_tr_b16): within each 16-lane group, the
// lane that receives column d0 + i gets the four 16-bit values at rows kv0 .. kv0 + 3 when
// lane j of the group points at row kv0 + j / 4, columns d0 + 4 (j % 4) .. + 3.
//
// LDS: two K slots and one V slot, each a tile of [64][128] bf16 (rows of 256 B = 16 pieces of
// 16 B): 48 KiB, so that three workgroups share a CU (three waves per SIMD; two left the
// matrix pipes idle while both waves ran their softmax). K tiles store logical piece p of row r
// at p ^ (r & 15) (a ds_read_b128 phase reads one piece of 16 consecutive rows); V tiles at
// p ^ 4 (r & 3) (a transposing read touches four consecutive rows, four pieces each). Both
// arrive by direct buffer -> LDS loads with the swizzle applied on the global side. Per K/V
// tile j: S' from K slot j % 2, a barrier, K tile j + 2 into that slot; the softmax; V tile j
// waited for and a barrier; O' from the V slot; K tile j + 1 waited for, a barrier, V tile
// j + 1 into the V slot. K tiles are loaded about one and a half tiles ahead, V tiles one S'
// and softmax ahead.
//
// Epilogue: O = O' / rowsum, packed to bf16 with the hardware conversion and stored four
// columns per 8-byte store, either to the local output or, fused, into the destination
// window of the tile's sequence chunk; the next tile's Q-loop is the drain window of these
// stores (no extra wait, no dedicated communication wave).
#include <algorithm>
#include <cmath>

#include "xs_common.hpp"

namespace xs {

namespace attn {

typedef __attribute__((address_space(3))) char lds_char;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));

constexpr int kD = 128;                    // head_dim
constexpr int kBQ = 128;                   // queries per output tile (4 waves x 32)
constexpr int kBKV = 64;                   // keys per K/V tile
constexpr int kRowBytes = kD * 2;          // 256
constexpr int kTileBytes = kBKV * kRowBytes;   // 16 KiB
constexpr int kLds = 3 * kTileBytes;       // two K slots and one V slot: 48 KiB
constexpr int kThreads = 256;
// a query's running maximum is raised (and its sums rescaled) only when a block's maximum
// exceeds it by more than this many powers of two; until then probabilities stay <= 2^8
constexpr float kRescaleSlack = 8.f;
constexpr int kBufDword3 = 0x00020000;     // raw buffer resource: 32-bit data, no swizzle

typedef int v4i __attribute__((ext_vector_type(4)));
// A raw buffer descriptor over [base, base + bytes): 32-bit data, no stride, no swizzle.
__device__ __forceinline__ v4i buffer_rsrc(const void* base, int bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const v4i r = {static_cast<int>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b))),
                 static_cast<int>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)) & 0xFFFF),
                 bytes, kBufDword3};
  return r;
}
// One 16-byte piece per lane from the buffer at voff + soff into LDS at dst + 16 lane. Issued
// from assembly so that the compiler does not count it: it would otherwise wait for every
// load in flight before each transposing LDS read (it cannot tell the two apart), and the
// kernel orders these loads itself, with vmcnt waits and workgroup barriers.
__device__ __forceinline__ void load_lds16(v4i rsrc, uint32_t voff, int soff, const lds_char* dst) {
  const uint32_t m0v = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(dst));
  asm volatile("buffer_load_dwordx4 %0, %1, %2 offen lds" :: "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(m0v) : "memory");
}

__device__ __forceinline__ int k_swz(int r) { return r & 15; }
__device__ __forceinline__ int v_swz(int r) { return 4 * (r & 3); }

struct Args {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  WinSet win;
  int heads, M, chunk;
  int mode;
  float scale_log2e;
  xs_trace tr;
};

__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }
__device__ __forceinline__ void wait_vm4() { __builtin_amdgcn_s_waitcnt(0x0F74); }

// The two halves of a wave hold the two key halves of the same 32 queries: lanes l and
// l + 32 combine through one half swap (v_permlane32_swap: a's upper half <-> b's lower half),
// after which one result holds every lane's lower-half value and the other its upper-half
// value. The two results are reinterpreted as floats through one two-element vector: a bit
// cast of each result on its own was compiled to read the first result twice.
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ f32x2_t both_halves(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const u32x2_t t = {r[0], r[1]};
  return __builtin_bit_cast(f32x2_t, t);
}
__device__ __forceinline__ float max_halves(float x) {
  const f32x2_t h = both_halves(x);
  return fmaxf(h.x, h.y);
}
__device__ __forceinline__ float add_halves(float x) {
  const f32x2_t h = both_halves(x);
  return h.x + h.y;
}

__global__ __launch_bounds__(kThreads, 3) void attn_kernel(Args a) {
  __shared__ __attribute__((aligned(16))) char lds_raw[kLds];
  lds_char* const lds = (lds_char*)lds_raw;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int up = lane >> 5;                 // which half of the wave
  const int qtiles = a.M / kBQ;
  const int ntiles = a.heads * qtiles;
  const int nkv = a.M / kBKV;
  // direct loads: instruction i of wave w fills rows 4 (4 i + w) .. + 3 of a tile; lane ->
  // row + lane / 16, physical piece lane % 16, fetching logical piece (lane % 16) ^ swz(row)
  uint32_t ko[4], vo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * (4 * i + w) + (lane >> 4);
    ko[i] = static_cast<uint32_t>(r * kRowBytes + (((lane & 15) ^ k_swz(r)) << 4));
    vo[i] = static_cast<uint32_t>(r * kRowBytes + (((lane & 15) ^ v_swz(r)) << 4));
  }
  // K fragment reads: row 32 b + lane % 32, logical piece 2 kk + up, at piece ^ (row & 15)
  // (the row's low bits do not depend on b, so b is an immediate offset)
  const int krow = lane & 31;
  uint32_t kofs[8];
#pragma unroll
  for (int kk = 0; kk < 8; ++kk)
    kofs[kk] = static_cast<uint32_t>(krow * kRowBytes + (((2 * kk + up) ^ k_swz(krow)) << 4));
  // transposing reads of the value columns: for key step s (16 keys), column block db (32
  // columns) and half hf (keys +0 / +4) this lane addresses row 16 s + tr_k + 4 hf, columns
  // 32 db + tr_d .. + 3; the row's low two bits (the swizzle) do not depend on s or hf
  const int grp = lane >> 4, j16 = lane & 15;
  const int tr_d = 16 * (grp & 1) + 4 * (j16 & 3);
  const int tr_k = 8 * (grp >> 1) + (j16 >> 2);
  uint32_t vofs[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) {
    const int phys_piece = (4 * db + (tr_d >> 3)) ^ v_swz(tr_k);
    vofs[db] = static_cast<uint32_t>(tr_k * kRowBytes + (phys_piece << 4) + ((tr_d >> 2) & 1) * 8);
  }

  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int h = t / qtiles, qt = t - h * qtiles;
    const uint64_t t0 = a.tr.buf ? wall_ticks() : 0;
    const int64_t hoff = static_cast<int64_t>(h) * a.M * kD;
    const char* kh = reinterpret_cast<const char*>(a.k + hoff);
    const char* vh = reinterpret_cast<const char*>(a.v + hoff);
    const int qrow = qt * kBQ + 32 * w + (lane & 31);
    bf16x8 qf[8];
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
      qf[kk] = *reinterpret_cast<const bf16x8*>(a.q + hoff + static_cast<int64_t>(qrow) * kD + 16 * kk + 8 * up);
    const v4i krs = buffer_rsrc(kh, a.M * kRowBytes);
    const v4i vrs = buffer_rsrc(vh, a.M * kRowBytes);
    // K tile j into K slot j % 2, V tile j into the V slot: four 1 KiB pieces per wave each
    auto issue_k = [&](int j) {
      lds_char* st = lds + (j & 1) * kTileBytes;
      const int so = j * kTileBytes;
#pragma unroll
      for (int i = 0; i < 4; ++i) load_lds16(krs, ko[i], so, st + (4 * i + w) * 1024);
    };
    auto issue_v = [&](int j) {
      lds_char* st = lds + 2 * kTileBytes;
      const int so = j * kTileBytes;
#pragma unroll
      for (int i = 0; i < 4; ++i) load_lds16(vrs, vo[i], so, st + (4 * i + w) * 1024);
    };
    f32x16 oacc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) oacc[db][e] = 0.f;
    float m = -INFINITY, l = 0.f;
    issue_k(0);
    issue_v(0);
    if (nkv > 1) issue_k(1);
    wait_vm0();
    asm volatile("s_barrier" ::: "memory");
    for (int j = 0; j < nkv; ++j) {
      lds_char* const ks = lds + (j & 1) * kTileBytes;
      lds_char* const vs = lds + 2 * kTileBytes;
      // S' = K Q^T over two 32-key blocks
      f32x16 sacc[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[b][e] = 0.f;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
          const bf16x8 kf = *(const lds_bf16x8*)(ks + b * 32 * kRowBytes + kofs[kk]);
          sacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], sacc[b], 0, 0, 0);
        }
      }
      // every wave is done with K slot j % 2: K tile j + 2 goes there
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      const bool k2 = j + 2 < nkv;
      if (k2) issue_k(j + 2);
      // online softmax in base 2 for query lane % 32
      float mx = fmaxf(sacc[0][0], sacc[0][1]);
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int e = (b ? 0 : 2); e < 16; ++e) mx = fmaxf(mx, sacc[b][e]);
      const float mxs = max_halves(mx) * a.scale_log2e;
      if (__builtin_amdgcn_ballot_w64(mxs > m + kRescaleSlack)) {    // wave-uniform
        const float m_new = fmaxf(m, mxs);
        const float corr = __builtin_amdgcn_exp2f(m - m_new);
        l *= corr;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[db][e] *= corr;
        m = m_new;
      }
      // probabilities, packed to bf16; the row sum adds the packed values themselves, so the
      // normaliser is the sum of exactly the weights the second product uses
      uint32_t pk[2][8];
      float rs = 0.f;
      const bf16x2_v ones = __builtin_bit_cast(bf16x2_v, 0x3F803F80u);
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[b][2 * e], a.scale_log2e, -m));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[b][2 * e + 1], a.scale_log2e, -m));
          pk[b][e] = pack_bf16x2(p0, p1);
          rs = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, pk[b][e]), ones, rs, false);
        }
      l += add_halves(rs);
      // P^T fragments: key step s covers keys 16 s .. 16 s + 15 of block s / 2; the lower
      // half needs keys +0..7 (its own pairs o, o + 1 and the upper half's), the upper half
      // keys +8..15 (the lower half's pairs o + 2, o + 3 and its own): two half swaps
      bf16x8 pf[4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int b = s >> 1, o = 4 * (s & 1);
        const auto x = __builtin_amdgcn_permlane32_swap(pk[b][o], pk[b][o + 2], false, false);
        const auto y = __builtin_amdgcn_permlane32_swap(pk[b][o + 1], pk[b][o + 3], false, false);
        const u32x4 pv = {x[0], y[0], x[1], y[1]};
        pf[s] = __builtin_bit_cast(bf16x8, pv);
      }
      // V tile j has landed in every wave's share (only K tile j + 2 may still be in flight)
      if (k2) wait_vm4(); else wait_vm0();
      asm volatile("s_barrier" ::: "memory");
      // O' += V^T P^T
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const s16x4 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vs + (16 * s) * kRowBytes + vofs[db]));
          const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vs + (16 * s + 4) * kRowBytes + vofs[db]));
          const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(r0, r1, 0, 1, 2, 3, 4, 5, 6, 7));
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[s], oacc[db], 0, 0, 0);
        }
      if (j + 1 < nkv) {
        // K tile j + 1 has landed in every wave's share, and no wave reads the V slot any more
        if (k2) wait_vm4(); else wait_vm0();
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        issue_v(j + 1);
      }
    }
    const uint64_t t1 = a.tr.buf ? wall_ticks() : 0;
    // epilogue: O[q][d] for d = 32 db + 8 g + 4 up + 0..3
    const float inv = 1.f / l;
    char* dst;
    if (a.mode != XS_ATTN_LOCAL) {
      const int g = (qt * kBQ) / a.chunk;    // uniform: a tile lies in one sequence chunk
      dst = a.win.base[g] + static_cast<int64_t>(qrow - g * a.chunk) * a.win.stride[g] +
            static_cast<int64_t>(h) * kD * 2;
    } else {
      dst = reinterpret_cast<char*>(a.o + hoff + static_cast<int64_t>(qrow) * kD);
    }
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 v = {pack_bf16x2(oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv),
                         pack_bf16x2(oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv)};
        *(__attribute__((address_space(1))) u32x2*)(dst + (32 * db + 8 * g + 4 * up) * 2) = v;
      }
    // completion-coupled counterfactual: the producer waits until its stores are visible at
    // system scope before it starts the next Q-loop
    if (a.mode == XS_ATTN_WINDOWS_COUPLED) __threadfence_system();
    // the next tile's loads overwrite both stages: every wave must be done with them (the
    // stores above may still drain)
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (a.tr.buf && tid == 0) {
      uint32_t i = atomicAdd(a.tr.count, 1u);
      if (static_cast<int64_t>(i) < a.tr.capacity) {
        uint64_t* r = a.tr.buf + static_cast<int64_t>(i) * 4;
        r[0] = (4ull << 56) | (static_cast<uint64_t>(blockIdx.x) << 32) | static_cast<uint32_t>(t);
        r[1] = t0;
        r[2] = t1;
        r[3] = wall_ticks();
      }
    }
  }
}

// Serial post-attention exchange: one thread per 16-byte piece of o.
__global__ __launch_bounds__(256) void ulysses_copy_kernel(const uint16_t* __restrict__ o, int heads,
                                                           int M, int D, int chunk, WinSet win) {
  const int per_row = D / 8;
  const int64_t total = static_cast<int64_t>(heads) * M * per_row;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int pc = static_cast<int>(i % per_row);
    const int64_t rt = i / per_row;
    const int t = static_cast<int>(rt % M);
    const int h = static_cast<int>(rt / M);
    const int g = t / chunk;
    const u32x4 v = reinterpret_cast<const u32x4*>(o + rt * D)[pc];
    char* dst = win.base[g] + static_cast<int64_t>(t - g * chunk) * win.stride[g] +
                (static_cast<int64_t>(h) * D + pc * 8) * 2;
    *reinterpret_cast<u32x4*>(dst) = v;
  }
}

}  // namespace attn
}  // namespace xs

using namespace xs;

namespace xs_host {
int signal_windows(const WinSet& ws, hipStream_t st);
int persistent_grid(int max_producers);
}  // namespace xs_host

static int attn_windows(const xs_window* win, int32_t W, int32_t heads, int32_t M, int32_t D, WinSet* ws) {
  if (!win || W < 1 || W > XS_MAX_WINDOWS || M % W) return XS_EINVAL;
  int rc = xs_host::make_winset(win, W, static_cast<int64_t>(heads) * D * 2, ws);
  if (rc) return rc;
  for (int g = 0; g < W; ++g)
    if (ws->cap[g] < M / W) return XS_EINVAL;
  return XS_OK;
}

extern "C" int xs_attention(const xs_attn* A, int32_t mode, const xs_trace* trace, void* stream) {
  if (!A || !A->q || !A->k || !A->v || A->heads < 1 || A->M < 1 || A->head_dim < 1 ||
      !(A->scale >= 0.f) || A->max_producers < 0)
    return XS_EINVAL;
  if (mode != XS_ATTN_LOCAL && mode != XS_ATTN_WINDOWS && mode != XS_ATTN_WINDOWS_COUPLED) return XS_EINVAL;
  const auto misaligned = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; };
  if (misaligned(A->q) || misaligned(A->k) || misaligned(A->v)) return XS_EINVAL;
  if (A->head_dim != attn::kD || A->M % attn::kBQ || A->M > INT32_MAX / attn::kRowBytes) return XS_EUNSUPPORTED;
  attn::Args a{};
  a.q = static_cast<const uint16_t*>(A->q);
  a.k = static_cast<const uint16_t*>(A->k);
  a.v = static_cast<const uint16_t*>(A->v);
  a.heads = A->heads;
  a.M = A->M;
  a.mode = mode;
  const float scale = A->scale > 0.f ? A->scale : 1.f / std::sqrt(static_cast<float>(A->head_dim));
  a.scale_log2e = scale * 1.4426950408889634f;
  a.tr = xs_trace{nullptr, 0, nullptr};
  if (trace && trace->buf && trace->count) a.tr = *trace;
  if (mode == XS_ATTN_LOCAL) {
    if (!A->o || misaligned(A->o)) return XS_EINVAL;
    a.o = static_cast<uint16_t*>(A->o);
    a.chunk = A->M;
  } else {
    int rc = attn_windows(A->win, A->W, A->heads, A->M, A->head_dim, &a.win);
    if (rc) return rc;
    a.chunk = A->M / A->W;
    if (a.chunk % attn::kBQ) return XS_EUNSUPPORTED;
  }
  const int tiles = A->heads * (A->M / attn::kBQ);
  int grid = A->max_producers > 0 ? A->max_producers : 3 * xs_host::persistent_grid(0);
  if (grid > tiles) grid = tiles;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(attn::attn_kernel, dim3(grid), dim3(attn::kThreads), 0, st, a);
  if (xs_host::launch_status()) return XS_EHIP;
  if (mode != XS_ATTN_LOCAL) return xs_host::signal_windows(a.win, st);
  return XS_OK;
}

extern "C" int xs_ulysses_copy(const void* o, int32_t heads, int32_t M, int32_t head_dim,
                               const xs_window* win, int32_t W, void* stream) {
  if (!o || (reinterpret_cast<uintptr_t>(o) & 15) || heads < 1 || M < 1 || head_dim < 8 || head_dim % 8) return XS_EINVAL;
  WinSet ws;
  int rc = attn_windows(win, W, heads, M, head_dim, &ws);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t pieces = static_cast<int64_t>(heads) * M * (head_dim / 8);
  const int grid = static_cast<int>(std::min<int64_t>((pieces + 255) / 256, 8192));
  hipLaunchKernelGGL(attn::ulysses_copy_kernel, dim3(grid), dim3(256), 0, st,
                     static_cast<const uint16_t*>(o), heads, M, head_dim, M / W, ws);
  if (xs_host::launch_status()) return XS_EHIP;
  return xs_host::signal_windows(ws, st);
}
