// MFMA bf16 GEMM core for gfx950: 256x256 output tile, K step 64, 512 threads = 8 waves, two
// per SIMD, as 2 (M) x 4 (N) waves of 128 x 64 each = 4 x 2 blocks of
// v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per lane). Two waves per SIMD let one
// wave's LDS or memory wait be covered by the other's MFMAs; measured on an 8192^3 GEMM this
// beats one wave per SIMD of 128 x 128 (fewer LDS reads per MFMA, but every stall idles the
// matrix pipe) by about 20 %.
//
// Operands move global -> LDS with gfx950's direct 128-bit loads (global_load_lds_dwordx4):
// no staging registers and no LDS store instructions. LDS holds two stages of the A tile
// ([256][64] bf16 each) and three of the B tile, 160 KiB in all: A (activations, shared by
// every tile of a row block and mostly L2-resident) is loaded one K step ahead, B (weights,
// streamed from HBM) two K steps ahead, so a weight load has two K steps of MFMA work to
// land in. (Measured alternatives that lost: four or five stages of K step 32, whose extra
// barriers cost more than the deeper prefetch gains, and loads through registers with LDS
// stores.)
//
// LDS operand layout: 128 B per row in eight 16-byte pieces; logical piece c of row r sits at
// physical position c ^ ((r >> 1) & 7). A direct load writes 64 consecutive pieces (8 rows)
// per wave instruction, so the swizzle is applied on the global side: the lane that fills
// physical piece p of row r fetches logical piece p ^ ((r >> 1) & 7). The 16 lanes of each
// ds_read_b128 phase then hit 16 distinct 16-byte bank groups (no bank conflicts measured).
//
// C = A B^T: A rows are K-contiguous and B is output-major ([N][K], K-contiguous), so both
// MFMA operands are 16-byte contiguous reads from LDS. The MFMA is issued with the B
// fragment as its first operand, so each lane's accumulators hold four consecutive output
// columns of one row per group (8-byte epilogue writes instead of 2-byte ones).
//
// Partial tiles (an expert's last 256-row block) skip the MFMAs and fragment reads of the
// 32-row blocks that hold no valid row: each wave runs the pipeline instantiated for its
// number of valid 32-row blocks (0 to 4); every instantiation issues the same loads and
// barriers, so the workgroup stays in step.
#pragma once
#include <type_traits>

#include "xs_common.hpp"

namespace xs {

constexpr int kBM = 256, kBN = 256, kBK = 64, kThreads = 512;
constexpr int kOpBytes = kBM * kBK * 2;                      // one operand stage: 32 KiB
// LDS operand stages: A in two buffers [0, 64 KiB), B in three [64 KiB, 160 KiB)
constexpr int kAStages = 2, kBStages = 3;
constexpr int kBBase = kAStages * kOpBytes;
constexpr int kLdsOpBytes = (kAStages + kBStages) * kOpBytes;   // 160 KiB
constexpr int kEpiPitch = kBN + 8;                           // bf16 per staged output row
constexpr int kEpiPitchH = kBN / 2 + 8;                      // SwiGLU output rows (128 wide)
constexpr int kLdsEpiBytes = kBM * kEpiPitch * 2;            // 135168
constexpr int kLdsRowPtrOff = kLdsEpiBytes;                  // 256 row pointers
constexpr int kLdsMiscOff = kLdsRowPtrOff + kBM * 8;         // small scheduler scratch
constexpr int kLdsBytes = kLdsOpBytes;
// The epilogue tile, the row pointers and the scheduler scratch reuse the operand stages:
// they are only touched between a mainloop's final barrier and the next mainloop's loads.
static_assert(kLdsMiscOff + 64 <= kLdsBytes, "epilogue area must fit in the operand stages");
static_assert(kLdsBytes <= 160 * 1024, "gfx950 LDS per workgroup");

// address-space-qualified pointees for the direct-load builtin (C-style casts convert)
typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void glob_void;

// B tile row r -> weight row. SwiGLU tiles interleave gate and up rows in blocks of 32 so
// that each wave's 64 columns hold the gate and up rows of the same 32 output columns.
__device__ __forceinline__ int b_row_map(int r, int n0, int half, bool swiglu) {
  return swiglu ? n0 + ((r >> 5) & 1) * half + (r >> 6) * 32 + (r & 31) : n0 + r;
}

typedef f32x16 Acc[4][2];

__device__ __forceinline__ void zero_acc(Acc& acc) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
}

// s_waitcnt vmcnt(0) only (expcnt and lgkmcnt left at their maxima).
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Workgroup barrier that orders LDS only: every wave's LDS reads and writes have completed,
// outstanding global stores may still drain (__syncthreads would wait for them, vmcnt(0)).
// Used after an epilogue whose stores need no ordering before the next tile's work.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
}

// Per-wave operand addressing, computed once per tile.
struct TileAddr {
  const char* a;          // A tile base (row 0, k 0)
  const char* b;          // B base
  uint32_t oa[4], ob[4];  // per-lane byte offsets of the four direct loads of each operand
  int arow, brow;         // LDS byte offsets of this lane's fragment rows (A, B)
  int w;                  // wave index (uniform)
};

// The software pipeline for a wave that multiplies NI of its four 32-row blocks.
//
// Fragments are double-buffered in registers: the reads of k sub-step kk + 1 are in flight
// while the MFMAs of sub-step kk issue. The order is pinned one MFMA at a time between
// scheduling fences (left alone, the scheduler reuses one fragment register set and waits out
// every LDS read): in sub-steps 0-2 each MFMA is followed by one fragment read of the next
// sub-step; the stage barrier comes before sub-step 3, whose MFMAs are each followed by one
// fragment read of the next stage's sub-step 0 and one direct load, so the matrix pipe works
// while the loads are issued and the next stage's first fragments arrive.
//
// kLateB moves the weight loads out of that burst: B(kt + 3) is issued one stage later, over
// sub-steps 0-2 of stage kt + 1 (its slot is free from stage kt's barrier on), so sub-step 3
// issues only the four A loads. The wait at each barrier stays vmcnt(4) (the B loads of the
// stage after next are the only newer ones); a weight load then has 1 to 1.75 K steps to land
// instead of about 1.75. Measured in one process on three boxes: the persistent EP FFN 1.6-1.9 %
// faster, plain GEMMs with K of 7168 or more 0-1.5 % slower (where every CU streams weights at
// once and the longer lead pays), K = 1024 unchanged; the EP kernels use it, the plain and
// scatter GEMMs do not. Output is bit-identical either way.
template <int NI, bool kLateB>
__device__ __forceinline__ void mainloop_ni(const TileAddr& ta, int nk, Acc& acc, char* lds) {
  const int lane = threadIdx.x & 63;
  const int w = ta.w;
  const int swz = (lane >> 1) & 7;
  const int khalf = lane >> 5;
  auto issue_a = [&](int kt) {
    char* st = lds + (kt & 1) * kOpBytes;
    const char* a0 = ta.a + kt * kBK * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_global_load_lds((glob_void*)(a0 + ta.oa[i]), (lds_void*)(st + (8 * i + w) * 1024),
                                       16, 0, 0);
  };
  auto issue_b = [&](int kt, int slot) {
    char* st = lds + kBBase + slot * kOpBytes;
    const char* b0 = ta.b + kt * kBK * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_global_load_lds((glob_void*)(b0 + ta.ob[i]), (lds_void*)(st + (8 * i + w) * 1024),
                                       16, 0, 0);
  };
  bf16x8 af[2][4], bfr[2][2];
  auto frags = [&](const char* ca, const char* cb, int kk, int buf) {
    if (NI == 0) return;
    const int piece = (((kk * 2 + khalf) ^ swz) << 4);
#pragma unroll
    for (int i = 0; i < NI; ++i)
      af[buf][i] = *reinterpret_cast<const bf16x8*>(ca + ta.arow + i * 32 * kBK * 2 + piece);
#pragma unroll
    for (int j = 0; j < 2; ++j)
      bfr[buf][j] = *reinterpret_cast<const bf16x8*>(cb + ta.brow + j * 32 * kBK * 2 + piece);
  };
  auto mma = [&](int buf, int i0, int i1) {
#pragma unroll
    for (int i = i0; i < i1; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[buf][j], af[buf][i], acc[i][j], 0, 0, 0);
  };
  // per sub-step: 2 NI MFMAs and NI + 2 fragment reads
  constexpr int kReads = NI + 2, kMfma = 2 * NI;
  // Issue order: A(0), B(0), B(1) | A(1), B(2) | A(2), B(3) | ... At the boundary into
  // stage s + 1 the loads newer than A(s + 1) are only B(s + 2) (4 per wave), so waiting for
  // stage s + 1 is vmcnt(4), or vmcnt(0) when B(s + 2) does not exist.
  issue_a(0);
  issue_b(0, 0);
  if (nk > 1) {
    issue_b(1, 1);
    __builtin_amdgcn_s_waitcnt(0x0F74);   // vmcnt(4): A(0) and B(0) have landed
  } else {
    wait_vm0();
  }
  __builtin_amdgcn_s_barrier();
  if (nk > 1) issue_a(1);
  if (!kLateB && nk > 2) issue_b(2, 2);
  frags(lds, lds + kBBase, 0, 0);
  // One stage. NEXT: a stage follows; IA: A(kt + 2) exists (then B(kt + 2) is the only newer
  // load at the boundary: vmcnt(4)); IB: B(kt + 3) exists. Compile-time, so the steady loop
  // body is one basic block: with the boundary's conditions inside the loop the register
  // allocator split the accumulators' live ranges and copied all of them every stage.
  // one fragment read r of sub-step kk into buffer buf: 0, 1 = B blocks, 2.. = A blocks
  auto read_one = [&](const char* ca, const char* cb, int kk, int buf, int r) {
    const int piece = (((kk * 2 + khalf) ^ swz) << 4);
    if (r < 2)
      bfr[buf][r] = *reinterpret_cast<const bf16x8*>(cb + ta.brow + r * 32 * kBK * 2 + piece);
    else
      af[buf][r - 2] = *reinterpret_cast<const bf16x8*>(ca + ta.arow + (r - 2) * 32 * kBK * 2 + piece);
  };
  auto mma_one = [&](int buf, int g) {
    const int i = g >> 1, j = g & 1;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[buf][j], af[buf][i], acc[i][j], 0, 0, 0);
  };
  // one direct load n of stage kt + 2 (A, n < 4) or kt + 3 (B, n >= 4, into slot bs)
  auto load_one = [&](int kt, int bs, int n) {
    if (n < 4) {
      char* st = lds + (kt & 1) * kOpBytes;
      const char* a0 = ta.a + (kt + 2) * kBK * 2;
      __builtin_amdgcn_global_load_lds((glob_void*)(a0 + ta.oa[n]), (lds_void*)(st + (8 * n + w) * 1024), 16, 0, 0);
    } else {
      char* st = lds + kBBase + bs * kOpBytes;
      const char* b0 = ta.b + (kt + 3) * kBK * 2;
      __builtin_amdgcn_global_load_lds((glob_void*)(b0 + ta.ob[n - 4]), (lds_void*)(st + (8 * (n - 4) + w) * 1024),
                                       16, 0, 0);
    }
  };
  // kLateB: direct load n of B(kt + 2) into its slot bs2 (that of B(kt - 1))
  auto load_b_late = [&](int kt, int bs2, int n) {
    char* st = lds + kBBase + bs2 * kOpBytes;
    const char* b0 = ta.b + (kt + 2) * kBK * 2;
    __builtin_amdgcn_global_load_lds((glob_void*)(b0 + ta.ob[n]), (lds_void*)(st + (8 * n + w) * 1024), 16, 0, 0);
  };
  auto stage = [&](int kt, int bs, auto next_c, auto ia_c, auto ib_c) {
    constexpr bool kNext = decltype(next_c)::value;
    constexpr bool kIA = decltype(ia_c)::value;
    constexpr bool kIB = decltype(ib_c)::value;
    const char* ca = lds + (kt & 1) * kOpBytes;
    const char* cb = lds + kBBase + bs * kOpBytes;
    const int bs_next = bs == 2 ? 0 : bs + 1;
    const char* na = lds + ((kt + 1) & 1) * kOpBytes;
    const char* nb = lds + kBBase + bs_next * kOpBytes;
    // kLateB: B(kt + 2) exists exactly when A(kt + 2) does
    constexpr bool kLate = kLateB && kIA;
    const int bs_prev = bs == 0 ? 2 : bs - 1;
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < kMfma; ++g) {
        mma_one(kk & 1, g);
        if (g < kReads) read_one(ca, cb, kk + 1, (kk + 1) & 1, g);
        if constexpr (kLate) {   // loads kk after the first MFMA of sub-step kk, load 3 mid sub-step 0
          if (g == 0) load_b_late(kt, bs_prev, kk);
          if (kk == 0 && g == kMfma / 2) load_b_late(kt, bs_prev, 3);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int r = kMfma; r < kReads; ++r) read_one(ca, cb, kk + 1, (kk + 1) & 1, r);
      if constexpr (kLate && kMfma == 0) {
        load_b_late(kt, bs_prev, kk);
        if (kk == 0) load_b_late(kt, bs_prev, 3);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kNext) {
      // this wave's reads of stage kt are done and its loads of stage kt + 1 have landed (only
      // B(kt + 2) may still be in flight) ... and every wave's (bare s_barrier, see above);
      // kLateB issues B(kt + 2) in this stage, after A(kt + 1), so the count is the same
      __builtin_amdgcn_s_waitcnt(kIA ? 0x0074 : 0x0070);   // vmcnt(4 or 0) lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
    }
    __builtin_amdgcn_sched_barrier(0);
    // Sub-step 3 runs at raised wave priority: the wave that has passed the barrier issues its
    // MFMAs, next-stage reads and loads ahead of the SIMD's other wave (measured on the EP FFN:
    // -1.1 %, output unchanged; placing it over sub-steps 0-2 instead was slower).
    __builtin_amdgcn_s_setprio(1);
    constexpr int kLoads = (kIA ? 4 : 0) + (kIB && !kLateB ? 4 : 0);
    // sub-step 3: each MFMA followed by one read of the next stage's sub-step 0 and one load
#pragma unroll
    for (int g = 0; g < kMfma; ++g) {
      mma_one(1, g);
      if constexpr (kNext) {
        if (g < kReads) read_one(na, nb, 0, 0, g);
      }
      if (g < kLoads) load_one(kt, bs, kIA ? g : g + 4);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (kNext) {
#pragma unroll
      for (int r = kMfma; r < kReads; ++r) read_one(na, nb, 0, 0, r);
    }
    __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int n = kMfma; n < kLoads; ++n) load_one(kt, bs, kIA ? n : n + 4);
  };
  const std::true_type yes;
  const std::false_type no;
  int kt = 0, bs = 0;   // bs: B slot of stage kt (kt mod 3)
  for (; kt + 3 < nk; ++kt, bs = bs == 2 ? 0 : bs + 1) stage(kt, bs, yes, yes, yes);
  if (kt + 2 < nk) {
    stage(kt, bs, yes, yes, no);
    ++kt;
    bs = bs == 2 ? 0 : bs + 1;
  }
  if (kt + 1 < nk) {
    stage(kt, bs, yes, no, no);
    ++kt;
    bs = bs == 2 ? 0 : bs + 1;
  }
  stage(kt, bs, no, no, no);
}

// acc = A[0:256, 0:K] * B[rows(0:256), 0:K]^T. Rows of A at or beyond a_rows read row
// a_rows - 1 and their 32-row blocks are skipped where a whole block is past a_rows (their
// results are zero or stale and are never stored). Ends with a block barrier, after which the
// LDS may be reused. Accumulator layout: acc[i][j][q] is output
//   row wm*128 + 32 i + lane % 32, column wn*64 + 32 j + 8 (q / 4) + 4 (lane / 32) + q % 4.
template <bool kLateB = false>
__device__ __forceinline__ void gemm_mainloop(const uint16_t* __restrict__ A, int64_t lda,
                                              int a_rows, const uint16_t* __restrict__ B,
                                              int64_t ldb, int b_n0, int b_half, bool swiglu,
                                              int K, Acc& acc, char* lds) {
  const int lane = threadIdx.x & 63;
  // the wave index is uniform: keep it scalar so the LDS destinations (M0) are scalar math
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 2, wn = w & 3;
  TileAddr ta;
  ta.a = reinterpret_cast<const char*>(A);
  ta.b = reinterpret_cast<const char*>(B);
  ta.w = w;
  // direct-load sources: instruction i of wave w fills rows [64 i + 8 w, +8) of a stage; the
  // swizzle term of those rows does not depend on i. 32-bit byte offsets from the
  // wave-uniform bases keep the per-lane state small and let the loads use the
  // scalar-base + vector-offset addressing form.
  const int lr = lane >> 3, lp = lane & 7;
  const int c16 = (lp ^ ((4 * w + (lr >> 1)) & 7)) * 16;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 64 * i + 8 * w + lr;
    const int ar = r < a_rows ? r : a_rows - 1;
    ta.oa[i] = static_cast<uint32_t>(ar * lda * 2 + c16);
    ta.ob[i] = static_cast<uint32_t>(b_row_map(r, b_n0, b_half, swiglu) * ldb * 2 + c16);
  }
  // fragment reads: row (wm*128 + i*32 + lane%32) of A, (wn*64 + j*32 + lane%32) of B, as
  // byte offsets inside a stage buffer
  ta.arow = (wm * 128 + (lane & 31)) * kBK * 2;
  ta.brow = (wn * 64 + (lane & 31)) * kBK * 2;
  zero_acc(acc);
  const int nk = K / kBK;
  const int valid = a_rows - wm * 128;
  const int ni = valid >= 128 ? 4 : (valid <= 0 ? 0 : (valid + 31) >> 5);
  switch (__builtin_amdgcn_readfirstlane(ni)) {
    case 4: mainloop_ni<4, kLateB>(ta, nk, acc, lds); break;
    case 3: mainloop_ni<3, kLateB>(ta, nk, acc, lds); break;
    case 2: mainloop_ni<2, kLateB>(ta, nk, acc, lds); break;
    case 1: mainloop_ni<1, kLateB>(ta, nk, acc, lds); break;
    default: mainloop_ni<0, kLateB>(ta, nk, acc, lds); break;
  }
  __syncthreads();
}

// Accumulators -> bf16 tile in LDS, row-major [256][kEpiPitch]; four columns per 8-byte write.
__device__ __forceinline__ void stage_tile(const Acc& acc, char* lds) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 2, wn = w & 3;
  const int row0 = wm * 128 + (lane & 31);
  const int col0 = wn * 64 + 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 v;
        v.x = pack_bf16x2(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
        v.y = pack_bf16x2(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
        const int row = row0 + 32 * i, col = col0 + 32 * j + 8 * g;
        *reinterpret_cast<uint2*>(lds + (row * kEpiPitch + col) * 2) = v;
      }
}

// SwiGLU of a gate/up tile -> bf16 h tile [256][kEpiPitchH] in LDS (128 columns): B block 0
// of a wave holds the gate rows and block 1 the up rows of the same 32 output columns, so
// gate and up of one output sit in the same lane and register index.
__device__ __forceinline__ void stage_swiglu(const Acc& acc, char* lds) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 2, wn = w & 3;
  const int row0 = wm * 128 + (lane & 31);
  const int col0 = wn * 32 + 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float h[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float gt = acc[i][0][4 * g + q], up = acc[i][1][4 * g + q];
        // silu(g) = g / (1 + e^-g), with the hardware reciprocal (about 1 ulp) in place of an
        // IEEE division sequence
        h[q] = gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up;
      }
      uint2 v;
      v.x = pack_bf16x2(h[0], h[1]);
      v.y = pack_bf16x2(h[2], h[3]);
      const int row = row0 + 32 * i, col = col0 + 8 * g;
      *reinterpret_cast<uint2*>(lds + (row * kEpiPitchH + col) * 2) = v;
    }
}

// Stores staged rows [0, rows) through the per-row destination pointers in LDS (null rows are
// skipped). cols = 256 (plain) or 128 (SwiGLU). Every piece is one 128-bit store.
__device__ __forceinline__ void store_rows(const char* lds_bytes, int pitch, int cols, int rows,
                                           char* const* rowptr) {
  typedef __attribute__((address_space(1))) u32x4 global_u32x4;
  const uint16_t* lds = reinterpret_cast<const uint16_t*>(lds_bytes);
  const int tid = threadIdx.x;
  const int per_row = cols / 8;                // 16-byte pieces per row
  const int rows_per_pass = kThreads / per_row;
  const int pc = tid % per_row;
  // global-address stores (a generic pointer would make them flat stores, which also count
  // against the LDS wait counter); no unrolling, so no per-row LDS addresses are held (and
  // spilled) across the loop. (Measured: nontemporal stores here slow the next tiles'
  // mainloops by about 5 %.)
#pragma unroll 1
  for (int r = tid / per_row; r < rows; r += rows_per_pass) {
    char* p = rowptr[r];
    if (!p) continue;
    const u32x4 v = *reinterpret_cast<const u32x4*>(lds + r * pitch + pc * 8);
    *(global_u32x4*)(p + pc * 16) = v;
  }
}

}  // namespace xs
