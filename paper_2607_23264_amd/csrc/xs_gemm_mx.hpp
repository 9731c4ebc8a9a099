// MXFP8 GEMM core for gfx950: E4M3 operands with one E8M0 scale per 32 elements along K, on
// v_mfma_scale_f32_32x32x64_f8f6f4. 256 x 256 output tile, 256 threads = 4 waves, one per
// SIMD, as 2 (M) x 2 (N) waves of 128 x 128 each = 4 x 4 blocks of 32 x 32 (256 fp32
// accumulators per lane). An fp8 fragment is twice a bf16 one, so the bf16 core's two waves
// per SIMD (128 x 64 each) cannot hold double-buffered fragments and the block scales within
// their 256 registers; one wave per SIMD has 512, and a 128 x 128 wave reads half the LDS
// bytes per MFMA.
//
// LDS: two stages, each with an A and a B operand tile of 256 rows x 128 bytes (here 128 K
// elements; logical piece c of row r at c ^ ((r >> 1) & 7), as in the bf16 core), 128 KiB,
// and two scale groups at the top of the LDS. A group holds, per A and per B row, the 16
// bytes of block scales of four stages (K elements [512 g, 512 g + 512): stage kt reads the
// 32-bit word kt % 4 of group kt / 4). Everything arrives by direct global -> LDS loads, the
// swizzle applied on the global side (instruction i of wave w fills operand rows 32 i + 8 w
// .. + 7). A row's scale bytes are contiguous in memory, so loading one 4-byte word per row
// and stage would touch a different cache line in every lane (64 lines per instruction, as
// many as all of the stage's code loads together). Instead each stage loads one quarter of
// the next group: wave w's scale instruction covers rows 64 w + 16 q .. + 15 of quarter q,
// four lanes per row reading its 16 contiguous bytes, which divides those line touches by
// four with every lane active (no branch in the K loop). A stage is 32
// MFMAs of 64 cycles per wave (one wave per SIMD), so loading it one stage ahead gives the
// loads about as long to land as the bf16 core's three-deep weight pipeline does.
//
// Operand layout of the scaled MFMA (measured on gfx950): lane 32 h + i holds row i's K
// elements [16 h, 16 h + 16) in bytes 0..15 and [32 + 16 h, 48 + 16 h) in bytes 16..31 of its
// eight dwords (an fp4 operand: elements [32 h, 32 h + 32), two per byte, in the first four
// dwords), and the scale of K block b (32 elements) of row i comes from lane 32 b + i, in
// the byte op_sel names. Sub-step kk of a stage (K elements [64 kk, 64 kk + 64)) reads pieces
// 4 kk + h and 4 kk + 2 + h of an fp8 row, or piece 2 kk + h of an fp4 row; a lane's scale
// word for the stage holds the row's four block scales, and one byte permute puts the scale
// of block 2 kk + h into byte kk.
//
// B may be E2M1 (W4A8): its tile rows are then 64 bytes per stage (four 16-byte pieces,
// piece c at c ^ ((row >> 2) & 3), so the 16 rows of each ds_read_b128 phase hit 16 distinct
// bank groups) in the first half of the B area; the MFMA rate is that of fp8.
#pragma once
#include <type_traits>

#include "xs_gemm.hpp"

namespace xs {

// The lane index, computed where it is used: the asm is volatile, so the value (and the LDS
// addresses derived from it) is not hoisted into a register kept live across the mainloop,
// where these kernels are short of registers and would spill it to scratch.
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// The thread index, with its lane part computed where it is used (lane_id_here) and its wave
// part uniform.
__device__ __forceinline__ int tid_here() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x & ~63u) + lane_id_here();
}

constexpr int kMxThreads = 256;
constexpr int kMxStage = 2 * kOpBytes;             // A tile and B tile of one stage: 64 KiB
constexpr int kMxScaleBuf = 2 * kBM * 16;          // one scale group: 16 bytes per A and B row
constexpr int kMxScaleOff = kLdsBytes - 2 * kMxScaleBuf;
static_assert(2 * kMxStage <= kMxScaleOff, "the MX stages and scale groups fit the LDS");
// the epilogue's row pointers and the scheduler scratch (touched between mainloops) lie below
static_assert(kLdsMiscOff + 64 <= kMxScaleOff, "scale groups clear of the scheduler scratch");
typedef int v8i_t __attribute__((ext_vector_type(8)));
typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef f32x16 AccMx[4][4];

struct MxTile {
  const char* a;          // A code base (tile row 0, k 0)
  const char* b;          // B code base
  const char* sa;         // A scale base (tile row 0)
  const char* sb;         // B scale base
  uint32_t oa[8], ob[8];  // per-lane byte offsets of the eight direct loads of each operand
  // scale word this lane loads in quarter q: A at min(sa0 + q * sa16, samax), B at sb0 +
  // (q % 2) * sbq1 + (q / 2) * sbq2 (row offsets are linear in q; uniform strides); group g
  // of either operand starts g * sa_grp / sb_grp bytes further
  uint32_t sa0, samax, sb0;
  uint32_t sa16, sbq1, sbq2;
  int64_t sa_grp, sb_grp;
  int ar, br;             // this lane's fragment rows in the A and B tiles
  int arow, brow;         // their LDS byte offsets within an operand tile
  int w;
};

template <int NI, bool BF4>
__device__ __forceinline__ void mainloop_mx_ni(const MxTile& t, int nk, AccMx& acc, char* lds) {
  const int lane = threadIdx.x & 63;
  const int w = t.w;
  const int swz = (lane >> 1) & 7;          // fp8 rows: 8 pieces, piece c at c ^ ((row >> 1) & 7)
  const int swz4 = (lane >> 2) & 3;         // fp4 rows: 4 pieces, piece c at c ^ ((row >> 2) & 3)
  const int h = lane >> 5;
  const uint32_t sel = h ? 0x0C0C0301u : 0x0C0C0200u;
  // B as E2M1 (BF4): 64-byte tile rows per stage (four direct loads per wave instead of
  // eight), one 16-byte fragment read per sub-step, and the MFMA told its first operand is fp4
  constexpr int kBLoads = BF4 ? 4 : 8;
  constexpr int kLoads = 8 + kBLoads;                  // operand loads per wave and stage
  constexpr uint32_t kBStep = BF4 ? 64u : 128u;        // B bytes per row and stage
  constexpr int kBRow = BF4 ? 64 : 128;                // B tile row pitch in LDS
  constexpr int kFmtB = BF4 ? 4 : 0;
  // Addresses are the uniform base plus a 32-bit per-lane offset that includes the stage
  // (a 32-bit sum that may wrap is not folded into loop-invariant 64-bit per-lane pointers,
  // which would cost two registers per load): the loads keep the scalar-base + vector-offset
  // form. Direct load n of stage kt: 0..7 A pieces, 8.. B pieces; then, in a stage that issues
  // loads, the two scale loads (A rows, B rows) of one quarter of a group.
  auto issue_one = [&](int kt, int n) {
    char* st = lds + (kt & 1) * kMxStage;
    if (n < 8)
      __builtin_amdgcn_global_load_lds((glob_void*)(t.a + (t.oa[n] + static_cast<uint32_t>(kt) * 128u)),
                                       (lds_void*)(st + (4 * n + w) * 1024), 16, 0, 0);
    else
      __builtin_amdgcn_global_load_lds((glob_void*)(t.b + (t.ob[n - 8] + static_cast<uint32_t>(kt) * kBStep)),
                                       (lds_void*)(st + kOpBytes + (4 * (n - 8) + w) * 1024), 16, 0, 0);
  };
  auto issue = [&](int kt) {
#pragma unroll
    for (int n = 0; n < kLoads; ++n) issue_one(kt, n);
  };
  // scale load n (0: A rows, 1: B rows) of quarter q of group g, into group buffer g % 2 (row
  // r's 16 bytes at r * 16, so the lanes' words land in order). A group past the last one
  // reads the last group's bytes (in bounds; that buffer is no longer read).
  const int last_group = (nk >> 2) - 1;
  auto issue_scale = [&](int g, int n, int q) {
    char* sb = lds + kMxScaleOff + (g & 1) * kMxScaleBuf + n * (kBM * 16) + (64 * w + 16 * q) * 16;
    const uint32_t uq = static_cast<uint32_t>(q);
    const uint32_t oq = n ? t.sb0 + (uq & 1u) * t.sbq1 + (uq >> 1) * t.sbq2 : min(t.sa0 + uq * t.sa16, t.samax);
    const char* base = (n ? t.sb : t.sa) + min(g, last_group) * (n ? t.sb_grp : t.sa_grp);
    __builtin_amdgcn_global_load_lds((glob_void*)(base + oq), (lds_void*)sb, 4, 0, 0);
  };
  uint32_t sw[8];         // a stage's scale words as read: A blocks 0..3, B blocks 0..3
  int sc[8];              // the same, byte kk = scale of K block 2 kk + h (the MFMA's op_sel)
  auto read_s = [&](int ks) {   // the scale words of stage ks
    const char* sg = lds + kMxScaleOff + ((ks >> 2) & 1) * kMxScaleBuf + (ks & 3) * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      sw[i] = *reinterpret_cast<const uint32_t*>(sg + (t.ar + 32 * i) * 16);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      sw[4 + j] = *reinterpret_cast<const uint32_t*>(sg + kBM * 16 + (t.br + 32 * j) * 16);
  };
  auto perm_s = [&]() {
#pragma unroll
    for (int n = 0; n < 8; ++n) sc[n] = static_cast<int>(__builtin_amdgcn_perm(sw[n], sw[n], sel));
  };
  // fragments of sub-step 0 (K elements [0, 64) of a stage) and of sub-step 1 ([64, 128))
  v8i_t a0[4], b0[4], a1[4], b1[4];
  auto frag = [&](const char* base, int row_off, int kk) {
    const v4i_t lo = *reinterpret_cast<const v4i_t*>(base + row_off + (((4 * kk + h) ^ swz) << 4));
    const v4i_t hi = *reinterpret_cast<const v4i_t*>(base + row_off + (((4 * kk + 2 + h) ^ swz) << 4));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  // B fragment j of sub-step kk: an fp4 operand is 32 codes (16 bytes) per lane, in the low
  // four registers (the MFMA ignores the upper four)
  auto frag_b = [&](const char* st, int j, int kk) {
    if constexpr (BF4) {
      const char* base = st + kOpBytes + t.brow + j * 32 * kBRow;
      const v4i_t v = *reinterpret_cast<const v4i_t*>(base + (((2 * kk + h) ^ swz4) << 4));
      return __builtin_shufflevector(v, v, 0, 1, 2, 3, -1, -1, -1, -1);
    } else {
      return frag(st + kOpBytes, t.brow + j * 32 * kBRow, kk);
    }
  };
  auto read_frags = [&](const char* st, int kk, v8i_t (&a)[4], v8i_t (&b)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) b[j] = frag_b(st, j, kk);
#pragma unroll
    for (int i = 0; i < NI; ++i) a[i] = frag(st, t.arow + i * 32 * 128, kk);
  };
  constexpr int kMfma = 4 * NI;             // MFMAs per sub-step
  // One stage. The schedule is fixed by hand, one MFMA and what follows it per fenced group
  // (left alone, the compiler sinks every MFMA of the stage below the barrier, leaves the
  // fragment reads exposed and issues the global loads in one burst):
  //   A: sub-step 0's MFMAs, the first eight each followed by one fragment read of sub-step 1;
  //   barrier: this wave's reads of the stage are done and the next stage has landed in every
  //     wave's share;
  //   B: sub-step 1's MFMAs, each followed by two global loads of the stage after next (into
  //     this stage's buffers, which no wave reads any more) and one read of the next stage's
  //     scale words or sub-step-0 fragments. Among the loads are the scale loads of quarter
  //     (kt + 1) % 4 of group (kt + 1) / 4 + 1: its buffer last held group (kt + 1) / 4 - 1,
  //     whose final words were read in stage 4 ((kt + 1) / 4) - 2 or earlier, before this
  //     stage's barrier; its last quarter lands by the barrier of stage 4 ((kt + 1) / 4) + 3,
  //     before the group's first words are read. Past the last group the loads repeat the
  //     last group into the other buffer, which is no longer read (no branch).
  // NEXT: a stage follows; ISSUE: the stage after next exists. Compile-time, so the steady
  // loop body has no branches.
  auto stage = [&](int kt, auto next_c, auto issue_c) {
    constexpr bool kNext = decltype(next_c)::value;
    constexpr bool kIssue = decltype(issue_c)::value;
    const char* st = lds + (kt & 1) * kMxStage;
    const char* nx = lds + ((kt + 1) & 1) * kMxStage;
    const int sg = ((kt + 1) >> 2) + 1;
    const int sq = (kt + 1) & 3;
    // load n of this stage's issue: 0..7 A pieces, 8 / 9 scale quarter (A / B rows), 10.. B
    auto load_n = [&](int n) {
      if (n < 8) issue_one(kt + 2, n);
      else if (n < 10) issue_scale(sg, n - 8, sq);
      else issue_one(kt + 2, n - 2);
    };
    constexpr int kAll = kLoads + 2;
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NI > 0) {
#pragma unroll
      for (int g = 0; g < kMfma; ++g) {
        const int i = g >> 2, j = g & 3;   // B fragment first: a lane's accumulators hold 4 columns
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(b0[j], a0[i], acc[i][j], kFmtB, 0, 0,
                                                                    sc[4 + j], 0, sc[i]);
        if (g < 4) b1[g] = frag_b(st, g, 1);
        else if (g - 4 < NI) a1[g - 4] = frag(st, t.arow + (g - 4) * 32 * 128, 1);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int r = kMfma; r < 4 + NI; ++r) {   // reads left over when there are few MFMAs
        if (r < 4) b1[r] = frag_b(st, r, 1);
        else a1[r - 4] = frag(st, t.arow + (r - 4) * 32 * 128, 1);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kNext) {
      __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0)
      __builtin_amdgcn_s_barrier();
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NI > 0) {
#pragma unroll
      for (int g = 0; g < kMfma; ++g) {
        const int i = g >> 2, j = g & 3;
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(b1[j], a1[i], acc[i][j], kFmtB, 0, 1,
                                                                    sc[4 + j], 1, sc[i]);
        if constexpr (kIssue) {
          if (2 * g < kAll) load_n(2 * g);
          if (2 * g + 1 < kAll) load_n(2 * g + 1);
        }
        if constexpr (kNext) {
          if (g == 0) read_s(kt + 1);
          else if (g - 1 < 4) b0[g - 1] = frag_b(nx, g - 1, 0);
          else if (g - 5 < NI) a0[g - 5] = frag(nx, t.arow + (g - 5) * 32 * 128, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // what did not fit beside the MFMAs
      if constexpr (kIssue) {
#pragma unroll
        for (int n = 2 * kMfma; n < kAll; ++n) load_n(n);
      }
      if constexpr (kNext) {
#pragma unroll
        for (int r = kMfma; r < 5 + NI; ++r) {
          if (r == 0) read_s(kt + 1);
          else if (r - 1 < 4) b0[r - 1] = frag_b(nx, r - 1, 0);
          else a0[r - 5] = frag(nx, t.arow + (r - 5) * 32 * 128, 0);
        }
      }
    } else if constexpr (kIssue) {
#pragma unroll
      for (int n = 0; n < kAll; ++n) load_n(n);
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kNext && NI > 0) perm_s();
  };
  // prologue: stage 0 and scale group 0 resident, stage 1 and the first quarter of group 1
  // in flight, stage 0's sub-step-0 operands in registers
  issue(0);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    issue_scale(0, 0, q);
    issue_scale(0, 1, q);
  }
  wait_vm0();
  __builtin_amdgcn_s_barrier();
  if (nk > 1) issue(1);
  issue_scale(1, 0, 0);   // group 1, or (K = 512) group 0 again into the unused buffer
  issue_scale(1, 1, 0);
  if constexpr (NI > 0) {
    read_s(0);
    read_frags(lds, 0, a0, b0);
    perm_s();
  }
  const std::true_type yes;
  const std::false_type no;
  int kt = 0;
  for (; kt + 2 < nk; ++kt) stage(kt, yes, yes);
  if (kt + 1 < nk) {
    stage(kt, yes, no);
    ++kt;
  }
  stage(kt, no, no);
}

// acc = deq(A)[0:256, 0:K] deq(B)[rows(0:256), 0:K]^T. A: E4M3 code rows (lda bytes apart,
// 16-byte aligned); B: E4M3 code rows, or with BF4 E2M1 codes packed two per byte (low nibble
// first, K / 2 bytes per row), ldb bytes apart, 16-byte aligned; As / Bs: E8M0 scales, the 16
// bytes of row r's blocks [16 g, 16 g + 16) (K elements [512 g, 512 g + 512)) at r * srow + g
// * sgrp: row-major scale rows are (srow = row bytes, sgrp = 16), the grouped layout [K / 512]
// [rows][16] is (16, 16 * rows). 16-byte aligned. K a multiple of 512. B rows map
// through b_row_map (SwiGLU interleave). Rows of A at or beyond a_rows read row a_rows - 1; a
// wave skips the MFMAs of 32-row blocks past a_rows. Ends with a block barrier. Accumulator
// acc[i][j][q] is output
//   row wm*128 + 32 i + lane % 32, column wn*128 + 32 j + 8 (q / 4) + 4 (lane / 32) + q % 4.
template <bool BF4 = false>
__device__ __forceinline__ void gemm_mainloop_mx(const uint8_t* __restrict__ A, int64_t lda,
                                                 const uint8_t* __restrict__ As, int64_t a_srow,
                                                 int64_t a_sgrp, int a_rows,
                                                 const uint8_t* __restrict__ B, int64_t ldb,
                                                 const uint8_t* __restrict__ Bs, int64_t b_srow,
                                                 int64_t b_sgrp, int b_n0, int b_half, bool swiglu,
                                                 int K, AccMx& acc, char* lds) {
  const int lane = lane_id_here();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  MxTile t;
  t.a = reinterpret_cast<const char*>(A);
  t.b = reinterpret_cast<const char*>(B);
  t.sa = reinterpret_cast<const char*>(As);
  t.sb = reinterpret_cast<const char*>(Bs);
  t.w = w;
  // fp8 rows: instruction i of wave w fills rows 32 i + 8 w .. + 7, lane -> (row lane / 8,
  // physical piece lane % 8) holding logical piece (lane % 8) ^ ((row >> 1) & 7)
  const int lr = lane >> 3, lp = lane & 7;
  const int c16 = (lp ^ ((4 * w + (lr >> 1)) & 7)) * 16;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = 32 * i + 8 * w + lr;
    const int ar = r < a_rows ? r : a_rows - 1;
    t.oa[i] = static_cast<uint32_t>(ar * lda + c16);
    if constexpr (!BF4) t.ob[i] = static_cast<uint32_t>(b_row_map(r, b_n0, b_half, swiglu) * ldb + c16);
  }
  if constexpr (BF4) {
    // fp4 rows (64 bytes): instruction i of wave w fills rows 16 (4 i + w) .. + 15, lane ->
    // (row lane / 4, physical piece lane % 4) holding logical piece (lane % 4) ^ ((row >> 2) & 3)
    const int c4 = ((lane & 3) ^ ((lane >> 4) & 3)) * 16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * (4 * i + w) + (lane >> 2);
      t.ob[i] = static_cast<uint32_t>(b_row_map(r, b_n0, b_half, swiglu) * ldb + c4);
    }
  }
  // scale words: quarter q covers wave w's rows 64 w + 16 q + lane / 4, four lanes per row.
  // B rows through b_row_map move by 16 rows from q = 0 to 1 and by b_half (SwiGLU) or 32
  // rows from q = 0 to 2.
  const int rs = 64 * w + (lane >> 2);
  t.sa0 = static_cast<uint32_t>(rs * a_srow + (lane & 3) * 4);
  t.samax = static_cast<uint32_t>((a_rows - 1) * a_srow + (lane & 3) * 4);
  t.sa16 = static_cast<uint32_t>(16 * a_srow);
  t.sb0 = static_cast<uint32_t>(b_row_map(rs, b_n0, b_half, swiglu) * b_srow + (lane & 3) * 4);
  t.sbq1 = static_cast<uint32_t>(16 * b_srow);
  t.sbq2 = static_cast<uint32_t>((swiglu ? b_half : 32) * b_srow);
  t.sa_grp = a_sgrp;
  t.sb_grp = b_sgrp;
  t.ar = wm * 128 + (lane & 31);
  t.br = wn * 128 + (lane & 31);
  t.arow = t.ar * 128;
  t.brow = t.br * (BF4 ? 64 : 128);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  const int nk = K / 128;
  const int valid = a_rows - wm * 128;
  const int ni = valid >= 128 ? 4 : (valid <= 0 ? 0 : (valid + 31) >> 5);
  switch (__builtin_amdgcn_readfirstlane(ni)) {
    case 4: mainloop_mx_ni<4, BF4>(t, nk, acc, lds); break;
    case 3: mainloop_mx_ni<3, BF4>(t, nk, acc, lds); break;
    case 2: mainloop_mx_ni<2, BF4>(t, nk, acc, lds); break;
    case 1: mainloop_mx_ni<1, BF4>(t, nk, acc, lds); break;
    default: mainloop_mx_ni<0, BF4>(t, nk, acc, lds); break;
  }
  __syncthreads();
}

// Accumulators -> bf16 tile in LDS, row-major [256][kEpiPitch].
__device__ __forceinline__ void stage_tile_mx(const AccMx& acc, char* lds) {
  const int lane = lane_id_here(), w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int row0 = wm * 128 + (lane & 31);
  const int col0 = wn * 128 + 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 v;
        v.x = pack_bf16x2(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
        v.y = pack_bf16x2(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
        const int row = row0 + 32 * i, col = col0 + 32 * j + 8 * g;
        *reinterpret_cast<uint2*>(lds + (row * kEpiPitch + col) * 2) = v;
      }
}

// Shared exponent of an MXFP8 (E4M3) block from the bits of its largest magnitude as an fp32
// value: the smallest e with amax <= 448 2^e (448 = 1.75 2^8), i.e. e = E - 8 + [M > 1.75] for
// amax = M 2^E; 0 for an all-zero block; clamped to [-127, 127]. Integer arithmetic only.
__device__ __forceinline__ int mx_exp_e4m3_f32(uint32_t amax_bits) {
  if (amax_bits == 0) return 0;
  const int F = static_cast<int>(amax_bits >> 23);
  const uint32_t m = amax_bits & 0x7FFFFFu;
  int E, above;
  if (F != 0) {
    E = F - 127;
    above = m > 0x600000u;
  } else {                                       // fp32 subnormal: m 2^-149
    const int p = 31 - __builtin_clz(m);
    E = p - 149;
    above = static_cast<uint64_t>(m) * 4 > (7ull << p);
  }
  const int e = E - 8 + above;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// Staged MXFP8 h tile: 256 rows of 128 codes (pitch kHqPitch bytes) and, after them, 256
// rows of 4 scale bytes.
constexpr int kHqPitch = 144;
constexpr int kHqScaleOff = kBM * kHqPitch;

// SwiGLU of a gate/up tile, quantized to MXFP8 along its 128 output columns (four blocks of
// 32). B blocks 2 jj and 2 jj + 1 of a wave hold the gate and up rows of the same 32 output
// columns (block 2 wn + jj of the tile); a lane holds 16 of a row's 32 values of that block
// and lane ^ 32 the other 16, so the block maximum takes one half swap. Codes: the exact
// power-of-two scaling and the hardware round-to-nearest-even E4M3 conversion.
__device__ __forceinline__ void stage_swiglu_mxq(const AccMx& acc, char* lds) {
  const int lane = lane_id_here(), w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int up = lane >> 5;
  typedef uint32_t u32x2_ __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = wm * 128 + 32 * i + (lane & 31);
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      float hv[16];
      uint32_t amax = 0;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const float gt = acc[i][2 * jj][q], u = acc[i][2 * jj + 1][q];
        hv[q] = gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * u;
        amax = max(amax, __builtin_bit_cast(uint32_t, hv[q]) & 0x7FFFFFFFu);
      }
      const auto r = __builtin_amdgcn_permlane32_swap(amax, amax, false, false);
      const u32x2_ both = {r[0], r[1]};
      const int e = mx_exp_e4m3_f32(max(both.x, both.y));
      const int col0 = 32 * (2 * wn + jj) + 4 * up;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint32_t c = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(
            __builtin_amdgcn_ldexpf(hv[4 * g], -e), __builtin_amdgcn_ldexpf(hv[4 * g + 1], -e), 0, false));
        c = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(
            __builtin_amdgcn_ldexpf(hv[4 * g + 2], -e), __builtin_amdgcn_ldexpf(hv[4 * g + 3], -e),
            static_cast<int>(c), true));
        *reinterpret_cast<uint32_t*>(lds + row * kHqPitch + col0 + 8 * g) = c;
      }
      if (up == 0) lds[kHqScaleOff + row * 4 + 2 * wn + jj] = static_cast<char>(e + 127);
    }
  }
}

// Stores staged rows [0, rows) through per-row destination pointers (null rows skipped):
// pieces of 16 bytes, per_row pieces per row, pitch bytes between staged rows; NT threads.
// U rows' pointers and data are read from LDS before their U stores, so a pass waits for one
// LDS round trip instead of U.
template <int NT, int U = 4>
__device__ __forceinline__ void store_rows_n(const char* lds, int pitch, int per_row, int rows,
                                             char* const* rowptr) {
  typedef __attribute__((address_space(1))) u32x4 global_u32x4;
  const int tid = tid_here();
  const int rows_per_pass = NT / per_row;
  const int pc = tid % per_row;
#pragma unroll 1
  for (int r = tid / per_row; r < rows; r += U * rows_per_pass) {
    char* p[U];
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int ru = r + u * rows_per_pass;
      p[u] = nullptr;
      if (ru < rows) {
        p[u] = rowptr[ru];
        v[u] = *reinterpret_cast<const u32x4*>(lds + ru * pitch + pc * 16);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (p[u]) *(global_u32x4*)(p[u] + pc * 16) = v[u];
  }
}

}  // namespace xs
