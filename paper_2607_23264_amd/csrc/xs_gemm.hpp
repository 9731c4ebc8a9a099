// MFMA bf16 GEMM core for gfx950: 256x256 output tile, K step 64, 512 threads = 8 waves, two
// per SIMD, as 2 (M) x 4 (N) waves of 128 x 64 each = 4 x 2 blocks of
// v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per lane). Two waves per SIMD let one
// wave's LDS or memory wait be covered by the other's MFMAs; measured on an 8192^3 GEMM this
// beats one wave per SIMD of 128 x 128 (fewer LDS reads per MFMA, but every stall idles the
// matrix pipe) by about 20 %.
//
// Operands move global -> LDS with gfx950's direct 128-bit loads (global_load_lds_dwordx4):
// no staging registers and no LDS store instructions. Two LDS stages of [256][64] bf16 per
// operand (2 x 64 KiB); the loads of stage k+1 are issued right after the barrier that
// opens stage k and land while stage k is multiplied.
//
// LDS operand layout: 128 B per row in eight 16-byte pieces; logical piece c of row r sits at
// physical position c ^ ((r >> 1) & 7). A direct load writes 64 consecutive pieces (8 rows)
// per wave instruction, so the swizzle is applied on the global side: the lane that fills
// physical piece p of row r fetches logical piece p ^ ((r >> 1) & 7). The 16 lanes of each
// ds_read_b128 phase then hit 16 distinct 16-byte bank groups (no bank conflicts measured).
//
// C = A B^T: A rows are K-contiguous and B is output-major ([N][K], K-contiguous), so both
// MFMA operands are 16-byte contiguous reads from LDS.
#pragma once
#include "xs_common.hpp"

namespace xs {

constexpr int kBM = 256, kBN = 256, kBK = 64, kThreads = 512;
constexpr int kOpBytes = kBM * kBK * 2;                      // one operand stage: 32 KiB
constexpr int kStageBytes = 2 * kOpBytes;                    // A + B: 64 KiB
constexpr int kEpiPitch = kBN + 8;                           // bf16 per staged output row
constexpr int kEpiPitchH = kBN / 2 + 8;                      // SwiGLU output rows (128 wide)
constexpr int kLdsEpiBytes = kBM * kEpiPitch * 2;            // 135168
constexpr int kLdsRowPtrOff = kLdsEpiBytes;                  // 256 row pointers
constexpr int kLdsMiscOff = kLdsRowPtrOff + kBM * 8;         // small scheduler scratch
constexpr int kLdsBytes = kLdsMiscOff + 64;
static_assert(2 * kStageBytes <= kLdsEpiBytes, "operand stages must fit under the epilogue tile");

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

// acc = A[0:256, 0:K] * B[rows(0:256), 0:K]^T. Rows of A at or beyond a_rows read row
// a_rows - 1 (their results are never stored). Ends with a block barrier, after which the
// LDS may be reused.
__device__ __forceinline__ void gemm_mainloop(const uint16_t* __restrict__ A, int64_t lda,
                                              int a_rows, const uint16_t* __restrict__ B,
                                              int64_t ldb, int b_n0, int b_half, bool swiglu,
                                              int K, Acc& acc, char* lds) {
  const int lane = threadIdx.x & 63;
  // the wave index is uniform: keep it scalar so the LDS destinations (M0) are scalar math
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 2, wn = w & 3;
  // direct-load sources: instruction i of wave w fills rows [64 i + 8 w, +8) of a stage; the
  // swizzle term of those rows does not depend on i. 32-bit byte offsets from the
  // wave-uniform bases keep the per-lane state small and let the loads use the
  // scalar-base + vector-offset addressing form.
  const int lr = lane >> 3, lp = lane & 7;
  const int c16 = (lp ^ ((4 * w + (lr >> 1)) & 7)) * 16;
  uint32_t oa[4], ob[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 64 * i + 8 * w + lr;
    const int ar = r < a_rows ? r : a_rows - 1;
    oa[i] = static_cast<uint32_t>(ar * lda * 2 + c16);
    ob[i] = static_cast<uint32_t>(b_row_map(r, b_n0, b_half, swiglu) * ldb * 2 + c16);
  }
  // fragment reads: row (wm*128 + i*32 + lane%32) of A, (wn*64 + j*32 + lane%32) of B
  const int swz = (lane >> 1) & 7;
  const int khalf = lane >> 5;
  const int arow = (wm * 128 + (lane & 31)) * kBK * 2;
  const int brow = kOpBytes + (wn * 64 + (lane & 31)) * kBK * 2;

  zero_acc(acc);
  const int nk = K / kBK;
  auto issue = [&](int kt) {
    char* st = lds + (kt & 1) * kStageBytes;
    const char* a0 = reinterpret_cast<const char*>(A + kt * kBK);
    const char* b0 = reinterpret_cast<const char*>(B + kt * kBK);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int off = (8 * i + w) * 1024;   // 64 pieces of 16 B
      __builtin_amdgcn_global_load_lds((glob_void*)(a0 + oa[i]), (lds_void*)(st + off), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((glob_void*)(b0 + ob[i]), (lds_void*)(st + kOpBytes + off), 16,
                                       0, 0);
    }
  };
  // Software pipeline. Fragments are double-buffered in registers: the reads of k sub-step
  // kk + 1 are in flight while the 8 MFMAs of sub-step kk issue (sched_group_barrier pins the
  // MFMA / ds_read alternation; left alone the scheduler reuses one fragment register set and
  // waits out every LDS read). At a stage boundary half the MFMAs of the last sub-step are
  // issued before the vmcnt wait and the barrier, so the matrix pipe keeps working while the
  // workgroup synchronises; the reads of the next stage's first sub-step then overlap the
  // remaining MFMAs.
  bf16x8 af[2][4], bfr[2][2];
  auto frags = [&](const char* cur, int kk, int buf) {
    const int piece = (((kk * 2 + khalf) ^ swz) << 4);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      af[buf][i] = *reinterpret_cast<const bf16x8*>(cur + arow + i * 32 * kBK * 2 + piece);
#pragma unroll
    for (int j = 0; j < 2; ++j)
      bfr[buf][j] = *reinterpret_cast<const bf16x8*>(cur + brow + j * 32 * kBK * 2 + piece);
  };
  auto mma = [&](int buf, int i0, int i1) {
#pragma unroll
    for (int i = i0; i < i1; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[buf][i], bfr[buf][j], acc[i][j], 0, 0, 0);
  };
  issue(0);
  wait_vm0();
  __syncthreads();
  if (nk > 1) issue(1);
  frags(lds, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    const char* cur = lds + (kt & 1) * kStageBytes;
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
      frags(cur, kk + 1, (kk + 1) & 1);
      mma(kk & 1, 0, 4);
#pragma unroll
      for (int g = 0; g < 6; ++g) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one ds_read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    // sub-step 3 (fragments in buffer 1): half the MFMAs, then the stage boundary
    mma(1, 0, 2);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    if (kt + 1 < nk) {
      wait_vm0();          // this wave's loads of stage kt + 1 have landed
      __syncthreads();     // every wave's have, and stage kt is no longer read
      if (kt + 2 < nk) issue(kt + 2);
      frags(lds + ((kt + 1) & 1) * kStageBytes, 0, 0);
    }
    mma(1, 2, 4);
  }
  __syncthreads();
}

// Accumulators -> bf16 tile in LDS, row-major [256][kEpiPitch].
__device__ __forceinline__ void stage_tile(const Acc& acc, char* lds_bytes) {
  uint16_t* lds = reinterpret_cast<uint16_t*>(lds_bytes);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 2, wn = w & 3;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int row = wm * 128 + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
        const int col = wn * 64 + j * 32 + (lane & 31);
        lds[row * kEpiPitch + col] = static_cast<uint16_t>(f2bf(acc[i][j][q]));
      }
}

// SwiGLU of a gate/up tile -> bf16 h tile [256][kEpiPitchH] in LDS (128 columns): block 0 of
// a wave holds the gate values and block 1 the up values of the same 32 output columns.
__device__ __forceinline__ void stage_swiglu(const Acc& acc, char* lds_bytes) {
  uint16_t* lds = reinterpret_cast<uint16_t*>(lds_bytes);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 2, wn = w & 3;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const float g = acc[i][0][q], u = acc[i][1][q];
      const float h = g / (1.f + __expf(-g)) * u;
      const int row = wm * 128 + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
      const int col = wn * 32 + (lane & 31);
      lds[row * kEpiPitchH + col] = static_cast<uint16_t>(f2bf(h));
    }
}

// Stores staged rows [0, rows) through the per-row destination pointers in LDS (null rows are
// skipped). cols = 256 (plain) or 128 (SwiGLU). Every piece is one 128-bit store.
__device__ __forceinline__ void store_rows(const char* lds_bytes, int pitch, int cols, int rows,
                                           char* const* rowptr) {
  const uint16_t* lds = reinterpret_cast<const uint16_t*>(lds_bytes);
  const int tid = threadIdx.x;
  const int per_row = cols / 8;                // 16-byte pieces per row
  const int rows_per_pass = kThreads / per_row;
  const int pc = tid % per_row;
  for (int r = tid / per_row; r < rows; r += rows_per_pass) {
    char* p = rowptr[r];
    if (!p) continue;
    u32x4 v = *reinterpret_cast<const u32x4*>(lds + r * pitch + pc * 8);
    *reinterpret_cast<u32x4*>(p + pc * 16) = v;
  }
}

}  // namespace xs
