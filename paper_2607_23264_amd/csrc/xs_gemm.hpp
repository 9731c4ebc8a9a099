// MFMA bf16 GEMM core for gfx950: 256x256 output tile, K step 64, 512 threads (8 waves as
// 2 (M) x 4 (N), each wave 128 x 64 = 4 x 2 blocks of v_mfma_f32_32x32x16_bf16), operands
// double-buffered in LDS (2 x 64 KiB) and staged through registers one K step ahead.
//
// LDS operand layout: row-major [256][64] bf16 per operand, 128 B per row split into eight
// 16-byte pieces; piece c of row r sits at position c ^ ((r >> 1) & 7), so the 16 lanes of a
// ds_read_b128 / ds_write_b128 phase touch 16 distinct 16-byte bank groups.
//
// C = A B^T: A rows are K-contiguous, B is output-major ([N][K], K-contiguous), so both MFMA
// operands are 16-byte contiguous loads from LDS.
#pragma once
#include "xs_common.hpp"

namespace xs {

constexpr int kBM = 256, kBN = 256, kBK = 64, kThreads = 512;
constexpr int kOpElems = (kBM + kBN) * kBK;                 // one LDS stage, elements
constexpr int kLdsOperandBytes = 2 * kOpElems * 2;           // 131072
constexpr int kEpiPitch = kBN + 8;                           // bf16 per staged output row
constexpr int kEpiPitchH = kBN / 2 + 8;                      // SwiGLU output rows (128 wide)
constexpr int kLdsEpiBytes = kBM * kEpiPitch * 2;            // 135168
constexpr int kLdsRowPtrOff = kLdsEpiBytes;                  // 256 row pointers
constexpr int kLdsMiscOff = kLdsRowPtrOff + kBM * 8;         // small scheduler scratch
constexpr int kLdsBytes = kLdsMiscOff + 64;

// B tile row r -> weight row. SwiGLU tiles interleave gate and up rows in blocks of 32 so
// that each wave's 64 columns hold 32 gate columns and the 32 matching up columns.
__device__ __forceinline__ int b_row_map(int r, int n0, int half, bool swiglu) {
  return swiglu ? n0 + ((r >> 5) & 1) * half + (r >> 6) * 32 + (r & 31) : n0 + r;
}

__device__ __forceinline__ void zero_acc(f32x16 (&acc)[4][2]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
}

// acc += A[0:256, 0:K] * B[rows(0:256), 0:K]^T. Rows of A at or beyond a_rows read row
// a_rows - 1 (their results are never stored). Ends with a block barrier.
__device__ __forceinline__ void gemm_mainloop(const uint16_t* __restrict__ A, int64_t lda,
                                              int a_rows, const uint16_t* __restrict__ B,
                                              int64_t ldb, int b_n0, int b_half, bool swiglu,
                                              int K, f32x16 (&acc)[4][2], uint16_t* lds) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 2, wn = w & 3;
  const int pc = tid & 7, pr = tid >> 3;        // load piece / row of this thread
  const uint16_t* ga[4];
  const uint16_t* gb[4];
  int soff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int r = pr + 64 * i;
    int ar = r < a_rows ? r : a_rows - 1;
    ga[i] = A + static_cast<int64_t>(ar) * lda + pc * 8;
    gb[i] = B + static_cast<int64_t>(b_row_map(r, b_n0, b_half, swiglu)) * ldb + pc * 8;
    soff[i] = r * kBK + ((pc ^ ((r >> 1) & 7)) << 3);
  }
  // fragment read offsets (elements) inside one operand stage
  const int swz = (lane >> 1) & 7;
  const int khalf = lane >> 5;
  int aoff[4], boff[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) aoff[i] = (wm * 128 + i * 32 + (lane & 31)) * kBK;
#pragma unroll
  for (int j = 0; j < 2; ++j) boff[j] = kBM * kBK + (wn * 64 + j * 32 + (lane & 31)) * kBK;

  zero_acc(acc);
  const int nk = K / kBK;
  u32x4 ra[4], rb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ra[i] = *reinterpret_cast<const u32x4*>(ga[i]);
    rb[i] = *reinterpret_cast<const u32x4*>(gb[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<u32x4*>(lds + soff[i]) = ra[i];
    *reinterpret_cast<u32x4*>(lds + kBM * kBK + soff[i]) = rb[i];
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    uint16_t* cur = lds + (kt & 1) * kOpElems;
    const bool more = kt + 1 < nk;
    if (more) {
      const int k0 = (kt + 1) * kBK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ra[i] = *reinterpret_cast<const u32x4*>(ga[i] + k0);
        rb[i] = *reinterpret_cast<const u32x4*>(gb[i] + k0);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int piece = ((kk * 2 + khalf) ^ swz) << 3;
      bf16x8 af[4], bfr[2];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(cur + aoff[i] + piece);
#pragma unroll
      for (int j = 0; j < 2; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(cur + boff[j] + piece);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      uint16_t* nxt = lds + ((kt + 1) & 1) * kOpElems;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<u32x4*>(nxt + soff[i]) = ra[i];
        *reinterpret_cast<u32x4*>(nxt + kBM * kBK + soff[i]) = rb[i];
      }
    }
    __syncthreads();
  }
}

// Accumulators -> bf16 tile in LDS, row-major [256][kEpiPitch].
__device__ __forceinline__ void stage_tile(const f32x16 (&acc)[4][2], uint16_t* lds) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 2, wn = w & 3;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        int row = wm * 128 + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
        int col = wn * 64 + j * 32 + (lane & 31);
        lds[row * kEpiPitch + col] = static_cast<uint16_t>(f2bf(acc[i][j][q]));
      }
}

// SwiGLU of a gate/up tile -> bf16 h tile [256][kEpiPitchH] in LDS (128 columns).
__device__ __forceinline__ void stage_swiglu(const f32x16 (&acc)[4][2], uint16_t* lds) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 2, wn = w & 3;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      float g = acc[i][0][q], u = acc[i][1][q];
      float h = g / (1.f + __expf(-g)) * u;
      int row = wm * 128 + i * 32 + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
      int col = wn * 32 + (lane & 31);
      lds[row * kEpiPitchH + col] = static_cast<uint16_t>(f2bf(h));
    }
}

// Stores staged rows [0, rows) through the per-row destination pointers in LDS.
// cols = 256 (plain) or 128 (SwiGLU). Every piece is one 128-bit store.
__device__ __forceinline__ void store_rows(const uint16_t* lds, int pitch, int cols, int rows,
                                           char* const* rowptr) {
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
