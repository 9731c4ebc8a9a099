// Microscaled (MX) formats of the quantized EP path: the block quantizer (bf16 -> E4M3 or
// E2M1 codes with one E8M0 scale per 32 elements) and the MXFP8 GEMM. The paper runs its EP
// kernel at W8A8 and W4A8 (Sec. 5.2) without fixing the formats; these are the OCP microscaled
// formats the gfx950 matrix cores take natively.
#include <algorithm>

#include "xs_gemm_mx.hpp"

namespace xs {

namespace mx {

// Shared exponent of a block from the bits of its largest magnitude (a bf16 value, sign
// cleared): the smallest e with amax <= fmax 2^e, where fmax = Mf 2^Ef (448 = 1.75 2^8 for
// E4M3, 6 = 1.5 2^2 for E2M1). amax = M 2^E with 1 <= M < 2 gives e = E - Ef + [M > Mf].
// Integer arithmetic only, so the decision is the same on every implementation.
template <int FMT>
__device__ __forceinline__ int shared_exp(uint32_t amax_bits) {
  constexpr int Ef = FMT == XS_FMT_E4M3 ? 8 : 2;
  if (amax_bits == 0) return 0;
  const int F = static_cast<int>(amax_bits >> 7);       // biased exponent
  const int m = static_cast<int>(amax_bits & 0x7F);     // 7 mantissa bits
  int E, above;
  if (F != 0) {
    E = F - 127;
    above = FMT == XS_FMT_E4M3 ? (m > 96) : (m > 64);  // 1 + m/128 > 1.75 or 1.5
  } else {                                              // subnormal: m 2^-133
    const int p = 31 - __builtin_clz(static_cast<uint32_t>(m));
    E = p - 133;
    above = FMT == XS_FMT_E4M3 ? (4 * m > 7 << p) : (2 * m > 3 << p);
  }
  const int e = E - Ef + above;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// E2M1 code of |v| <= 6, round to nearest, ties to the even code; the sign is kept also when
// the magnitude rounds to zero (as the hardware E4M3 conversion does).
__device__ __forceinline__ uint32_t e2m1_code(float v) {
  const float a = fabsf(v);
  uint32_t c;
  if (a <= 0.25f) c = 0;
  else if (a < 0.75f) c = 1;
  else if (a <= 1.25f) c = 2;
  else if (a < 1.75f) c = 3;
  else if (a <= 2.5f) c = 4;
  else if (a < 3.5f) c = 5;
  else if (a <= 5.f) c = 6;
  else c = 7;
  return (__builtin_bit_cast(uint32_t, v) >> 31) ? (c | 8u) : c;
}

// One lane per 8 consecutive elements; four lanes per 32-element block. Codes: E4M3 one byte
// per element, E2M1 two per byte (element 2 i in the low nibble). The scale of row r, block j
// goes to byte r * s_row + (j / 16) * s_grp + j % 16: row-major rows with s_grp = 16, or
// groups of 16 blocks (512 columns) [cols / 512][rows][16] with s_row = 16, s_grp = 16 rows.
template <int FMT>
__global__ __launch_bounds__(256) void quantize_kernel(const uint16_t* __restrict__ x, int64_t ldx,
                                                       int64_t rows, int cols,
                                                       uint8_t* __restrict__ codes, int64_t ldc,
                                                       uint8_t* __restrict__ scales, int64_t s_row,
                                                       int64_t s_grp) {
  const int per_row = cols / 8;
  const int64_t total = rows * per_row;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t r = i / per_row;
    const int pc = static_cast<int>(i - r * per_row);
    const u32x4 raw = *reinterpret_cast<const u32x4*>(x + r * ldx + pc * 8);
    uint32_t bits[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      bits[2 * q] = raw[q] & 0xFFFFu;
      bits[2 * q + 1] = raw[q] >> 16;
    }
    uint32_t amax = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) amax = max(amax, bits[q] & 0x7FFFu);   // magnitudes order as integers
    // the block's four lanes are consecutive (cols is a multiple of 32 and rows start on a block)
    amax = max(amax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(amax), 1)));
    amax = max(amax, static_cast<uint32_t>(__shfl_xor(static_cast<int>(amax), 2)));
    const int e = shared_exp<FMT>(amax);
    float v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q)
      v[q] = __builtin_amdgcn_ldexpf(__builtin_bit_cast(float, bits[q] << 16), -e);   // exact
    if (FMT == XS_FMT_E4M3) {
      uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(v[0], v[1], 0, false));
      lo = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(v[2], v[3], static_cast<int>(lo), true));
      uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(v[4], v[5], 0, false));
      hi = static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(v[6], v[7], static_cast<int>(hi), true));
      typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
      *reinterpret_cast<u32x2*>(codes + r * ldc + pc * 8) = u32x2{lo, hi};
    } else {
      uint32_t p = 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) p |= e2m1_code(v[q]) << (4 * q);
      *reinterpret_cast<uint32_t*>(codes + r * ldc + pc * 4) = p;
    }
    if ((pc & 3) == 0) {
      const int j = pc / 4;
      scales[r * s_row + (j >> 4) * s_grp + (j & 15)] = static_cast<uint8_t>(e + 127);
    }
  }
}

// Plain MX GEMM, persistent over 256 x 256 output tiles: C (bf16) = deq(A) deq(B)^T; A E4M3,
// B E4M3 or (BF4) packed E2M1.
template <bool BF4>
__global__ __launch_bounds__(kMxThreads, 1) void gemm_mx_kernel(
    const uint8_t* __restrict__ A, int64_t lda, const uint8_t* __restrict__ As, int64_t lda_s,
    const uint8_t* __restrict__ B, int64_t ldb, const uint8_t* __restrict__ Bs, int64_t ldb_s,
    char* __restrict__ C, int64_t ldc_bytes, int M, int N, int K, xs_trace tr) {
  __shared__ __attribute__((aligned(16))) char smem[kLdsBytes];
  char* lds = smem;
  char** rowptr = reinterpret_cast<char**>(smem + kLdsRowPtrOff);
  const int tid = threadIdx.x;
  const int tm = (M + kBM - 1) / kBM, tn = N / kBN, ntiles = tm * tn;
  for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int mb = t % tm, nb = t / tm;
    const int m0 = mb * kBM, n0 = nb * kBN;
    const int rows = min(kBM, M - m0);
    const uint64_t t0 = tr.buf ? wall_ticks() : 0;
    AccMx acc;
    gemm_mainloop_mx<BF4>(A + static_cast<int64_t>(m0) * lda, lda, As + static_cast<int64_t>(m0) * lda_s,
                          lda_s, 16, rows, B, ldb, Bs, ldb_s, 16, n0, 0, false, K, acc, lds);
    const uint64_t t1 = tr.buf ? wall_ticks() : 0;
    if (tid < rows) rowptr[tid] = C + static_cast<int64_t>(m0 + tid) * ldc_bytes + static_cast<int64_t>(n0) * 2;
    stage_tile_mx(acc, lds);
    __syncthreads();
    store_rows_n<kMxThreads>(lds, kEpiPitch * 2, kBN * 2 / 16, rows, rowptr);
    lds_barrier();
    if (tr.buf && tid == 0) {
      uint32_t i = atomicAdd(tr.count, 1u);
      if (static_cast<int64_t>(i) < tr.capacity) {
        uint64_t* rec = tr.buf + static_cast<int64_t>(i) * 4;
        rec[0] = (5ull << 56) | (static_cast<uint64_t>(blockIdx.x) << 32) | static_cast<uint32_t>(t);
        rec[1] = t0;
        rec[2] = t1;
        rec[3] = wall_ticks();
      }
    }
  }
}

}  // namespace mx
}  // namespace xs

using namespace xs;

namespace xs_host {
int persistent_grid(int max_producers);
}  // namespace xs_host

static bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

namespace {

int quantize_mx(const void* x, int64_t rows, int32_t cols, int64_t ldx, int32_t fmt, void* codes,
                int64_t ld_codes, void* scales, int64_t s_row, int64_t s_grp, void* stream) {
  const int64_t pieces = rows * (cols / 8);
  const int grid = static_cast<int>(std::min<int64_t>((pieces + 255) / 256, 16384));
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (fmt == XS_FMT_E4M3)
    hipLaunchKernelGGL(mx::quantize_kernel<XS_FMT_E4M3>, dim3(grid), dim3(256), 0, st,
                       static_cast<const uint16_t*>(x), ldx, rows, cols, static_cast<uint8_t*>(codes),
                       ld_codes, static_cast<uint8_t*>(scales), s_row, s_grp);
  else
    hipLaunchKernelGGL(mx::quantize_kernel<XS_FMT_E2M1>, dim3(grid), dim3(256), 0, st,
                       static_cast<const uint16_t*>(x), ldx, rows, cols, static_cast<uint8_t*>(codes),
                       ld_codes, static_cast<uint8_t*>(scales), s_row, s_grp);
  return xs_host::launch_status();
}

int quantize_args_ok(const void* x, int64_t rows, int32_t cols, int64_t ldx, int32_t fmt, const void* codes,
                     int64_t ld_codes, const void* scales) {
  if (!x || !codes || !scales || rows < 0 || cols <= 0) return XS_EINVAL;
  if (fmt != XS_FMT_E4M3 && fmt != XS_FMT_E2M1) return XS_EINVAL;
  const int64_t code_bytes = fmt == XS_FMT_E4M3 ? cols : cols / 2;
  if (cols % 32 || ldx < cols || ldx % 8 || ld_codes < code_bytes) return XS_EINVAL;
  if (!aligned(x, 16) || ld_codes % (fmt == XS_FMT_E4M3 ? 8 : 4) || !aligned(codes, fmt == XS_FMT_E4M3 ? 8 : 4))
    return XS_EINVAL;
  return XS_OK;
}

}  // namespace

extern "C" int xs_quantize_mx(const void* x, int64_t rows, int32_t cols, int64_t ldx, int32_t fmt,
                              void* codes, int64_t ld_codes, void* scales, int64_t ld_scales,
                              void* stream) {
  int rc = quantize_args_ok(x, rows, cols, ldx, fmt, codes, ld_codes, scales);
  if (rc) return rc;
  if (ld_scales < cols / 32) return XS_EINVAL;
  if (rows == 0) return XS_OK;
  return quantize_mx(x, rows, cols, ldx, fmt, codes, ld_codes, scales, ld_scales, 16, stream);
}

extern "C" int xs_quantize_mx_grouped(const void* x, int64_t rows, int32_t cols, int64_t ldx, int32_t fmt,
                                      void* codes, int64_t ld_codes, void* scales, void* stream) {
  int rc = quantize_args_ok(x, rows, cols, ldx, fmt, codes, ld_codes, scales);
  if (rc) return rc;
  if (cols % 512 || !aligned(scales, 16)) return XS_EINVAL;
  if (rows == 0) return XS_OK;
  return quantize_mx(x, rows, cols, ldx, fmt, codes, ld_codes, scales, 16, rows * 16, stream);
}

extern "C" int xs_gemm_mx(const void* a, int64_t lda, const void* a_scales, int64_t lda_s,
                          const void* b, int64_t ldb, const void* b_scales, int64_t ldb_s,
                          int32_t b_fmt, void* c, int64_t ldc, int32_t M, int32_t N, int32_t K,
                          const xs_trace* trace, void* stream) {
  if (!a || !a_scales || !b || !b_scales || !c || M < 0 || N <= 0 || K <= 0) return XS_EINVAL;
  if (b_fmt != XS_FMT_E4M3 && b_fmt != XS_FMT_E2M1) return XS_EINVAL;
  const bool bf4 = b_fmt == XS_FMT_E2M1;
  if (N % kBN || K % 512 || lda < K || ldb < (bf4 ? K / 2 : K) || lda % 16 || ldb % 16 || lda_s < K / 32 ||
      ldb_s < K / 32 || lda_s % 16 || ldb_s % 16 || ldc < N || ldc % 8)
    return XS_EUNSUPPORTED;
  if (!aligned(a, 16) || !aligned(b, 16) || !aligned(a_scales, 16) || !aligned(b_scales, 16) ||
      !aligned(c, 16))
    return XS_EINVAL;
  if (M == 0) return XS_OK;
  xs_trace tr{nullptr, 0, nullptr};
  if (trace && trace->buf && trace->count) tr = *trace;
  const int tiles = ((M + kBM - 1) / kBM) * (N / kBN);
  const int grid = std::min(tiles, xs_host::persistent_grid(0));
  hipLaunchKernelGGL(bf4 ? mx::gemm_mx_kernel<true> : mx::gemm_mx_kernel<false>, dim3(grid), dim3(kMxThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint8_t*>(a), lda,
                     static_cast<const uint8_t*>(a_scales), lda_s, static_cast<const uint8_t*>(b), ldb,
                     static_cast<const uint8_t*>(b_scales), ldb_s, static_cast<char*>(c), ldc * 2, M, N, K, tr);
  return xs_host::launch_status();
}
