// Shared device/host helpers of the gfx950 store-path library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "xstage.h"

namespace xs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Window set passed by value to kernels (host xs_window array, copied into the kernel
// arguments so that device code never dereferences host memory).
struct WinSet {
  char* base[XS_MAX_WINDOWS];
  int64_t cap[XS_MAX_WINDOWS];
  int64_t stride[XS_MAX_WINDOWS];
  uint32_t* flag[XS_MAX_WINDOWS];
  int n;
};

// First error wins.
__device__ __forceinline__ void set_status(int32_t* st, int32_t code) {
  if (st) atomicCAS(st, 0, code);
}

// fp32 -> bf16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 (lo in bits 0..15) with gfx950's v_cvt_pk_bf16_f32: round to
// nearest even, as f2bf, in one instruction and without a branch.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t b = __builtin_convertvector(f32x2{lo, hi}, bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ uint64_t wall_ticks() { return wall_clock64(); }

// Busy-wait for `ticks` wall-clock ticks without touching memory.
__device__ __forceinline__ void spin_ticks(uint64_t ticks) {
  if (!ticks) return;
  uint64_t t0 = wall_clock64();
  while (wall_clock64() - t0 < ticks) __builtin_amdgcn_s_sleep(1);
}

}  // namespace xs

// ------------------------------------------------------------------------------ host side
namespace xs_host {

// Validates a host window array and copies it into a kernel-argument WinSet.
// row_bytes: bytes each row must hold. Returns XS_OK or XS_EINVAL.
int make_winset(const xs_window* win, int32_t W, int64_t row_bytes, xs::WinSet* out);

int launch_status();                      // XS_OK, or XS_EHIP if the last launch failed
double wall_rate_hz();                    // wall-clock tick rate of the current device
int num_cus();                            // compute units of the current device
int64_t ns_to_ticks(int64_t ns);

}  // namespace xs_host
