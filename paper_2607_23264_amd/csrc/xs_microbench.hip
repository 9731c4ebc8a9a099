// Remote-store microbenchmark (Sec. 3.1): K producer workgroups each issue bursts of B bytes
// of 128-bit stores into a target window, separated by a producer-side gap with no stores.
// The issue span of a burst ends when its last store has been issued (a workgroup barrier
// that does not wait for store completion), i.e. when the stores are sender-accepted.
// In completion mode every wave also waits for its stores to complete (a release fence at
// system scope) before the gap: the completion-coupled counterfactual.
#include "xs_common.hpp"

namespace xs {

constexpr int kMaxBursts = 256;

// Timestamps stay in LDS while the bursts run; one slot reservation per producer after the
// last burst, so recording never sits between two bursts.
__global__ void xstage_mb_kernel(char* __restrict__ target, int64_t target_bytes, int B,
                                 int n_bursts, int64_t gap_ticks, int mode, xs_trace tr) {
  __shared__ uint64_t ts[3][kMaxBursts];
  const int p = blockIdx.x, tid = threadIdx.x;
  const int pieces = B / 16;
  for (int b = 0; b < n_bursts; ++b) {
    __syncthreads();
    if (tid == 0) ts[0][b] = wall_ticks();
    const int64_t off = ((static_cast<int64_t>(p) * n_bursts + b) * B) % target_bytes;
    u32x4* dst = reinterpret_cast<u32x4*>(target + off);
    u32x4 v;
    v[0] = static_cast<uint32_t>(p);
    v[1] = static_cast<uint32_t>(b);
    v[2] = 0x58535447u;
    for (int i = tid; i < pieces; i += blockDim.x) {
      v[3] = static_cast<uint32_t>(i);
      dst[i] = v;
    }
    if (mode == XS_MB_COMPLETION) __threadfence_system();
    __syncthreads();
    if (tid == 0) {
      ts[1][b] = wall_ticks();
      spin_ticks(static_cast<uint64_t>(gap_ticks));
      ts[2][b] = wall_ticks();
    }
  }
  __syncthreads();
  if (tid == 0) {
    const uint32_t base = atomicAdd(tr.count, static_cast<uint32_t>(n_bursts));
    for (int b = 0; b < n_bursts; ++b) {
      const int64_t i = static_cast<int64_t>(base) + b;
      if (i < tr.capacity) {
        uint64_t* r = tr.buf + i * 4;
        r[0] = (static_cast<uint64_t>(p) << 32) | static_cast<uint32_t>(b);
        r[1] = ts[0][b];
        r[2] = ts[1][b];
        r[3] = ts[2][b];
      }
    }
  }
}

}  // namespace xs

extern "C" int xs_xstage_microbench(const xs_microbench_args* a, const xs_trace* trace,
                                    void* stream) {
  if (!a || !trace || !trace->buf || !trace->count || !a->target) return XS_EINVAL;
  if (a->K < 1 || a->K > 65535 || a->B_bytes < 1024 || a->B_bytes % 1024 || a->n_bursts < 1 || a->n_bursts > xs::kMaxBursts ||
      a->gap_ns < 0 || (a->mode != XS_MB_PERIODIC && a->mode != XS_MB_COMPLETION) ||
      a->store_waves < 1 || a->store_waves > 8)
    return XS_EINVAL;
  if (a->target_bytes < a->B_bytes || a->target_bytes % a->B_bytes ||
      (reinterpret_cast<uintptr_t>(a->target) & 15))
    return XS_EINVAL;
  hipLaunchKernelGGL(xs::xstage_mb_kernel, dim3(a->K), dim3(64 * a->store_waves), 0,
                     static_cast<hipStream_t>(stream), static_cast<char*>(a->target),
                     a->target_bytes, a->B_bytes, a->n_bursts, xs_host::ns_to_ticks(a->gap_ns),
                     a->mode, *trace);
  return xs_host::launch_status();
}
