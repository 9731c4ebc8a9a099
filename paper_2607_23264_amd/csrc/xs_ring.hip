// Dispatch through bounded destination rings (Sec. 4.3: an eligible Linear-1 tile needs a free
// destination ring slot; App. A.2: the scheduler checks ring-slot readiness before emission).
//
// Each destination d owns a ring of S slots. An entry is one token row plus a header listing
// the rows of d's dispatch window it goes to: every (token, k) slot of that destination when
// deduplicating, one slot otherwise. Entries of a ring are numbered by an atomic head counter
// in the order producers claim them; entry n lives in slot n mod S.
//
// Lifetime protocol (per slot two words, counting completed uses):
//   pub[s] = u + 1  entry n = u S + s is written (system-scope release by its producer);
//   rel[s] = u + 1  it has been copied out (release by its consumer).
// The producer of entry n waits for rel[n mod S] == n / S (entry n - S released), writes the
// row and header, then publishes. A consumer claims entries in order from an atomic tail
// counter, waits for pub == n / S + 1 (acquire), copies the row into every listed window row,
// then releases the slot.
//
// Progress: a producer waiting for its slot helps: while the tail has not passed n - S it
// claims and consumes the oldest entries itself, so the entry it waits for is always either
// being consumed or consumable by it. Those entries were claimed by earlier producers, which
// never wait on this one. A workgroup that has produced all its entries drains the rings
// until every entry is consumed. Every wait is bounded: on time-out a workgroup reports
// XS_ETIMEOUT and raises an abort word that makes every other wait give up, so the grid
// always drains.
#include <algorithm>

#include "xs_common.hpp"

namespace xs {
namespace ring {

constexpr int kThreads = 256;
constexpr int kMaxK = 32;

struct RingArgs {
  const char* x;               // token rows, x_stride bytes apart
  int64_t x_stride;
  int row_bytes;               // payload bytes per entry (a multiple of 16)
  int T, k, E, S, dedup;
  const int* idx;              // [T][k] routed experts
  const int* slot_row;         // [T][k] window row of each (token, k) slot
  WinSet win;                  // dispatch windows
  char* ring[XS_MAX_WINDOWS];  // ring memory per destination: S slots of slot_bytes
  int64_t slot_bytes;          // payload, then 1 + k header ints
  int* head;                   // [W] producer claim counters
  int* tail;                   // [W] consumer claim counters
  int* total;                  // [W] entries per destination
  int* abort_word;
  int* pub;                    // [W][S]
  int* rel;                        // [W][S]
  int* stats;                  // optional [2W]: entries, producer stalls
  int* status;
  int64_t timeout_ticks;
};

// Entries per destination and a clean control block (one workgroup).
__global__ __launch_bounds__(1024) void ring_plan_kernel(RingArgs a) {
  __shared__ int cnt[XS_MAX_WINDOWS];
  const int W = a.win.n;
  const int epw = a.E / W;
  for (int i = threadIdx.x; i < W; i += blockDim.x) {
    cnt[i] = 0;
    a.head[i] = 0;
    a.tail[i] = 0;
  }
  if (threadIdx.x == 0) *a.abort_word = 0;
  for (int64_t i = threadIdx.x; i < static_cast<int64_t>(W) * a.S; i += blockDim.x) {
    a.pub[i] = 0;
    a.rel[i] = 0;
  }
  __syncthreads();
  for (int t = threadIdx.x; t < a.T; t += blockDim.x) {
    uint64_t seen = 0;
    for (int j = 0; j < a.k; ++j) {
      const int e = a.idx[static_cast<int64_t>(t) * a.k + j];
      if (e < 0 || e >= a.E) continue;
      const int d = e / epw;
      if (!a.dedup) {
        atomicAdd(&cnt[d], 1);
      } else if (!(seen >> d & 1ull)) {
        seen |= 1ull << d;
        atomicAdd(&cnt[d], 1);
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < W; i += blockDim.x) {
    a.total[i] = cnt[i];
    if (a.stats) {
      a.stats[i] = cnt[i];
      a.stats[W + i] = 0;
    }
  }
}

struct Shared {
  int d[kMaxK], r[kMaxK];      // this token's (destination, window row) pairs, by destination
  int nent, ent_first[kMaxK], ent_n[kMaxK];
  int state, value;            // broadcast words
  int hdr[kMaxK + 1];          // header of the entry being consumed
};

__device__ __forceinline__ bool aborted(const RingArgs& a) {
  return __hip_atomic_load(a.abort_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}

__device__ __forceinline__ void give_up(const RingArgs& a) {
  set_status(a.status, XS_ETIMEOUT);
  __hip_atomic_store(a.abort_word, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 16-byte copy of one payload by the whole workgroup.
__device__ __forceinline__ void copy_row(char* dst, const char* src, int bytes) {
  typedef __attribute__((address_space(1))) u32x4 gv;
  for (int o = threadIdx.x * 16; o < bytes; o += kThreads * 16)
    *(gv*)(dst + o) = *(const gv*)(src + o);
}

// Consume entry m of ring d (already claimed by this workgroup). False on abort.
__device__ bool consume(const RingArgs& a, int d, int m, Shared& sh) {
  const int s = m % a.S;
  const int u = m / a.S;
  int* pub = a.pub + static_cast<int64_t>(d) * a.S + s;
  int* rel = a.rel + static_cast<int64_t>(d) * a.S + s;
  const char* slot = a.ring[d] + static_cast<int64_t>(s) * a.slot_bytes;
  if (threadIdx.x == 0) {
    int ok = 1;
    if (__hip_atomic_load(pub, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != u + 1) {
      const uint64_t t0 = wall_ticks();
      while (__hip_atomic_load(pub, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) != u + 1) {
        if (aborted(a)) { ok = 0; break; }
        if (wall_ticks() - t0 > static_cast<uint64_t>(a.timeout_ticks)) { give_up(a); ok = 0; break; }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (ok) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
      const int* h = reinterpret_cast<const int*>(slot + a.row_bytes);
      int n = h[0];
      if (n < 0 || n > a.k) {                 // never written by a producer: report, copy nothing
        set_status(a.status, XS_EBADINPUT);
        n = 0;
      }
      sh.hdr[0] = n;
      for (int i = 0; i < n; ++i) sh.hdr[1 + i] = h[1 + i];
    }
    sh.state = ok;
  }
  __syncthreads();
  const bool ok = sh.state != 0;
  const int n = sh.hdr[0];
  __syncthreads();
  if (!ok) return false;
  for (int i = 0; i < n; ++i) {
    const int r = sh.hdr[1 + i];
    if (r < 0 || r >= a.win.cap[d]) {
      if (threadIdx.x == 0) set_status(a.status, XS_ECAPACITY);
      continue;
    }
    copy_row(a.win.base[d] + static_cast<int64_t>(r) * a.win.stride[d], slot, a.row_bytes);
  }
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(rel, u + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  return true;
}

// Produce one entry of token t into ring d with window rows sh.r[first, first + n).
__device__ bool produce(const RingArgs& a, int t, int d, int first, int n, Shared& sh) {
  int* head = a.head + d;
  if (threadIdx.x == 0) sh.value = atomicAdd(head, 1);
  __syncthreads();
  const int e = sh.value;
  __syncthreads();
  const int s = e % a.S;
  const int u = e / a.S;
  int* rel = a.rel + static_cast<int64_t>(d) * a.S + s;
  int* pub = a.pub + static_cast<int64_t>(d) * a.S + s;
  bool stalled = false;
  const uint64_t t0 = wall_ticks();
  for (;;) {
    // state: 1 slot free, 0 abort, 2 help with entry value, 3 wait
    if (threadIdx.x == 0) {
      int st;
      if (__hip_atomic_load(rel, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) == u) {
        st = 1;
      } else if (aborted(a)) {
        st = 0;
      } else if (wall_ticks() - t0 > static_cast<uint64_t>(a.timeout_ticks)) {
        give_up(a);
        st = 0;
      } else {
        st = 3;
        int m = __hip_atomic_load(a.tail + d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (m <= e - a.S && m < a.total[d] &&
            __hip_atomic_compare_exchange_strong(a.tail + d, &m, m + 1, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT)) {
          st = 2;
          sh.value = m;
        } else {
          __builtin_amdgcn_s_sleep(1);
        }
      }
      sh.state = st;
    }
    __syncthreads();
    const int st = sh.state;
    const int m = sh.value;
    __syncthreads();
    if (st == 1) break;
    if (st == 0) return false;
    stalled = true;
    if (st == 2 && !consume(a, d, m, sh)) return false;
  }
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");   // the slot's last reader is done
    if (stalled && a.stats) atomicAdd(a.stats + a.win.n + d, 1);
  }
  __syncthreads();
  char* slot = a.ring[d] + static_cast<int64_t>(s) * a.slot_bytes;
  copy_row(slot, a.x + static_cast<int64_t>(t) * a.x_stride, a.row_bytes);
  if (threadIdx.x == 0) {
    int* h = reinterpret_cast<int*>(slot + a.row_bytes);
    h[0] = n;
    for (int i = 0; i < n; ++i) h[1 + i] = sh.r[first + i];
  }
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(pub, u + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  return true;
}

__global__ __launch_bounds__(kThreads) void ring_dispatch_kernel(RingArgs a) {
  __shared__ Shared sh;
  const int W = a.win.n;
  const int epw = a.E / W;
  for (int t = blockIdx.x; t < a.T; t += gridDim.x) {
    if (threadIdx.x == 0) {
      // (destination, window row) pairs of the valid slots, stably ordered by destination
      int n = 0;
      for (int j = 0; j < a.k; ++j) {
        const int e = a.idx[static_cast<int64_t>(t) * a.k + j];
        if (e < 0 || e >= a.E) {
          set_status(a.status, XS_EBADINPUT);
          continue;
        }
        const int d = e / epw, r = a.slot_row[static_cast<int64_t>(t) * a.k + j];
        int p = n++;
        if (a.dedup)
          for (; p > 0 && sh.d[p - 1] > d; --p) {
            sh.d[p] = sh.d[p - 1];
            sh.r[p] = sh.r[p - 1];
          }
        sh.d[p] = d;
        sh.r[p] = r;
      }
      int ne = 0;
      for (int p = 0; p < n; ++p) {
        if (a.dedup && ne > 0 && sh.d[sh.ent_first[ne - 1]] == sh.d[p]) {
          ++sh.ent_n[ne - 1];
        } else {
          sh.ent_first[ne] = p;
          sh.ent_n[ne] = 1;
          ++ne;
        }
      }
      sh.nent = ne;
    }
    __syncthreads();
    const int ne = sh.nent;
    for (int i = 0; i < ne; ++i) {
      const int first = sh.ent_first[i];
      if (!produce(a, t, sh.d[first], first, sh.ent_n[i], sh)) return;
    }
  }
  // drain: consume whatever is left, ring by ring
  for (int i = 0; i < W; ++i) {
    const int d = (blockIdx.x + i) % W;
    for (;;) {
      if (threadIdx.x == 0) {
        const int m = __hip_atomic_load(a.tail + d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        sh.value = m < a.total[d] ? atomicAdd(a.tail + d, 1) : a.total[d];
        sh.state = aborted(a) ? 0 : 1;
      }
      __syncthreads();
      const int m = sh.value;
      const int ok = sh.state;
      __syncthreads();
      if (!ok) return;
      if (m >= a.total[d]) break;
      if (!consume(a, d, m, sh)) return;
    }
  }
}

}  // namespace ring
}  // namespace xs

// ------------------------------------------------------------------------------ host side
namespace xs_host {
int signal_windows(const xs::WinSet& ws, hipStream_t st);
int persistent_grid(int max_producers);
}  // namespace xs_host

namespace {

int64_t align16(int64_t v) { return (v + 15) / 16 * 16; }

// Control block in the workspace: head, tail, total [W] each, the abort word, then pub and rel
// [W][S] each.
int64_t ctrl_ints(int32_t W, int32_t S) { return 4 * static_cast<int64_t>(XS_MAX_WINDOWS) + 2 * static_cast<int64_t>(W) * S; }

}  // namespace

extern "C" int xs_ring_slot_bytes(int32_t H, int32_t k, int64_t* bytes) {
  if (!bytes || H < 8 || H % 8 || k < 1 || k > xs::ring::kMaxK) return XS_EINVAL;
  *bytes = align16(static_cast<int64_t>(H) * 2 + 4 * (1 + static_cast<int64_t>(k)));
  return XS_OK;
}

extern "C" int xs_dispatch_ring_workspace_bytes(int32_t W, int32_t slots, int64_t* bytes) {
  if (!bytes || W < 1 || W > XS_MAX_WINDOWS || slots < 1) return XS_EINVAL;
  *bytes = ctrl_ints(W, slots) * 4;
  return XS_OK;
}

extern "C" int xs_dispatch_ring(const void* x, int32_t T, int32_t H, const int32_t* topk_idx,
                                const int32_t* slot_row, int32_t k, int32_t E, const xs_window* win,
                                int32_t W, const xs_window* rings, int32_t dedup, int32_t max_producers,
                                int64_t spin_timeout_us, void* workspace, int64_t workspace_bytes,
                                int32_t* stats, int32_t* dev_status, void* stream) {
  using namespace xs;
  if (!x || !topk_idx || !slot_row || !win || !rings || !dev_status || T < 0 || k < 1 ||
      k > ring::kMaxK || k > E || E < 1 || W < 1 || W > XS_MAX_WINDOWS || E % W || (dedup != 0 && dedup != 1) ||
      max_producers < 0 || spin_timeout_us < 0)
    return XS_EINVAL;
  if (H < 8 || H % 8 || (reinterpret_cast<uintptr_t>(x) & 15)) return XS_EUNSUPPORTED;
  int64_t slot_bytes = 0;
  xs_ring_slot_bytes(H, k, &slot_bytes);
  const int32_t S = static_cast<int32_t>(rings[0].capacity_rows);
  if (S < 1 || rings[0].capacity_rows > (1 << 20)) return XS_EINVAL;
  ring::RingArgs a{};
  for (int d = 0; d < W; ++d) {
    if (!rings[d].base || rings[d].capacity_rows != S || rings[d].row_stride_bytes < slot_bytes ||
        rings[d].row_stride_bytes % 16 || (reinterpret_cast<uintptr_t>(rings[d].base) & 15))
      return XS_EINVAL;
    a.ring[d] = static_cast<char*>(rings[d].base);
  }
  if (rings[0].row_stride_bytes != rings[W - 1].row_stride_bytes) return XS_EINVAL;
  for (int d = 0; d < W; ++d)
    if (rings[d].row_stride_bytes != rings[0].row_stride_bytes) return XS_EINVAL;
  int64_t need = 0;
  xs_dispatch_ring_workspace_bytes(W, S, &need);
  if (!workspace || workspace_bytes < need) return XS_EWORKSPACE;
  const int rc = xs_host::make_winset(win, W, static_cast<int64_t>(H) * 2, &a.win);
  if (rc) return rc;
  int* ctrl = static_cast<int*>(workspace);
  a.x = static_cast<const char*>(x);
  a.x_stride = static_cast<int64_t>(H) * 2;
  a.row_bytes = H * 2;
  a.T = T;
  a.k = k;
  a.E = E;
  a.S = S;
  a.dedup = dedup;
  a.idx = topk_idx;
  a.slot_row = slot_row;
  a.slot_bytes = rings[0].row_stride_bytes;
  a.head = ctrl;
  a.tail = ctrl + XS_MAX_WINDOWS;
  a.total = ctrl + 2 * XS_MAX_WINDOWS;
  a.abort_word = ctrl + 3 * XS_MAX_WINDOWS;
  a.pub = ctrl + 4 * XS_MAX_WINDOWS;
  a.rel = a.pub + static_cast<int64_t>(W) * S;
  a.stats = stats;
  a.status = dev_status;
  a.timeout_ticks = xs_host::ns_to_ticks((spin_timeout_us > 0 ? spin_timeout_us : 2000000) * 1000);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(ring::ring_plan_kernel, dim3(1), dim3(1024), 0, st, a);
  if (xs_host::launch_status()) return XS_EHIP;
  if (T > 0) {
    const int grid = std::min(T, xs_host::persistent_grid(max_producers));
    hipLaunchKernelGGL(ring::ring_dispatch_kernel, dim3(grid), dim3(ring::kThreads), 0, st, a);
    if (xs_host::launch_status()) return XS_EHIP;
  }
  return xs_host::signal_windows(a.win, st);
}
