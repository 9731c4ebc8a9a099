// Dispatch through bounded destination rings (Sec. 4.3: an eligible Linear-1 tile needs a free
// destination ring slot; App. A.2: the scheduler checks ring-slot readiness before emission).
//
// Each destination d owns a ring of S slots. An entry is one token row plus a header listing
// the rows of d's dispatch window it goes to: every (token, k) slot of that destination when
// deduplicating, one slot otherwise. Entries of a ring are numbered in token order (then k slot
// order) by a prefix scan before the dispatch; entry n lives in slot n mod S.
//
// Lifetime protocol (per slot two words, counting completed uses):
//   pub[s] = u + 1  entry n = u S + s is written (system-scope release by its producer);
//   rel[s] = u + 1  it has been copied out (release by its consumer).
// The producer of entry n waits for rel[n mod S] == n / S (entry n - S released), writes the
// row and header, then publishes. A consumer claims entries in order from an atomic tail
// counter, waits for pub == n / S + 1 (acquire), copies the row into every listed window row,
// then releases the slot.
//
// Agents are waves: each produces its tokens' entries and consumes entries on its own, with no
// workgroup barrier in the protocol, so about two thousand entries are in flight at once.
// Each claim counter sits on a 128-byte line of its own (counters sharing a line serialise
// every claim of every ring at one L2 atomic unit).
//
// Progress: a producer waiting for its slot helps: while the tail has not passed n - S it
// claims and consumes the oldest entries itself, so the entry it waits for is always either
// being consumed or consumable by it. Those entries belong to earlier tokens, whose producers
// are behind this one in token order and so never wait on it. An agent that has produced all
// its entries drains the rings until every entry is consumed. Every wait is bounded: on
// time-out an agent reports XS_ETIMEOUT and raises an abort word that makes every other wait
// give up, so the grid always drains. Same-address device-scope atomics are slow on this
// GPU (measured: ~0.4 us each, serialised, when every entry took one): producers take no
// atomic, and a draining agent claims eight entries per atomic.
#include <algorithm>

#include "xs_common.hpp"

namespace xs {
namespace ring {

constexpr int kThreads = 256;         // four waves; every wave is an independent agent
constexpr int kMaxK = 32;
constexpr int kLine = 32;             // ints per 128-byte line: one counter per line
constexpr int kBatch = 8;             // entries a draining agent claims per atomic
// Rings of at least kWideRing slots drain in batches of kBatchWide: one acquire and one release
// per batch, and with slots to spare fewer, larger batches pay fewer fences (measured on one
// source of the DeepSeek-V3 share: 256 slots 5.5 -> 2.4 ms, 4096 slots 0.97 -> 0.85 ms); in small
// rings a wide batch holds slots the producers are waiting for (16 slots: 19.5 -> 65 ms).
constexpr int kBatchWide = 32, kWideRing = 256;

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
  int* entry_no;               // [T][k] entry number of each (token, k) slot in its ring
  int* tail;                   // [W] consumer claim counters, one per line
  int* total;                  // [W] entries per destination, one per line
  int* abort_word;
  int* pub;                    // [W][S]
  int* rel;                    // [W][S]
  int* stats;                  // optional [2W]: entries, producer stalls
  int* status;
  int64_t timeout_ticks;
};

// Exclusive prefix sum of v over the block's threads in order (1024 threads, 16 waves): a
// shuffle scan inside each wave, then each thread adds the totals of the waves before it.
// `total` receives the block's sum. Two barriers; wsum is 16 ints of LDS.
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum, int& total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wv] = x;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int w = wsum[i];
    before += i < wv ? w : 0;
    all += w;
  }
  total = all;
  __syncthreads();
  return before + x - v;
}

constexpr int kPlanInts = 32768;   // expert indices staged in LDS per round (128 KiB)

// Entry numbers, entries per destination and a clean control block (one workgroup of 1024).
// Entries of ring d are numbered in token order (and k slot order within a token without
// dedup): for each destination an exclusive scan over contiguous token chunks, one per thread.
__global__ __launch_bounds__(1024) void ring_plan_kernel(RingArgs a) {
  __shared__ int sidx[kPlanInts];
  __shared__ int wsum[16];
  __shared__ int base[XS_MAX_WINDOWS];
  const int W = a.win.n;
  const int epw = a.E / W;
  const int tid = threadIdx.x;
  for (int i = tid; i < W; i += blockDim.x) {
    a.tail[i * kLine] = 0;
    base[i] = 0;
  }
  if (tid == 0) *a.abort_word = 0;
  for (int64_t i = tid; i < static_cast<int64_t>(W) * a.S; i += blockDim.x) {
    a.pub[i] = 0;
    a.rel[i] = 0;
  }
  // Rounds of R tokens: their k indices are staged in LDS by coalesced loads, then each thread
  // numbers a contiguous run of the round's tokens per destination (entries in token order,
  // k slots ascending), continuing from the destination's count of earlier rounds.
  const int R = kPlanInts / a.k;
  for (int r0 = 0; r0 < a.T; r0 += R) {
    const int nr = min(R, a.T - r0);
    __syncthreads();   // the previous round's reads of sidx and base are done
    for (int i = tid; i < nr * a.k; i += blockDim.x) sidx[i] = a.idx[static_cast<int64_t>(r0) * a.k + i];
    __syncthreads();
    const int chunk = (nr + blockDim.x - 1) / blockDim.x;
    const int t0 = min(nr, tid * chunk), t1 = min(nr, t0 + chunk);
    for (int d = 0; d < W; ++d) {
      const int lo = d * epw, hi = lo + epw;   // destination d's experts
      int n = 0;
      for (int t = t0; t < t1; ++t) {
        int c = 0;
        for (int j = 0; j < a.k; ++j) {
          const int e = sidx[t * a.k + j];
          c += e >= lo && e < hi;
        }
        n += a.dedup ? (c > 0) : c;
      }
      int round_total;
      const int b = base[d];   // read before the scan's barriers; thread 0 advances it after them
      int next = b + block_exclusive_scan(n, wsum, round_total);
      for (int t = t0; t < t1; ++t) {
        bool any = false;
        for (int j = 0; j < a.k; ++j) {
          const int e = sidx[t * a.k + j];
          if (e >= lo && e < hi) {
            a.entry_no[static_cast<int64_t>(r0 + t) * a.k + j] = a.dedup ? next : next++;
            any = true;
          }
        }
        if (a.dedup && any) ++next;
      }
      if (tid == 0) base[d] = b + round_total;
    }
  }
  __syncthreads();
  for (int d = tid; d < W; d += blockDim.x) {
    a.total[d * kLine] = base[d];
    if (a.stats) {
      a.stats[d] = base[d];
      a.stats[W + d] = 0;
    }
  }
}

__device__ __forceinline__ bool aborted(const RingArgs& a) {
  return __hip_atomic_load(a.abort_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}

__device__ __forceinline__ void give_up(const RingArgs& a) {
  set_status(a.status, XS_ETIMEOUT);
  __hip_atomic_store(a.abort_word, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int bcast(int v) { return __builtin_amdgcn_readfirstlane(v); }

typedef __attribute__((address_space(1))) u32x4 gv4;

// Consume entries [m0, m0 + nb) of ring d (claimed by this wave, nb <= min(64, S)): wait
// until all are published, one acquire, one read of each ring row with one store per listed
// window row, one release, then the nb slot releases. nb <= S, so no entry of the batch
// waits on a slot the batch itself holds. False on abort. Wave-uniform control flow.
__device__ bool consume(const RingArgs& a, int d, int m0, int nb, int lane) {
  const int m = m0 + min(lane, nb - 1);
  const int* pub_i = a.pub + static_cast<int64_t>(d) * a.S + m % a.S;
  const int want = m / a.S + 1;
  if (__ballot(lane < nb && __hip_atomic_load(pub_i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want)) {
    const uint64_t t0 = wall_ticks();
    for (int it = 1;; ++it) {
      const bool pending =
          __ballot(lane < nb && __hip_atomic_load(pub_i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want) != 0;
      if (!pending) break;
      int stop = 0;
      if (lane == 0) {
        if ((it & 15) == 0 && aborted(a)) stop = 1;
        else if (wall_ticks() - t0 > static_cast<uint64_t>(a.timeout_ticks)) { give_up(a); stop = 1; }
      }
      if (bcast(stop)) return false;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");
  const int pieces = a.row_bytes >> 4;
  for (int b = 0; b < nb; ++b) {
    const int mb = m0 + b;
    const char* slot = a.ring[d] + static_cast<int64_t>(mb % a.S) * a.slot_bytes;
    const int* h = reinterpret_cast<const int*>(slot + a.row_bytes);
    int n = bcast(lane == 0 ? h[0] : 0);
    if (n < 0 || n > a.k) {               // never written by a producer: report, copy nothing
      if (lane == 0) set_status(a.status, XS_EBADINPUT);
      n = 0;
    }
    const int my_row = lane < n ? h[1 + lane] : -1;
    for (int p0 = 0; p0 < pieces; p0 += 64 * 8) {
      u32x4 v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int p = p0 + q * 64 + lane;
        if (p < pieces) v[q] = *(const gv4*)(slot + p * 16);
      }
      for (int i = 0; i < n; ++i) {
        const int r = __shfl(my_row, i);
        if (r < 0 || r >= a.win.cap[d]) {
          if (lane == 0 && p0 == 0) set_status(a.status, XS_ECAPACITY);
          continue;
        }
        char* dst = a.win.base[d] + static_cast<int64_t>(r) * a.win.stride[d];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int p = p0 + q * 64 + lane;
          if (p < pieces) *(gv4*)(dst + p * 16) = v[q];
        }
      }
    }
  }
  // every lane's reads of the slots are done before they are released
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
  if (lane < nb)
    __hip_atomic_store(a.rel + static_cast<int64_t>(d) * a.S + m % a.S, m / a.S + 1, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_SYSTEM);
  return true;
}

// Entries a producer has written but not yet published: lane i < n holds the i-th flag and
// its value. One release fence makes all of them visible; a producer publishes before it
// ever waits, so no consumer waits on an entry whose producer is itself waiting.
constexpr int kPend = 32;
struct Pending {
  int* flag;
  int val;
  int n;
};

__device__ __forceinline__ void publish(Pending& p, int lane) {
  if (p.n == 0) return;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "");
  if (lane < p.n) __hip_atomic_store(p.flag, p.val, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  p.n = 0;
}

// Produce entry e of token t into ring d: the window rows of the lanes in `mask` (each lane j
// holds slot j's row in my_row). The entry is left pending. False on abort.
__device__ bool produce(const RingArgs& a, int t, int d, int e, uint64_t mask, int my_row, int lane, Pending& pend) {
  const int s = e % a.S;
  const int u = e / a.S;
  int* rel = a.rel + static_cast<int64_t>(d) * a.S + s;
  int* pub = a.pub + static_cast<int64_t>(d) * a.S + s;
  bool stalled = false;
  const uint64_t t0 = wall_ticks();
  for (int it = 0;; ++it) {
    // 1 slot free, 0 abort, 2 help with entry m, 3 wait
    int st = 3, m = 0;
    if (lane == 0) {
      if (__hip_atomic_load(rel, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == u) {
        st = 1;
      } else if ((it & 15) == 15 && aborted(a)) {
        st = 0;
      } else if (wall_ticks() - t0 > static_cast<uint64_t>(a.timeout_ticks)) {
        give_up(a);
        st = 0;
      } else {
        m = __hip_atomic_load(a.tail + d * kLine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (m <= e - a.S && m < a.total[d * kLine] &&
            __hip_atomic_compare_exchange_strong(a.tail + d * kLine, &m, m + 1, __ATOMIC_RELAXED,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
          st = 2;
        else
          __builtin_amdgcn_s_sleep(1);
      }
    }
    st = bcast(st);
    m = bcast(m);
    if (st == 1) break;
    if (st == 0) return false;
    if (!stalled) publish(pend, lane);     // never wait holding unpublished entries
    stalled = true;
    if (st == 2 && !consume(a, d, m, 1, lane)) return false;
  }
  // only orders this wave's stores below after the observation (a write after the last
  // reader's reads): nothing is read here, so no cache maintenance
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  if (stalled && lane == 0 && a.stats) atomicAdd(a.stats + a.win.n + d, 1);
  char* slot = a.ring[d] + static_cast<int64_t>(s) * a.slot_bytes;
  const char* src = a.x + static_cast<int64_t>(t) * a.x_stride;
  const int pieces = a.row_bytes >> 4;
  for (int p0 = 0; p0 < pieces; p0 += 64 * 8) {
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int p = p0 + q * 64 + lane;
      if (p < pieces) v[q] = *(const gv4*)(src + p * 16);
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int p = p0 + q * 64 + lane;
      if (p < pieces) *(gv4*)(slot + p * 16) = v[q];
    }
  }
  // header: the number of rows, then the rows in ascending k slot order
  int* hdr = reinterpret_cast<int*>(slot + a.row_bytes);
  if ((mask >> lane) & 1ull) hdr[1 + __builtin_popcountll(mask & ((1ull << lane) - 1))] = my_row;
  if (lane == 0) hdr[0] = __builtin_popcountll(mask);
  if (lane == pend.n) {
    pend.flag = pub;
    pend.val = u + 1;
  }
  if (++pend.n == kPend) publish(pend, lane);
  return true;
}

__global__ __launch_bounds__(kThreads) void ring_dispatch_kernel(RingArgs a) {
  const int lane = threadIdx.x & 63;
  const int agents = gridDim.x * (kThreads / 64);
  const int me = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  const int W = a.win.n;
  const int epw = a.E / W;
  // Odd waves consume from the start (the receivers), even waves produce in token order: a
  // full ring then drains at the consumers' rate rather than through stalled producers'
  // help. Both drain at the end.
  const bool consumer = agents > 1 && (me & 1);
  const int producers = agents > 1 ? agents / 2 : 1;
  Pending pend{nullptr, 0, 0};
  for (int t = consumer ? a.T : (agents > 1 ? me / 2 : me); t < a.T; t += producers) {
    // lane j < k holds slot j's destination, window row and entry number
    int d = -1, r = -1, en = 0;
    if (lane < a.k) {
      const int64_t q = static_cast<int64_t>(t) * a.k + lane;
      const int e = a.idx[q];
      if (e < 0 || e >= a.E) {
        set_status(a.status, XS_EBADINPUT);
      } else {
        d = e / epw;
        r = a.slot_row[q];
        en = a.entry_no[q];
      }
    }
    uint64_t todo = __ballot(d >= 0);
    while (todo) {
      const int lead = __builtin_ctzll(todo);
      const int dd = __shfl(d, lead);
      // the entry's lanes: this slot alone, or every slot of the token on destination dd
      const uint64_t mask = a.dedup ? __ballot(d == dd) : (1ull << lead);
      todo &= ~mask;
      if (!produce(a, t, dd, __shfl(en, lead), mask, r, lane, pend)) return;
    }
  }
  publish(pend, lane);
  // drain: consume whatever is left, ring by ring, claiming up to kBatch (kBatchWide in wide
  // rings) entries per atomic (never more than S: see consume)
  const int batch = min(a.S >= kWideRing ? kBatchWide : kBatch, a.S);
  for (int i = 0; i < W; ++i) {
    const int d = (me + i) % W;
    const int tot = a.total[d * kLine];
    for (;;) {
      int m = 0, ok = 1;
      if (lane == 0) {
        ok = aborted(a) ? 0 : 1;
        m = __hip_atomic_load(a.tail + d * kLine, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        m = m < tot ? atomicAdd(a.tail + d * kLine, batch) : tot;
      }
      if (!bcast(ok)) return;
      m = bcast(m);
      if (m >= tot) break;
      if (!consume(a, d, m, min(batch, tot - m), lane)) return;
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

// Control block in the workspace: tail and total [W] each, one counter per 128-byte line, the
// abort word on a line of its own, then pub and rel [W][S] each.
constexpr int64_t kCtrlTail = 0, kCtrlTotal = XS_MAX_WINDOWS * 32, kCtrlAbort = 2 * XS_MAX_WINDOWS * 32,
                  kCtrlPub = 2 * XS_MAX_WINDOWS * 32 + 32;
// control words, then the entry numbers [T][k]
int64_t ctrl_ints(int32_t T, int32_t k, int32_t W, int32_t S) {
  return kCtrlPub + 2 * static_cast<int64_t>(W) * S + static_cast<int64_t>(T) * k;
}

}  // namespace

extern "C" int xs_ring_slot_bytes(int32_t H, int32_t k, int64_t* bytes) {
  if (!bytes || H < 8 || H % 8 || k < 1 || k > xs::ring::kMaxK) return XS_EINVAL;
  *bytes = align16(static_cast<int64_t>(H) * 2 + 4 * (1 + static_cast<int64_t>(k)));
  return XS_OK;
}

extern "C" int xs_dispatch_ring_workspace_bytes(int32_t T, int32_t k, int32_t W, int32_t slots, int64_t* bytes) {
  if (!bytes || T < 0 || k < 1 || W < 1 || W > XS_MAX_WINDOWS || slots < 1) return XS_EINVAL;
  *bytes = ctrl_ints(T, k, W, slots) * 4;
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
  xs_dispatch_ring_workspace_bytes(T, k, W, S, &need);
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
  a.tail = ctrl + kCtrlTail;
  a.total = ctrl + kCtrlTotal;
  a.abort_word = ctrl + kCtrlAbort;
  a.pub = ctrl + kCtrlPub;
  a.rel = a.pub + static_cast<int64_t>(W) * S;
  a.entry_no = a.rel + static_cast<int64_t>(W) * S;
  a.stats = stats;
  a.status = dev_status;
  a.timeout_ticks = xs_host::ns_to_ticks((spin_timeout_us > 0 ? spin_timeout_us : 2000000) * 1000);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(ring::ring_plan_kernel, dim3(1), dim3(1024), 0, st, a);
  if (xs_host::launch_status()) return XS_EHIP;
  if (T > 0) {
    // two workgroups (eight agent waves) per CU, all resident
    const int grid = std::min((T + 3) / 4, 2 * xs_host::persistent_grid(max_producers));
    hipLaunchKernelGGL(ring::ring_dispatch_kernel, dim3(grid), dim3(ring::kThreads), 0, st, a);
    if (xs_host::launch_status()) return XS_EHIP;
  }
  return xs_host::signal_windows(a.win, st);
}
