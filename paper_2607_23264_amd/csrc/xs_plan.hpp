// The expert FFN's scheduler plan, computed from the local experts' row counts: scheduler rows
// of up to 256 rows per expert, the Expert-Wave boundaries (App. A.2), the h row offsets, and
// the cleared readiness and claim counters. Shared by the plan kernel and by the layout's
// scan kernel, which plans right after it has the expert totals.
#pragma once
#include "xs_common.hpp"

namespace xs {

struct PlanArgs {
  int e_begin, n_experts, cap, P1, P2, wave_tiles;
  int* meta;           // [0] rows P, [1] waves, [2] wave-list length, [3] computed rows,
                       // [8], [9] claim counters, [10] workgroups done (FFN), [11] blocks done
                       // (dispatch)
  int* row_expert;
  int* exp_m;
  int* exp_rowfirst;
  int* exp_hrow;
  int* wave_pos;
  int* wave_row;
  int* l1_done;
};

// s_m[x] (LDS): local expert x's rows, clipped to its window; s_first (LDS, n_experts) and
// s_rows are this function's scratch. Called by every thread of one block of at least
// n_experts threads; begins with a block barrier.
__device__ __forceinline__ void plan_rows(const PlanArgs& pa, int bm, const int* s_m, int* s_first, int* s_rows) {
  const int i = threadIdx.x;
  __syncthreads();
  if (i == 0) {
    int rows = 0, hrow = 0, nw = 0, wl1 = 0;
    pa.wave_row[0] = 0;
    pa.wave_pos[0] = 0;
    for (int x = 0; x < pa.n_experts; ++x) {
      const int mt = (s_m[x] + bm - 1) / bm;
      pa.exp_m[x] = s_m[x];
      pa.exp_rowfirst[x] = rows;
      s_first[x] = rows;
      pa.exp_hrow[x] = hrow;
      rows += mt;
      hrow += s_m[x];
      wl1 += mt * pa.P1;
      if (wl1 >= pa.wave_tiles && rows > pa.wave_row[nw]) {
        ++nw;
        pa.wave_row[nw] = rows;
        pa.wave_pos[nw] = rows * (pa.P1 + pa.P2);
        wl1 = 0;
      }
    }
    if (rows > pa.wave_row[nw]) {
      ++nw;
      pa.wave_row[nw] = rows;
      pa.wave_pos[nw] = rows * (pa.P1 + pa.P2);
    }
    pa.meta[0] = rows;
    pa.meta[1] = nw;
    pa.meta[2] = rows * (pa.P1 + pa.P2);
    pa.meta[3] = hrow;
    pa.meta[8] = 0;    // claim counters (dynamic claiming)
    pa.meta[9] = 0;
    pa.meta[10] = 0;   // workgroups done (the FFN's window signal)
    pa.meta[11] = 0;   // blocks done (the dispatch's window signal)
    *s_rows = rows;
  }
  __syncthreads();
  if (i < pa.n_experts) {
    const int mt = (s_m[i] + bm - 1) / bm;
    for (int p = s_first[i]; p < s_first[i] + mt; ++p) pa.row_expert[p] = i;
  }
  for (int p = i; p < *s_rows; p += blockDim.x) pa.l1_done[p] = 0;
}

// The rest of the layout, done by the dispatch launch of the fused layer (see dispatch_kernel).
struct FinArgs {
  int src, n_src, cap, n_chunks, n_disp_blocks;
  const int* idx_all;          // [n_src][T][k]; null: plain dispatch
  int* slot_row_all;
  const int* chunk_base;
  const int* src_base;
  const int* expert_offsets;
  int* row_src;
  int* done;
};

}  // namespace xs
