/*
 * xstage.h — C ABI of the MI355X (gfx950) fused store-path library.
 *
 * The library implements, at one GPU's share, the communication–computation fusion
 * studied in "X-Stage: Modeling Post-Issue Backpressure in GPU Communication–Computation
 * Fusion": a compute pipeline that issues one-sided stores into per-destination windows.
 *   - expert parallelism (Sec. 4.3, Sec. 5.3): route -> dispatch -> local-expert SwiGLU
 *     grouped GEMM -> combine-send stores (the Linear-2 epilogue bursts) -> combine-reduce;
 *   - tensor parallelism (Sec. 4.5): GEMM whose output row blocks are stored into
 *     per-destination windows as tiles complete;
 *   - Ulysses sequence parallelism (Sec. 5.4, GEMM-All-to-All): QKV projection whose
 *     epilogue stores head groups into per-destination windows;
 *   - store pacing: the tile order of the persistent EP kernel (Expert-Wave, cross-wave
 *     interleaving of Alg. 1, chunked bursts) and the Burst-Gap model of Sec. 3
 *     (Eqs. 1-6) with its calibration microbenchmark (Sec. 3.1).
 *
 * Conventions (every entry point):
 *   - Pointers named "device" point to GPU memory (hipMalloc / torch CUDA tensors) or, for
 *     windows, to fine-grained host-coherent memory (hipHostMalloc coherent). Host pointers
 *     are marked "host". bf16 tensors are passed as void* (16-bit storage, row-major).
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream). Every call is
 *     asynchronous on that stream; it only enqueues work.
 *   - Ownership: the caller owns every buffer; the library only borrows pointers for the
 *     stream-ordered duration of the call and never allocates on these calls. Scratch is
 *     passed in as `workspace` (size from the matching *_workspace_bytes query).
 *   - Errors: the return value reports argument problems synchronously (XS_EINVAL,
 *     XS_EUNSUPPORTED, XS_EWORKSPACE) and launch failures (XS_EHIP). Data-dependent errors
 *     (a window over capacity, a bad expert id, a dependency wait that timed out) are
 *     written to the caller's device word `dev_status` (first error wins, via atomic
 *     compare-and-swap from 0). The library never clears `dev_status`: zero it before the
 *     first call. No exception crosses the ABI and the library prints nothing.
 *   - Calls on one stream are ordered; calls on different streams that share buffers race.
 */
#ifndef XSTAGE_H
#define XSTAGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ----------------------------------------------------------------------------- status */
enum {
  XS_OK = 0,
  XS_EINVAL = 1,        /* bad argument (null pointer, k > E, E % W != 0, ...) */
  XS_EUNSUPPORTED = 2,  /* valid but not implemented (e.g. H not a multiple of 256) */
  XS_EHIP = 3,          /* a HIP launch or runtime call failed */
  XS_EWORKSPACE = 4,    /* workspace missing or too small */
  XS_ECAPACITY = 5,     /* device: a window received more rows than capacity_rows */
  XS_ETIMEOUT = 6,      /* device: a bounded dependency wait expired */
  XS_EBADINPUT = 7      /* device: an expert id outside [0, E), or listed twice by one token */
};

/* Text for a status code (static storage; never NULL). */
const char* xs_strerror(int code);
/* Library version, major * 10000 + minor * 100 + patch. */
int xs_version(void);

/* ----------------------------------------------------------------------------- windows
 * A destination window (Sec. 2.1: the memory a one-sided store lands in). On one GPU a
 * "remote" window is a buffer in local HBM, or in host-coherent memory for a slow sink.
 * Row r starts at base + r * row_stride_bytes. row_stride_bytes must be a multiple of 16
 * and at least the row size in bytes. If ready_flag is non-NULL, the call that stores into
 * the window sets *ready_flag = 1 after its last store, behind a release fence at system
 * scope (consumer readiness, Sec. 2.1; sender progress alone is not readiness). */
typedef struct xs_window {
  void* base;
  int64_t capacity_rows;
  int64_t row_stride_bytes;
  uint32_t* ready_flag;
} xs_window;

#define XS_MAX_WINDOWS 64

/* ----------------------------------------------------------------------------- routing
 * Top-k softmax gating (routing is fixed by the model and unchanged by the method:
 * Related Work, "MoE communication").
 *   logits   device fp32 [T][E], finite or -inf (a masked expert), at least one finite
 *            value per row.
 *   topk_idx device int32 [T][k] out: the k largest logits in descending order, ties to
 *            the lower expert index (selection is exact on the fp32 logits).
 *   topk_w   device fp32 [T][k] out: softmax over all E experts taken at topk_idx; with
 *            renormalize != 0 divided by the sum of the k weights.
 * Requires 1 <= k <= min(E, 32), E <= 1024. */
int xs_route_topk_softmax(const float* logits, int32_t T, int32_t E, int32_t k,
                          int32_t renormalize, int32_t* topk_idx, float* topk_w, void* stream);

/* ----------------------------------------------------------------------------- layout
 * Destination-window layout of every (source, token, slot) (the Dispatch exchange,
 * Sec. 2.2 and Sec. 4.3: expert-parallel tokens go to the ranks owning their experts).
 * Expert e lives in window d(e) = e / (E / W). Rows of window d are the slots routed to
 * its experts ordered by (expert, source, token), unpadded, one row per slot.
 *   topk_idx       device int32 [n_src][T][k]; the k experts of a token are distinct (an id
 *                  outside [0, E) or listed twice by one token sets XS_EBADINPUT, and the
 *                  rows of that token are then unspecified)
 *   expert_counts  device int32 [n_src][E] out: slots of source s routed to expert e
 *   src_base       device int32 [n_src][E] out: rows of expert e from sources < s
 *   expert_offsets device int32 [E] out: first row of expert e inside window d(e)
 *   dest_counts    device int32 [W] out: rows per window (may exceed cap: XS_ECAPACITY)
 *   slot_row       device int32 [n_src][T][k] out: row of each slot inside its window
 *   row_src        device int32 [W][cap] out: inverse map, (src << 24) | (t * k + j), for
 *                  rows < cap (rows at or beyond cap are not recorded)
 *   workspace      device, xs_dispatch_layout_workspace_bytes() bytes
 * Requires E % W == 0, E <= 1024, W <= XS_MAX_WINDOWS, n_src <= 127, T * k < 2^24. */
int xs_dispatch_layout_workspace_bytes(int32_t n_src, int32_t T, int32_t E, int64_t* bytes);
int xs_dispatch_layout(const int32_t* topk_idx, int32_t n_src, int32_t T, int32_t k, int32_t E,
                       int32_t W, int32_t cap, int32_t* expert_counts, int32_t* src_base,
                       int32_t* expert_offsets, int32_t* dest_counts, int32_t* slot_row,
                       int32_t* row_src, void* workspace, int64_t workspace_bytes,
                       int32_t* dev_status, void* stream);

/* ----------------------------------------------------------------------------- dispatch
 * Store one source's token rows into the destination windows (one-sided stores, Sec. 2.1):
 * window d(topk_idx[t][j]) row slot_row[t][j] <- x[t], a bit-exact bf16 copy of H values.
 *   x        device bf16 [T][H] (row-major, rows contiguous)
 *   topk_idx, slot_row  device int32 [T][k] of this source (a slice of the layout outputs)
 *   win      host array of W windows (capacity_rows >= largest row + 1, else XS_ECAPACITY
 *            and the row is skipped)
 * Requires H % 8 == 0 (128-bit stores). */
int xs_dispatch(const void* x, int32_t T, int32_t H, const int32_t* topk_idx,
                const int32_t* slot_row, int32_t k, int32_t E, const xs_window* win, int32_t W,
                int32_t* dev_status, void* stream);

/* The same one-sided row stores (Sec. 2.1; the quantized EP runs of Sec. 5.2 dispatch quantized
 * token rows) for rows of any byte length (a multiple of 16, rows row_stride bytes apart,
 * 16-byte aligned): e.g. MXFP8 token rows of H codes then H / 32 scales (xs_quantize_mx into
 * caller staging, then this). Windows need row_stride_bytes >= row_bytes. Errors as
 * xs_dispatch. */
int xs_dispatch_rows(const void* rows, int64_t row_stride, int32_t row_bytes, int32_t T,
                     const int32_t* topk_idx, const int32_t* slot_row, int32_t k, int32_t E,
                     const xs_window* win, int32_t W, int32_t* dev_status, void* stream);

/* Dispatch through bounded destination rings (Sec. 4.3: an eligible Linear-1 tile needs ready
 * dispatch input and a free destination ring slot; App. A.2: ring-slot readiness is checked
 * before a tile is emitted). Reading: destination d owns a ring of S slots (rings[d]: base,
 * capacity_rows = S, equal for every d; row_stride_bytes >= xs_ring_slot_bytes(H, k), a
 * multiple of 16; 16-byte aligned; device or host-coherent memory). An entry is one bf16
 * token row of x [T][H] plus a header naming the rows of window d it is copied into: with
 * dedup = 1 one entry per (token, destination) listing every k slot of the token there, with
 * dedup = 0 one entry per (token, k) slot. Lifetime protocol: the producer of entry n
 * (numbered per ring in token order, then k slot order) fills slot n mod S only after entry
 * n - S has been copied out and released; the consumer copies an entry into its window rows
 * (slot_row[t][j] of win[d]) and then releases the slot. Workgroups produce their tokens'
 * entries and consume entries, a stalled producer draining the entries it waits on, so the
 * call completes for any S >= 1. The windows end equal to xs_dispatch's.
 * max_producers: workgroups (0 = one per CU). spin_timeout_us: bound of every wait (0 = 2 s);
 * on expiry XS_ETIMEOUT goes to dev_status and the kernel exits. workspace: device bytes from
 * xs_dispatch_ring_workspace_bytes(T, k, W, S) (control words and entry numbers; rewritten
 * by every call). stats:
 * optional device int32 [2W]: entries per destination, then productions that found their
 * slot still occupied. Status words as xs_dispatch (XS_ECAPACITY for rows beyond a window,
 * XS_EBADINPUT for bad experts). Argument errors: XS_EINVAL / XS_EUNSUPPORTED /
 * XS_EWORKSPACE, nothing launched. */
int xs_ring_slot_bytes(int32_t H, int32_t k, int64_t* bytes);
int xs_dispatch_ring_workspace_bytes(int32_t T, int32_t k, int32_t W, int32_t slots, int64_t* bytes);
int xs_dispatch_ring(const void* x, int32_t T, int32_t H, const int32_t* topk_idx,
                     const int32_t* slot_row, int32_t k, int32_t E, const xs_window* win, int32_t W,
                     const xs_window* rings, int32_t dedup, int32_t max_producers,
                     int64_t spin_timeout_us, void* workspace, int64_t workspace_bytes,
                     int32_t* stats, int32_t* dev_status, void* stream);

/* ----------------------------------------------------------------------------- EP layer
 * One rank's share of an expert-parallel MoE layer (Sec. 4.3). Experts
 * [e_begin, e_begin + n_experts) are computed here; they must be whole windows
 * (e_begin and n_experts multiples of E / W). "This GPU" is source rank `src`: its
 * tokens are dispatched and its output is reduced; routing and layout cover all n_src
 * sources (standing in for the count exchange between ranks).
 * Expert FFN (SwiGLU): h = bf16(silu(x Wg^T) * (x Wu^T)), y = bf16(h W2^T), fp32
 * accumulation; W1 rows [0, I) are the gate Wg and rows [I, 2I) the up projection Wu.
 * Precision (the paper's EP runs also at W8A8, Sec. 5.2):
 *   XS_PREC_BF16   as above.
 *   XS_PREC_MXFP8  MX formats (see "MX formats" below). Token rows are quantized once, in
 *                  the dispatch phase, into workspace staging and dispatched as rows of H
 *                  E4M3 codes followed by H / 32 E8M0 scales (dispatch window rows >= H +
 *                  H / 32 bytes; a row stride that is a multiple of 128 bytes keeps every
 *                  row on whole cache lines, which the Linear-1 loads run faster on);
 *                  w1 / w2 hold E4M3 codes ([n_experts][2I][H] and
 *                  [n_experts][H][I] bytes) and w1_scale / w2_scale their scales grouped
 *                  by 512 K elements, as xs_quantize_mx_grouped writes them over all of
 *                  the weight rows: [H / 512][n_experts * 2I][16] and
 *                  [I / 512][n_experts * H][16] bytes. Linear-1 runs on the scaled MFMA,
 *                  SwiGLU in fp32, and h is stored as MXFP8: h_ws holds h_rows code rows of
 *                  I bytes, then the scales in groups [I / 512][h_rows][16] (h_rows * (I +
 *                  I / 32) bytes in all); Linear-2 likewise, its
 *                  output y rounded to bf16 for the unchanged combine. Requires H and I
 *                  multiples of 512. Only xs_fused_ep_layer takes it (the unfused phase calls
 *                  return XS_EUNSUPPORTED).
 *   XS_PREC_W4A8   as XS_PREC_MXFP8 with E2M1 weights: w1 / w2 hold packed E2M1 codes
 *                  ([n_experts][2I][H / 2] and [n_experts][H][I / 2] bytes, element 2 i in the
 *                  low nibble) under the same E8M0 scales; token rows and h stay MXFP8. */
enum { XS_PREC_BF16 = 0, XS_PREC_MXFP8 = 1, XS_PREC_W4A8 = 2 };

typedef struct xs_ep_layer {
  int32_t n_src, T, H, E, k, I, W;
  int32_t e_begin, n_experts;
  int32_t src;
  int32_t renormalize;
  int32_t expert_mode;        /* XS_EXPERT_SWIGLU, or XS_EXPERT_IDENTITY (y = x) */
  int32_t cap;                /* capacity_rows of every dispatch window */
  const float* logits;        /* device fp32 [n_src][T][E] */
  const void* x;              /* device bf16 [T][H], tokens of source `src` */
  const void* w1;             /* device bf16 [n_experts][2I][H] */
  const void* w2;             /* device bf16 [n_experts][H][I] */
  int32_t* topk_idx;          /* device int32 [n_src][T][k] (out of route, in to layout) */
  float* topk_w;              /* device fp32  [n_src][T][k] */
  int32_t* expert_counts;     /* device int32 [n_src][E] */
  int32_t* src_base;          /* device int32 [n_src][E] */
  int32_t* expert_offsets;    /* device int32 [E] */
  int32_t* dest_counts;       /* device int32 [W] */
  int32_t* slot_row;          /* device int32 [n_src][T][k] */
  int32_t* row_src;           /* device int32 [W][cap] */
  const xs_window* dispatch_win; /* host array [W]; rows of H bf16 */
  const xs_window* combine_win;  /* host array [n_src]; window s holds [T*k] rows of H bf16 */
  void* h_ws;                 /* device bf16 [h_rows][I], SwiGLU activations */
  int64_t h_rows;             /* >= (n_experts / (E / W)) * cap */
  void* y_ws;                 /* device bf16 [h_rows][H]; only used by the unfused path */
  void* out;                  /* device bf16 [T][H], combined output of source `src` */
  void* events[8];            /* optional hipEvent_t per phase boundary (NULL = not recorded),
                                 recorded on `stream`; see XS_EV_* */
  int32_t precision;          /* XS_PREC_BF16 (0), XS_PREC_MXFP8 or XS_PREC_W4A8 */
  int32_t reserved;           /* 0 */
  const void* w1_scale;       /* MX precisions: device E8M0 [H / 512][n_experts * 2I][16], 16-byte aligned */
  const void* w2_scale;       /* MX precisions: device E8M0 [I / 512][n_experts * H][16], 16-byte aligned */
} xs_ep_layer;

/* Phase boundaries of the EP entry points: events[XS_EV_x] is recorded right before the
 * first launch of phase x (XS_EV_FFN_END right after the expert-FFN kernel(s), XS_EV_END
 * after the last launch). xs_fused_ep_layer records all of them; xs_expert_ffn records
 * XS_EV_PLAN, XS_EV_FFN and XS_EV_FFN_END. */
enum {
  XS_EV_ROUTE = 0, XS_EV_LAYOUT = 1, XS_EV_DISPATCH = 2, XS_EV_PLAN = 3, XS_EV_FFN = 4,
  XS_EV_FFN_END = 5, XS_EV_REDUCE = 6, XS_EV_END = 7
};

enum { XS_EXPERT_SWIGLU = 0, XS_EXPERT_IDENTITY = 1 };

/* Store pacing of the persistent EP kernel: the order of Linear-1 / Linear-2 tiles.
 *   XS_POLICY_BURST      Expert-Wave (Sec. 4.3): per wave of experts, all Linear-1 tiles
 *                        then all Linear-2 tiles (whose epilogues are the store bursts).
 *   XS_POLICY_INTERLEAVE cross-wave interleaving (App. A.2, Alg. 1) with lead D =
 *                        lead_rows rows of Linear-1 over Linear-2; lead_rows = 0 takes the
 *                        anti-starvation knee of App. A.2, ceil(grid / P1) with P1 = I / 128
 *                        Linear-1 tiles per row.
 *   XS_POLICY_CHUNK      Alg. 1 with at most chunk_tiles consecutive Linear-2 tiles before
 *                        a ready Linear-1 tile is forced.
 *   XS_POLICY_AUTO       the order xs_pacing_audit_run picks with `model` (Sec. 4.1, Eqs. 3-6
 *                        over each candidate order's burst sequence: BURST, INTERLEAVE at
 *                        lead_rows, CHUNK 1..32; the least predicted stall, ties to
 *                        INTERLEAVE); INTERLEAVE without a model.
 * max_producers caps the persistent grid (0 = one workgroup per CU); wave_tiles is the
 * minimum Linear-1 tile count of an expert wave (0 = the grid size); gap_ns inserts a
 * non-injecting wait of that many nanoseconds after every Linear-2 store burst.
 * claim selects how producers take tiles:
 *   XS_CLAIM_STATIC   producer g of G takes the entries g, g + G, ... of each tile stream
 *                     (the per-instance cursors of Alg. 1);
 *   XS_CLAIM_DYNAMIC  producers take the next entry of a stream from a shared counter when
 *                     they finish a tile, under the same rule (a Linear-2 tile of row p is
 *                     taken only when every Linear-1 tile of rows <= p + D - 1 has been
 *                     taken; BURST: the next entry of the Expert-Wave list). Same tiles and
 *                     bytes; balances producers whose tiles differ in length.
 * Every policy computes the same tiles and stores the same bytes; outputs are
 * bit-identical across policies. */
enum { XS_POLICY_BURST = 0, XS_POLICY_INTERLEAVE = 1, XS_POLICY_CHUNK = 2, XS_POLICY_AUTO = 3 };
enum { XS_CLAIM_STATIC = 0, XS_CLAIM_DYNAMIC = 1 };

struct xs_model;
typedef struct xs_pacing {
  int32_t policy;
  int32_t lead_rows;
  int32_t chunk_tiles;
  int32_t max_producers;
  int32_t wave_tiles;
  int32_t gap_ns;
  int32_t spin_timeout_us;        /* bound of each dependency wait; 0 = 2 s */
  int32_t withhold_row;           /* failure-path hook: this row never signals Linear-1
                                     completion, so its Linear-2 waits expire (-1 = none) */
  int32_t claim;                  /* XS_CLAIM_STATIC or XS_CLAIM_DYNAMIC */
  int32_t reserved;               /* must be 0 */
  double t_l1_us, t_l2_us;        /* mainloop time of one Linear-1 / Linear-2 tile for the
                                     model audit (xs_trace_tile_times gives them from a traced
                                     run); 0 = an estimate from the tile FLOPs at 40 % of one
                                     CU's share of the dense peak */
  const struct xs_model* model;   /* host, for XS_POLICY_AUTO and xs_pacing_audit; may be NULL */
  const int32_t* expert_rows;     /* host int32 [n_experts] or NULL: rows each local expert is
                                     expected to compute (for instance the last step's counts);
                                     NULL = the uniform expectation n_src T k / E */
  double sink_share;              /* share of each Linear-2 tile's stored bytes that reach the
                                     sink `model` describes (e.g. 2 / 8 with two of eight combine
                                     windows in host memory); 0 = all of them */
} xs_pacing;

/* Optional device trace of the persistent kernels: one 32-byte record per tile,
 *   rec[0] = kind << 56 | workgroup << 32 | tile index  (kind 1 = Linear-1, 2 = Linear-2,
 *            3 = plain / scatter GEMM tile)
 *   rec[1] = wall clock (s_memrealtime ticks, xs_clock_rate_hz) at tile start
 *   rec[2] = wall clock when the mainloop finished (epilogue starts)
 *   rec[3] = wall clock after the last store of the epilogue was issued (sender-visible
 *            issue end: the stores are accepted, not necessarily visible)
 * records are appended at atomicAdd(count, 1); records past `capacity` are dropped but
 * still counted. buf and count are device memory; the caller zeroes *count.
 * ext (nullable, device, 4 x uint64 per record, same index; EP kernels only):
 *   ext[0] = wall clock when the tile's dependency wait ended (= rec[1] for Linear-1 tiles)
 *   ext[1] = staging wait in ticks: how long the workgroup's first wave waited, before this
 *            tile's mainloop, for the stores of its previous epilogue to leave the wave (the
 *            local staging reuse point of App. A.2; taking it adds that wait to the wave)
 *   ext[2] = bytes the tile's epilogue stored, ext[3] = rows of the tile */
typedef struct xs_trace {
  uint64_t* buf;
  int64_t capacity;
  uint32_t* count;
  uint64_t* ext;
} xs_trace;

/* Workspace of the EP calls below (layout scratch, tile tables, readiness counters). */
int xs_ep_layer_workspace_bytes(const xs_ep_layer* L, int64_t* bytes);

/* Expert FFN of the computed experts, unfused: Linear-1 + SwiGLU into h_ws, then Linear-2
 * into y_ws, both indexed by "computed row" (window d_first's rows, then the next
 * window's, ...). Reads the layout outputs of L. */
int xs_expert_ffn(const xs_ep_layer* L, void* workspace, int64_t workspace_bytes,
                  int32_t* dev_status, void* stream);

/* Combine-send (the Combine exchange, Sec. 4.3): computed row r of window d goes to
 * combine window s at row t*k+j where row_src[d][r] = (s << 24) | (t*k+j). Unfused form of
 * the Linear-2 epilogue stores; reads y_ws. pacing (nullable) shapes the bursts the combine
 * windows see: max_producers workgroups (0 = eight per CU) each store bursts of chunk_tiles
 * blocks of 256 consecutive computed rows (chunk_tiles 0: bursts of 8 rows), burst b of
 * producer g being burst-sized block g + b * producers, with a non-injecting gap of gap_ns
 * after each burst; the other fields are ignored. Every setting stores the same bytes. */
int xs_combine_send(const xs_ep_layer* L, const xs_pacing* pacing, int32_t* dev_status, void* stream);

/* Combine-reduce (the receiving side of the Combine exchange, Sec. 4.3: the source rank weighs
 * the k expert outputs of each token by its gate weights once they are ready, Sec. 2.1):
 * out[t] = bf16(sum_{j<k} w[t][j] * C[t*k + j]), fp32 sum in ascending j.
 *   cbuf device bf16 [T*k][H] (row stride cbuf_stride_bytes), topk_w device fp32 [T][k],
 *   out device bf16 [T][H]. Requires H % 8 == 0. */
int xs_combine_reduce(const void* cbuf, int64_t cbuf_stride_bytes, const float* topk_w,
                      int32_t T, int32_t k, int32_t H, void* out, void* stream);

/* The whole layer: route (all sources) -> layout -> dispatch (source src) -> persistent
 * Linear-1 / Linear-2 kernel whose Linear-2 epilogue stores straight into the combine
 * windows, in the order set by `pacing` -> combine-reduce of source src. `trace` may be
 * NULL. Linear-2 tiles wait on per-row Linear-1 completion counters with a bounded spin
 * (XS_ETIMEOUT in dev_status if it expires; the kernel then skips the tile and exits). */
int xs_fused_ep_layer(const xs_ep_layer* L, const xs_pacing* pacing, const xs_trace* trace,
                      void* workspace, int64_t workspace_bytes, int32_t* dev_status,
                      void* stream);

/* The same layer for callers that cannot allocate (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): no workspace argument; the layer's scratch (layout
 * partial counts, tile tables, readiness and claim counters, MX token-row staging) lives in a
 * library-owned device array of XS_STATIC_SCRATCH_BYTES on each GPU the library runs on, held
 * until the process ends. Requires xs_ep_layer_workspace_bytes(L) <= XS_STATIC_SCRATCH_BYTES,
 * else XS_EWORKSPACE and nothing is launched (the DeepSeek-V3-like share needs under 1 MiB in
 * bf16 and about 31 MiB in the MX precisions). Calls no hipMalloc, hipFree or other allocating
 * routine. Every call on one GPU shares that GPU's array and the kernels rewrite or clear all of
 * it that they read, so consecutive calls on one stream are independent; calls that overlap on
 * one GPU (other streams, other host threads) race on it. Otherwise as xs_fused_ep_layer. */
#define XS_STATIC_SCRATCH_BYTES (48ll << 20)
int xs_fused_ep_layer_noalloc(const xs_ep_layer* L, const xs_pacing* pacing, const xs_trace* trace,
                              int32_t* dev_status, void* stream);

/* ----------------------------------------------------------------------------- GEMM
 * The plain local GEMM of row-parallel tensor parallelism (Sec. 4.5: each rank computes its
 * partial Y_r = X_r W_r) without a scatter epilogue, the compute-only baseline of the fused
 * calls: C = A B^T with bf16 operands and fp32 accumulation, bf16 output.
 *   a  device bf16 [M][K] (row stride lda elements), b device bf16 [N][K] (row stride ldb;
 *      the weight's output-major layout), c device bf16 [M][N] (row stride ldc).
 * Requires N % 256 == 0, K % 64 == 0, strides multiples of 8. */
int xs_gemm(const void* a, int64_t lda, const void* b, int64_t ldb, void* c, int64_t ldc,
            int32_t M, int32_t N, int32_t K, const xs_trace* trace, void* stream);

/* Grouped GEMM over row segments (the local-expert grouped GEMM of Sec. 4.3 as a library
 * call, with the Linear-1 SwiGLU epilogue of the expert FFN): for every segment s, rows
 * [seg_offsets[s], seg_offsets[s] + seg_rows[s]) of a times B_s^T, B_s = b + s N K elements, into
 * the same rows of c, fp32 accumulation, bf16 output:
 *   XS_EPI_STORE   c bf16 [M][N] (row stride ldc elements): c = bf16(a B_s^T)
 *   XS_EPI_SWIGLU  B_s holds the gate rows [0, N / 2) then the up rows [N / 2, N); c bf16
 *                  [M][N / 2]: c = bf16(silu(a Wg^T) * (a Wu^T))
 *   a         device bf16 [M][K], row stride lda elements
 *   seg_offsets, seg_rows  device int32 [n_seg] (n_seg <= 1024): a segment may be empty; one
 *             that does not lie inside [0, M) sets XS_EBADINPUT in dev_status and is skipped;
 *             overlapping segments race on their common rows
 *   b         device bf16 [n_seg][N][K] (output-major, K-contiguous)
 * Rows outside every segment are not written. Requires K % 64 == 0, N % 256 == 0 (STORE) or
 * N % 256 == 0 (SWIGLU: 128 output columns per tile), lda and ldc multiples of 8. Returns
 * XS_EINVAL / XS_EUNSUPPORTED on bad arguments (nothing launched), XS_EHIP if the launch fails.
 * The caller owns every buffer; nothing is allocated. */
enum { XS_EPI_STORE = 0, XS_EPI_SWIGLU = 1 };
int xs_grouped_gemm(const void* a, int64_t lda, int32_t M, const int32_t* seg_offsets, const int32_t* seg_rows,
                    int32_t n_seg, const void* b, int32_t N, int32_t K, void* c, int64_t ldc, int32_t epilogue,
                    int32_t* dev_status, void* stream);

/* GEMM with a scatter epilogue: every output tile is stored on completion into the
 * destination windows (no separate permutation pass).
 *   XS_SCATTER_ROW_BLOCK  (Sec. 4.5, row-parallel TP): output row m goes to window
 *                         m / rows_per_dest, row m % rows_per_dest (N values per row).
 *   XS_SCATTER_HEAD_GROUP (Sec. 5.4, Ulysses GEMM-All-to-All): column c of the
 *                         [n_proj * n_heads * head_dim] output is (p, head, dd) with
 *                         p = c / (n_heads*head_dim), head = (c / head_dim) % n_heads,
 *                         dd = c % head_dim; it goes to window g = head / heads_per_group
 *                         at element ((p * heads_per_group + head % heads_per_group) * M + m)
 *                         * head_dim + dd, i.e. window g is [n_proj][hpg][M][head_dim]
 *                         (row_stride_bytes = head_dim * 2).
 * Requires M % rows_per_dest == 0 and rows_per_dest % 256 == 0 (ROW_BLOCK); head_dim % 8 == 0
 * (HEAD_GROUP). Window capacity_rows must cover rows_per_dest (ROW_BLOCK) or
 * n_proj * heads_per_group * M (HEAD_GROUP). */
enum { XS_SCATTER_ROW_BLOCK = 0, XS_SCATTER_HEAD_GROUP = 1 };
typedef struct xs_scatter_desc {
  int32_t kind;
  int32_t rows_per_dest;
  int32_t n_proj, n_heads, head_dim, heads_per_group;
} xs_scatter_desc;

/* pacing (nullable) sets the order in which the persistent producers take tiles, and so the
 * bursts the windows see (Sec. 4.5: aligned producers push V_n = K_act B_c, with B_c one
 * 256 x 256 bf16 tile of 128 KiB; chunking makes bursts smaller but more frequent):
 *   NULL                  tiles in groups of 4 M-tiles (the L2-friendly order)
 *   XS_POLICY_BURST       destination-major: every tile of window 0, then of window 1, ...
 *   XS_POLICY_INTERLEAVE  round robin over the windows, one tile each
 *   XS_POLICY_CHUNK       chunk_tiles consecutive tiles of one window, then the next window
 *                         (the tiles per window must be a multiple of chunk_tiles)
 * plus max_producers (grid cap, 0 = one workgroup per CU) and gap_ns (a non-injecting wait
 * after every tile's stores); the other fields are ignored. With a pacing order, HEAD_GROUP
 * needs tile-aligned groups ((n_heads head_dim) % 256 == 0, (heads_per_group head_dim) % 256
 * == 0, 256 % head_dim == 0), else XS_EUNSUPPORTED. Every order stores the same bytes. */
int xs_gemm_scatter(const void* a, int64_t lda, const void* b, int64_t ldb, int32_t M, int32_t N,
                    int32_t K, const xs_scatter_desc* desc, const xs_window* win, int32_t W,
                    const xs_pacing* pacing, const xs_trace* trace, void* stream);

/* Serial counterpart of xs_gemm_scatter: a separate permutation pass that copies a plain
 * GEMM output c [M][N] into the windows with the same mapping (the "permutation before the
 * All-to-All" that fusion removes, Sec. 5.4). */
int xs_scatter_copy(const void* c, int64_t ldc, int32_t M, int32_t N, const xs_scatter_desc* desc,
                    const xs_window* win, int32_t W, void* stream);

/* ----------------------------------------------------------------------------- attention
 * Attention with the post-attention Ulysses exchange (Sec. 4.4, App. B; Table 4). One
 * rank's share after the pre-attention exchange: all M tokens of `heads` local heads.
 *   O[h][t][:] = sum_u softmax_u(scale * Q[h][t] . K[h][u]) V[h][u]   (full, non-causal)
 * computed as a flash-attention pass: every persistent workgroup takes 128-query output
 * tiles of one head and streams the head's K/V in 64-token tiles (the Q-loop), with an
 * online softmax in fp32 and bf16 probabilities for the second product.
 *   q, k, v  device bf16 [heads][M][head_dim]; head_dim must be 128.
 *   scale    0 = 1 / sqrt(head_dim).
 *   M        multiple of 128, at most 8,388,480 (one head's K or V rows within a 2 GiB
 *            buffer range); with windows, M / W must be a multiple of 128 (a tile never
 *            straddles two destinations).
 * Modes:
 *   XS_ATTN_LOCAL    output o, device bf16 [heads][M][head_dim] ("FA-only").
 *   XS_ATTN_WINDOWS  each finished output tile is stored by the workgroup that computed it
 *                    into window g = t / (M / W): row t % (M / W), head slot h, i.e. at
 *                    base + (t % (M / W)) * row_stride_bytes + h * head_dim * 2 (a window
 *                    holds [M / W][heads][head_dim]); the next Q-loop is the drain window.
 *                    Ready flags are set after the last tile.
 *   XS_ATTN_WINDOWS_COUPLED  as XS_ATTN_WINDOWS, but after each tile's stores the producer
 *                    waits until they are visible at system scope before its next Q-loop:
 *                    the completion-coupled issuer the paper argues against (Sec. 4.4, Fig. 7),
 *                    kept as the measured counterfactual.
 * max_producers caps the persistent grid (0 = three workgroups per CU). The optional trace
 * records one kind-4 record per output tile: rec[1] tile start, rec[2] end of its Q-loop,
 * rec[3] after its stores were issued. q, k, v and o are 16-byte aligned; windows as for the
 * other window calls (16-byte aligned base and row stride, stride >= heads * head_dim * 2,
 * capacity >= M / W rows). The caller owns every buffer; nothing is allocated. Returns
 * XS_EINVAL for null, misaligned or inconsistent arguments, XS_EUNSUPPORTED for a head_dim,
 * M or M / W the kernel does not tile, XS_EHIP if a launch fails; nothing is launched on an
 * argument error. Output tiles are computed in a fixed order of operations, so results do
 * not depend on the grid size or on the mode. */
enum { XS_ATTN_LOCAL = 0, XS_ATTN_WINDOWS = 1, XS_ATTN_WINDOWS_COUPLED = 2 };

typedef struct xs_attn {
  int32_t heads, M, head_dim, W;
  float scale;
  int32_t max_producers;
  const void* q;              /* device bf16 [heads][M][head_dim] */
  const void* k;
  const void* v;
  void* o;                    /* XS_ATTN_LOCAL: device bf16 [heads][M][head_dim] */
  const xs_window* win;       /* XS_ATTN_WINDOWS: host array [W] */
} xs_attn;

int xs_attention(const xs_attn* a, int32_t mode, const xs_trace* trace, void* stream);

/* The serial post-attention exchange: o (device bf16 [heads][M][head_dim], 16-byte aligned,
 * head_dim a multiple of 8) copied into the windows of XS_ATTN_WINDOWS, then their ready flags
 * set (the baseline the fused path is compared with). Returns XS_EINVAL for bad arguments,
 * XS_EHIP if a launch fails. */
int xs_ulysses_copy(const void* o, int32_t heads, int32_t M, int32_t head_dim,
                    const xs_window* win, int32_t W, void* stream);

/* ----------------------------------------------------------------------------- MX formats
 * Quantized EP precisions (W8A8, W4A8: Sec. 5.2, the MegaMoE sweep; the paper does not fix the
 * formats). Reading: OCP microscaling as the gfx950 matrix cores take it. A block of 32
 * consecutive elements along the reduction axis shares one E8M0 scale 2^(s - 127); elements
 * are E4M3 (OCP "FN": bias 7, largest 448, no infinities) or E2M1 (0, 0.5, 1, 1.5, 2, 3, 4, 6
 * and negatives). Quantization: e = the smallest integer with amax <= fmax 2^e (fmax 448 or
 * 6; e = 0 for an all-zero block; clamped to [-127, 127]), decided on the exponent and
 * mantissa bits of the block's largest magnitude; codes = round-to-nearest-even of
 * x / 2^e (never saturates). E2M1 codes pack two per byte, element 2 i in the low nibble. */
enum { XS_FMT_E4M3 = 0, XS_FMT_E2M1 = 1 };

/* Block quantizer: x bf16 [rows][cols] (ldx elements per row, 16-byte aligned rows) ->
 * codes [rows][cols] bytes (E4M3; ld_codes a multiple of 8) or [rows][cols / 2] (E2M1;
 * ld_codes a multiple of 4), scales [rows][cols / 32] bytes (ld_scales bytes per row).
 * cols is a multiple of 32. Device pointers, caller-owned; stream-ordered. XS_EINVAL on bad
 * arguments (nothing launched), XS_EHIP if the launch fails. */
int xs_quantize_mx(const void* x, int64_t rows, int32_t cols, int64_t ldx, int32_t fmt,
                   void* codes, int64_t ld_codes, void* scales, int64_t ld_scales, void* stream);

/* The same quantizer with the scales grouped by 512 columns, the layout the MX GEMM core of
 * the EP layer loads a run of rows from at once: the scale of row r, block j (columns
 * [32 j, 32 j + 32)) at byte ((j / 16) * rows + r) * 16 + j % 16, i.e. [cols / 512][rows][16].
 * cols a multiple of 512, scales 16-byte aligned; otherwise as xs_quantize_mx (the static
 * weights of an MX EP layer are quantized with it once, at upload). */
int xs_quantize_mx_grouped(const void* x, int64_t rows, int32_t cols, int64_t ldx, int32_t fmt,
                           void* codes, int64_t ld_codes, void* scales, void* stream);

/* MX GEMM: c (bf16 [M][N], ldc elements) = deq(a) deq(b)^T with a E4M3 codes [M][K] (lda
 * bytes per row) and scales [M][K / 32] (lda_s bytes per row), b codes in b_fmt, [N][K]
 * bytes (E4M3) or [N][K / 2] packed (E2M1, ldb >= K / 2), ldb bytes per row, and scales
 * [N][K / 32] (ldb_s). fp32 accumulation on v_mfma_scale_f32_32x32x64_f8f6f4, one bf16
 * rounding at the end. N a multiple of 256, K of 512; code and scale rows 16-byte aligned
 * (the kernel loads a row's scales for 512 K elements as one 16-byte piece). XS_EINVAL /
 * XS_EUNSUPPORTED on bad arguments (nothing launched), XS_EHIP if the launch fails. */
int xs_gemm_mx(const void* a, int64_t lda, const void* a_scales, int64_t lda_s, const void* b,
               int64_t ldb, const void* b_scales, int64_t ldb_s, int32_t b_fmt, void* c,
               int64_t ldc, int32_t M, int32_t N, int32_t K, const xs_trace* trace, void* stream);

/* ----------------------------------------------------------------------------- X-Stage
 * Burst-Gap model (Sec. 3.3-3.5). Units: bytes and microseconds.
 *   T0(V) = t0_a_us + t0_b_us_per_byte * V   recovered issue floor at K producers
 *   R_bytes_per_us                           effective aggregate drain rate
 *   Q_bytes                                  effective outstanding capacity (inf allowed) */
typedef struct xs_model {
  double t0_a_us;
  double t0_b_us_per_byte;
  double R_bytes_per_us;
  double Q_bytes;
  int32_t K;
  int32_t _pad;
} xs_model;

/* One burst of a sequence (Sec. 4.1): aggregate volume, recovered issue floor, the compute
 * gap before the next burst and, for App. A.2's MMA-side stall, the mainloop time T_cover
 * that runs before the burst's local staging must be reused (0 = none). */
typedef struct xs_burst { double V_bytes, T0_us, G_us, cover_us; } xs_burst;

/* Per-burst audit: rho and delta_b (Eqs. 3-4), backlog before the burst, b_iso and the
 * capacity guard (Eq. 6), and the predicted issue time: T0 while the guard holds, else
 * (q + V - Q) / R (a fluid queue capped at Q); the backlog then follows
 * q' = [q + V - R (T_iss + G)]_+, which is Eq. 5 whenever the guard holds. stall_us =
 * T_iss - T0; mma_stall_us = [T_iss - cover]_+ (App. A.2, with T_RS = T_iss). */
typedef struct xs_burst_pred {
  double rho, delta_b, q_before, b_iso, T_iss_us, stall_us, mma_stall_us;
  int32_t guard_ok;
  int32_t _pad;
} xs_burst_pred;

/* Host-only, synchronous. q0 is the backlog before the first burst. */
int xs_model_predict(const xs_model* m, const xs_burst* bursts, int32_t n, double q0,
                     xs_burst_pred* out);

/* Calibration points (host arrays): recovered large-gap issue times, zero-gap periodic
 * periods, isolated-burst issue times, each against the aggregate volume V (Sec. 3.3).
 * T0 is a least-squares line, R the through-origin slope of period vs V, and Q the median
 * of V - R T_iss over isolated bursts whose issue exceeds T0(V) by more than knee_excess
 * (relative): the knee where the floor meets the stalled branch (Sec. 3.5). */
typedef struct xs_calib {
  const double* rec_V; const double* rec_T; int32_t n_rec;
  const double* zg_V; const double* zg_T; int32_t n_zg;
  const double* iso_V; const double* iso_T; int32_t n_iso;
  int32_t K;
  double knee_excess;
} xs_calib;

int xs_model_fit(const xs_calib* c, xs_model* out);

/* The calibration procedure around xs_model_fit (Sec. 3.1, 3.3, 3.5), host-only:
 *   xs_drain_rate   R = sum V^2 / sum V T over zero-gap periodic runs (T = V / R through the
 *                   origin), the estimate used to size the recovery gaps of later runs;
 *   xs_calib_knee   the isolated-burst knee: the first index i >= 2 whose issue time exceeds
 *                   (1 + knee_excess) times the line through bursts 0 and i - 1 (n if none);
 *                   iso_V ascending;
 *   xs_model_calibrate  xs_model_fit on c, plus the knee of c's isolated bursts and the capacity
 *                   bracket it gives: Q between V - R T0(V) at the last isolated burst on the
 *                   floor and at the first one off it (lo = hi = +inf without a knee). A sharp
 *                   knee whose stalled bursts issue at about V / R makes the fluid Q of
 *                   xs_model_fit come out <= 0; the bracket's lower end is then the capacity to
 *                   use (the largest volume seen absorbed without stalling). */
typedef struct xs_calib_summary {
  xs_model model;                 /* xs_model_fit's T0, R and fluid Q */
  int32_t knee;                   /* index of the first isolated burst past the knee, n_iso if none */
  int32_t _pad;
  double Q_bracket_lo, Q_bracket_hi;
} xs_calib_summary;

int xs_drain_rate(const double* zg_V, const double* zg_T, int32_t n, double* R_bytes_per_us);
int xs_calib_knee(const double* iso_V, const double* iso_T, int32_t n, double knee_excess, int32_t* knee);
int xs_model_calibrate(const xs_calib* c, xs_calib_summary* out);

/* Eq. 1 for periodic bursts of aggregate volume V separated by a non-injecting gap G:
 * T_period = max(T0(V) + G, V / R) and T_iss = max(T0(V), V / R - G), with T0(V) from m.
 * Host-only. */
int xs_burst_gap(const xs_model* m, double V_bytes, double G_us, double* T_period_us, double* T_iss_us);

/* Recovery audit of a producer's output bursts (App. B, App. C): n_bursts aligned bursts of V
 * bytes, each followed by the gap G (the next Q-loop); the recurrence of xs_model_predict over
 * them; G* = [V / R - T0(V)]_+ (Eq. 2); with sigma_us the compute per K/V tile of b_n keys, the
 * smallest sequence length whose Q-loop covers G*, M_ub* = b_n ceil(G* / sigma) (App. C.2); the
 * drain left after the last burst, [(q_last + V) / R - T0]_+ (no compute follows it); and the
 * completion-coupled issuer's extra time, n_bursts max(T0, V / R) (Sec. 3.2). Host-only. */
typedef struct xs_recovery {
  double T0_us, G_star_us, rho, delta_b, b_iso, stall_us, tail_us, coupled_us;
  int32_t guard_ok;               /* the capacity guard held at every burst */
  int32_t M_ub_star;              /* 0 when sigma_us <= 0 */
} xs_recovery;

int xs_recovery_audit(const xs_model* m, double V_bytes, int32_t n_bursts, double G_us, double sigma_us,
                      int32_t b_n, xs_recovery* out);

/* ----------------------------------------------------------------------------- pacing audit
 * The audit of Sec. 4.1 applied to the persistent EP kernel's tile orders, and the choice
 * XS_POLICY_AUTO makes with it (App. A.1: the average-rate bound of Eq. 9 is necessary but
 * not sufficient; the concrete order must pass the backlog recurrence and capacity guard).
 * For one order the burst sequence is rebuilt from the schedule (Sec. 4.2): producer 0's own
 * tile stream (static claiming, the grid's G producers); its n-th Linear-2 epilogue is the n-th
 * burst, issued together with every other producer's n-th Linear-2 epilogue (full alignment),
 * V_n = K_act V_t summed over those producers' tiles (V_t a tile's stored bytes times
 * sink_share; K_act < G once some producers have no n-th Linear-2 tile); G_n = producer 0's
 * mainloops before its next burst (T_L1 per Linear-1 tile, T_L2 for the next Linear-2 tile);
 * cover = T0 (a workgroup issues its own epilogue stores, so only the floor issue is covered). Rows per local expert come from
 * pacing->expert_rows (else the uniform expectation), split into blocks as the kernel does.
 * Candidates: the given policy alone, or for XS_POLICY_AUTO: BURST (Expert-Wave), INTERLEAVE
 * at the given lead, and CHUNK c = 1, 2, 4, ..., 32. AUTO takes the least predicted stall;
 * among the candidates within 1 % of BURST's mainloop time of it, INTERLEAVE first, then the
 * largest chunk, then BURST (the compute side of the choice, Sec. 5.3: Expert-Wave's Linear-2
 * tiles wait for their wave's Linear-1 tiles, which the audit does not price).
 * Host-only and synchronous; needs the current device only for the grid size. */
#define XS_AUDIT_MAX 16
typedef struct xs_pacing_audit {
  int32_t policy;                 /* chosen policy: XS_POLICY_BURST, _INTERLEAVE or _CHUNK */
  int32_t chunk;                  /* chosen chunk (CHUNK), else 0 */
  int32_t lead_rows;              /* lead D the order uses */
  int32_t producers;              /* G = K_act */
  int32_t rows;                   /* scheduler rows P (expert row blocks) */
  int32_t rate_feasible;          /* Eq. 9 at the whole share's tile mix */
  int32_t n_cand;
  int32_t _pad;
  double t_l1_us, t_l2_us;        /* mainloop times used */
  double V_full_bytes;            /* V of a burst of full tiles */
  int32_t cand_policy[XS_AUDIT_MAX], cand_chunk[XS_AUDIT_MAX];
  int32_t cand_bursts[XS_AUDIT_MAX], cand_guard_fail[XS_AUDIT_MAX];
  double cand_stall_us[XS_AUDIT_MAX];       /* sum of predicted issue stall over the bursts */
  double cand_mma_stall_us[XS_AUDIT_MAX];   /* sum of App. A.2's MMA-side stall */
  double cand_compute_us[XS_AUDIT_MAX];     /* producer 0's mainloop time */
} xs_pacing_audit;

int xs_pacing_audit_run(const xs_ep_layer* L, const xs_pacing* pacing, xs_pacing_audit* out);

/* Mainloop times from a device trace copied to the host (records as xs_trace, n of them, with
 * their ext records, or ext = NULL): medians over Linear-1 tiles of (mainloop end - start) and
 * over Linear-2 tiles of (mainloop end - dependency-wait end), in microseconds, and the
 * median epilogue issue span of Linear-2 tiles (rec[3] - rec[2]). Tiles with fewer than
 * min_rows rows are left out when ext is given (partial tiles run shorter). Host-only. */
int xs_trace_tile_times(const uint64_t* recs, const uint64_t* ext, int64_t n, int32_t min_rows,
                        double* t_l1_us, double* t_l2_us, double* l2_issue_us);

/* Remote-store microbenchmark (Sec. 3.1): K producer workgroups each store B bytes per
 * burst into `target` (HBM window or host-coherent sink), separated by a non-injecting
 * gap of gap_ns nanoseconds; n_bursts (1..256) bursts per producer. Timestamps are kept
 * on chip while the bursts run and written after the last one.
 *   mode XS_MB_PERIODIC   bursts back to back with the gap in between
 *   mode XS_MB_COMPLETION after each burst the producer waits for its stores to complete
 *                         (the completion-coupled counterfactual) before the gap
 * Each producer writes one record per burst into trace->buf: [0] = producer << 32 | burst,
 * [1] = clock at burst start, [2] = clock after the last store was issued, [3] = clock
 * after the gap. Clocks are wall-clock ticks; xs_clock_rate_hz() converts.
 * Producer p writes bytes [p * B * n_bursts ...) of target, wrapping at target_bytes. */
enum { XS_MB_PERIODIC = 0, XS_MB_COMPLETION = 1 };
typedef struct xs_microbench_args {
  void* target;
  int64_t target_bytes;
  int32_t K;
  int32_t B_bytes;        /* multiple of 1024 */
  int32_t n_bursts;
  int32_t gap_ns;
  int32_t mode;
  int32_t store_waves;    /* waves per producer issuing the stores (1..8) */
} xs_microbench_args;

int xs_xstage_microbench(const xs_microbench_args* args, const xs_trace* trace, void* stream);

/* Frequency of the wall clock used by trace records (Hz), from the current device. */
double xs_clock_rate_hz(void);

#ifdef __cplusplus
}
#endif
#endif /* XSTAGE_H */
