"""Oracle for the expert-parallel MoE path: route, dispatch layout, dispatch,
expert SwiGLU FFN, combine-send and combine-reduce (test infrastructure only).

The X-Stage paper treats routing, placement and the bytes moved as fixed by the
model: its MegaMoE scheduler only reorders ready Linear-1 / Linear-2 tiles and
changes neither routing nor communication volume (Related Work, "MoE
communication"; Sec. 5.3 "Kernel performance": only the tile order changes).
Every function below is therefore a plain definition of what the layer computes;
the fused, paced GPU kernels must reach the same result.

Readings where the paper is silent (listed again in the design notes):
  * gating: softmax over all E experts (fp64, stored fp32), top-k chosen on the
    fp32 logits in descending order, ties to the lower expert index, no
    renormalisation unless asked;
  * expert e lives in window d(e) = e // (E / W) (contiguous expert blocks);
  * rows inside a window are ordered by (expert, source, token), unpadded, one row
    per (token, k) slot (no per-destination dedup);
  * row_src encodes a window row's origin as (src << 24) | (t * k + j);
  * SwiGLU: h = silu(x Wg^T) * (x Wu^T), W1 rows [0, I) are gate and [I, 2I) up;
    h and y are stored in bf16, the gate weight is applied in combine-reduce,
    which sums the k slots in ascending j.
"""
from __future__ import annotations

import numpy as np

STATUS_OK = 0
STATUS_CAPACITY = 5      # a window received more rows than its capacity
STATUS_BADINPUT = 7      # a token lists one expert twice
SENTINEL_BF16 = np.uint16(0xFFFF)  # a NaN pattern no correct kernel ever writes

__all__ = [
    "bf16_bits_to_f64", "round_bf16", "f64_to_bf16_bits", "route_topk_softmax",
    "dispatch_layout", "dispatch", "expert_ffn", "grouped_gemm", "grouped_ffn", "combine_send",
    "combine_reduce", "ep_layer", "ep_layer_dense", "encode_row_src", "decode_row_src",
]


# ----------------------------------------------------------------------------- bf16
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> exact fp64 values."""
    u = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def round_bf16(v: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bf16 value, ties to even (no double rounding).

    v = m * 2**ex with 0.5 <= |m| < 1; bf16 keeps 8 significant bits, so the
    representable neighbours are integers times 2**(ex-8). Exponents below the
    bf16 normal range use the fixed subnormal spacing 2**-133.
    """
    v = np.asarray(v, dtype=np.float64)
    m, ex = np.frexp(v)
    ex = np.maximum(ex, -125)          # subnormal spacing 2**-133 = 2**(-125-8)
    scaled = np.ldexp(v, -(ex - 8))    # exact power-of-two scaling
    return np.ldexp(np.rint(scaled), ex - 8)  # rint rounds half to even


def f64_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    r = round_bf16(v).astype(np.float32)   # exact: r is a bf16 value
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ----------------------------------------------------------------------------- route
def route_topk_softmax(logits: np.ndarray, k: int, renormalize: bool = False):
    """Top-k softmax gating.

    idx[t] lists the k experts with the largest fp32 logits in descending order,
    ties broken toward the lower expert index; w[t, j] = softmax(logits[t])[idx[t, j]]
    with the softmax over all E experts in fp64, stored as fp32. With
    ``renormalize`` the k weights are divided by their sum (fp64) before storing.
    """
    logits = np.asarray(logits, dtype=np.float32)
    T, E = logits.shape
    if not (1 <= k <= E):
        raise ValueError("k must be in [1, E]")
    # a stable sort of the negated keys keeps the lower index first among ties
    order = np.argsort(-logits.astype(np.float64), axis=1, kind="stable")
    idx = order[:, :k].astype(np.int32)
    l64 = logits.astype(np.float64)
    z = np.exp(l64 - l64.max(axis=1, keepdims=True))
    p = z / z.sum(axis=1, keepdims=True)
    w = np.take_along_axis(p, idx.astype(np.int64), axis=1)
    if renormalize:
        w = w / w.sum(axis=1, keepdims=True)
    return idx, w.astype(np.float32)


# ----------------------------------------------------------------------------- layout
def encode_row_src(src, slot):
    return (np.asarray(src, dtype=np.int64) << 24) | np.asarray(slot, dtype=np.int64)


def decode_row_src(code):
    code = np.asarray(code, dtype=np.int64)
    return code >> 24, code & ((1 << 24) - 1)


def dispatch_layout(idx: np.ndarray, E: int, W: int, cap: int | None = None):
    """Window layout of every (source, token, k) slot.

    idx: int [n_src, T, k] expert ids. Expert e belongs to window d(e) = e // (E/W).
    Rows of window d are the slots routed to its experts, ordered by
    (expert, source, token); each slot gets exactly one row.

    Returns a dict with
      expert_counts  [n_src, E]  slots of source s routed to expert e
      src_base       [n_src, E]  rows of expert e contributed by sources < s
      expert_offsets [E]         first row of expert e inside window d(e)
      dest_counts    [W]         rows in each window
      slot_row       [n_src, T, k] row of the slot inside its window
      row_src        list of W int64 arrays, the inverse map (src << 24 | t*k + j)
      status         STATUS_CAPACITY if some window exceeds ``cap`` rows, STATUS_BADINPUT
                     if a token lists one expert twice
    """
    idx = np.asarray(idx, dtype=np.int64)
    if idx.ndim == 2:
        idx = idx[None]
    n_src, T, k = idx.shape
    if E % W != 0:
        raise ValueError("E must be a multiple of W")
    epw = E // W
    s_id = np.broadcast_to(np.arange(n_src)[:, None, None], idx.shape).ravel()
    t_id = np.broadcast_to(np.arange(T)[None, :, None], idx.shape).ravel()
    j_id = np.broadcast_to(np.arange(k)[None, None, :], idx.shape).ravel()
    e_id = idx.ravel()
    if e_id.size and (e_id.min() < 0 or e_id.max() >= E):
        raise ValueError("expert id out of range")

    counts = np.zeros((n_src, E), dtype=np.int64)
    np.add.at(counts, (s_id, e_id), 1)
    total = counts.sum(axis=0)
    src_base = np.cumsum(counts, axis=0) - counts
    expert_offsets = np.zeros(E, dtype=np.int64)
    dest_counts = np.zeros(W, dtype=np.int64)
    for d in range(W):
        blk = total[d * epw:(d + 1) * epw]
        expert_offsets[d * epw:(d + 1) * epw] = np.cumsum(blk) - blk
        dest_counts[d] = blk.sum()

    # order all slots by (expert, source, token); lexsort's last key is primary
    order = np.lexsort((t_id, s_id, e_id))
    slot_row = np.empty(idx.size, dtype=np.int64)
    row_src = [np.empty(int(dest_counts[d]), dtype=np.int64) for d in range(W)]
    start = 0
    for d in range(W):
        n = int(dest_counts[d])
        sel = order[start:start + n]
        slot_row[sel] = np.arange(n)
        row_src[d][:] = encode_row_src(s_id[sel], t_id[sel] * k + j_id[sel])
        start += n
    status = STATUS_OK
    if cap is not None and dest_counts.size and dest_counts.max() > cap:
        status = STATUS_CAPACITY
    # the k experts of a token must be distinct: a repeated one is invalid input (the rows are
    # still assigned one per slot here, but callers must not rely on them)
    if k > 1 and np.any(np.sort(idx, axis=2)[:, :, 1:] == np.sort(idx, axis=2)[:, :, :-1]):
        status = STATUS_BADINPUT
    return {
        "expert_counts": counts.astype(np.int32),
        "src_base": src_base.astype(np.int32),
        "expert_offsets": expert_offsets.astype(np.int32),
        "dest_counts": dest_counts.astype(np.int32),
        "slot_row": slot_row.reshape(idx.shape).astype(np.int32),
        "row_src": row_src,
        "status": status,
    }


# ----------------------------------------------------------------------------- dispatch
def dispatch(x_bits: np.ndarray, idx: np.ndarray, slot_row: np.ndarray, E: int, W: int,
             cap: int, sources=None, windows: np.ndarray | None = None):
    """Copy each token row into the window row of each of its k slots.

    x_bits uint16 [n_src, T, H]. Rows at or beyond ``cap`` are not written and the
    status becomes STATUS_CAPACITY. Unwritten rows keep their previous contents
    (a sentinel pattern for a fresh window set). Returns (windows [W, cap, H], status).
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    if x_bits.ndim == 2:
        x_bits = x_bits[None]
    idx = np.asarray(idx).reshape(x_bits.shape[0], x_bits.shape[1], -1)
    slot_row = np.asarray(slot_row).reshape(idx.shape)
    n_src, T, H = x_bits.shape
    k = idx.shape[2]
    epw = E // W
    if windows is None:
        windows = np.full((W, cap, H), SENTINEL_BF16, dtype=np.uint16)
    status = STATUS_OK
    for s in (range(n_src) if sources is None else sources):
        for t in range(T):
            for j in range(k):
                d = int(idx[s, t, j]) // epw
                r = int(slot_row[s, t, j])
                if r >= cap:
                    status = STATUS_CAPACITY
                    continue
                windows[d, r] = x_bits[s, t]
    return windows, status


# ----------------------------------------------------------------------------- expert FFN
def expert_ffn(x_bits: np.ndarray, w1_bits: np.ndarray, w2_bits: np.ndarray):
    """One expert's SwiGLU FFN on its rows.

    g = X Wg^T and u = X Wu^T (Wg = W1[:I], Wu = W1[I:]), h = bf16(silu(g) * u),
    y = h W2^T. Products and sums in fp64 from the bf16 operands.
    Returns (h_bits [M, I], y64 [M, H] before rounding, y_bits [M, H]).
    """
    X = bf16_bits_to_f64(x_bits)
    W1 = bf16_bits_to_f64(w1_bits)
    W2 = bf16_bits_to_f64(w2_bits)
    I = W1.shape[0] // 2
    g = X @ W1[:I].T
    u = X @ W1[I:].T
    with np.errstate(over="ignore"):
        silu = g / (1.0 + np.exp(-g))
    h = round_bf16(silu * u)
    y64 = h @ W2.T
    return f64_to_bf16_bits(h), y64, f64_to_bf16_bits(y64)


def grouped_gemm(a_bits: np.ndarray, seg_offsets, seg_rows, b_bits: np.ndarray, swiglu: bool = False):
    """Grouped GEMM over row segments (the local-expert grouped GEMM of Sec. 4.3): rows
    [seg_offsets[s], seg_offsets[s] + seg_rows[s]) of A times segment s's own B_s^T
    (b_bits [n_seg][N][K]). Plain: C = A B_s^T. SwiGLU: B_s's rows [0, N/2) are the gate and
    [N/2, N) the up projection, C = silu(A Wg^T) * (A Wu^T). In fp64 from the bf16 operands.
    Returns (c64 [M][N or N/2] with NaN in rows outside every segment, c bits with the sentinel
    there)."""
    A = bf16_bits_to_f64(a_bits)
    M = A.shape[0]
    n_out = b_bits.shape[1] // 2 if swiglu else b_bits.shape[1]
    c64 = np.full((M, n_out), np.nan)
    for s, (o, r) in enumerate(zip(seg_offsets, seg_rows)):
        o, r = int(o), int(r)
        if r == 0:
            continue
        B = bf16_bits_to_f64(b_bits[s])
        X = A[o:o + r]
        if swiglu:
            g = X @ B[:n_out].T
            u = X @ B[n_out:].T
            with np.errstate(over="ignore"):
                c64[o:o + r] = g / (1.0 + np.exp(-g)) * u
        else:
            c64[o:o + r] = X @ B.T
    bits = np.full(c64.shape, SENTINEL_BF16, dtype=np.uint16)
    inside = ~np.isnan(c64[:, 0]) if n_out else np.zeros(M, bool)
    bits[inside] = f64_to_bf16_bits(c64[inside])
    return c64, bits


def grouped_ffn(windows: np.ndarray, layout: dict, w1_bits: np.ndarray, w2_bits: np.ndarray,
                experts, E: int, W: int, identity: bool = False):
    """Run every listed expert on its rows of its window.

    w1_bits/w2_bits are indexed by position in ``experts``. Returns, per window d,
    (y64 [dest_counts[d], H] with NaN for rows of experts not computed here,
     y_bits [dest_counts[d], H] with the sentinel for such rows).
    With ``identity`` every expert returns its input row unchanged.
    """
    epw = E // W
    H = windows.shape[2]
    total = layout["expert_counts"].sum(axis=0)
    out = {}
    for d in range(W):
        n = int(layout["dest_counts"][d])
        out[d] = (np.full((n, H), np.nan), np.full((n, H), SENTINEL_BF16, dtype=np.uint16))
    for i, e in enumerate(experts):
        d = e // epw
        r0 = int(layout["expert_offsets"][e])
        r1 = r0 + int(total[e])
        rows = windows[d, r0:r1]
        if identity:
            y_bits = rows.copy()
            y64 = bf16_bits_to_f64(rows)
        else:
            _, y64, y_bits = expert_ffn(rows, w1_bits[i], w2_bits[i])
        out[d][0][r0:r1] = y64
        out[d][1][r0:r1] = y_bits
    return out


# ----------------------------------------------------------------------------- combine
def combine_send(y_bits: np.ndarray, row_src: np.ndarray, combine: np.ndarray, k: int,
                 rows=None):
    """Store each computed window row into its source's combine buffer at slot t*k + j.

    combine: uint16 [n_src, T*k, H], updated in place and returned. ``rows`` limits
    the copy to those window rows (default: all).
    """
    src, slot = decode_row_src(row_src)
    for r in (range(len(row_src)) if rows is None else rows):
        combine[src[r], slot[r]] = y_bits[r]
    return combine


def combine_reduce(c_bits: np.ndarray, w: np.ndarray):
    """out[t] = sum_j w[t, j] * C[t*k + j], summed in ascending j.

    c_bits uint16 [T*k, H], w fp32 [T, k]. Returns (out64 [T, H], out_bits [T, H]).
    """
    w = np.asarray(w, dtype=np.float32)
    T, k = w.shape
    C = bf16_bits_to_f64(c_bits).reshape(T, k, -1)
    out = np.zeros((T, C.shape[2]), dtype=np.float64)
    for j in range(k):
        out += w[:, j].astype(np.float64)[:, None] * C[:, j, :]
    return out, f64_to_bf16_bits(out)


# ----------------------------------------------------------------------------- whole layer
def ep_layer(x_bits, logits, w1_bits, w2_bits, k, E, W, cap, experts=None, identity=False,
             renormalize=False, combine_fill=None, out_src=0):
    """Route -> layout -> dispatch -> expert FFN -> combine-send -> combine-reduce.

    x_bits [n_src, T, H], logits [n_src, T, E]. ``experts`` are computed here (default:
    all). ``combine_fill`` pre-fills source ``out_src``'s combine buffer (rows that
    other ranks would write). Returns a dict with every intermediate.
    """
    x_bits = np.asarray(x_bits)
    logits = np.asarray(logits, dtype=np.float32)
    if x_bits.ndim == 2:
        x_bits, logits = x_bits[None], logits[None]
    n_src, T, H = x_bits.shape
    experts = list(range(E)) if experts is None else list(experts)
    idx = np.empty((n_src, T, k), dtype=np.int32)
    w = np.empty((n_src, T, k), dtype=np.float32)
    for s in range(n_src):
        idx[s], w[s] = route_topk_softmax(logits[s], k, renormalize)
    lay = dispatch_layout(idx, E, W, cap)
    win, st = dispatch(x_bits, idx, lay["slot_row"], E, W, cap)
    ys = grouped_ffn(win, lay, w1_bits, w2_bits, experts, E, W, identity=identity)
    comb = np.full((n_src, T * k, H), SENTINEL_BF16, dtype=np.uint16)
    if combine_fill is not None:
        comb[out_src] = combine_fill
    epw = E // W
    for d in sorted({e // epw for e in experts}):
        total = lay["expert_counts"].sum(axis=0)
        rows = []
        for e in experts:
            if e // epw == d:
                r0 = int(lay["expert_offsets"][e])
                rows.extend(range(r0, r0 + int(total[e])))
        combine_send(ys[d][1], lay["row_src"][d], comb, k, rows=rows)
    out64, out_bits = combine_reduce(comb[out_src], w[out_src])
    return {"idx": idx, "w": w, "layout": lay, "windows": win, "status": st, "y": ys,
            "combine": comb, "out64": out64, "out_bits": out_bits}


def ep_layer_dense(x_bits, logits, w1_bits, w2_bits, k, renormalize=False):
    """Brute-force single-source layer with no permutation:
    out[t] = sum over experts e in top-k(t), in ascending slot order, of w[t, e] * bf16(FFN_e(x_t)).

    Loops over every expert and every token; for tiny shapes only.
    """
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    T, H = x_bits.shape
    E = w1_bits.shape[0]
    idx, w = route_topk_softmax(logits, k, renormalize)
    y_all = np.empty((E, T, H), dtype=np.float64)
    for e in range(E):
        _, _, yb = expert_ffn(x_bits, w1_bits[e], w2_bits[e])
        y_all[e] = bf16_bits_to_f64(yb)
    out = np.zeros((T, H), dtype=np.float64)
    for t in range(T):
        for j in range(k):
            out[t] += np.float64(w[t, j]) * y_all[idx[t, j], t]
    return out, f64_to_bf16_bits(out)
