"""Oracle for the quantized EP layer, W8A8 (MXFP8) and W4A8 (test infrastructure only).

The paper runs its EP kernel at W8A8 as well as W4A8 (Sec. 5.2); the path is the same
route -> dispatch -> grouped SwiGLU FFN -> combine, with narrower operands. Readings:
  * token rows are quantized once, at dispatch, to MXFP8 along H (E4M3 codes, one E8M0
    scale per 32 elements; oracle/mx.py); a dispatch window row holds the H codes followed by
    the H / 32 scales;
  * W1 [2I][H] and W2 [H][I] are quantized along their reduction axis (H for W1, I for W2)
    with one E8M0 scale per 32 elements, to E4M3 (W8A8) or to E2M1 (W4A8: MXFP4 weights,
    8-bit activations); codes are kept one per element here (the GPU packs E2M1 two per
    byte, low nibble first);
  * Linear-1 in fp64 from the dequantized operands, SwiGLU in fp64, and the activation h is
    quantized to MXFP8 along I straight from that value (the quantized path stores h as MXFP8
    where the bf16 path stores bf16);
  * Linear-2 in fp64 from dequantized h and W2; the expert output y is rounded to bf16, and
    combine-send / combine-reduce are those of the bf16 layer (oracle/ep.py).
"""
from __future__ import annotations

import numpy as np

from . import ep, mx

__all__ = ["quantize_rows", "expert_ffn_mx", "ep_layer_mx", "ep_layer_mx_dense"]


def quantize_rows(bits, fmt=mx.E4M3):
    """bf16 bits [..., K] -> (codes [..., K] of format fmt, scales [..., K / 32])."""
    return mx.quantize_mx(ep.bf16_bits_to_f64(np.asarray(bits)), fmt)


def expert_ffn_mx(xq, w1q, w2q, wfmt=mx.E4M3):
    """One expert's SwiGLU FFN on MXFP8 rows. xq = (codes, scales) of [M][H]; w1q of
    [2I][H] and w2q of [H][I] in format wfmt. Returns (h codes, h scales, y64 [M][H],
    y bits)."""
    X = mx.dequantize_mx(*xq, mx.E4M3)
    W1 = mx.dequantize_mx(*w1q, wfmt)
    W2 = mx.dequantize_mx(*w2q, wfmt)
    I = W1.shape[0] // 2
    g = X @ W1[:I].T
    u = X @ W1[I:].T
    with np.errstate(over="ignore"):
        silu = g / (1.0 + np.exp(-g))
    hc, hs = mx.quantize_mx(silu * u, mx.E4M3)
    y64 = mx.dequantize_mx(hc, hs, mx.E4M3) @ W2.T
    return hc, hs, y64, ep.f64_to_bf16_bits(y64)


def ep_layer_mx(x_bits, logits, w1_bits, w2_bits, k, E, W, cap, experts=None, renormalize=False,
                combine_fill=None, out_src=0, wfmt=mx.E4M3):
    """The layer of oracle/ep.ep_layer with MXFP8 rows and activations and weights in format
    wfmt (E4M3: W8A8, E2M1: W4A8).

    x_bits [n_src][T][H], logits [n_src][T][E], w1_bits [n_exp][2I][H], w2_bits [n_exp][H][I]
    (indexed by position in ``experts``). Returns every intermediate, including the dispatch
    windows' codes [W][cap][H] and scales [W][cap][H / 32] (unwritten rows 0)."""
    x_bits = np.asarray(x_bits)
    logits = np.asarray(logits, dtype=np.float32)
    if x_bits.ndim == 2:
        x_bits, logits = x_bits[None], logits[None]
    n_src, T, H = x_bits.shape
    experts = list(range(E)) if experts is None else list(experts)
    idx = np.empty((n_src, T, k), dtype=np.int32)
    w = np.empty((n_src, T, k), dtype=np.float32)
    for s in range(n_src):
        idx[s], w[s] = ep.route_topk_softmax(logits[s], k, renormalize)
    lay = ep.dispatch_layout(idx, E, W, cap)
    xc, xs = quantize_rows(x_bits)
    win_c = np.zeros((W, cap, H), dtype=np.uint8)
    win_s = np.zeros((W, cap, H // 32), dtype=np.uint8)
    epw = E // W
    status = ep.STATUS_OK
    for s in range(n_src):
        for t in range(T):
            for j in range(k):
                d, r = int(idx[s, t, j]) // epw, int(lay["slot_row"][s, t, j])
                if r >= cap:
                    status = ep.STATUS_CAPACITY
                    continue
                win_c[d, r], win_s[d, r] = xc[s, t], xs[s, t]
    total = lay["expert_counts"].sum(axis=0)
    comb = np.full((n_src, T * k, H), ep.SENTINEL_BF16, dtype=np.uint16)
    if combine_fill is not None:
        comb[out_src] = combine_fill
    h = {}
    for i, e in enumerate(experts):
        d, r0 = e // epw, int(lay["expert_offsets"][e])
        r1 = r0 + int(total[e])
        if r1 == r0:
            continue
        w1q = quantize_rows(w1_bits[i], wfmt)
        w2q = quantize_rows(w2_bits[i], wfmt)
        hc, hs, _, yb = expert_ffn_mx((win_c[d, r0:r1], win_s[d, r0:r1]), w1q, w2q, wfmt)
        h[e] = (hc, hs)
        ep.combine_send(np.concatenate([np.zeros((r0, H), np.uint16), yb]), lay["row_src"][d], comb, k,
                        rows=range(r0, r1))
    out64, out_bits = ep.combine_reduce(comb[out_src], w[out_src])
    return {"idx": idx, "w": w, "layout": lay, "win_codes": win_c, "win_scales": win_s, "status": status,
            "h": h, "combine": comb, "out64": out64, "out_bits": out_bits}


def ep_layer_mx_dense(x_bits, logits, w1_bits, w2_bits, k, renormalize=False, wfmt=mx.E4M3):
    """Brute force for one source with no layout or windows: each token's row is quantized,
    run through each of its top-k experts on its own, and the bf16 outputs are summed with
    the routing weights in ascending slot order. Tiny shapes only."""
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    T, H = x_bits.shape
    idx, w = ep.route_topk_softmax(logits, k, renormalize)
    out = np.zeros((T, H), dtype=np.float64)
    for t in range(T):
        xq = quantize_rows(x_bits[t:t + 1])
        for j in range(k):
            e = int(idx[t, j])
            _, _, _, yb = expert_ffn_mx(xq, quantize_rows(w1_bits[e], wfmt), quantize_rows(w2_bits[e], wfmt), wfmt)
            out[t] += np.float64(w[t, j]) * ep.bf16_bits_to_f64(yb[0])
    return out, ep.f64_to_bf16_bits(out)
