"""Oracle for attention with the post-attention Ulysses All-to-All (test infrastructure only).

Ulysses parallelism (Sec. 4.4 and App. B; measured in Sec. 5.4, Table 4): before attention
each rank holds all tokens of its own heads; after
attention the All-to-All returns every token's output to the rank that owns that token's
sequence chunk. The fused kernel of the paper attaches these stores to the output boundary
of a FlashAttention kernel. What is computed is a plain definition:

  O[h, t, :] = sum_u softmax_u(scale * Q[h, t, :] . K[h, u, :]) V[h, u, :]

(full, non-causal attention; scale = 1 / sqrt(head_dim) unless given), stored in bf16, then a
pure re-indexing of O into destination windows. Arithmetic is fp64 from the bf16 operands.
Readings: Q, K, V are [heads][M][head_dim] (head-major, one rank's heads after the
pre-attention exchange); the sequence is split into W equal chunks and window g receives
tokens [g M / W, (g + 1) M / W) of every local head as [M / W][heads][head_dim] (token-major,
so a destination rank sees its tokens with this rank's heads side by side).
"""
from __future__ import annotations

import math

import numpy as np

from .ep import bf16_bits_to_f64, f64_to_bf16_bits

__all__ = ["attention", "ulysses_scatter", "ulysses_window_index", "attention_reference_loops"]


def attention(q_bits, k_bits, v_bits, scale: float | None = None):
    """Softmax attention per head in fp64. Inputs bf16 bits [h][M][d] (K, V may have another
    length Mk). Returns (o64 [h][M][d], o_bits)."""
    q = bf16_bits_to_f64(np.asarray(q_bits))
    k = bf16_bits_to_f64(np.asarray(k_bits))
    v = bf16_bits_to_f64(np.asarray(v_bits))
    d = q.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.empty(q.shape, dtype=np.float64)
    for h in range(q.shape[0]):
        s = (q[h] @ k[h].T) * scale                 # [M, Mk]
        s -= s.max(axis=1, keepdims=True)           # row shift: leaves the softmax unchanged
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)           # normalise over the keys of each query
        out[h] = p @ v[h]
    return out, f64_to_bf16_bits(out)


def attention_reference_loops(q, k, v, scale):
    """The same definition with explicit loops over float lists (tiny inputs only): the
    brute-force cross-check of ``attention``."""
    H, M, D = len(q), len(q[0]), len(q[0][0])
    Mk = len(k[0])
    out = [[[0.0] * D for _ in range(M)] for _ in range(H)]
    for h in range(H):
        for t in range(M):
            logits = [scale * sum(q[h][t][i] * k[h][u][i] for i in range(D)) for u in range(Mk)]
            mx = max(logits)
            w = [math.exp(x - mx) for x in logits]
            z = sum(w)
            for i in range(D):
                out[h][t][i] = sum(w[u] * v[h][u][i] for u in range(Mk)) / z
    return out


def ulysses_window_index(h: int, t: int, M: int, W: int):
    """Destination of output row (head h, token t): (window g, row in the window, head slot)."""
    chunk = M // W
    return t // chunk, t % chunk, h


def ulysses_scatter(o, W: int):
    """Post-attention exchange: o [h][M][d] -> windows [W][M / W][h][d]."""
    o = np.asarray(o)
    H, M, D = o.shape
    if M % W:
        raise ValueError("sequence length must split evenly over the windows")
    return np.ascontiguousarray(o.reshape(H, W, M // W, D).transpose(1, 2, 0, 3))
