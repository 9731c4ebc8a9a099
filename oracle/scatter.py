"""Oracle for the GEMM scatter epilogues (test infrastructure only).

Tensor parallelism (Sec. 4.5): in a row-parallel linear layer each rank computes a
partial output Y_r = X_r W_r; the fused kernel pushes ready output chunks to their
destinations while the GEMM continues. On one GPU the "push" is a store of output
row block d into window d.

Ulysses sequence parallelism (Sec. 5.4, "GEMM-All-to-All fusion"): the projection
GEMM before attention is fused with the All-to-All that moves its output from the
sequence partition to head partitions, which also removes the separate
permutation before the exchange. On one GPU the exchange is a store of each head
group into its window.

Both are plain definitions: C = A B in fp64 from bf16 operands, then a pure
re-indexing of C, stored in bf16. Readings: B is given logically [K, N]; QKV
columns are ordered Q heads 0..n_heads-1, then K heads, then V heads, head_dim
each; window g holds heads [g*hpg, (g+1)*hpg) as [3][hpg][S][head_dim].
"""
from __future__ import annotations

import numpy as np

from .ep import bf16_bits_to_f64, f64_to_bf16_bits

__all__ = ["gemm", "tp_row_block_scatter", "sp_head_group_scatter", "sp_window_index"]


def gemm(a_bits: np.ndarray, b_bits: np.ndarray) -> np.ndarray:
    """C = A B in fp64; A [M, K], B [K, N] as bf16 bits."""
    return bf16_bits_to_f64(a_bits) @ bf16_bits_to_f64(b_bits)


def tp_row_block_scatter(a_bits, b_bits, rows_per_dest: int):
    """Rows [d*rpd, (d+1)*rpd) of C = A B go to window d.

    Returns (c64 [M, N], windows_bits [M // rpd, rpd, N]).
    """
    c = gemm(a_bits, b_bits)
    M, N = c.shape
    if M % rows_per_dest:
        raise ValueError("M must be a multiple of rows_per_dest")
    W = M // rows_per_dest
    win = np.empty((W, rows_per_dest, N), dtype=np.uint16)
    for d in range(W):
        win[d] = f64_to_bf16_bits(c[d * rows_per_dest:(d + 1) * rows_per_dest])
    return c, win


def sp_window_index(col: int, n_heads: int, head_dim: int, heads_per_group: int):
    """Output column -> (window g, projection q/k/v, head within group, dim)."""
    which, rem = divmod(col, n_heads * head_dim)
    head, dd = divmod(rem, head_dim)
    g, lh = divmod(head, heads_per_group)
    return g, which, lh, dd


def sp_head_group_scatter(x_bits, w_bits, n_heads: int, head_dim: int, heads_per_group: int):
    """QKV = X Wqkv; window g[which][lh][s][dd] = QKV[s, which*n_heads*head_dim + (g*hpg+lh)*head_dim + dd].

    Returns (qkv64 [S, 3*n_heads*head_dim], windows_bits [G, 3, hpg, S, head_dim]).
    """
    qkv = gemm(x_bits, w_bits)
    S, N = qkv.shape
    if N != 3 * n_heads * head_dim or n_heads % heads_per_group:
        raise ValueError("bad QKV shape")
    G = n_heads // heads_per_group
    win = np.empty((G, 3, heads_per_group, S, head_dim), dtype=np.uint16)
    bits = f64_to_bf16_bits(qkv)
    for which in range(3):
        for head in range(n_heads):
            g, lh = divmod(head, heads_per_group)
            c0 = which * n_heads * head_dim + head * head_dim
            win[g, which, lh] = bits[:, c0:c0 + head_dim]
    return qkv, win
