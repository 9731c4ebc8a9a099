"""Pins of the TP / Ulysses scatter oracle: identity and permutation operands, and a
hand-written expected window table for the head-group reading."""
import numpy as np

import synth
from oracle import scatter


def _bits(v):
    return synth.to_bf16_bits(np.asarray(v, np.float32))


def test_tp_identity_b_copies_row_blocks():
    a = synth.normal_bf16(0, 5, (64, 32))
    b = _bits(np.eye(32))
    _, win = scatter.tp_row_block_scatter(a, b, 16)
    assert win.shape == (4, 16, 32)
    for d in range(4):
        assert np.array_equal(win[d], a[16 * d:16 * (d + 1)])


def test_tp_hand_worked_example():
    # A = [[1,2],[3,4],[5,6],[7,8]], B = [[1,1],[0,1]] -> C = [[1,3],[3,7],[5,11],[7,15]]
    a = _bits([[1, 2], [3, 4], [5, 6], [7, 8]])
    b = _bits([[1, 1], [0, 1]])
    c, win = scatter.tp_row_block_scatter(a, b, 2)
    assert c.tolist() == [[1, 3], [3, 7], [5, 11], [7, 15]]
    assert synth.bf16_bits_to_f32(win[0]).tolist() == [[1, 3], [3, 7]]
    assert synth.bf16_bits_to_f32(win[1]).tolist() == [[5, 11], [7, 15]]


def test_tp_permutation_b_permutes_columns():
    g = np.random.default_rng(0)
    perm = g.permutation(16)
    b = np.zeros((16, 16), np.float32)
    b[perm, np.arange(16)] = 1     # C[:, n] = A[:, perm[n]]
    a = synth.normal_bf16(0, 5, (8, 16))
    _, win = scatter.tp_row_block_scatter(a, _bits(b), 8)
    assert np.array_equal(win[0], a[:, perm])


def test_sp_head_groups_hand_written():
    # S=2, 4 heads of dim 2, groups of 2 heads -> 2 windows; X[s, c] = 100 s + c, Wqkv = I
    S, nh, hd, hpg = 2, 4, 2, 2
    N = 3 * nh * hd
    x = _bits([[100 * s + c for c in range(N)] for s in range(S)])
    _, win = scatter.sp_head_group_scatter(x, _bits(np.eye(N)), nh, hd, hpg)
    v = synth.bf16_bits_to_f32(win)
    assert v.shape == (2, 3, 2, 2, 2)
    # window 0 holds heads 0,1; window 1 heads 2,3; columns: Q 0-7, K 8-15, V 16-23
    assert v[0, 0, 0].tolist() == [[0, 1], [100, 101]]      # Q head 0
    assert v[0, 0, 1].tolist() == [[2, 3], [102, 103]]      # Q head 1
    assert v[1, 0, 0].tolist() == [[4, 5], [104, 105]]      # Q head 2
    assert v[1, 0, 1].tolist() == [[6, 7], [106, 107]]      # Q head 3
    assert v[0, 1, 0].tolist() == [[8, 9], [108, 109]]      # K head 0
    assert v[1, 1, 1].tolist() == [[14, 15], [114, 115]]    # K head 3
    assert v[0, 2, 1].tolist() == [[18, 19], [118, 119]]    # V head 1
    assert v[1, 2, 1].tolist() == [[22, 23], [122, 123]]    # V head 3


def test_sp_unscatter_roundtrip():
    cfg = synth.SPConfig("t", S=8, Dm=16, n_heads=4, head_dim=4, heads_per_group=2)
    inp = synth.sp_inputs(cfg, 0)
    qkv, win = scatter.sp_head_group_scatter(inp["x"], inp["w"], cfg.n_heads, cfg.head_dim, cfg.heads_per_group)
    back = np.empty((cfg.S, 3 * cfg.Dm), np.uint16)
    for c in range(3 * cfg.Dm):
        g, which, lh, dd = scatter.sp_window_index(c, cfg.n_heads, cfg.head_dim, cfg.heads_per_group)
        back[:, c] = win[g, which, lh, :, dd]
    from oracle.ep import f64_to_bf16_bits
    assert np.array_equal(back, f64_to_bf16_bits(qkv))
