"""Pins of the EP oracle against things other than itself: brute force with a
different algorithm, crafted ties, closed forms, invariants, library routines and
exact integer arithmetic."""
import numpy as np
import pytest
import scipy.special

import synth
from oracle import ep


# ----------------------------------------------------------------------------- bf16
def test_round_bf16_matches_integer_bit_trick():
    # two independent implementations: frexp/rint on fp64 vs the integer carry trick on fp32
    g = np.random.default_rng(1)
    v = np.concatenate([g.standard_normal(200000).astype(np.float32),
                        (g.standard_normal(1000) * 1e-38).astype(np.float32),
                        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0, -0.0], np.float32)])
    a = ep.f64_to_bf16_bits(v.astype(np.float64))
    b = synth.to_bf16_bits(v)
    assert np.array_equal(a, b)


def test_round_bf16_ties_and_no_double_rounding():
    assert ep.round_bf16(np.array([1 + 2 ** -8]))[0] == 1.0            # tie -> even
    assert ep.round_bf16(np.array([1 + 3 * 2 ** -8]))[0] == 1 + 2 ** -6  # tie -> even (up)
    # an fp64 value just above a bf16 tie rounds up; going through fp32 first would not
    v = 1 + 2 ** -8 + 2 ** -40
    assert ep.round_bf16(np.array([v]))[0] == 1 + 2 ** -7
    assert synth.bf16_bits_to_f32(synth.to_bf16_bits(np.float32(v)))[()] == 1.0


# ----------------------------------------------------------------------------- route
def _route_by_selection(logits, k):
    """Repeated arg-max with masking, scanning experts in ascending order."""
    T, E = logits.shape
    idx = np.zeros((T, k), np.int32)
    for t in range(T):
        taken = set()
        for j in range(k):
            best = None
            for e in range(E):
                if e in taken:
                    continue
                if best is None or logits[t, e] > logits[t, best]:
                    best = e
            taken.add(best)
            idx[t, j] = best
    return idx


def test_route_matches_selection_brute_force():
    g = np.random.default_rng(2)
    for E, k in [(8, 2), (16, 5), (32, 8)]:
        lg = g.standard_normal((40, E)).astype(np.float32)
        lg[::7, 3] = lg[::7, 1]                 # sprinkle ties
        lg = np.round(lg * 4) / 4               # many more ties
        idx, _ = ep.route_topk_softmax(lg, k)
        assert np.array_equal(idx, _route_by_selection(lg, k))


def test_route_all_equal_row_and_weights():
    lg = np.zeros((3, 8), np.float32)
    idx, w = ep.route_topk_softmax(lg, 3)
    assert np.array_equal(idx, np.tile(np.arange(3), (3, 1)))
    assert np.allclose(w, 1 / 8, rtol=0, atol=1e-8)


def test_route_worked_example_closed_form():
    lg = np.log(np.array([[1.0, 2.0, 3.0, 4.0]], np.float32))
    idx, w = ep.route_topk_softmax(lg, 2)
    assert idx.tolist() == [[3, 2]]
    assert np.allclose(w, [[0.4, 0.3]], rtol=1e-6)
    _, wr = ep.route_topk_softmax(lg, 2, renormalize=True)
    assert np.allclose(wr, [[4 / 7, 3 / 7]], rtol=1e-6)


def test_route_softmax_matches_scipy_and_invariants():
    g = np.random.default_rng(3)
    lg = g.standard_normal((64, 256)).astype(np.float32)
    idx, w = ep.route_topk_softmax(lg, 8)
    p = scipy.special.softmax(lg.astype(np.float64), axis=1)
    assert np.allclose(w, np.take_along_axis(p, idx.astype(np.int64), 1), rtol=1e-6, atol=0)
    assert all(len(set(r)) == 8 for r in idx.tolist())
    assert np.all(np.diff(w, axis=1) <= 0)
    assert np.all(w.sum(1) <= 1 + 1e-6)
    _, wr = ep.route_topk_softmax(lg, 8, renormalize=True)
    assert np.allclose(wr.sum(1), 1, atol=1e-6)


# ----------------------------------------------------------------------------- layout
def _layout_brute(idx, E, W):
    """Nested loops appending slots window by window, expert by expert, source by source."""
    n_src, T, k = idx.shape
    epw = E // W
    slot_row = np.full(idx.shape, -1)
    rows = []
    for d in range(W):
        r = []
        for e in range(d * epw, (d + 1) * epw):
            for s in range(n_src):
                for t in range(T):
                    for j in range(k):
                        if idx[s, t, j] == e:
                            slot_row[s, t, j] = len(r)
                            r.append((s, t * k + j))
        rows.append(r)
    return slot_row, rows


@pytest.mark.parametrize("n_src,T,k,E,W", [(1, 8, 2, 8, 4), (3, 6, 3, 12, 3), (2, 5, 4, 8, 8), (1, 1, 1, 4, 1)])
def test_layout_matches_brute_force(n_src, T, k, E, W):
    g = np.random.default_rng(4 + T)
    idx = np.stack([[g.permutation(E)[:k] for _ in range(T)] for _ in range(n_src)])
    lay = ep.dispatch_layout(idx, E, W)
    sr, rows = _layout_brute(idx, E, W)
    assert np.array_equal(lay["slot_row"], sr)
    for d in range(W):
        src, slot = ep.decode_row_src(lay["row_src"][d])
        assert list(zip(src.tolist(), slot.tolist())) == rows[d]


def test_layout_invariants_multi_source():
    g = np.random.default_rng(5)
    n_src, T, k, E, W = 4, 300, 8, 64, 8
    idx = np.stack([[g.permutation(E)[:k] for _ in range(T)] for _ in range(n_src)])
    lay = ep.dispatch_layout(idx, E, W)
    c = lay["expert_counts"]
    assert np.all(c.sum(1) == T * k)
    tot = c.sum(0)
    epw = E // W
    assert np.array_equal(lay["dest_counts"], tot.reshape(W, epw).sum(1))
    for d in range(W):
        blk = tot[d * epw:(d + 1) * epw]
        assert lay["expert_offsets"][d * epw] == 0
        assert np.array_equal(np.diff(lay["expert_offsets"][d * epw:(d + 1) * epw]), blk[:-1])
    assert np.array_equal(lay["src_base"][0], np.zeros(E))
    assert np.array_equal(lay["src_base"][1:], np.cumsum(c, 0)[:-1])
    # slot_row is a bijection onto [0, dest_counts[d]) for each window
    for d in range(W):
        m = (idx // epw) == d
        r = np.sort(lay["slot_row"][m])
        assert np.array_equal(r, np.arange(lay["dest_counts"][d]))


def test_route_masked_experts_rank_last_in_index_order():
    # -inf logits (masked experts) come after every finite one, ties to the lower index,
    # with zero weight; checked against the selection brute force
    lg = np.full((4, 10), -np.inf, np.float32)
    lg[0, [2, 7]] = [0.5, 1.5]
    lg[1, :] = 0.0
    lg[1, 3:6] = -np.inf
    lg[2, 9] = 2.0
    lg[3, [0, 4, 8]] = [1.0, 1.0, 3.0]
    idx, w = ep.route_topk_softmax(lg, 5)
    assert np.array_equal(idx, _route_by_selection(lg, 5))
    assert idx[0].tolist() == [7, 2, 0, 1, 3] and idx[2].tolist() == [9, 0, 1, 2, 3]
    assert np.all(w[np.isneginf(np.take_along_axis(lg, idx.astype(np.int64), 1))] == 0)


def test_layout_repeated_expert_is_bad_input():
    idx = np.array([[[0, 1], [2, 2], [1, 3]]])
    assert ep.dispatch_layout(idx, 4, 2)["status"] == ep.STATUS_BADINPUT
    assert ep.dispatch_layout(idx[:, [0, 2]], 4, 2)["status"] == ep.STATUS_OK


def test_layout_capacity_status():
    idx = np.array([[[0, 1], [0, 1], [0, 1]]])
    assert ep.dispatch_layout(idx, 4, 2, cap=3)["status"] == ep.STATUS_CAPACITY
    assert ep.dispatch_layout(idx, 4, 2, cap=6)["status"] == ep.STATUS_OK


# ----------------------------------------------------------------------------- dispatch
def test_dispatch_every_slot_lands_once_and_bitexact():
    g = np.random.default_rng(6)
    n_src, T, H, k, E, W = 2, 20, 16, 3, 8, 4
    idx = np.stack([[g.permutation(E)[:k] for _ in range(T)] for _ in range(n_src)])
    x = synth.normal_bf16(0, 1, (n_src, T, H))
    lay = ep.dispatch_layout(idx, E, W)
    cap = int(lay["dest_counts"].max()) + 2
    win, st = ep.dispatch(x, idx, lay["slot_row"], E, W, cap)
    assert st == ep.STATUS_OK
    for d in range(W):
        n = lay["dest_counts"][d]
        src, slot = ep.decode_row_src(lay["row_src"][d])
        assert np.array_equal(win[d, :n], x[src, slot // k])
        assert np.all(win[d, n:] == ep.SENTINEL_BF16)


def test_dispatch_capacity_overflow_leaves_rows_unwritten():
    idx = np.array([[[0], [0], [0], [1]]])
    x = synth.normal_bf16(0, 1, (1, 4, 8))
    lay = ep.dispatch_layout(idx, 2, 1, cap=2)
    win, st = ep.dispatch(x, idx, lay["slot_row"], 2, 1, cap=2)
    assert st == ep.STATUS_CAPACITY and lay["status"] == ep.STATUS_CAPACITY
    assert np.array_equal(win[0, 0], x[0, 0]) and np.array_equal(win[0, 1], x[0, 1])


# ----------------------------------------------------------------------------- expert FFN
def test_ffn_one_hot_selects_gate_up_and_down():
    g = np.random.default_rng(7)
    M, H, I = 5, 8, 4
    xv = g.integers(-3, 4, size=(M, H)).astype(np.float32) / 2
    x = synth.to_bf16_bits(xv)
    a_col = [1, 4, 6, 0]   # gate row i reads feature a_col[i]
    b_col = [2, 2, 7, 5]   # up row i reads feature b_col[i]
    w1 = np.zeros((2 * I, H), np.float32)
    for i in range(I):
        w1[i, a_col[i]] = 1
        w1[I + i, b_col[i]] = 1
    w2 = np.zeros((H, I), np.float32)
    pick = [3, 0, 1, 2, 2, 0, 3, 1]  # output o reads h column pick[o]
    for o in range(H):
        w2[o, pick[o]] = 1
    h, y64, y = ep.expert_ffn(x, synth.to_bf16_bits(w1), synth.to_bf16_bits(w2))
    gate = xv[:, a_col].astype(np.float64)
    up = xv[:, b_col].astype(np.float64)
    href = gate * scipy.special.expit(gate) * up
    href_bits = synth.to_bf16_bits(href.astype(np.float32))  # values far from ties here
    assert np.array_equal(h, href_bits)
    hv = synth.bf16_bits_to_f32(h).astype(np.float64)
    assert np.array_equal(y64, hv[:, pick])
    assert np.array_equal(y, h[:, pick])


def test_ffn_silu_closed_form():
    # g = ln 3 -> sigmoid = 3/4; u = 2 -> h = 1.5 ln 3
    x = synth.to_bf16_bits(np.array([[1.0, 2.0]], np.float32))
    w1 = np.array([[np.log(3.0), 0.0], [0.0, 1.0]], np.float32)  # gate = ln3 * x0, up = x1
    w1b = synth.to_bf16_bits(w1)
    g = synth.bf16_bits_to_f32(w1b)[0, 0].astype(np.float64)
    h, _, _ = ep.expert_ffn(x, w1b, synth.to_bf16_bits(np.ones((2, 1), np.float32)))
    hv = synth.bf16_bits_to_f32(h)[0, 0]
    assert abs(hv - 2 * g / (1 + np.exp(-g))) <= 2 ** -7 * abs(hv)
    assert abs(hv - 1.5 * np.log(3)) < 0.02


def test_ffn_integer_operands_exact():
    # integer x and W1 make g, u exact integers; fp64 sums of products of bf16 values are exact
    g = np.random.default_rng(8)
    M, H, I = 6, 32, 16
    x = synth.int_valued_bf16(0, 1, (M, H))
    w1 = synth.int_valued_bf16(0, 2, (2 * I, H))
    w2 = synth.int_valued_bf16(0, 3, (H, I))
    h, y64, _ = ep.expert_ffn(x, w1, w2)
    X = synth.bf16_bits_to_f32(x).astype(np.int64)
    W1 = synth.bf16_bits_to_f32(w1).astype(np.int64)
    gi = X @ W1[:I].T
    ui = X @ W1[I:].T
    hv = synth.bf16_bits_to_f32(h).astype(np.float64)
    ref = gi * scipy.special.expit(gi.astype(np.float64)) * ui
    assert np.all(np.abs(hv - ref) <= 2 ** -8 * np.abs(ref) + 1e-300)
    # y = h W2^T with exact integer W2: exact in fp64 (small magnitudes)
    W2 = synth.bf16_bits_to_f32(w2).astype(np.float64)
    assert np.array_equal(y64, hv @ W2.T)


# ----------------------------------------------------------------------------- combine
def test_combine_reduce_one_hot_and_identity():
    g = np.random.default_rng(9)
    T, k, H = 7, 3, 16
    c = synth.normal_bf16(0, 4, (T * k, H))
    w = np.zeros((T, k), np.float32)
    w[np.arange(T), g.integers(0, k, T)] = 1.0
    _, out = ep.combine_reduce(c, w)
    sel = c.reshape(T, k, H)[np.arange(T), w.argmax(1)]
    assert np.array_equal(out, sel)


def test_identity_experts_scale_input_by_summed_gates():
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0, with_weights=False)
    res = ep.ep_layer(inp["x"], inp["logits"], None, None, cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k,
                      identity=True)
    x = synth.bf16_bits_to_f32(inp["x"][0]).astype(np.float64)
    wsum = res["w"][0].astype(np.float64).sum(1, keepdims=True)
    ref = x * wsum
    assert np.allclose(res["out64"], ref, rtol=1e-15, atol=1e-300)
    got = synth.bf16_bits_to_f32(res["out_bits"]).astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2 ** -8 * np.abs(ref))   # within one bf16 rounding


def test_permuted_layer_equals_dense_brute_force():
    # c1-shaped layer at reduced size: permutation path vs the no-permutation dense path
    cfg = synth.EPConfig("t", T=48, H=64, E=8, k=2, I=32, W=4, n_src=1, compute_all=True)
    inp = synth.ep_inputs(cfg, 3)
    res = ep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W,
                      cap=cfg.T * cfg.k)
    dense64, dense_bits = ep.ep_layer_dense(inp["x"][0], inp["logits"][0], inp["w1"], inp["w2"], cfg.k)
    assert np.allclose(res["out64"], dense64, rtol=1e-13, atol=1e-15)
    assert np.mean(res["out_bits"] == dense_bits) > 0.999


def test_multi_source_layer_combine_targets():
    # every computed row lands in the combine buffer of its own source at slot t*k+j
    cfg = synth.EPConfig("t", T=16, H=32, E=8, k=2, I=16, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 1)
    experts = synth.computed_experts(cfg)
    res = ep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W,
                      cap=cfg.n_src * cfg.T * cfg.k, experts=experts, identity=True)
    comb = res["combine"]
    for s in range(cfg.n_src):
        for t in range(cfg.T):
            for j in range(cfg.k):
                e = res["idx"][s, t, j]
                row = comb[s, t * cfg.k + j]
                if e in experts:
                    assert np.array_equal(row, inp["x"][s, t])
                else:
                    assert np.all(row == ep.SENTINEL_BF16)


def test_grouped_gemm_integer_exact_and_swiglu_matches_expert_ffn():
    g = np.random.default_rng(12)
    M, K, N = 40, 64, 32
    a = synth.int_valued_bf16(0, 7, (M, K))
    b = synth.int_valued_bf16(0, 8, (3, N, K))
    offs, rows = [0, 10, 30], [7, 0, 10]
    c64, bits = ep.grouped_gemm(a, offs, rows, b)
    A, B = ep.bf16_bits_to_f64(a), ep.bf16_bits_to_f64(b)
    for s, (o, r) in enumerate(zip(offs, rows)):
        for i in range(o, o + r):                 # explicit dot products of integers: exact
            for n in range(N):
                assert c64[i, n] == sum(A[i, kk] * B[s, n, kk] for kk in range(K))
    outside = np.ones(M, bool)
    outside[0:7] = outside[30:40] = False
    assert np.isnan(c64[outside]).all() and (bits[outside] == ep.SENTINEL_BF16).all()
    # the SwiGLU epilogue is the expert FFN's Linear-1 + activation, h before rounding
    x = synth.normal_bf16(0, 9, (12, 64))
    w1 = synth.normal_bf16(0, 10, (2, 2 * 16, 64), std=0.1)
    c64, bits = ep.grouped_gemm(x, [0, 5], [5, 7], w1, swiglu=True)
    for s, (o, r) in enumerate([(0, 5), (5, 7)]):
        h_bits, _, _ = ep.expert_ffn(x[o:o + r], w1[s], np.zeros((64, 16), np.uint16))
        assert np.array_equal(bits[o:o + r], h_bits)
