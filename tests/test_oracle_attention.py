"""Pins of the attention / Ulysses oracle against brute force, closed forms and invariants."""
import math

import numpy as np

import synth
from oracle import attention as oa
from oracle.ep import bf16_bits_to_f64


def _bits(a):
    return synth.to_bf16_bits(np.asarray(a, dtype=np.float32))


def test_matches_explicit_loops_on_tiny_inputs():
    g = np.random.default_rng(3)
    q, k, v = (_bits(g.standard_normal((2, n, 3))) for n in (5, 7, 7))
    o64, _ = oa.attention(q, k, v, scale=0.7)
    ref = oa.attention_reference_loops(bf16_bits_to_f64(q).tolist(), bf16_bits_to_f64(k).tolist(),
                                       bf16_bits_to_f64(v).tolist(), 0.7)
    assert np.allclose(o64, np.array(ref), rtol=0, atol=1e-12)


def test_zero_queries_average_the_values():
    # equal scores: every key gets weight 1 / Mk, so each output row is the mean of V
    g = np.random.default_rng(4)
    q = _bits(np.zeros((3, 6, 8)))
    k, v = _bits(g.standard_normal((3, 9, 8))), _bits(g.standard_normal((3, 9, 8)))
    o64, _ = oa.attention(q, k, v)
    mean = bf16_bits_to_f64(v).mean(axis=1, keepdims=True)
    assert np.allclose(o64, np.broadcast_to(mean, o64.shape), rtol=0, atol=1e-14)


def test_softmax_is_over_keys_per_query():
    # shifting every key by the same vector adds a per-query constant to the scores: the
    # output must not change (a softmax taken over queries instead of keys would)
    g = np.random.default_rng(5)
    q = g.standard_normal((1, 6, 4))
    k = g.standard_normal((1, 5, 4))
    v = g.standard_normal((1, 5, 4))
    c = np.array([0.5, -1.0, 0.25, 2.0])
    a, _ = oa.attention(_bits(q), _bits(k), _bits(v))
    b, _ = oa.attention(_bits(q), _bits(k + c), _bits(v))
    ks = bf16_bits_to_f64(_bits(k + c)) - bf16_bits_to_f64(_bits(k))
    if np.allclose(ks, c):          # the shift survived bf16 rounding exactly
        assert np.allclose(a, b, rtol=0, atol=1e-12)
    # and the same output through explicit weights
    qd, kd, vd = (bf16_bits_to_f64(_bits(x))[0] for x in (q, k, v))
    s = qd @ kd.T / math.sqrt(4)
    w = np.exp(s - s.max(axis=1, keepdims=True))
    w /= w.sum(axis=1, keepdims=True)
    assert np.allclose(w.sum(axis=1), 1.0)
    assert np.allclose(a[0], w @ vd, atol=1e-12)


def test_a_dominant_key_selects_its_value_row():
    d = 16
    q = np.zeros((1, 3, d))
    k = np.zeros((1, 4, d))
    v = np.arange(4 * d, dtype=np.float64).reshape(1, 4, d) / 64.0
    q[0, :, 0] = 8.0
    k[0, 2, 0] = 8.0            # score 64 / sqrt(16) = 16 for key 2, 0 for the others
    o64, _ = oa.attention(_bits(q), _bits(k), _bits(v))
    expect = bf16_bits_to_f64(_bits(v))[0, 2]
    w_other = math.exp(-16.0) / (1 + 3 * math.exp(-16.0))
    assert np.allclose(o64[0], expect, atol=4 * w_other * np.abs(v).max())


def test_scale_defaults_to_inverse_sqrt_head_dim():
    g = np.random.default_rng(6)
    q, k, v = (_bits(g.standard_normal((1, 4, 32))) for _ in range(3))
    a, _ = oa.attention(q, k, v)
    b, _ = oa.attention(q, k, v, scale=1.0 / math.sqrt(32))
    assert np.array_equal(a, b)


def test_ulysses_windows_by_hand():
    H, M, D, W = 2, 8, 3, 4
    o = np.arange(H * M * D, dtype=np.float64).reshape(H, M, D)
    win = oa.ulysses_scatter(o, W)
    assert win.shape == (W, M // W, H, D)
    # token 5 of head 1: chunk 2 (tokens 4..5), row 1, head slot 1
    assert oa.ulysses_window_index(1, 5, M, W) == (2, 1, 1)
    assert np.array_equal(win[2, 1, 1], o[1, 5])
    assert np.array_equal(win[0, 0, 0], o[0, 0])
    assert np.array_equal(win[3, 1, 0], o[0, 7])
    # every output row lands exactly once
    seen = np.zeros((H, M), dtype=int)
    for h in range(H):
        for t in range(M):
            g_, r, s = oa.ulysses_window_index(h, t, M, W)
            assert np.array_equal(win[g_, r, s], o[h, t])
            seen[h, t] += 1
    assert (seen == 1).all()


def test_synth_attention_inputs_shapes():
    cfg = synth.AttnConfig("t", M=64, heads=2, head_dim=16, W=4)
    inp = synth.attn_inputs(cfg, 0)
    assert all(inp[n].shape == (2, 64, 16) for n in ("q", "k", "v"))
    assert inp["q"].dtype == np.uint16
