"""Pins of the quantized (W8A8 MXFP8 and W4A8) EP layer oracle: its layout / dispatch / combine
plumbing against a dense per-token brute force (bit-exact on operands the formats hold
exactly), the dispatch windows' contents, and its distance from the bf16 layer (the size of
the quantization error)."""
import numpy as np
import pytest

import synth
from oracle import ep, ep_mx, mx


def _int_bits(g, shape):
    return synth.to_bf16_bits(g.integers(-8, 9, shape).astype(np.float32))


def _e2m1_int_bits(g, shape):
    # integers that E2M1 holds under any block scale: amax 6 or 4 takes scale 1, amax 3 or 2
    # scale 1/2, amax 1 scale 1/4, and every smaller member stays on the grid
    return synth.to_bf16_bits(g.choice([0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6], shape).astype(np.float32))


@pytest.mark.parametrize("wfmt", [mx.E4M3, mx.E2M1])
def test_layer_equals_dense_brute_force_bitexact(wfmt):
    # integers in [-8, 8] are exact in E4M3 under any block scale (and the E2M1 set above in
    # E2M1), so every product and sum is exact and the two paths round h and y identically
    g = np.random.default_rng(0)
    T, H, E, k, I = 24, 64, 6, 2, 64
    x = _int_bits(g, (T, H))
    logits = g.standard_normal((T, E)).astype(np.float32)
    wbits = _int_bits if wfmt == mx.E4M3 else _e2m1_int_bits
    w1 = wbits(g, (E, 2 * I, H))
    w2 = wbits(g, (E, H, I))
    res = ep_mx.ep_layer_mx(x, logits, w1, w2, k, E, 3, T * k, wfmt=wfmt)
    dense64, dense_bits = ep_mx.ep_layer_mx_dense(x, logits, w1, w2, k, wfmt=wfmt)
    assert res["status"] == ep.STATUS_OK
    assert np.array_equal(res["out_bits"], dense_bits)
    assert np.array_equal(res["out64"], dense64)


def test_dispatch_windows_hold_the_quantized_token_rows():
    g = np.random.default_rng(1)
    n_src, T, H, E, k, W = 2, 16, 96, 4, 2, 2
    x = synth.to_bf16_bits(g.standard_normal((n_src, T, H)).astype(np.float32))
    logits = g.standard_normal((n_src, T, E)).astype(np.float32)
    w1 = synth.normal_bf16(0, 1, (E, 64, H), std=0.05)
    w2 = synth.normal_bf16(0, 2, (E, H, 32), std=0.05)
    res = ep_mx.ep_layer_mx(x, logits, w1, w2, k, E, W, n_src * T * k)
    xc, xs = ep_mx.quantize_rows(x)
    epw = E // W
    seen = 0
    for s in range(n_src):
        for t in range(T):
            for j in range(k):
                d, r = res["idx"][s, t, j] // epw, res["layout"]["slot_row"][s, t, j]
                assert np.array_equal(res["win_codes"][d, r], xc[s, t])
                assert np.array_equal(res["win_scales"][d, r], xs[s, t])
                seen += 1
    assert seen == n_src * T * k


def test_quantized_layer_is_within_the_format_error_of_the_bf16_layer():
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    ref = ep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k)
    rl2 = {}
    for wfmt in (mx.E4M3, mx.E2M1):
        q = ep_mx.ep_layer_mx(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cfg.T * cfg.k,
                              wfmt=wfmt)
        a, b = q["out64"], ref["out64"]
        rl2[wfmt] = np.linalg.norm(a - b) / np.linalg.norm(b)
    # E4M3 keeps 3 mantissa bits: each quantized operand carries a relative rounding error of
    # up to 2^-4 (about 2^-4 / sqrt(3) rms); x, W1, h and W2 are quantized, so the output's
    # relative error is a few percent, and clearly nonzero
    assert 0.005 < rl2[mx.E4M3] < 0.12, rl2
    # E2M1 weights keep 1 mantissa bit (steps of up to 2^-2 relative, and values below a
    # twelfth of the block maximum flush to 0 or 0.5 steps): a larger error, still bounded
    assert 2 * rl2[mx.E4M3] < rl2[mx.E2M1] < 0.5, rl2


def test_h_is_the_quantized_swiglu_output():
    g = np.random.default_rng(2)
    M, H, I = 5, 64, 96
    xq = mx.quantize_mx(g.standard_normal((M, H)), mx.E4M3)
    w1q = mx.quantize_mx(g.standard_normal((2 * I, H)) * 0.1, mx.E4M3)
    w2q = mx.quantize_mx(g.standard_normal((H, I)) * 0.1, mx.E4M3)
    hc, hs, y64, yb = ep_mx.expert_ffn_mx(xq, w1q, w2q)
    X = mx.dequantize_mx(*xq, mx.E4M3)
    W1 = mx.dequantize_mx(*w1q, mx.E4M3)
    gg, uu = X @ W1[:I].T, X @ W1[I:].T
    h = gg * uu / (1 + np.exp(-gg))
    assert hc.shape == (M, I) and hs.shape == (M, I // 32)
    # every h value is within half an E4M3 step of its block's grid
    hd = mx.dequantize_mx(hc, hs, mx.E4M3)
    step = np.repeat(np.ldexp(1.0, hs.astype(int) - 127 - 9), 32, axis=1)   # subnormal step of the block
    rel = np.abs(hd - h) <= np.maximum(np.abs(h) * 2.0 ** -4, step / 2) * (1 + 1e-12)
    assert rel.all()
    assert np.allclose(y64, hd @ mx.dequantize_mx(*w2q, mx.E4M3).T)
