"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

# bf16-input / fp32-accumulate outputs against the oracle's fp64 value before its final
# rounding: per element |gpu - ref| / max(1, |ref|) <= 2e-2 and relative L2 <= 1e-2.
ELEM_TOL = 2e-2
L2_TOL = 1e-2


def require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def xs():
    from paper_2607_23264_amd import xstage
    return xstage


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint16)


def dev_bits(a: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


def bits_f64(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_close(gpu_bits: np.ndarray, ref64: np.ndarray, what: str, slack=None):
    """Reading 11's bounds; `slack` (same shape, optional) is a derived allowance added to
    |gpu - ref| before the scaled bound applies (quantization decisions that fp32 may take
    either way, see mx_y_slack)."""
    g = bits_f64(gpu_bits)
    r = np.asarray(ref64, dtype=np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite values"
    d = np.abs(g - r)
    if slack is not None:
        d = np.maximum(0.0, d - slack)
    err = d / np.maximum(1.0, np.abs(r))
    worst = float(err.max()) if err.size else 0.0
    rl2 = float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-300)) if r.size else 0.0
    assert worst <= ELEM_TOL, f"{what}: max scaled error {worst:.3e} at {np.unravel_index(err.argmax(), err.shape)}"
    assert rl2 <= L2_TOL, f"{what}: relative L2 {rl2:.3e}"
    return worst, rl2


# ----------------------------------------------------------------------------- MX h bounds
def mx_h_admissible(xq, w1q, wfmt):
    """The quantized SwiGLU activations h the GPU may legitimately produce for one expert.

    The GPU accumulates Linear-1 in fp32 and evaluates SwiGLU in fp32, so its h differs from
    the exact value h of the dequantized operands by at most bh = |dh/dg| bg + |dh/du| bu +
    (8 + 2|g|) 2^-24 |h|, with bg, bu = 2 (64 + K / 64) 2^-24 sum_k |x_k w_k| the bounds of
    the gate and up sums: the scaled MFMA adds 64 products per instruction into its fp32
    accumulator, so a product passes through at most 64 rounded additions inside an
    instruction and K / 64 accumulator updates (the blocked-summation bound, doubled for the
    block-scale products); the last term covers the exp, reciprocal and products. A
    block's scale may be the shared exponent of any values within that bound (e_lo .. e_hi),
    and a code the round-to-nearest-even of any value within it.
    Returns (h exact [M][I], lo, hi, e_lo, e_hi [M][I / 32], vmin, vmax): vmin / vmax bound
    the dequantized value of every admissible (scale, code)."""
    from oracle import mx as omxf
    X = omxf.dequantize_mx(*xq, omxf.E4M3)
    W1 = omxf.dequantize_mx(*w1q, wfmt)
    I = W1.shape[0] // 2
    K = X.shape[1]
    g, u = X @ W1[:I].T, X @ W1[I:].T
    u_eps = 2.0 ** -24
    aX = np.abs(X)
    n_round = 2 * (64 + K // 64)
    bg = n_round * u_eps * (aX @ np.abs(W1[:I]).T)
    bu = n_round * u_eps * (aX @ np.abs(W1[I:]).T)
    with np.errstate(over="ignore"):
        sig = 1.0 / (1.0 + np.exp(-g))
    h = g * sig * u
    dh_dg = np.abs(u * sig * (1 + g * (1 - sig)))
    bh = dh_dg * bg + np.abs(g * sig) * bu + (8 + 2 * np.abs(g)) * u_eps * np.abs(h)
    lo, hi = h - bh, h + bh
    m = h.shape[0]
    amax_lo = np.where((lo > 0) | (hi < 0), np.minimum(np.abs(lo), np.abs(hi)), 0.0)
    amax_hi = np.maximum(np.abs(lo), np.abs(hi))
    e_lo = omxf.shared_exponent(amax_lo.reshape(m, -1, 32).max(-1), omxf.E4M3)
    e_hi = omxf.shared_exponent(amax_hi.reshape(m, -1, 32).max(-1), omxf.E4M3)
    vmin = np.full(h.shape, np.inf)
    vmax = np.full(h.shape, -np.inf)
    for de in range(int((e_hi - e_lo).max()) + 1):
        e = np.minimum(e_lo + de, e_hi)
        sc = np.repeat(np.ldexp(1.0, e), 32, axis=1)
        vmin = np.minimum(vmin, omxf.decode(omxf.encode(lo / sc, omxf.E4M3), omxf.E4M3) * sc)
        vmax = np.maximum(vmax, omxf.decode(omxf.encode(hi / sc, omxf.E4M3), omxf.E4M3) * sc)
    return h, lo, hi, e_lo, e_hi, vmin, vmax


def mx_y_slack(adm, w2q, wfmt, h_codes, h_scales):
    """Allowance on each expert output y of the quantized layer beyond reading 11's bound.

    Where an h code is decided differently within the fp32 bound (mx_h_admissible), y moves
    by that code's change times the W2 column: the allowance of output (m, n) is
    sum_i dev_mi |W2_ni|, dev_mi the largest distance between an admissible dequantized h and
    the oracle's (zero where only the oracle's code is admissible), plus the fp32 accumulation
    bound of Linear-2, 2 (64 + I / 64) 2^-24 sum_i |h_mi W2_ni|. adm is mx_h_admissible's
    result; h_codes / h_scales are the oracle's."""
    from oracle import mx as omxf
    vmin, vmax = adm[5], adm[6]
    v = omxf.dequantize_mx(h_codes, h_scales, omxf.E4M3)
    dev = np.maximum(vmax - v, v - vmin)
    W2 = np.abs(omxf.dequantize_mx(*w2q, wfmt))
    I = W2.shape[1]
    return dev @ W2.T + 2 * (64 + I // 64) * 2.0 ** -24 * (np.abs(v) @ W2.T)


def check_h_admissible(got_codes, got_scales, adm, what):
    """Every GPU h scale and code is admissible (adm = mx_h_admissible's result); returns how
    many codes differ from the oracle's own quantization of the exact h."""
    from oracle import mx as omxf
    h, lo, hi, e_lo, e_hi, _, _ = adm
    es = got_scales.astype(np.int64) - 127
    bad_scale = (es < e_lo) | (es > e_hi)
    assert not bad_scale.any(), f"{what}: {bad_scale.sum()} block scales outside the fp32 bound"
    sc = np.repeat(np.ldexp(1.0, es), 32, axis=1)
    vals = omxf.decode(got_codes, omxf.E4M3)
    c_lo = omxf.decode(omxf.encode(lo / sc, omxf.E4M3), omxf.E4M3)
    c_hi = omxf.decode(omxf.encode(hi / sc, omxf.E4M3), omxf.E4M3)
    bad = (vals < c_lo) | (vals > c_hi)
    assert not bad.any(), f"{what}: {bad.sum()} codes outside the fp32 bound, first at {np.argwhere(bad)[0]}"
    want, _ = omxf.quantize_mx(h, omxf.E4M3)
    return int((got_codes != want).sum())


def h_codes_scales(lay, I):
    """h code rows [h_rows][I] and row-major h scales [h_rows][I / 32] from an MX layer's h
    workspace (code rows, then the scale groups [I / 512][h_rows][16])."""
    flat = lay.h_ws.cpu().numpy().reshape(-1)
    rows = lay.h_ws.shape[0]
    codes = flat[:rows * I].reshape(rows, I)
    g = flat[rows * I:rows * I + (I // 512) * rows * 16].reshape(I // 512, rows, 16)
    return codes, np.ascontiguousarray(g.transpose(1, 0, 2).reshape(rows, I // 32))
