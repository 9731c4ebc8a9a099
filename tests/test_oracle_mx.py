"""Pins of the MX-format oracle: the OCP element tables, round-to-nearest-even encoding (against
torch's own float8_e4m3fn conversion and hand-worked E2M1 ties), the shared-exponent rule by
brute force, the quantizer's error bound and the dequantized GEMM."""
import numpy as np
import pytest
import torch

from oracle import mx


def test_e4m3_table_against_torch_decode():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = mx.decode(np.arange(256, dtype=np.uint8), mx.E4M3)
    nan = np.isnan(ref)
    assert nan.sum() == 2 and (np.isnan(ours) == nan).all()       # 0x7F and 0xFF
    assert np.array_equal(ours[~nan], ref[~nan])
    t = mx.fmt_values(mx.E4M3)
    assert t[-1] == 448.0 and t[1] == 2.0 ** -9 and (np.diff(t) > 0).all()


def test_e4m3_encode_matches_torch_rne():
    g = np.random.default_rng(0)
    t = mx.fmt_values(mx.E4M3)
    mids = (t[1:] + t[:-1]) / 2                       # exact ties between neighbours
    v = np.concatenate([g.uniform(-448, 448, 20000), g.standard_normal(20000) * 2.0 ** g.integers(-12, 6, 20000),
                        mids, -mids, t, -t, [0.0, -0.0, 2.0 ** -10, 3 * 2.0 ** -10]])
    ref = torch.from_numpy(v.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    ours = mx.encode(v.astype(np.float32).astype(np.float64), mx.E4M3)
    assert np.array_equal(ours, ref)                  # including -0 (0x80) for negative underflow


def test_e2m1_table_and_ties_by_hand():
    assert list(mx.fmt_values(mx.E2M1)) == [0, 0.5, 1, 1.5, 2, 3, 4, 6]
    # halfway cases go to the even code: (value, expected value)
    cases = [(0.25, 0), (0.75, 1), (1.25, 1), (1.75, 2), (2.5, 2), (3.5, 4), (5.0, 4),
             (0.3, 0.5), (2.6, 3), (5.1, 6), (6.0, 6), (-1.75, -2), (-0.25, 0)]
    for v, want in cases:
        got = mx.decode(mx.encode(np.array([v]), mx.E2M1), mx.E2M1)[0]
        assert got == want, (v, got, want)
    # the sign survives a zero result: -0.25 -> code 0x8 (-0)
    assert mx.encode(np.array([-0.25, -0.0, 0.0]), mx.E2M1).tolist() == [8, 8, 0]


@pytest.mark.parametrize("fmt,fmax", [(mx.E4M3, 448.0), (mx.E2M1, 6.0)])
def test_shared_exponent_is_the_smallest_that_fits(fmt, fmax):
    g = np.random.default_rng(1)
    amax = np.concatenate([np.abs(g.standard_normal(5000)) * 2.0 ** g.integers(-30, 30, 5000),
                           [fmax, fmax * 2, fmax / 2, np.nextafter(fmax, 1e9), 1.0, 2.0 ** -20]])
    e = mx.shared_exponent(amax, fmt)
    assert (amax <= fmax * np.ldexp(1.0, e)).all()
    assert (amax > fmax * np.ldexp(1.0, e - 1)).all()
    assert mx.shared_exponent(np.array([0.0]), fmt)[0] == 0
    assert mx.shared_exponent(np.array([fmax]), fmt)[0] == 0


def test_quantize_error_bound_and_no_saturation():
    g = np.random.default_rng(2)
    x = g.standard_normal((64, 256)) * np.exp(g.uniform(-3, 3, (64, 1)))
    x[3, 32:64] = 0.0                                   # an all-zero block
    for fmt, mant_bits in ((mx.E4M3, 3), (mx.E2M1, 1)):
        codes, scales = mx.quantize_mx(x, fmt)
        assert codes.shape == x.shape and scales.shape == (64, 8)
        y = mx.dequantize_mx(codes, scales, fmt)
        s = np.ldexp(1.0, scales.astype(np.int64) - 127)
        blk = np.abs(x).reshape(64, 8, 32)
        # no element saturates: every scaled value is within the format
        assert (blk / s[..., None] <= mx.fmt_values(fmt)[-1]).all()
        # round-to-nearest error: half a unit in the last place of the element's binade,
        # or half the smallest subnormal step of the block
        err = np.abs(y - x).reshape(64, 8, 32)
        min_step = {mx.E4M3: 2.0 ** -9, mx.E2M1: 0.5}[fmt] * s[..., None]
        ulp = np.where(blk > 0, np.ldexp(1.0, np.floor(np.log2(np.maximum(blk, 1e-300))).astype(int) - mant_bits), 0)
        assert (err <= np.maximum(ulp, min_step) / 2 * (1 + 1e-12)).all()
        assert (y[3, 32:64] == 0).all() and scales[3, 1] == 127


def test_representable_values_survive_exactly():
    g = np.random.default_rng(3)
    for fmt in (mx.E4M3, mx.E2M1):
        t = mx.fmt_values(fmt)
        codes = g.integers(0, len(t), (16, 64))
        sign = np.where(g.random((16, 64)) < 0.5, -1.0, 1.0)
        e = g.integers(-20, 20, (16, 2))
        x = (sign * t[codes]).reshape(16, 2, 32)
        x[:, :, 0] = t[-1] * np.sign(x[:, :, 0] + 0.5)     # each block reaches fmax exactly
        x = (x * np.ldexp(1.0, e)[..., None]).reshape(16, 64)
        c, s = mx.quantize_mx(x, fmt)
        assert np.array_equal(mx.dequantize_mx(c, s, fmt), x)
        assert np.array_equal(s.astype(int) - 127, e)


def test_e2m1_packing_roundtrip():
    g = np.random.default_rng(4)
    c = g.integers(0, 16, (5, 64)).astype(np.uint8)
    p = mx.pack_e2m1(c)
    assert p.shape == (5, 32) and (p[:, 0] & 0xF == c[:, 0]).all() and (p[:, 0] >> 4 == c[:, 1]).all()
    assert np.array_equal(mx.unpack_e2m1(p), c)


def test_gemm_mx_is_the_product_of_dequantized_operands():
    g = np.random.default_rng(5)
    a = g.standard_normal((9, 96))
    b = g.standard_normal((7, 96))
    ac, as_ = mx.quantize_mx(a, mx.E4M3)
    bc, bs = mx.quantize_mx(b, mx.E2M1)
    c = mx.gemm_mx(ac, as_, mx.E4M3, bc, bs, mx.E2M1)
    ref = np.array([[sum(mx.dequantize_mx(ac, as_, mx.E4M3)[i, k] * mx.dequantize_mx(bc, bs, mx.E2M1)[j, k]
                         for k in range(96)) for j in range(7)] for i in range(9)])
    assert np.allclose(c, ref, rtol=0, atol=1e-12)
