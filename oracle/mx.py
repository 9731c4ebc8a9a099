"""Oracle for the microscaled (MX) number formats of the quantized EP path (test infrastructure
only: nothing in the product path imports it).

The paper runs its EP kernel at W8A8 and W4A8 (Sec. 5.2, the MegaMoE sweep) without fixing the
formats. Reading: OCP microscaling, as the gfx950 matrix cores take it natively. A block of 32
consecutive elements along the reduction axis shares one power-of-two scale (E8M0: 2^(c - 127),
code 255 is NaN); the elements are
  * E4M3 (OCP "FN"): 1 sign, 4 exponent bits (bias 7), 3 mantissa bits; normals
    (1 + m/8) 2^(E - 7) for E = 1..15 except E = 15, m = 7 (NaN); subnormals (m/8) 2^-6;
    largest finite 448, no infinities;
  * E2M1: 1 sign, 2 exponent bits (bias 1), 1 mantissa bit: 0, 0.5, 1, 1.5, 2, 3, 4, 6.
Encoding is round to nearest, ties to the even code (the code whose mantissa ends in 0), and
keeps the sign, also when the magnitude rounds to zero (-0 = the sign bit alone), as an IEEE
round-to-nearest-even conversion does.
Shared exponent (reading): the smallest integer e with amax <= fmax 2^e (fmax = 448 or 6), so
no element of the block saturates; e is clamped to [-127, 127], and an all-zero block takes
e = 0. With amax = M 2^E (1 <= M < 2) and fmax = Mf 2^Ef this is e = E - Ef + [M > Mf], an
integer decision the GPU takes on the same bits.
Quantized values are exact in fp64, so the GEMM oracle is the plain fp64 product of the
dequantized operands.
"""
from __future__ import annotations

import concurrent.futures as cf
import math
import os

import numpy as np

__all__ = ["E4M3", "E2M1", "fmt_values", "encode", "decode", "shared_exponent", "quantize_mx",
           "dequantize_mx", "pack_e2m1", "unpack_e2m1", "gemm_mx", "GROUP"]

GROUP = 32
E4M3, E2M1 = "e4m3", "e2m1"


def _e4m3_table():
    """Value of every non-negative E4M3 code 0..126 (127 is NaN)."""
    vals = []
    for c in range(127):
        E, m = c >> 3, c & 7
        vals.append(m / 8 * 2.0 ** -6 if E == 0 else (1 + m / 8) * 2.0 ** (E - 7))
    return np.array(vals)


def _e2m1_table():
    vals = []
    for c in range(8):
        E, m = c >> 1, c & 1
        vals.append(m / 2 if E == 0 else (1 + m / 2) * 2.0 ** (E - 1))
    return np.array(vals)


_TABLES = {E4M3: _e4m3_table(), E2M1: _e2m1_table()}
_SIGN = {E4M3: 0x80, E2M1: 0x8}
_FMAX = {E4M3: (1.75, 8), E2M1: (1.5, 2)}        # fmax = Mf 2^Ef: 448, 6


def fmt_values(fmt):
    """Non-negative finite values of the format, indexed by code."""
    return _TABLES[fmt]


def decode(codes, fmt):
    """Codes (uint8; E2M1 in the low nibble) -> fp64 (E4M3 NaN codes -> nan)."""
    c = np.asarray(codes).astype(np.int64)
    sign_bit = _SIGN[fmt]
    mag = c & (sign_bit - 1)
    t = _TABLES[fmt]
    out = np.where(mag < len(t), t[np.minimum(mag, len(t) - 1)], np.nan)
    return np.where(c & sign_bit, -out, out)


def encode(v, fmt):
    """fp64 -> codes, round to nearest with ties to the even code, sign kept (also for -0).
    |v| above the largest finite value saturates to it (the quantizer below never produces
    such values)."""
    v = np.asarray(v, dtype=np.float64)
    t = _TABLES[fmt]
    a = np.minimum(np.abs(v), t[-1])
    hi = np.clip(np.searchsorted(t, a, side="left"), 0, len(t) - 1)   # t[hi] >= a
    lo = np.maximum(hi - 1, 0)
    dlo, dhi = a - t[lo], t[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0) & (hi != lo))
    mag = np.where(pick_hi, hi, lo)
    mag = np.where(a == t[hi], hi, mag)
    return (mag | np.where(np.signbit(v), _SIGN[fmt], 0)).astype(np.uint8)


def shared_exponent(amax, fmt):
    """Smallest integer e with amax <= fmax 2^e (0 for amax = 0), clamped to [-127, 127]."""
    amax = np.asarray(amax, dtype=np.float64)
    Mf, Ef = _FMAX[fmt]
    m, E = np.frexp(amax)                  # amax = m 2^E with 0.5 <= m < 1
    M, E = 2.0 * m, E - 1                  # 1 <= M < 2
    e = E - Ef + (M > Mf).astype(np.int64)
    e = np.where(amax == 0, 0, e)
    return np.clip(e, -127, 127).astype(np.int64)


def _quantize_block_rows(x, fmt, group):
    g = x.reshape(*x.shape[:-1], x.shape[-1] // group, group)
    e = shared_exponent(np.abs(g).max(axis=-1), fmt)
    codes = encode(g / np.ldexp(1.0, e)[..., None], fmt)
    return codes.reshape(x.shape), (e + 127).astype(np.uint8)


def quantize_mx(x, fmt, group=GROUP):
    """x: fp64 values [..., K] with K % group == 0. Returns (codes uint8 [..., K], scale codes
    uint8 [..., K / group] = e + 127).

    Every block is quantized on its own, so large inputs are split into row chunks handled on
    a thread pool (numpy releases the interpreter lock in these element-wise steps); the
    arithmetic of each element is the same either way."""
    x = np.asarray(x, dtype=np.float64)
    K = x.shape[-1]
    if K % group:
        raise ValueError("reduction length must be a multiple of the group")
    rows = x.reshape(-1, K)
    if rows.size <= 1 << 20:
        c, s = _quantize_block_rows(rows, fmt, group)
    else:
        step = max(1, (1 << 16) // K)
        with cf.ThreadPoolExecutor(max(1, len(os.sched_getaffinity(0)))) as ex:
            parts = list(ex.map(lambda r0: _quantize_block_rows(rows[r0:r0 + step], fmt, group),
                                range(0, rows.shape[0], step)))
        c = np.concatenate([p[0] for p in parts])
        s = np.concatenate([p[1] for p in parts])
    return c.reshape(x.shape), s.reshape(*x.shape[:-1], K // group)


def dequantize_mx(codes, scales, fmt, group=GROUP):
    c = decode(codes, fmt)
    K = c.shape[-1]
    g = c.reshape(*c.shape[:-1], K // group, group)
    s = np.ldexp(1.0, np.asarray(scales).astype(np.int64) - 127)
    return (g * s[..., None]).reshape(c.shape)


def pack_e2m1(codes):
    """E2M1 codes [..., K] -> bytes [..., K / 2]: element 2i in the low nibble, 2i + 1 high."""
    c = np.asarray(codes, dtype=np.uint8)
    return (c[..., 0::2] & 0xF) | ((c[..., 1::2] & 0xF) << 4)


def unpack_e2m1(packed):
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.uint8)
    out[..., 0::2] = p & 0xF
    out[..., 1::2] = p >> 4
    return out


def gemm_mx(a_codes, a_scales, a_fmt, b_codes, b_scales, b_fmt):
    """C = deq(A) deq(B)^T in fp64; A [M][K], B [N][K] (codes unpacked)."""
    A = dequantize_mx(a_codes, a_scales, a_fmt)
    B = dequantize_mx(b_codes, b_scales, b_fmt)
    return A @ B.T


def bf16_to_mx(bits, fmt):
    """Convenience: bf16 bits -> (codes, scales) through the exact fp64 values."""
    v = (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return quantize_mx(v, fmt)


assert math.isclose(_TABLES[E4M3][-1], 448.0) and _TABLES[E2M1][-1] == 6.0
