"""GPU parity of the MX (microscaled) quantizer and GEMM against the CPU oracle, through the C
ABI: codes and scales bit-exact, the GEMM (E4M3 x E4M3 and E4M3 x packed E2M1) within the
fp32-accumulation tolerance of the fp64 product of the dequantized operands."""
import numpy as np
import pytest
import torch

import synth
from oracle import mx
from gpu_helpers import assert_close, dev_bits, host_bits, require_gpu, xs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _bits_f64(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _quantize(x_bits, fmt, pad_codes=0, pad_scales=0):
    X = xs()
    rows, cols = x_bits.shape
    cb = cols if fmt == X.XS_FMT_E4M3 else cols // 2
    ldc, lds = cb + pad_codes, cols // 32 + pad_scales
    x = dev_bits(x_bits)
    codes = torch.full((rows, ldc), 0x5A, dtype=torch.uint8, device="cuda")
    scales = torch.full((rows, lds), 0xA5, dtype=torch.uint8, device="cuda")
    X.check(X.xs_quantize_mx(x.data_ptr(), rows, cols, cols, fmt, codes.data_ptr(), ldc,
                             scales.data_ptr(), lds, _stream()))
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy(), cb


@pytest.mark.parametrize("fmt_name", ["E4M3", "E2M1"])
@pytest.mark.parametrize("rows,cols", [(1, 512), (37, 1536), (300, 7168)])
def test_quantize_grouped_is_the_oracle_regrouped(fmt_name, rows, cols):
    # the grouped quantizer writes the oracle's codes bit for bit and its scales regrouped as
    # [cols / 512][rows][16]: scale (r, j) at ((j / 16) * rows + r) * 16 + j % 16
    X = xs()
    fmt = getattr(X, f"XS_FMT_{fmt_name}")
    g = np.random.default_rng(rows * 7 + cols)
    x = synth.to_bf16_bits((g.standard_normal((rows, cols)) * np.exp(g.uniform(-6, 6, (rows, 1)))).astype(np.float32))
    want_c, want_s = mx.quantize_mx(_bits_f64(x), getattr(mx, fmt_name))
    if fmt_name == "E2M1":
        want_c = mx.pack_e2m1(want_c)
    cb = want_c.shape[1]
    codes = torch.full((rows, cb), 0x5A, dtype=torch.uint8, device="cuda")
    scales = torch.full((cols // 512, rows, 16), 0xA5, dtype=torch.uint8, device="cuda")
    dx = dev_bits(x)
    X.check(X.xs_quantize_mx_grouped(dx.data_ptr(), rows, cols, cols, fmt, codes.data_ptr(), cb,
                                     scales.data_ptr(), _stream()))
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), want_c)
    got_s = scales.cpu().numpy().transpose(1, 0, 2).reshape(rows, cols // 32)
    assert np.array_equal(got_s, want_s)
    # arguments: columns not a multiple of 512, a misaligned scale base
    assert X.xs_quantize_mx_grouped(dx.data_ptr(), rows, 480, 480, fmt, codes.data_ptr(), cb, scales.data_ptr(),
                                    _stream()) == X.XS_EINVAL
    assert X.xs_quantize_mx_grouped(dx.data_ptr(), rows, cols, cols, fmt, codes.data_ptr(), cb,
                                    scales.data_ptr() + 4, _stream()) == X.XS_EINVAL
    torch.cuda.synchronize()


def _special_rows(cols):
    """Rows that hit the exponent rule's edges and the encoder's ties."""
    t = mx.fmt_values(mx.E4M3)
    rows = [np.zeros(cols),                                    # all-zero blocks
            np.full(cols, 448.0), np.full(cols, 449.0),        # amax exactly fmax / just above
            np.tile((t[1:] + t[:-1])[:32] / 2, cols // 32),     # exact midpoints of E4M3
            np.tile(np.r_[1.75, np.linspace(-1, 1, 31)], cols // 32),
            np.tile(np.r_[2.0 ** -130, np.zeros(31)], cols // 32)]   # a bf16 subnormal maximum
    return synth.to_bf16_bits(np.array(rows, dtype=np.float32))


@pytest.mark.parametrize("fmt_name", ["E4M3", "E2M1"])
@pytest.mark.parametrize("rows,cols", [(1, 32), (7, 96), (130, 7168), (257, 2048)])
def test_quantize_bitexact(fmt_name, rows, cols):
    X = xs()
    fmt = getattr(X, f"XS_FMT_{fmt_name}")
    ofmt = getattr(mx, fmt_name)
    g = np.random.default_rng(rows + cols)
    x = synth.to_bf16_bits((g.standard_normal((rows, cols)) * np.exp(g.uniform(-4, 4, (rows, 1)))).astype(np.float32))
    if rows >= 6:
        x[:6] = _special_rows(cols)
    codes, scales, cb = _quantize(x, fmt, pad_codes=16, pad_scales=4)
    ref_c, ref_s = mx.quantize_mx(_bits_f64(x), ofmt)
    if ofmt == mx.E2M1:
        ref_c = mx.pack_e2m1(ref_c)
    assert np.array_equal(scales[:, :cols // 32], ref_s)
    assert np.array_equal(codes[:, :cb], ref_c)
    assert (codes[:, cb:] == 0x5A).all() and (scales[:, cols // 32:] == 0xA5).all()   # padding untouched


def _gemm_mx(a_bits, b_bits, b_fmt="E4M3"):
    """Quantize both operands on the GPU (B as E4M3 or packed E2M1), multiply; returns (c bits,
    oracle fp64)."""
    X = xs()
    M, K = a_bits.shape
    N = b_bits.shape[0]
    fmt = getattr(X, f"XS_FMT_{b_fmt}")
    ac, as_, _ = _quantize(a_bits, X.XS_FMT_E4M3)
    bc, bs, ldb = _quantize(b_bits, fmt)
    da, das = torch.from_numpy(ac).cuda(), torch.from_numpy(as_).cuda()
    db, dbs = torch.from_numpy(bc).cuda(), torch.from_numpy(bs).cuda()
    c = torch.full((M, N), -1, dtype=torch.int16, device="cuda")
    X.check(X.xs_gemm_mx(da.data_ptr(), K, das.data_ptr(), K // 32, db.data_ptr(), ldb, dbs.data_ptr(), K // 32,
                         fmt, c.data_ptr(), N, M, N, K, None, _stream()))
    torch.cuda.synchronize()
    ofmt = getattr(mx, b_fmt)
    ref = mx.gemm_mx(ac, as_, mx.E4M3, mx.unpack_e2m1(bc) if ofmt == mx.E2M1 else bc, bs, ofmt)
    return host_bits(c), ref


@pytest.mark.parametrize("b_fmt", ["E4M3", "E2M1"])
@pytest.mark.parametrize("M,N,K", [(256, 256, 512), (300, 512, 1536), (1, 256, 512), (513, 768, 1024), (77, 256, 7168),
                                   (260, 256, 2560)])
def test_gemm_mx_matches_oracle(M, N, K, b_fmt):
    a = synth.normal_bf16(0, 20, (M, K))
    b = synth.normal_bf16(0, 21, (N, K), std=0.05)
    c, ref = _gemm_mx(a, b, b_fmt)
    assert_close(c, ref, f"gemm_mx {M}x{N}x{K} B {b_fmt}")


@pytest.mark.parametrize("b_fmt", ["E4M3", "E2M1"])
def test_gemm_mx_integer_operands_bitexact(b_fmt):
    # small integers are exact in E4M3 with scale 2^0 when every block holds a value of 256..448
    # (scale exponent 0) - here A blocks are integers in [-8, 8] plus one 256: scale 2^0, exact
    # codes. B likewise, or for E2M1 integers that E2M1 holds ({0, 1, 2, 3, 4, 6} and negatives)
    # with one 6 per block (scale 2^0). |sums| < 2^24, so fp32 accumulation is exact in any order
    g = np.random.default_rng(9)
    M, N, K = 300, 256, 512
    a = g.integers(-8, 9, (M, K)).astype(np.float32)
    a[:, ::32] = 256.0
    if b_fmt == "E4M3":
        b = g.integers(-8, 9, (N, K)).astype(np.float32)
        b[:, ::32] = 256.0
    else:
        b = g.choice([0, 1, -1, 2, -2, 3, -3, 4, -4, 6, -6], (N, K)).astype(np.float32)
        b[:, ::32] = 6.0
    c, ref = _gemm_mx(synth.to_bf16_bits(a), synth.to_bf16_bits(b), b_fmt)
    from oracle.ep import f64_to_bf16_bits
    assert np.array_equal(c, f64_to_bf16_bits(a.astype(np.float64) @ b.astype(np.float64).T))
    assert np.array_equal(c, f64_to_bf16_bits(ref))


def test_mx_bad_arguments():
    X = xs()
    x = torch.zeros((4, 64), dtype=torch.int16, device="cuda")
    c = torch.zeros((4, 64), dtype=torch.uint8, device="cuda")
    s = torch.zeros((4, 2), dtype=torch.uint8, device="cuda")
    assert X.xs_quantize_mx(x.data_ptr(), 4, 48, 64, X.XS_FMT_E4M3, c.data_ptr(), 64, s.data_ptr(), 2, _stream()) == X.XS_EINVAL
    assert X.xs_quantize_mx(x.data_ptr(), 4, 64, 64, 7, c.data_ptr(), 64, s.data_ptr(), 2, _stream()) == X.XS_EINVAL
    assert X.xs_quantize_mx(x.data_ptr(), 4, 64, 64, X.XS_FMT_E4M3, c.data_ptr(), 32, s.data_ptr(), 2, _stream()) == X.XS_EINVAL
    a = torch.zeros((256, 1024), dtype=torch.uint8, device="cuda")
    sc = torch.zeros((256, 32), dtype=torch.uint8, device="cuda")
    o = torch.zeros((256, 256), dtype=torch.int16, device="cuda")

    def gemm(K=512, N=256, fmt=X.XS_FMT_E4M3, lda=1024, ldb=1024, lds=32, sa=0, M=256):
        return X.xs_gemm_mx(a.data_ptr(), lda, sc.data_ptr() + sa, lds, a.data_ptr(), ldb, sc.data_ptr(), lds, fmt,
                            o.data_ptr(), 256, M, N, K, None, _stream())

    assert gemm(K=384) == X.XS_EUNSUPPORTED            # K % 512
    assert gemm(N=200) == X.XS_EUNSUPPORTED            # N % 256
    assert gemm(fmt=9) == X.XS_EINVAL
    assert gemm(lds=20) == X.XS_EUNSUPPORTED           # scale rows of 16-byte pieces
    assert gemm(sa=4) == X.XS_EINVAL                   # scale base 16-byte aligned
    # packed E2M1 rows need K / 2 bytes: 256 bytes cover K = 512 but not K = 1024
    assert gemm(K=1024, fmt=X.XS_FMT_E2M1, ldb=256, M=0) == X.XS_EUNSUPPORTED
    assert gemm(K=512, fmt=X.XS_FMT_E2M1, ldb=256, M=0) == X.XS_OK
    torch.cuda.synchronize()
