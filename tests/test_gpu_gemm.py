"""GPU parity of the MFMA GEMM and its scatter epilogues (TP row blocks, Ulysses head
groups) against the CPU oracle, through the C ABI."""
import numpy as np
import pytest
import torch

import synth
from oracle import ep as oep
from oracle import scatter as osc
from oracle.ep import f64_to_bf16_bits
from gpu_helpers import assert_close, dev_bits, host_bits, require_gpu, xs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _gemm(a_bits, bt_bits):
    X = xs()
    M, K = a_bits.shape
    N = bt_bits.shape[0]
    a, b = dev_bits(a_bits), dev_bits(bt_bits)
    c = torch.full((M, N), -1, dtype=torch.int16, device="cuda")
    X.check(X.xs_gemm(a.data_ptr(), K, b.data_ptr(), K, c.data_ptr(), N, M, N, K, None, _stream()))
    torch.cuda.synchronize()
    return host_bits(c)


@pytest.mark.parametrize("M,N,K", [(300, 512, 192), (1, 256, 64), (256, 256, 64), (513, 768, 1024)])
def test_gemm_ragged_matches_oracle(M, N, K):
    a = synth.normal_bf16(0, 5, (M, K))
    b = synth.normal_bf16(0, 6, (K, N), std=0.05)
    c = _gemm(a, np.ascontiguousarray(b.T))
    assert_close(c, osc.gemm(a, b), f"gemm {M}x{N}x{K}")


def test_gemm_integer_operands_bitexact():
    # |sums| < 2^24: fp32 accumulation is exact in any order, so the rounded bits are unique
    a = synth.int_valued_bf16(0, 1, (384, 320))
    b = synth.int_valued_bf16(0, 2, (320, 512))
    c = _gemm(a, np.ascontiguousarray(b.T))
    assert np.array_equal(c, f64_to_bf16_bits(osc.gemm(a, b)))


def _windows_rowblock(W, rpd, N):
    X = xs()
    win = torch.full((W, rpd, N), -1, dtype=torch.int16, device="cuda")
    return win, X.windows([X.window(win[d]) for d in range(W)])


def _tp(a_bits, b_bits, rpd, serial=False, pacing=None):
    X = xs()
    M, K = a_bits.shape
    N = b_bits.shape[1]
    W = M // rpd
    a, bt = dev_bits(a_bits), dev_bits(np.ascontiguousarray(b_bits.T))
    win, wins = _windows_rowblock(W, rpd, N)
    desc = X.xs_scatter_desc(X.XS_SCATTER_ROW_BLOCK, rpd, 0, 0, 0, 0)
    if serial:
        c = torch.empty((M, N), dtype=torch.int16, device="cuda")
        X.check(X.xs_gemm(a.data_ptr(), K, bt.data_ptr(), K, c.data_ptr(), N, M, N, K, None, _stream()))
        X.check(X.xs_scatter_copy(c.data_ptr(), N, M, N, desc, wins, W, _stream()))
    else:
        X.check(X.xs_gemm_scatter(a.data_ptr(), K, bt.data_ptr(), K, M, N, K, desc, wins, W, pacing, None, _stream()))
    torch.cuda.synchronize()
    return host_bits(win)


def test_tp_identity_b_copies_row_blocks_bitexact():
    a = synth.normal_bf16(0, 5, (1024, 256))
    b = synth.to_bf16_bits(np.eye(256, dtype=np.float32))
    win = _tp(a, b, 256)
    assert np.array_equal(win, a.reshape(4, 256, 256))


def test_tp_full_size_every_element_and_fused_equals_serial():
    cfg = synth.TP_ROWBLOCK
    inp = synth.tp_inputs(cfg, 0)
    rpd = cfg.M // cfg.W
    fused = _tp(inp["a"], inp["b"], rpd)
    serial = _tp(inp["a"], inp["b"], rpd, serial=True)
    assert np.array_equal(fused, serial)
    # every element of every window against the oracle's fp64 product before rounding
    c64, win_ref = osc.tp_row_block_scatter(inp["a"], inp["b"], rpd)
    assert_close(fused.reshape(cfg.M, cfg.N), c64, "tp windows")
    assert np.mean(fused == win_ref) > 0.99      # nearly every element rounds like the oracle's


def _sp(x_bits, w_bits, nh, hd, hpg, serial=False, pacing=None):
    X = xs()
    S, Dm = x_bits.shape
    N = w_bits.shape[1]
    G = nh // hpg
    x, wt = dev_bits(x_bits), dev_bits(np.ascontiguousarray(w_bits.T))
    win = torch.full((G, 3, hpg, S, hd), -1, dtype=torch.int16, device="cuda")
    wins = X.windows([X.xs_window(win[g].data_ptr(), 3 * hpg * S, hd * 2, None) for g in range(G)])
    desc = X.xs_scatter_desc(X.XS_SCATTER_HEAD_GROUP, 0, 3, nh, hd, hpg)
    if serial:
        c = torch.empty((S, N), dtype=torch.int16, device="cuda")
        X.check(X.xs_gemm(x.data_ptr(), Dm, wt.data_ptr(), Dm, c.data_ptr(), N, S, N, Dm, None, _stream()))
        X.check(X.xs_scatter_copy(c.data_ptr(), N, S, N, desc, wins, G, _stream()))
    else:
        X.check(X.xs_gemm_scatter(x.data_ptr(), Dm, wt.data_ptr(), Dm, S, N, Dm, desc, wins, G, pacing, None, _stream()))
    torch.cuda.synchronize()
    return host_bits(win)


@pytest.mark.parametrize("S,nh,hd,hpg", [(300, 8, 32, 2),     # heads straddle tile groups: generic path
                                          (300, 8, 64, 4),     # one group per tile, 4 heads per tile
                                          (257, 4, 256, 1)])   # one head per tile, ragged rows
def test_sp_small_matches_oracle_bitexact_on_identity(S, nh, hd, hpg):
    N = 3 * nh * hd
    x = synth.normal_bf16(0, 7, (S, N))
    w = synth.to_bf16_bits(np.eye(N, dtype=np.float32))
    win = _sp(x, w, nh, hd, hpg)
    _, ref = osc.sp_head_group_scatter(x, w, nh, hd, hpg)
    assert np.array_equal(win, ref)


def test_sp_full_size_every_element_and_fused_equals_serial():
    cfg = synth.SP_QKV
    inp = synth.sp_inputs(cfg, 0)
    fused = _sp(inp["x"], inp["w"], cfg.n_heads, cfg.head_dim, cfg.heads_per_group)
    serial = _sp(inp["x"], inp["w"], cfg.n_heads, cfg.head_dim, cfg.heads_per_group, serial=True)
    assert np.array_equal(fused, serial)
    qkv64, win_ref = osc.sp_head_group_scatter(inp["x"], inp["w"], cfg.n_heads, cfg.head_dim,
                                               cfg.heads_per_group)
    G = cfg.n_heads // cfg.heads_per_group
    # column (which, g, lh, dd) of the product is element [g][which][lh][s][dd] of the windows
    ref64 = qkv64.reshape(cfg.S, 3, G, cfg.heads_per_group, cfg.head_dim).transpose(2, 1, 3, 0, 4)
    assert np.array_equal(oep.f64_to_bf16_bits(ref64), win_ref)
    assert_close(fused, ref64, "sp windows")
    assert np.mean(fused == win_ref) > 0.99


def test_scatter_rejects_bad_descriptors():
    X = xs()
    a = torch.zeros((512, 64), dtype=torch.int16, device="cuda")
    b = torch.zeros((256, 64), dtype=torch.int16, device="cuda")
    win, wins = _windows_rowblock(2, 256, 256)
    bad = X.xs_scatter_desc(X.XS_SCATTER_ROW_BLOCK, 200, 0, 0, 0, 0)
    assert X.xs_gemm_scatter(a.data_ptr(), 64, b.data_ptr(), 64, 512, 256, 64, bad, wins, 2, None, None,
                             None) != X.XS_OK
    assert X.xs_gemm(a.data_ptr(), 64, b.data_ptr(), 64, a.data_ptr(), 64, 512, 100, 64, None,
                     None) == X.XS_EUNSUPPORTED


def _grouped(a_bits, offs, rows, b_bits, swiglu, M=None):
    X = xs()
    M = a_bits.shape[0] if M is None else M
    K = a_bits.shape[1]
    n_seg, N = b_bits.shape[0], b_bits.shape[1]
    n_out = N // 2 if swiglu else N
    a, b = dev_bits(a_bits), dev_bits(b_bits)
    c = torch.full((M, n_out), -1, dtype=torch.int16, device="cuda")
    so = torch.tensor(offs, dtype=torch.int32, device="cuda")
    sr = torch.tensor(rows, dtype=torch.int32, device="cuda")
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    X.check(X.xs_grouped_gemm(a.data_ptr(), K, M, so.data_ptr(), sr.data_ptr(), n_seg, b.data_ptr(), N, K,
                              c.data_ptr(), n_out, X.XS_EPI_SWIGLU if swiglu else X.XS_EPI_STORE, st.data_ptr(),
                              _stream()))
    torch.cuda.synchronize()
    return host_bits(c), int(st.item())


@pytest.mark.parametrize("swiglu", [False, True])
def test_grouped_gemm_matches_oracle(swiglu):
    # ragged segments with gaps, an empty one and one of a single row; K = 7168 as the expert FFN
    M, K, N = 1500, 7168, 512
    offs = [0, 300, 301, 700, 1200, 1499]
    rows = [257, 0, 399, 480, 299, 1]
    a = synth.normal_bf16(0, 20, (M, K))
    b = synth.normal_bf16(0, 21, (len(offs), N, K), std=0.02)
    got, st = _grouped(a, offs, rows, b, swiglu)
    assert st == 0
    c64, bits = oep.grouped_gemm(a, offs, rows, b, swiglu=swiglu)
    inside = ~np.isnan(c64[:, 0])
    assert_close(got[inside], c64[inside], f"grouped gemm swiglu={swiglu}")
    assert (got[~inside] == 0xFFFF).all()


def test_grouped_gemm_integer_operands_bitexact_and_bad_segment():
    X = xs()
    M, K, N = 600, 512, 256
    offs, rows = [0, 256, 512], [256, 256, 88]
    a = synth.int_valued_bf16(0, 22, (M, K))
    b = synth.int_valued_bf16(0, 23, (3, N, K))
    got, st = _grouped(a, offs, rows, b, False)
    _, bits = oep.grouped_gemm(a, offs, rows, b)
    assert st == 0 and np.array_equal(got, bits)
    # a segment past the rows is skipped and reported; the others are still computed
    got, st = _grouped(a, [0, 500], [256, 200], b[:2], False)
    assert st == X.XS_EBADINPUT
    _, bits = oep.grouped_gemm(a, [0], [256], b[:1])
    assert np.array_equal(got[:256], bits[:256]) and (got[256:] == 0xFFFF).all()
    # argument errors: nothing launched
    z = torch.zeros((16,), dtype=torch.int32, device="cuda")
    assert X.xs_grouped_gemm(z.data_ptr(), 64, 4, z.data_ptr(), z.data_ptr(), 1, z.data_ptr(), 100, 64, z.data_ptr(),
                             100, X.XS_EPI_STORE, None, None) == X.XS_EUNSUPPORTED
    assert X.xs_grouped_gemm(z.data_ptr(), 64, 4, z.data_ptr(), z.data_ptr(), 1, z.data_ptr(), 256, 64, z.data_ptr(),
                             256, 7, None, None) == X.XS_EINVAL


def _pacing(policy, chunk=0, max_producers=0, gap_ns=0):
    from paper_2607_23264_amd.layer import pacing
    return pacing(policy, lead=0, chunk=chunk, max_producers=max_producers, gap_ns=gap_ns)


def test_scatter_pacing_orders_store_the_same_windows():
    """Every pacing order of the scatter GEMM (destination-major bursts, round robin, chunks of
    tiles, a producer cap and a gap) fills the windows with the oracle's values, bit for bit equal
    to the default order."""
    X = xs()
    a = synth.normal_bf16(0, 30, (2048, 512))
    b = synth.normal_bf16(0, 31, (512, 1024), std=0.05)
    rpd = 512
    base = _tp(a, b, rpd)
    c64, _ = osc.tp_row_block_scatter(a, b, rpd)
    assert_close(base.reshape(2048, 1024), c64, "tp small")
    for pol in (_pacing(X.XS_POLICY_BURST), _pacing(X.XS_POLICY_INTERLEAVE, max_producers=7),
                _pacing(X.XS_POLICY_CHUNK, chunk=4, max_producers=16, gap_ns=3000)):
        assert np.array_equal(_tp(a, b, rpd, pacing=pol), base), pol.policy
    cfg = synth.SP_QKV
    x = synth.normal_bf16(0, 32, (512, 1024))
    w = synth.normal_bf16(0, 33, (1024, 3 * 16 * 64), std=0.05)
    base = _sp(x, w, 16, 64, 4)
    qkv64, _ = osc.sp_head_group_scatter(x, w, 16, 64, 4)
    ref64 = qkv64.reshape(512, 3, 4, 4, 64).transpose(2, 1, 3, 0, 4)
    assert_close(base, ref64, "sp small")
    for pol in (_pacing(X.XS_POLICY_BURST), _pacing(X.XS_POLICY_CHUNK, chunk=2, max_producers=5)):
        assert np.array_equal(_sp(x, w, 16, 64, 4, pacing=pol), base), pol.policy


def test_scatter_pacing_full_size_tp_equals_default():
    X = xs()
    cfg = synth.TP_ROWBLOCK
    inp = synth.tp_inputs(cfg, 0)
    rpd = cfg.M // cfg.W
    base = _tp(inp["a"], inp["b"], rpd)
    for pol in (_pacing(X.XS_POLICY_BURST), _pacing(X.XS_POLICY_INTERLEAVE), _pacing(X.XS_POLICY_CHUNK, chunk=8)):
        assert np.array_equal(_tp(inp["a"], inp["b"], rpd, pacing=pol), base), pol.policy


def test_scatter_pacing_rejects_bad_orders():
    X = xs()
    a = torch.zeros((1024, 64), dtype=torch.int16, device="cuda")
    b = torch.zeros((256, 64), dtype=torch.int16, device="cuda")
    win, wins = _windows_rowblock(2, 512, 256)
    desc = X.xs_scatter_desc(X.XS_SCATTER_ROW_BLOCK, 512, 0, 0, 0, 0)
    bad_chunk = _pacing(X.XS_POLICY_CHUNK, chunk=3)          # 2 tiles per window: 3 does not divide
    assert X.xs_gemm_scatter(a.data_ptr(), 64, b.data_ptr(), 64, 1024, 256, 64, desc, wins, 2, bad_chunk, None,
                             None) == X.XS_EINVAL
    neg = _pacing(X.XS_POLICY_BURST, gap_ns=-1)
    assert X.xs_gemm_scatter(a.data_ptr(), 64, b.data_ptr(), 64, 1024, 256, 64, desc, wins, 2, neg, None,
                             None) == X.XS_EINVAL
    torch.cuda.synchronize()
