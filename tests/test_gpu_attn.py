"""GPU parity of attention with the fused post-attention Ulysses exchange (Sec. 4.4, App. B;
Table 4) against the CPU oracle, through the C ABI."""
import numpy as np
import pytest
import torch

import synth
from oracle import attention as oa
from gpu_helpers import assert_close, dev_bits, host_bits, require_gpu, xs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _inputs(heads, M, seed, qstd=1.0, d=128):
    q = synth.normal_bf16(seed, 910, (heads, M, d), std=qstd)
    k = synth.normal_bf16(seed, 911, (heads, M, d))
    v = synth.normal_bf16(seed, 912, (heads, M, d))
    return q, k, v


def _desc(heads, M, q, k, v, o=None, win=None, W=0, max_producers=0, scale=0.0):
    X = xs()
    return X.xs_attn(heads, M, 128, W, scale, max_producers, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                     0 if o is None else o.data_ptr(), win)


def _local(q_bits, k_bits, v_bits, max_producers=0, scale=0.0, trace=None):
    X = xs()
    heads, M, _ = q_bits.shape
    q, k, v = dev_bits(q_bits), dev_bits(k_bits), dev_bits(v_bits)
    o = torch.full((heads, M, 128), -1, dtype=torch.int16, device="cuda")
    a = _desc(heads, M, q, k, v, o=o, max_producers=max_producers, scale=scale)
    X.check(X.xs_attention(a, X.XS_ATTN_LOCAL, trace, _stream()))
    torch.cuda.synchronize()
    return host_bits(o)


def _windows(heads, M, W, pad_cols=0):
    X = xs()
    rows = M // W
    buf = torch.full((W, rows, heads * 128 + pad_cols), -1, dtype=torch.int16, device="cuda")
    flags = torch.zeros(W, dtype=torch.int32, device="cuda")
    wins = X.windows([X.window(buf[g], flag=flags[g:g + 1]) for g in range(W)])
    return buf, flags, wins


def _fused(q_bits, k_bits, v_bits, W, pad_cols=0, max_producers=0, coupled=False):
    X = xs()
    heads, M, _ = q_bits.shape
    q, k, v = dev_bits(q_bits), dev_bits(k_bits), dev_bits(v_bits)
    buf, flags, wins = _windows(heads, M, W, pad_cols)
    a = _desc(heads, M, q, k, v, win=wins, W=W, max_producers=max_producers)
    mode = X.XS_ATTN_WINDOWS_COUPLED if coupled else X.XS_ATTN_WINDOWS
    X.check(X.xs_attention(a, mode, None, _stream()))
    torch.cuda.synchronize()
    return host_bits(buf), flags.cpu().numpy()


def _windows_as_heads(win_bits, heads):
    """[W][M/W][heads*128 (+pad)] -> [W][M/W][heads][128] (padding dropped)."""
    W, rows, _ = win_bits.shape
    return win_bits[:, :, :heads * 128].reshape(W, rows, heads, 128)


@pytest.mark.parametrize("heads,M,qstd", [(1, 128, 1.0), (2, 384, 1.0), (3, 1024, 1.0), (2, 640, 3.0)])
def test_attention_matches_oracle(heads, M, qstd):
    q, k, v = _inputs(heads, M, seed=heads * 7 + M, qstd=qstd)
    o = _local(q, k, v)
    ref64, _ = oa.attention(q, k, v)
    assert_close(o, ref64, f"attention h={heads} M={M} qstd={qstd}")


def test_explicit_scale_matches_oracle():
    q, k, v = _inputs(2, 256, seed=11)
    o = _local(q, k, v, scale=0.25)
    ref64, _ = oa.attention(q, k, v, scale=0.25)
    assert_close(o, ref64, "attention scale=0.25")


def test_dominant_keys_select_value_rows_bitexact():
    # keys 0..127 are 16 e_u, the rest 0; query t of head h is 16 e_c with c = (37 t + 5 h) mod
    # 128, so key c scores 256 / sqrt(128) = 22.6 and every other key 0 or less: the weights of
    # the others sum below 256 exp(-22.6) < 4e-8, under half a bf16 unit, so O[h][t] is exactly
    # V[h][c]. A wrong key, query or column index anywhere in either product breaks it.
    heads, M = 2, 256
    qf = np.zeros((heads, M, 128), dtype=np.float32)
    kf = np.zeros((heads, M, 128), dtype=np.float32)
    for h in range(heads):
        for u in range(128):
            kf[h, u, u] = 16.0
        for t in range(M):
            qf[h, t, (37 * t + 5 * h) % 128] = 16.0
    q, k = synth.to_bf16_bits(qf), synth.to_bf16_bits(kf)
    v = synth.normal_bf16(3, 913, (heads, M, 128))
    o = _local(q, k, v)
    pick = np.array([[(37 * t + 5 * h) % 128 for t in range(M)] for h in range(heads)])
    expect = np.stack([v[h, pick[h]] for h in range(heads)])
    assert np.array_equal(o, expect)


def test_grid_size_does_not_change_bits():
    q, k, v = _inputs(2, 512, seed=21)
    a = _local(q, k, v)
    b = _local(q, k, v, max_producers=1)
    c = _local(q, k, v, max_producers=3)
    assert np.array_equal(a, b) and np.array_equal(a, c)


@pytest.mark.parametrize("heads,M,W,pad", [(2, 512, 4, 0), (3, 768, 2, 8), (1, 256, 2, 0), (2, 1024, 8, 0)])
def test_fused_windows_equal_local_output_scattered(heads, M, W, pad):
    q, k, v = _inputs(heads, M, seed=31 + W)
    o = _local(q, k, v)
    win, flags = _fused(q, k, v, W, pad_cols=pad)
    assert np.array_equal(_windows_as_heads(win, heads), oa.ulysses_scatter(o, W))
    if pad:
        assert (win[:, :, heads * 128:] == 0xFFFF).all()     # the row padding is not written
    assert (flags == 1).all()
    ref64, _ = oa.attention(q, k, v)
    assert_close(_windows_as_heads(win, heads), oa.ulysses_scatter(ref64, W), "fused windows")


def test_completion_coupled_mode_stores_the_same_bits():
    q, k, v = _inputs(2, 1024, seed=61)
    a, fa = _fused(q, k, v, 4, max_producers=3)
    b, fb = _fused(q, k, v, 4, max_producers=3, coupled=True)
    assert np.array_equal(a, b) and (fa == 1).all() and (fb == 1).all()


def test_serial_copy_equals_fused():
    X = xs()
    heads, M, W = 2, 512, 4
    q, k, v = _inputs(heads, M, seed=41)
    o_bits = _local(q, k, v)
    buf, flags, wins = _windows(heads, M, W)
    o = dev_bits(o_bits)
    X.check(X.xs_ulysses_copy(o.data_ptr(), heads, M, 128, wins, W, _stream()))
    torch.cuda.synchronize()
    fused, _ = _fused(q, k, v, W)
    assert np.array_equal(host_bits(buf), fused)
    assert (flags.cpu().numpy() == 1).all()


def test_trace_records_every_tile_once():
    X = xs()
    heads, M = 3, 512
    q, k, v = _inputs(heads, M, seed=51)
    tiles = heads * M // 128
    buf = torch.zeros(4 * (tiles + 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    _local(q, k, v, max_producers=5, trace=X.trace(buf, cnt))
    n = int(cnt.item())
    assert n == tiles
    rec = buf.view(-1, 4)[:n].cpu().numpy().view(np.uint64)
    assert sorted((rec[:, 0] & 0xFFFFFFFF).tolist()) == list(range(tiles))
    assert ((rec[:, 0] >> 56) == 4).all()
    assert ((rec[:, 0] >> 32) & 0xFFFFFF < 5).all()          # producer ids within the grid
    assert (rec[:, 1] <= rec[:, 2]).all() and (rec[:, 2] <= rec[:, 3]).all()


def test_full_size_every_row():
    # the Ulysses shape of the fused-attention workload: 8 local heads, 8192 tokens, 8 windows,
    # the launch the benchmark times (default grid); every output element against the fp64
    # oracle (one head at a time, to bound host memory)
    cfg = synth.ATTN_UP_8K
    inp = synth.attn_inputs(cfg, 0)
    q, k, v = inp["q"], inp["k"], inp["v"]
    o = _local(q, k, v)
    win, flags = _fused(q, k, v, cfg.W)
    assert np.array_equal(_windows_as_heads(win, cfg.heads), oa.ulysses_scatter(o, cfg.W))
    assert (flags == 1).all()
    for h in range(cfg.heads):
        ref64, _ = oa.attention(q[h:h + 1], k[h:h + 1], v[h:h + 1])
        assert_close(o[h:h + 1], ref64, f"attention M=8192 head {h}")


@pytest.mark.parametrize("cfg", [synth.ATTN_UP_16K, synth.ATTN_UP_32K], ids=lambda c: c.name)
def test_long_sequences_at_the_default_grid(cfg):
    # the FA-only launch the benchmark times (default grid: several output tiles per workgroup,
    # a last round with idle slots) stores the same bits as a 100-workgroup grid, in which every
    # workgroup walks many tiles; sampled rows of every head (the first row of each of 16
    # tiles, the last tile, the first and last rows) against the fp64 oracle
    print(f"[attn long] {cfg.name}", flush=True)
    inp = synth.attn_inputs(cfg, 0)
    q, k, v = inp["q"], inp["k"], inp["v"]
    o = _local(q, k, v)
    assert np.array_equal(o, _local(q, k, v, max_producers=100))
    M = cfg.M
    rng = np.random.default_rng(7)
    for h in range(cfg.heads):
        tiles = rng.choice(M // 128, 16, replace=False)
        rows = np.unique(np.concatenate([tiles * 128, np.arange(M - 128, M, 8), [0, M - 1],
                                         rng.integers(0, M, 16)]))
        ref64, _ = oa.attention(q[h:h + 1, rows], k[h:h + 1], v[h:h + 1])
        assert_close(o[h:h + 1, rows], ref64, f"attention M={M} head {h} sampled rows")


def test_bad_arguments_are_rejected():
    X = xs()
    heads, M = 1, 256
    q = torch.zeros((heads, M, 128), dtype=torch.int16, device="cuda")
    o = torch.zeros_like(q)
    ok = _desc(heads, M, q, q, q, o=o)
    X.check(X.xs_attention(ok, X.XS_ATTN_LOCAL, None, _stream()))
    # head_dim other than 128, M not a multiple of 128, M past the kernel's buffer range
    # (rejected before any launch)
    for hd, m in ((64, 256), (128, 200), (128, 8388608)):
        a = _desc(heads, m, q, q, q, o=o)
        a.head_dim = hd
        assert X.xs_attention(a, X.XS_ATTN_LOCAL, None, _stream()) == X.XS_EUNSUPPORTED
    # bad mode, missing output, negative scale, misaligned input
    assert X.xs_attention(ok, 3, None, _stream()) == X.XS_EINVAL
    assert X.xs_attention(_desc(heads, M, q, q, q), X.XS_ATTN_LOCAL, None, _stream()) == X.XS_EINVAL
    a = _desc(heads, M, q, q, q, o=o, scale=-1.0)
    assert X.xs_attention(a, X.XS_ATTN_LOCAL, None, _stream()) == X.XS_EINVAL
    a = _desc(heads, M, q, q, q, o=o)
    a.q = q.data_ptr() + 2
    assert X.xs_attention(a, X.XS_ATTN_LOCAL, None, _stream()) == X.XS_EINVAL
    # windows: a chunk that straddles tiles, too few rows, too narrow a row
    buf, _, wins = _windows(heads, 384, 2)                  # chunk 192
    a = _desc(heads, 384, q, q, q, win=wins, W=2)
    assert X.xs_attention(a, X.XS_ATTN_WINDOWS, None, _stream()) == X.XS_EUNSUPPORTED
    small = torch.zeros((2, 64, 128), dtype=torch.int16, device="cuda")
    w2 = X.windows([X.window(small[g]) for g in range(2)])
    a = _desc(heads, M, q, q, q, win=w2, W=2)
    assert X.xs_attention(a, X.XS_ATTN_WINDOWS, None, _stream()) == X.XS_EINVAL
    narrow = torch.zeros((2, 128, 64), dtype=torch.int16, device="cuda")
    w3 = X.windows([X.window(narrow[g]) for g in range(2)])
    a = _desc(heads, M, q, q, q, win=w3, W=2)
    assert X.xs_attention(a, X.XS_ATTN_WINDOWS, None, _stream()) == X.XS_EINVAL
    assert X.xs_ulysses_copy(o.data_ptr(), heads, M, 128, w3, 2, _stream()) == X.XS_EINVAL
    torch.cuda.synchronize()
