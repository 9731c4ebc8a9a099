"""GPU parity of the quantized expert-parallel layer, W8A8 (MXFP8) and W4A8 (E2M1 weights),
against the CPU oracle, through the C ABI: dispatch windows of quantized token rows
(bit-exact), the quantized h rows, the combine rows and the combined output; every pacing
policy gives the same bits."""
import ctypes as C
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import ep as oep
from oracle import ep_mx as omx
from oracle import mx as omxf
from gpu_helpers import assert_close, bits_f64, check_h_admissible, host_bits, mx_h_admissible, require_gpu, xs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)


PRECISIONS = ["MXFP8", "W4A8"]


def _wfmt(prec):
    return omxf.E2M1 if prec == "W4A8" else omxf.E4M3


def _mx_layer(cfg, prec="MXFP8", **kw):
    from paper_2607_23264_amd.layer import EPLayer, Shape
    X = xs()
    experts = synth.computed_experts(cfg)
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=cfg.rank,
              **kw)
    return EPLayer(s, precision=getattr(X, f"XS_PREC_{prec}"))


def _policies():
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    return {"burst": pacing(X.XS_POLICY_BURST), "interleave_D1": pacing(X.XS_POLICY_INTERLEAVE, lead=1),
            "chunk2_p8": pacing(X.XS_POLICY_CHUNK, lead=2, chunk=2, max_producers=8),
            "auto_nomodel": pacing(X.XS_POLICY_AUTO),
            "interleave_dyn": pacing(X.XS_POLICY_INTERLEAVE, lead=1, claim=X.XS_CLAIM_DYNAMIC),
            "burst_w4_dyn": pacing(X.XS_POLICY_BURST, wave_tiles=4, claim=X.XS_CLAIM_DYNAMIC)}


def _window_bases(lay):
    """Row of the h workspace where each computed window's rows begin."""
    s = lay.s
    counts = lay.dest_counts.cpu().numpy()
    first = s.e_begin // s.epw
    base, out = 0, {}
    for d in range(first, first + s.n_cwin):
        out[d] = base
        base += min(int(counts[d]), lay.cap)
    return out


@pytest.mark.parametrize("prec", PRECISIONS)
def test_tiny_layer_matches_oracle_for_every_policy(prec):
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    ref = omx.ep_layer_mx(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k,
                          wfmt=_wfmt(prec))
    lay = _mx_layer(cfg, prec)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    outs = {}
    for name, p in _policies().items():
        lay.out.zero_()
        lay.cwin.fill_(-1)
        lay.fused(p)
        torch.cuda.synchronize()
        assert int(lay.status.item()) == 0, name
        outs[name] = host_bits(lay.out)
        assert_close(outs[name], ref["out64"], f"tiny {prec} layer {name}")
    first = next(iter(outs.values()))
    for name, o in outs.items():
        assert np.array_equal(o, first), f"policy {name} changed the output bits"
    assert np.array_equal(lay.topk_idx.cpu().numpy(), ref["idx"])
    assert np.array_equal(lay.slot_row.cpu().numpy(), ref["layout"]["slot_row"])
    # dispatch windows: the quantized token rows, codes then scales, bit for bit
    win = lay.dwin.cpu().numpy()
    H = cfg.H
    for d in range(cfg.W):
        n = int(ref["layout"]["dest_counts"][d])
        assert np.array_equal(win[d, :n, :H], ref["win_codes"][d, :n]), f"window {d} codes"
        assert np.array_equal(win[d, :n, H:H + H // 32], ref["win_scales"][d, :n]), f"window {d} scales"
        assert (win[d, n:] == 0xFF).all(), f"window {d} rows past the count were written"
    # h rows of every expert: I codes and I / 32 scales (code rows, then the scale groups)
    hcodes, hscales = _h_codes_scales(lay, cfg.I)
    bases = _window_bases(lay)
    epw = cfg.E // cfg.W
    flips = 0
    for e, (hc, hs) in ref["h"].items():
        d, r0 = e // epw, int(ref["layout"]["expert_offsets"][e])
        m = hc.shape[0]
        sl = slice(bases[d] + r0, bases[d] + r0 + m)
        xq = (ref["win_codes"][d, r0:r0 + m], ref["win_scales"][d, r0:r0 + m])
        adm = mx_h_admissible(xq, omx.quantize_rows(inp["w1"][e], _wfmt(prec)), _wfmt(prec))
        flips += check_h_admissible(hcodes[sl], hscales[sl], adm, f"h of expert {e}")
    print(f"h codes that differ from the oracle's (all within the fp32 bound): {flips}")
    # combine rows (bf16 expert outputs) against the oracle's rounded rows
    comb = host_bits(lay.cwin)
    assert_close(comb[0], bits_f64(ref["combine"][0]), "combine rows")


@pytest.mark.parametrize("prec", PRECISIONS)
def test_multi_source_ragged_share(prec):
    # 3 sources, this GPU = rank 1 owning experts 4..7; T not a multiple of the 256-row tile
    cfg = synth.EPConfig("t", T=300, H=512, E=16, k=3, I=512, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 7)
    experts = synth.computed_experts(cfg)
    fill = synth.normal_bf16(0, 200, (cfg.T * cfg.k, cfg.H))
    ref = omx.ep_layer_mx(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W,
                          cap=cfg.n_src * cfg.T * cfg.k, experts=experts, combine_fill=fill, out_src=cfg.rank,
                          wfmt=_wfmt(prec))
    lay = _mx_layer(cfg, prec)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(fill)
    from paper_2607_23264_amd.layer import pacing
    lay.fused(pacing(xs().XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    assert_close(host_bits(lay.out), ref["out64"], f"ragged {prec} share output")
    # the computed window holds every source's quantized rows bit for bit
    d = cfg.rank
    n = int(ref["layout"]["dest_counts"][d])
    win = lay.dwin.cpu().numpy()
    assert np.array_equal(win[d, :n, :cfg.H], ref["win_codes"][d, :n])
    assert np.array_equal(win[d, :n, cfg.H:cfg.H + cfg.H // 32], ref["win_scales"][d, :n])
    # combine windows of every source: computed rows close to the oracle's, the rest untouched
    comb = host_bits(lay.cwin)
    epw = cfg.E // cfg.W
    own = np.isin(ref["idx"] // epw, [cfg.rank]).reshape(cfg.n_src, cfg.T * cfg.k)
    for s in range(cfg.n_src):
        assert_close(comb[s][own[s]], bits_f64(ref["combine"][s][own[s]]), f"combine rows of source {s}")
        if s != cfg.rank:
            assert (comb[s][~own[s]] == 0xFFFF).all()


def _fused_rc(L, lay):
    X = xs()
    ws = lay.workspace
    return X.xs_fused_ep_layer(C.byref(L), None, None, ws.data_ptr(), ws.numel(), lay.status.data_ptr(),
                               lay.stream)


def test_bad_arguments():
    X = xs()
    cfg = synth.EP_TINY
    lay = _mx_layer(cfg)
    ws = lay.workspace

    def variant(**fields):
        L = X.xs_ep_layer.from_buffer_copy(lay.L)
        for k, v in fields.items():
            setattr(L, k, v)
        return L

    assert _fused_rc(variant(precision=3), lay) == X.XS_EINVAL
    assert _fused_rc(variant(reserved=1), lay) == X.XS_EINVAL
    assert _fused_rc(variant(w1_scale=None), lay) == X.XS_EINVAL
    assert _fused_rc(variant(w2_scale=None), lay) == X.XS_EINVAL
    assert _fused_rc(variant(expert_mode=X.XS_EXPERT_IDENTITY), lay) == X.XS_EUNSUPPORTED
    assert _fused_rc(variant(I=768), lay) == X.XS_EUNSUPPORTED
    assert _fused_rc(variant(w1=lay.w1q.data_ptr() + 8), lay) == X.XS_EINVAL
    assert _fused_rc(variant(w2_scale=lay.w2s.data_ptr() + 2), lay) == X.XS_EINVAL
    # the unfused phase calls take bf16 only
    assert X.xs_expert_ffn(C.byref(lay.L), ws.data_ptr(), ws.numel(), lay.status.data_ptr(),
                           lay.stream) == X.XS_EUNSUPPORTED
    assert X.xs_combine_send(C.byref(lay.L), None, lay.status.data_ptr(), lay.stream) == X.XS_EUNSUPPORTED
    # a workspace sized for bf16 is too small: the quantized rows are staged in it
    nb = C.c_int64()
    X.check(X.xs_ep_layer_workspace_bytes(C.byref(variant(precision=X.XS_PREC_BF16)), C.byref(nb)))
    assert X.xs_fused_ep_layer(C.byref(lay.L), None, None, ws.data_ptr(), nb.value, lay.status.data_ptr(),
                               lay.stream) == X.XS_EWORKSPACE
    # windows narrower than a quantized row
    narrow = X.windows([X.window(lay.dwin[w], row_bytes=cfg.H) for w in range(cfg.W)])
    assert _fused_rc(variant(dispatch_win=C.cast(narrow, C.POINTER(X.xs_window))), lay) != X.XS_OK
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0


def test_dispatch_rows_bitexact():
    X = xs()
    g = np.random.default_rng(3)
    T, k, E, W, row_bytes, stride = 301, 3, 12, 3, 80, 96
    idx = np.argsort(g.random((1, T, E)), axis=2)[:, :, :k].astype(np.int32)
    lay = oep.dispatch_layout(idx, E, W, T * k)
    rows = g.integers(0, 256, (T, stride), dtype=np.uint8)
    d_rows = torch.from_numpy(rows).cuda()
    d_idx = torch.from_numpy(idx[0]).cuda()
    d_slot = torch.from_numpy(np.ascontiguousarray(lay["slot_row"][0])).cuda()
    win = torch.full((W, T * k, 112), 0xAB, dtype=torch.uint8, device="cuda")
    wins = X.windows([X.window(win[d]) for d in range(W)])
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    X.check(X.xs_dispatch_rows(d_rows.data_ptr(), stride, row_bytes, T, d_idx.data_ptr(), d_slot.data_ptr(), k, E,
                               wins, W, st.data_ptr(), torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    want = np.full((W, T * k, 112), 0xAB, dtype=np.uint8)
    epw = E // W
    for t in range(T):
        for j in range(k):
            want[idx[0, t, j] // epw, lay["slot_row"][0, t, j], :row_bytes] = rows[t, :row_bytes]
    assert np.array_equal(win.cpu().numpy(), want)
    # argument checks
    cs = torch.cuda.current_stream().cuda_stream
    args = (d_idx.data_ptr(), d_slot.data_ptr(), k, E, wins, W, st.data_ptr(), cs)
    assert X.xs_dispatch_rows(d_rows.data_ptr(), stride, 8, T, *args) == X.XS_EINVAL
    assert X.xs_dispatch_rows(d_rows.data_ptr(), stride, 24, T, *args) == X.XS_EUNSUPPORTED
    assert X.xs_dispatch_rows(d_rows.data_ptr(), 72, row_bytes, T, *args) == X.XS_EINVAL
    assert X.xs_dispatch_rows(d_rows.data_ptr() + 8, stride, row_bytes, T, *args) == X.XS_EUNSUPPORTED
    assert X.xs_dispatch_rows(d_rows.data_ptr(), stride, 128, T, *args) != X.XS_OK   # windows too narrow
    assert X.xs_dispatch_rows(d_rows.data_ptr(), stride, row_bytes, 0, *args) == X.XS_OK
    torch.cuda.synchronize()


def _ungroup(groups, expert, rows):
    """Row-major scales [rows][K / 32] of one expert from the grouped layout [K / 512][experts *
    rows][16] (group g of row r holds the scales of blocks 16 g .. 16 g + 15)."""
    g = groups.cpu().numpy()[:, expert * rows:(expert + 1) * rows, :]
    return np.ascontiguousarray(g.transpose(1, 0, 2)).reshape(rows, -1)


def _h_codes_scales(lay, I):
    """h code rows [h_rows][I] and row-major h scales [h_rows][I / 32] from h_ws (code rows,
    then the scale groups [I / 512][h_rows][16])."""
    flat = lay.h_ws.cpu().numpy().reshape(-1)
    hr = flat.size // (I + I // 32)
    codes = flat[:hr * I].reshape(hr, I)
    sc = flat[hr * I:hr * (I + I // 32)].reshape(I // 512, hr, 16).transpose(1, 0, 2).reshape(hr, I // 32)
    return codes, sc


@pytest.mark.parametrize("prec", PRECISIONS)
def test_weight_quantization_matches_oracle(prec):
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 2)
    lay = _mx_layer(cfg, prec)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    pack = omxf.pack_e2m1 if prec == "W4A8" else (lambda c: c)
    for i in (0, cfg.E - 1):
        c1, s1 = omx.quantize_rows(inp["w1"][i], _wfmt(prec))
        c2, s2 = omx.quantize_rows(inp["w2"][i], _wfmt(prec))
        c1, c2 = pack(c1), pack(c2)
        assert np.array_equal(lay.w1q[i].cpu().numpy(), c1) and np.array_equal(_ungroup(lay.w1s, i, 2 * cfg.I), s1)
        assert np.array_equal(lay.w2q[i].cpu().numpy(), c2) and np.array_equal(_ungroup(lay.w2s, i, cfg.H), s2)


def _records(buf, count):
    n = min(int(count.item()), buf.shape[0])
    r = buf[:n].cpu().numpy().astype(np.uint64)
    kind = (r[:, 0] >> np.uint64(56)).astype(np.int64)
    wg = ((r[:, 0] >> np.uint64(32)) & np.uint64(0xFFFFFF)).astype(np.int64)
    tile = (r[:, 0] & np.uint64(0xFFFFFFFF)).astype(np.int64)
    return kind, wg, tile, r


@pytest.mark.parametrize("prec,policy", [("MXFP8", "interleave"), ("MXFP8", "burst"), ("W4A8", "chunk")])
def test_dynamic_claim_takes_every_tile_once_after_its_dependencies(prec, policy):
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    lay = _mx_layer(cfg, prec)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    G = 8
    pol = {"interleave": pacing(X.XS_POLICY_INTERLEAVE, lead=1, max_producers=G, claim=X.XS_CLAIM_DYNAMIC),
           "chunk": pacing(X.XS_POLICY_CHUNK, lead=1, chunk=1, max_producers=G, claim=X.XS_CLAIM_DYNAMIC),
           "burst": pacing(X.XS_POLICY_BURST, max_producers=G, wave_tiles=16, claim=X.XS_CLAIM_DYNAMIC)}[policy]
    buf = torch.zeros((4096, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
    lay.fused(pol, X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr()))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    kind, wg, tile, r = _records(buf, cnt)
    idx = oep.route_topk_softmax(inp["logits"][0], cfg.k)[0][None]
    counts = oep.dispatch_layout(idx, cfg.E, cfg.W)["expert_counts"].sum(0)
    P = sum((int(c) + 255) // 256 for c in counts)
    P1, P2 = cfg.I // 128, cfg.H // 256
    # every tile exactly once, on producers 0..G-1
    assert sorted(tile[kind == 1].tolist()) == list(range(P * P1))
    assert sorted(tile[kind == 2].tolist()) == list(range(P * P2))
    assert set(wg.tolist()) <= set(range(G))
    # a Linear-2 tile's mainloop ends after every Linear-1 tile of its row has stored h
    l1_end = {}
    for t, e in zip(tile[kind == 1], r[kind == 1, 3].astype(np.int64)):
        l1_end[int(t) // P1] = max(l1_end.get(int(t) // P1, 0), int(e))
    for t, m in zip(tile[kind == 2], r[kind == 2, 2].astype(np.int64)):
        assert int(m) >= l1_end[int(t) // P2], f"Linear-2 tile {int(t)} ran before its row"
    # and the output equals the static order's, bit for bit
    out_dyn = host_bits(lay.out)
    lay.out.zero_()
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    assert np.array_equal(out_dyn, host_bits(lay.out))


@pytest.mark.parametrize("claim", [0, 1])
def test_withheld_dependency_times_out_and_kernel_exits(claim):
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    lay = _mx_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1, withhold_row=0, spin_timeout_us=2000, claim=claim))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == X.XS_ETIMEOUT
    lay.status.zero_()
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0


@pytest.mark.parametrize("prec", PRECISIONS)
def test_degenerate_token_rows(prec):
    # all-zero rows (every block takes scale 2^0 and codes 0), rows scaled by 2^-40 and 2^20
    # (block exponents far from 0), and sparse rows (eight nonzero elements 61 apart: most
    # blocks all zero, the others with one nonzero code)
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 3)
    xf = ((inp["x"][0].astype(np.uint32) << 16).view(np.float32)).copy()
    xf[0:8] = 0.0
    xf[8:16] *= 2.0 ** -40
    xf[16:24] *= 2.0 ** 20
    xf[24:32] = 0.0
    xf[24:32, np.arange(8) * 61] = np.linspace(-3, 3, 8, dtype=np.float32)
    x = synth.to_bf16_bits(xf)[None]
    ref = omx.ep_layer_mx(x, inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k,
                          wfmt=_wfmt(prec))
    lay = _mx_layer(cfg, prec)
    lay.upload(inp["logits"], x, inp["w1"], inp["w2"])
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    out = host_bits(lay.out)
    assert np.all(out[0:8] & 0x7FFF == 0), "zero token rows must give zero outputs"
    # y grows as x^2 through SwiGLU: the scaled rows are compared at their own magnitude
    # (outputs times 2^80 and 2^-40, exact power-of-two rescalings), so reading 11's bound
    # applies relative to the row scale rather than to 1
    got, r = bits_f64(out), ref["out64"]
    for rows, k in ((slice(8, 16), 2.0 ** 80), (slice(16, 24), 2.0 ** -40), (slice(24, 32), 1.0),
                    (slice(32, None), 1.0)):
        g_, r_ = got[rows] * k, r[rows] * k
        err = np.abs(g_ - r_) / np.maximum(1.0, np.abs(r_))
        assert np.all(np.isfinite(g_)) and err.max() <= 2e-2, (prec, rows, float(err.max()))
        assert np.linalg.norm(g_ - r_) <= 1e-2 * np.linalg.norm(r_), (prec, rows)
    win = lay.dwin.cpu().numpy()
    for d in range(cfg.W):
        n = int(ref["layout"]["dest_counts"][d])
        assert np.array_equal(win[d, :n, :cfg.H], ref["win_codes"][d, :n])
        assert np.array_equal(win[d, :n, cfg.H:cfg.H + cfg.H // 32], ref["win_scales"][d, :n])


def test_share_without_local_rows():
    # no token of any source routes to this rank's experts: the layer computes nothing and the
    # output is the routing-weighted sum of the other ranks' combine rows
    from paper_2607_23264_amd.layer import pacing
    cfg = synth.EPConfig("t", T=300, H=512, E=16, k=3, I=512, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 5)
    experts = synth.computed_experts(cfg)
    logits = inp["logits"].copy()
    logits[:, :, experts] = -1e4
    fill = synth.normal_bf16(0, 201, (cfg.T * cfg.k, cfg.H))
    ref = omx.ep_layer_mx(inp["x"], logits, inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W,
                          cap=cfg.n_src * cfg.T * cfg.k, experts=experts, combine_fill=fill, out_src=cfg.rank)
    assert not ref["h"]
    lay = _mx_layer(cfg)
    lay.upload(logits, inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(fill)
    lay.fused(pacing(xs().XS_POLICY_INTERLEAVE, lead=1, claim=xs().XS_CLAIM_DYNAMIC))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    assert int(lay.dest_counts[cfg.rank].item()) == 0
    assert_close(host_bits(lay.out), ref["out64"], "share without local rows")
