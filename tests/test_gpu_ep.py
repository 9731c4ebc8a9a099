"""GPU parity of the expert-parallel path (route, layout, dispatch, expert FFN, combine)
against the CPU oracle, through the C ABI."""
import ctypes as C

import numpy as np
import pytest
import torch

import synth
from oracle import ep as oep
from oracle import schedule as osc
from gpu_helpers import assert_close, bits_f64, dev_bits, host_bits, require_gpu, xs

pytestmark = pytest.mark.gpu

# softmax weights: fp32 exp (about 1 ulp), a 6-level butterfly sum over 64 lane partials of
# at most 16 terms each and one division: relative error well below 2e-6
W_RTOL = 2e-6


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)


def _route_gpu(logits, k, renorm=0):
    X = xs()
    T, E = logits.shape
    lg = torch.from_numpy(np.ascontiguousarray(logits, np.float32)).cuda()
    idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    X.check(X.xs_route_topk_softmax(lg.data_ptr(), T, E, k, renorm, idx.data_ptr(), w.data_ptr(),
                                    torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    return idx.cpu().numpy(), w.cpu().numpy()


@pytest.mark.parametrize("case", ["tiny", "dsv3_uniform", "dsv3_zipf", "ties_E1000_k32", "one_token",
                                  "k_equals_E", "renorm", "ties_E200_k16", "E100_k3_T17",
                                  "masked_E256_k8", "masked_E300_k8", "loop_E256_T20001", "loop_E128_T9001",
                                  "loop_E64_T16385"])
def test_route_matches_oracle(case):
    g = np.random.default_rng(11)
    renorm = 0
    if case == "tiny":
        lg, k = synth.uniform_logits(0, 2, 256, 8), 2
    elif case == "dsv3_uniform":
        lg, k = synth.uniform_logits(0, 50, 4096, 256), 8
    elif case == "dsv3_zipf":
        lg, k = synth.zipf_logits(0, 0, 4096, 256), 8
    elif case == "ties_E1000_k32":
        lg, k = (np.round(g.standard_normal((37, 1000)) * 2) / 2).astype(np.float32), 32
        lg[5] = 0.0
    elif case == "one_token":
        lg, k = g.standard_normal((1, 64)).astype(np.float32), 4
    elif case == "k_equals_E":
        lg, k = g.standard_normal((9, 8)).astype(np.float32), 8
    elif case == "ties_E200_k16":   # sixteen-lane kernel: ties, E not a multiple of 64, k = 16
        lg, k = (np.round(g.standard_normal((41, 200)) * 2) / 2).astype(np.float32), 16
        lg[3] = 0.0
        lg[7, 150:] = 9.0
    elif case == "E100_k3_T17":     # sixteen-lane kernel with 8 logits per lane, T not a multiple of 16
        lg, k = g.standard_normal((17, 100)).astype(np.float32), 3
    elif case.startswith("masked"):   # -inf logits (masked experts), fewer finite ones than k
        E = 256 if case == "masked_E256_k8" else 300
        lg, k = g.standard_normal((33, E)).astype(np.float32), 8
        lg[g.random((33, E)) < 0.9] = -np.inf
        lg[:, 5] = 0.25                 # at least one finite logit per row
        lg[4, :] = -np.inf
        lg[4, [17, 200]] = [1.0, 1.0]   # two finite ones: six slots take -inf experts
    elif case.startswith("loop"):   # more tokens than one pass of the persistent grid covers
        E, T = (int(v) for v in case[6:].split("_T"))   # (several groups per workgroup, ragged tail)
        lg, k = g.standard_normal((T, E)).astype(np.float32), 8 if E > 64 else 4
        lg[T - 1] = 0.0                  # an all-tie row in the last group
    else:
        lg, k, renorm = synth.uniform_logits(0, 2, 200, 64), 6, 1
    idx, w = _route_gpu(lg, k, renorm)
    ridx, rw = oep.route_topk_softmax(lg, k, renormalize=bool(renorm))
    assert np.array_equal(idx, ridx)
    assert np.allclose(w, rw, rtol=W_RTOL, atol=0)


def _layout_gpu(idx, E, W, cap):
    X = xs()
    n_src, T, k = idx.shape
    d = "cuda"
    tidx = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(d)
    out = {n: torch.full(sh, -7, dtype=torch.int32, device=d) for n, sh in
           [("expert_counts", (n_src, E)), ("src_base", (n_src, E)), ("expert_offsets", (E,)),
            ("dest_counts", (W,)), ("slot_row", (n_src, T, k)), ("row_src", (W, cap))]}
    nb = C.c_int64()
    X.check(X.xs_dispatch_layout_workspace_bytes(n_src, T, E, C.byref(nb)))
    ws = torch.empty((nb.value,), dtype=torch.uint8, device=d)
    st = torch.zeros((1,), dtype=torch.int32, device=d)
    X.check(X.xs_dispatch_layout(tidx.data_ptr(), n_src, T, k, E, W, cap, out["expert_counts"].data_ptr(),
                                 out["src_base"].data_ptr(), out["expert_offsets"].data_ptr(),
                                 out["dest_counts"].data_ptr(), out["slot_row"].data_ptr(),
                                 out["row_src"].data_ptr(), ws.data_ptr(), nb.value, st.data_ptr(),
                                 torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    res = {n: v.cpu().numpy() for n, v in out.items()}
    res["status"] = int(st.item())
    return res


def _idx_random(n_src, T, k, E, seed):
    g = np.random.default_rng(seed)
    return np.argsort(g.random((n_src, T, E)), axis=2)[:, :, :k].astype(np.int32)


@pytest.mark.parametrize("n_src,T,k,E,W", [(1, 256, 2, 8, 4), (3, 300, 3, 12, 3), (8, 4096, 8, 256, 8),
                                           (2, 1, 1, 4, 2), (1, 257, 8, 1024, 64)])
def test_layout_matches_oracle(n_src, T, k, E, W):
    idx = _idx_random(n_src, T, k, E, seed=T + E)
    cap = n_src * T * k
    got = _layout_gpu(idx, E, W, cap)
    ref = oep.dispatch_layout(idx, E, W, cap)
    assert got["status"] == 0
    for n in ("expert_counts", "src_base", "expert_offsets", "dest_counts", "slot_row"):
        assert np.array_equal(got[n], ref[n]), n
    for d in range(W):
        nrow = ref["dest_counts"][d]
        assert np.array_equal(got["row_src"][d, :nrow], ref["row_src"][d]), d


def test_layout_from_routed_zipf_multi_source():
    cfg = synth.EP_DSV3_SHARE
    idx = np.stack([oep.route_topk_softmax(synth.zipf_logits(0, s, cfg.T, cfg.E), cfg.k)[0]
                    for s in range(cfg.n_src)])
    cap = cfg.n_src * cfg.T * cfg.k
    got = _layout_gpu(idx, cfg.E, cfg.W, cap)
    ref = oep.dispatch_layout(idx, cfg.E, cfg.W, cap)
    for n in ("expert_counts", "src_base", "expert_offsets", "dest_counts", "slot_row"):
        assert np.array_equal(got[n], ref[n]), n


def test_layout_capacity_and_bad_expert_status():
    idx = _idx_random(1, 64, 2, 4, seed=3)
    got = _layout_gpu(idx, 4, 2, cap=10)
    assert got["status"] == xs().XS_ECAPACITY
    ref = oep.dispatch_layout(idx, 4, 2, cap=10)
    assert np.array_equal(got["slot_row"], ref["slot_row"])      # rows stay defined past capacity
    bad = idx.copy()
    bad[0, 5, 1] = 9
    assert _layout_gpu(bad, 4, 2, cap=128)["status"] == xs().XS_EBADINPUT
    dup = idx.copy()
    dup[0, 7, 1] = dup[0, 7, 0]         # one token lists an expert twice
    assert oep.dispatch_layout(dup, 4, 2, cap=128)["status"] == xs().XS_EBADINPUT
    assert _layout_gpu(dup, 4, 2, cap=128)["status"] == xs().XS_EBADINPUT


def _ep_layer(cfg, seed=0, **kw):
    from paper_2607_23264_amd.layer import EPLayer, Shape
    experts = synth.computed_experts(cfg)
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=cfg.rank,
              **kw)
    return EPLayer(s)


def test_dispatch_bitexact_and_sentinel():
    cfg = synth.EPConfig("t", T=300, H=264, E=16, k=3, I=128, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 5, with_weights=False)
    lay = _ep_layer(cfg, expert_mode=1)
    lay.upload(inp["logits"], inp["x"])
    lay.route()
    lay.layout()
    for s in range(cfg.n_src):
        lay.dispatch(s)
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    idx = np.stack([oep.route_topk_softmax(inp["logits"][s], cfg.k)[0] for s in range(cfg.n_src)])
    ref = oep.dispatch_layout(idx, cfg.E, cfg.W, lay.cap)
    win, st = oep.dispatch(inp["x"], idx, ref["slot_row"], cfg.E, cfg.W, lay.cap)
    assert np.array_equal(host_bits(lay.dwin), win)


def test_dispatch_capacity_overflow_skips_rows():
    X = xs()
    T, H, k, E, W = 64, 64, 2, 4, 2
    idx = _idx_random(1, T, k, E, seed=9)[0]
    lay = oep.dispatch_layout(idx[None], E, W)
    cap = 20
    x = synth.normal_bf16(0, 1, (T, H))
    win = torch.full((W, cap, H), -1, dtype=torch.int16, device="cuda")
    wins = X.windows([X.window(win[d]) for d in range(W)])
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    ti = torch.from_numpy(idx).cuda()
    sr = torch.from_numpy(lay["slot_row"][0]).cuda()
    X.check(X.xs_dispatch(dev_bits(x).data_ptr(), T, H, ti.data_ptr(), sr.data_ptr(), k, E, wins, W,
                          st.data_ptr(), torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert int(st.item()) == X.XS_ECAPACITY
    ref, _ = oep.dispatch(x[None], idx[None], lay["slot_row"], E, W, cap)
    assert np.array_equal(host_bits(win), ref)


def test_combine_reduce_matches_oracle():
    X = xs()
    g = np.random.default_rng(4)
    for T, k, H in [(256, 2, 512), (97, 8, 7168), (5, 1, 8)]:
        c = synth.normal_bf16(0, 9, (T * k, H))
        w = g.random((T, k)).astype(np.float32)
        out = torch.empty((T, H), dtype=torch.int16, device="cuda")
        ct = dev_bits(c)
        wt = torch.from_numpy(w).cuda()
        X.check(X.xs_combine_reduce(ct.data_ptr(), H * 2, wt.data_ptr(), T, k, H, out.data_ptr(),
                                    torch.cuda.current_stream().cuda_stream))
        torch.cuda.synchronize()
        ref64, _ = oep.combine_reduce(c, w)
        assert_close(host_bits(out), ref64, f"combine T={T} k={k} H={H}")


def _policies():
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    return {"burst": pacing(X.XS_POLICY_BURST), "interleave_D1": pacing(X.XS_POLICY_INTERLEAVE, lead=1),
            "interleave_D3": pacing(X.XS_POLICY_INTERLEAVE, lead=3),
            "chunk1": pacing(X.XS_POLICY_CHUNK, lead=1, chunk=1),
            "chunk2_p8": pacing(X.XS_POLICY_CHUNK, lead=2, chunk=2, max_producers=8),
            "auto_nomodel": pacing(X.XS_POLICY_AUTO), "burst_p16_w4": pacing(X.XS_POLICY_BURST, max_producers=16,
                                                                              wave_tiles=4),
            "interleave_dyn": pacing(X.XS_POLICY_INTERLEAVE, lead=1, claim=X.XS_CLAIM_DYNAMIC),
            "chunk2_p8_dyn": pacing(X.XS_POLICY_CHUNK, lead=2, chunk=2, max_producers=8, claim=X.XS_CLAIM_DYNAMIC),
            "burst_w4_dyn": pacing(X.XS_POLICY_BURST, wave_tiles=4, claim=X.XS_CLAIM_DYNAMIC)}


def test_tiny_layer_all_policies_match_oracle_and_each_other():
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    ref = oep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k)
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    outs = {}
    for name, p in _policies().items():
        lay.out.zero_()
        lay.cwin.fill_(-1)
        lay.fused(p)
        torch.cuda.synchronize()
        assert int(lay.status.item()) == 0, name
        outs[name] = host_bits(lay.out)
        assert_close(outs[name], ref["out64"], f"tiny layer {name}")
    lay.out.zero_()
    lay.unfused()
    torch.cuda.synchronize()
    outs["unfused"] = host_bits(lay.out)
    first = next(iter(outs.values()))
    for name, o in outs.items():
        assert np.array_equal(o, first), f"policy {name} changed the output bits"
    # expert outputs of the unfused path against the oracle, row by row
    y = host_bits(lay.y_ws)
    base = 0
    for d in range(cfg.W):
        n = int(ref["layout"]["dest_counts"][d])
        assert_close(y[base:base + n], ref["y"][d][0], f"expert outputs window {d}")
        base += n
    # the layout the kernels used is the oracle's, bit for bit
    assert np.array_equal(lay.slot_row.cpu().numpy(), ref["layout"]["slot_row"])
    assert np.array_equal(lay.topk_idx.cpu().numpy(), ref["idx"])


def test_identity_experts_return_input_scaled_by_gate_sum():
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 1, with_weights=False)
    lay = _ep_layer(cfg, expert_mode=1)
    lay.upload(inp["logits"], inp["x"])
    lay.fused(None)
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    ref = oep.ep_layer(inp["x"], inp["logits"], None, None, cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k,
                       identity=True)
    x = bits_f64(inp["x"][0])
    wsum = ref["w"][0].astype(np.float64).sum(1, keepdims=True)
    got = bits_f64(host_bits(lay.out))
    assert np.all(np.abs(got - x * wsum) <= 2.0 ** -8 * np.abs(x * wsum) + 1e-30)
    # every (token, slot) lands exactly once: the combine buffer holds x row t at t*k+j
    assert np.array_equal(host_bits(lay.cwin[0]).reshape(cfg.T, cfg.k, cfg.H),
                          np.repeat(inp["x"][0][:, None, :], cfg.k, axis=1))


def test_multi_source_ragged_share():
    # 3 sources, this GPU = rank 1 owning experts 4..7; T not a multiple of 256 or 64
    cfg = synth.EPConfig("t", T=300, H=256, E=16, k=3, I=256, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 7)
    experts = synth.computed_experts(cfg)
    fill = synth.normal_bf16(0, 200, (cfg.T * cfg.k, cfg.H))
    ref = oep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W,
                       cap=cfg.n_src * cfg.T * cfg.k, experts=experts, combine_fill=fill, out_src=cfg.rank)
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(fill)
    from paper_2607_23264_amd.layer import pacing
    lay.fused(pacing(xs().XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    assert_close(host_bits(lay.out), ref["out64"], "ragged share output")
    # combine windows of every source: computed rows within tolerance, the rest untouched
    comb = host_bits(lay.cwin)
    for s in range(cfg.n_src):
        for t in range(cfg.T):
            for j in range(cfg.k):
                e = ref["idx"][s, t, j]
                row = comb[s, t * cfg.k + j]
                if e in experts:
                    d = e // (cfg.E // cfg.W)
                    r = ref["layout"]["slot_row"][s, t, j]
                    assert_close(row, ref["y"][d][0][r], "combine row")
                elif s != cfg.rank:
                    assert np.all(row == 0xFFFF)


def _records(buf, count):
    n = min(int(count.item()), buf.shape[0])
    r = buf[:n].cpu().numpy().astype(np.uint64)
    kind = (r[:, 0] >> np.uint64(56)).astype(np.int64)
    wg = ((r[:, 0] >> np.uint64(32)) & np.uint64(0xFFFFFF)).astype(np.int64)
    tile = (r[:, 0] & np.uint64(0xFFFFFFFF)).astype(np.int64)
    return kind, wg, tile, r


@pytest.mark.parametrize("policy", ["interleave", "chunk", "wave"])
def test_device_tile_order_matches_schedule_oracle(policy):
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    G = 8
    pol = {"interleave": pacing(X.XS_POLICY_INTERLEAVE, lead=2, max_producers=G),
           "chunk": pacing(X.XS_POLICY_CHUNK, lead=1, chunk=1, max_producers=G),
           "wave": pacing(X.XS_POLICY_BURST, max_producers=G, wave_tiles=16)}[policy]
    buf = torch.zeros((4096, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
    tr = X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr())
    lay.fused(pol, tr)
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    kind, wg, tile, _ = _records(buf, cnt)
    idx = np.stack([oep.route_topk_softmax(inp["logits"][0], cfg.k)[0]])
    counts = oep.dispatch_layout(idx, cfg.E, cfg.W)["expert_counts"].sum(0)
    mt = [(int(c) + 255) // 256 for c in counts]
    row_expert = [e for e in range(cfg.E) for _ in range(mt[e])]
    P, P1, P2 = len(row_expert), cfg.I // 128, cfg.H // 256
    if policy == "interleave":
        streams = osc.all_streams("interleave", G, P, P1, P2, D=2)
    elif policy == "chunk":
        streams = osc.all_streams("chunk", G, P, P1, P2, D=1, chunk=1)
    else:
        streams = osc.all_streams("wave", G, P, P1, P2, waves=osc.waves_by_tiles(row_expert, P1, 16))
    for b in range(G):
        got = [(int(kk), int(tt)) for kk, ww, tt in zip(kind, wg, tile) if ww == b]
        exp = [(kk, tt) for kk, _, tt in streams[b]]
        assert got == exp, f"workgroup {b}"


@pytest.mark.parametrize("policy", ["interleave", "chunk", "burst"])
def test_dynamic_claim_takes_every_tile_once_after_its_dependencies(policy):
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    lay = _ep_layer(cfg)
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
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1, withhold_row=0, spin_timeout_us=2000, claim=claim))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == X.XS_ETIMEOUT
    # the library never clears the status; a clean run after a reset reports ok again
    lay.status.zero_()
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0


def test_bad_arguments_rejected_synchronously():
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EP_TINY
    lay = _ep_layer(cfg)
    p = pacing(X.XS_POLICY_INTERLEAVE)
    p.policy = 9
    assert X.xs_fused_ep_layer(C.byref(lay.L), C.byref(p), None, lay.workspace.data_ptr(),
                               lay.workspace.numel(), lay.status.data_ptr(), None) == X.XS_EINVAL
    for field, value in (("claim", 2), ("reserved", 1), ("lead_rows", -1)):
        p = pacing(X.XS_POLICY_INTERLEAVE)
        setattr(p, field, value)
        assert X.xs_fused_ep_layer(C.byref(lay.L), C.byref(p), None, lay.workspace.data_ptr(),
                                   lay.workspace.numel(), lay.status.data_ptr(), None) == X.XS_EINVAL, field
    assert X.xs_fused_ep_layer(C.byref(lay.L), None, None, lay.workspace.data_ptr(), 16,
                               lay.status.data_ptr(), None) == X.XS_EWORKSPACE
    assert X.xs_route_topk_softmax(lay.logits.data_ptr(), 4, 8, 9, 0, lay.topk_idx.data_ptr(),
                                   lay.topk_w.data_ptr(), None) == X.XS_EINVAL


SKEWED = synth.EPConfig("skewed_T2048_H2048_E8_k2_I512_W4", T=2048, H=2048, E=8, k=2, I=512, W=4, n_src=1,
                        rank=0, compute_all=True, routing="zipf")


@pytest.mark.parametrize("D,Q,want", [(1, 1e6, "interleave"), (1, float("inf"), "interleave"), (4, 3e6, "wave")])
def test_auto_follows_the_audited_choice(D, Q, want):
    """AUTO with a model: the library audits every candidate order and runs the one with the least
    predicted stall; the traced tile order of every workgroup equals the schedule oracle's stream
    of the order the oracle's own audit picks."""
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = SKEWED
    inp = synth.ep_inputs(cfg, 0)
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    idx = oep.route_topk_softmax(inp["logits"][0], cfg.k)[0]
    counts = [int(c) for c in np.bincount(idx.ravel(), minlength=cfg.E)]
    G, tl1, tl2 = 8, 20.0, 10.0
    a, b, R = 1.0, 1e-7, 30000.0
    P1, P2 = cfg.I // 128, cfg.H // 256
    choice, _ = osc.pacing_audit(counts, True, P1, P2, G, D, G, 1.0, tl1, tl2, a, b, R, Q)
    assert choice[0] == want
    m = X.xs_model(a, b, R, Q, G, 0)
    pol = pacing(X.XS_POLICY_AUTO, lead=D, max_producers=G, model=m, t_l1_us=tl1, t_l2_us=tl2,
                 expert_rows=counts)
    buf = torch.zeros((8192, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
    lay.fused(pol, X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr()))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    kind, wg, tile, _ = _records(buf, cnt)
    sizes, owner = osc.expert_blocks(counts, True)
    P = len(sizes)
    if want == "wave":
        streams = osc.all_streams("wave", G, P, P1, P2, waves=osc.waves_by_tiles(owner, P1, G))
    else:
        streams = osc.all_streams("interleave", G, P, P1, P2, D=D)
    for g in range(G):
        got = [(int(kk), int(tt)) for kk, ww, tt in zip(kind, wg, tile) if ww == g]
        assert got == [(kk, tt) for kk, _, tt in streams[g]], f"workgroup {g}"
    ref = oep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k)
    assert_close(host_bits(lay.out), ref["out64"], f"skewed layer under AUTO ({want})")


def test_trace_ext_records_and_tile_times():
    """The ext trace records: dependency-wait end, staging wait, stored bytes and rows of every
    tile, consistent with the main records; and the library's tile-time medians of that trace."""
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = SKEWED
    inp = synth.ep_inputs(cfg, 0)
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    buf = torch.zeros((8192, 4), dtype=torch.int64, device="cuda")
    ext = torch.zeros((8192, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1, claim=X.XS_CLAIM_DYNAMIC),
              X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr(), ext.data_ptr()))
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    n = int(cnt.item())
    r = buf[:n].cpu().numpy().astype(np.uint64)
    x = ext[:n].cpu().numpy().astype(np.uint64)
    kind = (r[:, 0] >> np.uint64(56)).astype(np.int64)
    idx = oep.route_topk_softmax(inp["logits"][0], cfg.k)[0]
    sizes, _ = osc.expert_blocks(np.bincount(idx.ravel(), minlength=cfg.E), True)
    P1, P2 = cfg.I // 128, cfg.H // 256
    assert (kind == 1).sum() == len(sizes) * P1 and (kind == 2).sum() == len(sizes) * P2
    tile = (r[:, 0] & np.uint64(0xFFFFFFFF)).astype(np.int64)
    sz = np.array(sizes)
    rows = np.empty(n, np.int64)
    rows[kind == 1] = sz[tile[kind == 1] // P1]
    rows[kind == 2] = sz[tile[kind == 2] // P2]
    assert np.array_equal(x[:, 3].astype(np.int64), rows)
    assert np.array_equal(x[kind == 2, 2].astype(np.int64), rows[kind == 2] * 256 * 2)
    assert np.array_equal(x[kind == 1, 2].astype(np.int64), rows[kind == 1] * 128 * 2)
    assert np.all(x[kind == 1, 0] == r[kind == 1, 1])
    assert np.all((x[kind == 2, 0] >= r[kind == 2, 1]) & (x[kind == 2, 0] <= r[kind == 2, 2]))
    assert np.all(x[:, 1] <= r[:, 2] - r[:, 1])       # the staging wait lies inside the tile
    t1, t2, t3 = C.c_double(), C.c_double(), C.c_double()
    rc = np.ascontiguousarray(r)
    xc = np.ascontiguousarray(x)
    X.check(X.xs_trace_tile_times(rc.ctypes.data, xc.ctypes.data, n, 0, C.byref(t1), C.byref(t2), C.byref(t3)))
    us = 1e6 / X.xs_clock_rate_hz()
    assert t1.value == pytest.approx(np.median((r[kind == 1, 2] - r[kind == 1, 1]).astype(np.float64)) * us)
    assert t2.value == pytest.approx(np.median((r[kind == 2, 2] - x[kind == 2, 0]).astype(np.float64)) * us)
    assert t1.value > 0 and t2.value > 0 and t3.value > 0


def test_combine_send_pacing_stores_the_same_rows():
    """The unfused combine-send under pacing settings (producer caps, bursts of row blocks, gaps)
    writes the same combine windows as the fused layer, whose rows match the oracle."""
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    cfg = synth.EPConfig("t", T=300, H=256, E=16, k=3, I=256, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 7)
    experts = synth.computed_experts(cfg)
    ref = oep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W,
                       cap=cfg.n_src * cfg.T * cfg.k, experts=experts, out_src=cfg.rank)
    lay = _ep_layer(cfg)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources()
    lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=1))
    torch.cuda.synchronize()
    fused = host_bits(lay.cwin)
    own = (ref["idx"] // (cfg.E // cfg.W) == cfg.rank).reshape(cfg.n_src, -1)
    assert_close(fused[own], bits_f64(ref["combine"][own]), "fused combine rows")
    lay.expert_ffn()
    for p in (None, pacing(X.XS_POLICY_BURST, max_producers=3, chunk=1),
              pacing(X.XS_POLICY_BURST, max_producers=1, gap_ns=2000), pacing(X.XS_POLICY_BURST, chunk=2)):
        lay.cwin.fill_(-1)
        lay.combine_send(p)
        torch.cuda.synchronize()
        assert int(lay.status.item()) == 0
        assert np.array_equal(host_bits(lay.cwin), np.where(own[..., None], fused, np.uint16(0xFFFF)))
    bad = pacing(X.XS_POLICY_BURST, gap_ns=-5)
    assert X.xs_combine_send(C.byref(lay.L), C.byref(bad), lay.status.data_ptr(), lay.stream) == X.XS_EINVAL
