"""Full-size parity of one rank's DeepSeek-V3-like EP share (8 sources x 4096 tokens, H = 7168,
32 of 256 experts local, top-8, SwiGLU I = 2048, 8 windows) at bf16, MXFP8 (W8A8) and W4A8,
with uniform and Zipf(1.2) routing, under the benchmark's pacing (Alg. 1 interleave at a lead
of 64 rows, dynamic claiming), through the C ABI, against the CPU oracle:
  * routing indices (bit-exact) and weights, every layout table bit-exact;
  * every row of every dispatch window bit-exact (bf16 copies, or the oracle's MX codes and
    scales of the token row);
  * every computed row of all 8 combine windows within the tolerance of the oracle's value
    before rounding, every other row untouched (sentinel) or the pre-filled remote rows;
  * the whole combined output of this rank within tolerance;
  * the ready flags of every dispatch and combine window set.
The oracle runs expert by expert, which bounds its host memory."""
import concurrent.futures as cf
import dataclasses
import gc

import numpy as np
import pytest
import torch

import synth
from oracle import ep as oep
from oracle import ep_mx as omx
from oracle import mx as omxf
from gpu_helpers import (assert_close, bits_f64, check_h_admissible, h_codes_scales, host_bits, mx_h_admissible,
                         mx_y_slack, require_gpu, xs)

pytestmark = pytest.mark.gpu

W_RTOL = 2e-6
BENCH_LEAD = 64          # the benchmark's lead D in rows (four anti-starvation knees)

_cache = {}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)
    yield
    _cache.clear()


def _share(routing):
    """Inputs and the oracle's routing and layout of the share (cached per routing)."""
    if routing in _cache:
        return _cache[routing]
    _cache.clear()
    gc.collect()
    cfg = dataclasses.replace(synth.EP_DSV3_SHARE, routing=routing)
    logits = synth.ep_logits(cfg, 0)
    idx = np.empty((cfg.n_src, cfg.T, cfg.k), np.int32)
    w = np.empty((cfg.n_src, cfg.T, cfg.k), np.float32)
    for s in range(cfg.n_src):
        idx[s], w[s] = oep.route_topk_softmax(logits[s], cfg.k)
    if routing == "zipf":
        # "this GPU" is the most loaded destination (the max across ranks)
        loads = np.bincount((idx // cfg.E_local).ravel(), minlength=cfg.W)
        cfg = dataclasses.replace(cfg, rank=int(loads.argmax()))
    experts = synth.computed_experts(cfg)
    w1, w2 = synth.ep_weights(cfg, experts, 0)
    d = {"cfg": cfg, "logits": logits, "x": synth.ep_x(cfg, 0), "w1": w1, "w2": w2, "idx": idx, "w": w,
         "experts": experts, "fill": synth.ep_remote_combine_fill(cfg, 0),
         "layout": oep.dispatch_layout(idx, cfg.E, cfg.W)}
    _cache[routing] = d
    return d


CASES = [("uniform", "BF16"), ("uniform", "MXFP8"), ("uniform", "W4A8"),
         ("zipf", "BF16"), ("zipf", "MXFP8"), ("zipf", "W4A8")]


@pytest.mark.parametrize("routing,prec", CASES)
def test_dsv3_share_every_row_at_bench_pacing(routing, prec):
    from paper_2607_23264_amd.layer import EPLayer, Shape, pacing
    X = xs()
    ref = _share(routing)
    cfg, experts, lref = ref["cfg"], ref["experts"], ref["layout"]
    r, k, H, epw = cfg.rank, cfg.k, cfg.H, cfg.E_local
    mx = prec != "BF16"
    wfmt = omxf.E2M1 if prec == "W4A8" else omxf.E4M3
    s = Shape(cfg.n_src, cfg.T, H, cfg.E, k, cfg.I, cfg.W, experts[0], len(experts), src=r)
    print(f"[full-size] {routing} {prec}: rank {r}, {int(ref['layout']['dest_counts'][r])} rows", flush=True)
    lay = EPLayer(s, precision=getattr(X, f"XS_PREC_{prec}"), ready_flags=True)
    try:
        lay.upload(ref["logits"], ref["x"], ref["w1"], ref["w2"])
        lay.prefill_other_sources(ref["fill"])
        lay.flags.zero_()
        lay.fused(pacing(X.XS_POLICY_INTERLEAVE, lead=BENCH_LEAD, claim=X.XS_CLAIM_DYNAMIC))
        torch.cuda.synchronize()
        assert int(lay.status.item()) == 0
        # every window signalled ready after its last store
        assert lay.flags.cpu().numpy().tolist() == [1] * (cfg.W + cfg.n_src)
        # routing of every source and the layout tables, bit for bit
        assert np.array_equal(lay.topk_idx.cpu().numpy(), ref["idx"])
        assert np.allclose(lay.topk_w.cpu().numpy(), ref["w"], rtol=W_RTOL, atol=0)
        for name in ("expert_counts", "src_base", "expert_offsets", "dest_counts", "slot_row"):
            assert np.array_equal(getattr(lay, name).cpu().numpy(), lref[name]), name
        dc = lref["dest_counts"]
        xq = omx.quantize_rows(ref["x"]) if mx else None      # the oracle's MXFP8 token rows
        # every dispatch window row: the token row of its (source, token)
        for d in range(cfg.W):
            n = int(dc[d])
            assert np.array_equal(lay.row_src[d, :n].cpu().numpy(), lref["row_src"][d]), d
            src, slot = oep.decode_row_src(lref["row_src"][d])
            got = lay.dwin[d, :n].cpu().numpy()
            if mx:
                assert np.array_equal(got[:, :H], xq[0][src, slot // k]), f"window {d} codes"
                assert np.array_equal(got[:, H:H + H // 32], xq[1][src, slot // k]), f"window {d} scales"
            else:
                assert np.array_equal(got.view(np.uint16), ref["x"][src, slot // k]), f"window {d}"
            del got
        print(f"[full-size] {routing} {prec}: dispatch windows bit-exact", flush=True)
        # every computed row of every combine window, expert by expert
        comb = host_bits(lay.cwin)
        own = (ref["idx"] // epw == r).reshape(cfg.n_src, cfg.T * k)
        comb_r = ref["fill"].copy()             # this rank's combine buffer as the oracle fills it
        slack_r = np.zeros(comb_r.shape, np.float32) if mx else None
        total = lref["expert_counts"].sum(0)
        if mx:
            gh_codes, gh_scales = h_codes_scales(lay, cfg.I)    # the GPU's h rows (window r first)
            flips = 0
        def check_expert(i, e):
            """The oracle's rows of one local expert against the GPU's combine rows (and, in the MX
            precisions, the GPU's h rows against the fp32 bound). Returns (slots of this rank,
            y bits there, their slack, h codes that differ)."""
            r0 = int(lref["expert_offsets"][e])
            r1 = r0 + int(total[e])
            if r1 == r0:
                return None
            src, slot = oep.decode_row_src(lref["row_src"][r][r0:r1])
            mine = src == r
            nflip, slack = 0, None
            if mx:
                w1q = omx.quantize_rows(ref["w1"][i], wfmt)
                w2q = omx.quantize_rows(ref["w2"][i], wfmt)
                xr = (xq[0][src, slot // k], xq[1][src, slot // k])
                hc, hs, y64, yb = omx.expert_ffn_mx(xr, w1q, w2q, wfmt)
                # h codes decided in fp32 may differ from the oracle's within the fp32 bound;
                # y then gets the matching allowance (reading 39)
                adm = mx_h_admissible(xr, w1q, wfmt)
                nflip = check_h_admissible(gh_codes[r0:r1], gh_scales[r0:r1], adm, f"h of expert {e}")
                slack = mx_y_slack(adm, w2q, wfmt, hc, hs)
                del adm
            else:
                _, y64, yb = oep.expert_ffn(ref["x"][src, slot // k], ref["w1"][i], ref["w2"][i])
            assert_close(comb[src, slot], y64, f"{prec} {routing} expert {e} combine rows", slack)
            return slot[mine], yb[mine], (slack[mine] if mx else None), nflip

        # experts are checked concurrently (their element-wise steps release the interpreter lock)
        with cf.ThreadPoolExecutor(4) as pool:
            for res in pool.map(lambda ie: check_expert(*ie), list(enumerate(experts))):
                if res is None:
                    continue
                sl, yb, sk, nflip = res
                comb_r[sl] = yb
                if mx:
                    slack_r[sl] = sk
                    flips += nflip
        for q in range(cfg.n_src):
            if q != r:
                assert (comb[q][~own[q]] == 0xFFFF).all(), f"combine window {q}: rows of other ranks touched"
        assert np.array_equal(comb[r][~own[r]], ref["fill"][~own[r]])
        del comb
        print(f"[full-size] {routing} {prec}: combine windows within tolerance", flush=True)
        out64, _ = oep.combine_reduce(comb_r, ref["w"][r])
        out_slack = None
        if mx:
            print(f"[full-size] {routing} {prec}: {flips} h codes differ from the oracle's, all within "
                  f"the fp32 bound", flush=True)
            wr = ref["w"][r].astype(np.float64)
            out_slack = np.einsum("tj,tjh->th", wr, slack_r.reshape(cfg.T, k, H).astype(np.float64))
        assert_close(host_bits(lay.out), out64, f"{prec} {routing} output", out_slack)
        # other orders store the same bits: Expert-Wave burst and static cursors at the knee
        out0, cw0 = lay.out.clone(), lay.cwin.clone()
        for pol in (pacing(X.XS_POLICY_BURST, claim=X.XS_CLAIM_DYNAMIC), pacing(X.XS_POLICY_INTERLEAVE, lead=0)):
            lay.out.zero_()
            lay.cwin.fill_(-1)
            lay.prefill_other_sources(ref["fill"])
            lay.fused(pol)
            torch.cuda.synchronize()
            assert int(lay.status.item()) == 0
            assert torch.equal(lay.out, out0) and torch.equal(lay.cwin, cw0), f"policy {pol.policy} changed bits"
        del out0, cw0
    finally:
        lay.close()
        del lay
        torch.cuda.empty_cache()
