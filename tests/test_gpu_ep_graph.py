"""The fused EP layer captured once in a HIP graph and replayed: each call is a plain sequence of
stream-ordered kernel launches (no host synchronisation, no memset, no allocation), so a replay
must reproduce the eager call's output bit for bit. The graph is replayed several times, with
eager work and synchronisations between replays, and every replay is checked."""
import numpy as np
import pytest
import torch

import synth
from gpu_helpers import host_bits, require_gpu, xs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)


@pytest.mark.parametrize("prec_name", ["BF16", "MXFP8"])
def test_fused_layer_graph_replays_equal_eager(prec_name):
    from paper_2607_23264_amd.layer import EPLayer, Shape, pacing
    X = xs()
    cfg = synth.EPConfig("g", T=300, H=512, E=16, k=3, I=512, W=4, n_src=3, rank=1)
    inp = synth.ep_inputs(cfg, 5)
    experts = synth.computed_experts(cfg)
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=cfg.rank)
    lay = EPLayer(s, sentinel=False, precision=getattr(X, f"XS_PREC_{prec_name}"))
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(synth.normal_bf16(0, 200, (cfg.T * cfg.k, cfg.H)))
    pol = pacing(X.XS_POLICY_INTERLEAVE, lead=1, claim=X.XS_CLAIM_DYNAMIC)
    for i in range(8):
        lay.L.events[i] = None
    lay.fused(pol)
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    want = host_bits(lay.out)
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        lay.fused(pol)            # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        lay.fused(pol)
    torch.cuda.synchronize()
    for rep in range(4):
        lay.out.fill_(0)
        lay.fused(pol)            # eager work between replays
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(lay.out), want), f"eager call {rep}"
        lay.out.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        assert int(lay.status.item()) == 0
        assert np.array_equal(host_bits(lay.out), want), f"replay {rep}"
