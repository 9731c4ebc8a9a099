"""The fused EP layer's no-alloc entry point (a library-owned scratch array per GPU) against the
workspace entry point, through the C ABI: two calls in a row, the second on a smaller layer, each
bit for bit equal to xs_fused_ep_layer on the same inputs (which the other tests hold to the
oracle), and the size limit."""
import ctypes as C

import numpy as np
import pytest
import torch

import synth
from gpu_helpers import assert_close, host_bits, require_gpu, xs
from oracle import ep as oep

pytestmark = pytest.mark.gpu


def _layer(cfg, precision=0):
    from paper_2607_23264_amd.layer import EPLayer, Shape
    experts = synth.computed_experts(cfg)
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=cfg.rank)
    lay = EPLayer(s, precision=precision)
    inp = synth.ep_inputs(cfg, 3)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    if cfg.n_src > 1:
        lay.prefill_other_sources()
    return lay, inp


def _run_both(cfg, precision, pol):
    X = xs()
    lay, inp = _layer(cfg, precision)
    lay.fused(pol)
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    want_out, want_comb = host_bits(lay.out), host_bits(lay.cwin)
    lay.out.zero_()
    lay.cwin.fill_(-1)
    if cfg.n_src > 1:
        lay.prefill_other_sources()
    rc = X.xs_fused_ep_layer_noalloc(C.byref(lay.L), C.byref(pol), None, lay.status.data_ptr(), lay.stream)
    assert rc == X.XS_OK, X.xs_strerror(rc)
    torch.cuda.synchronize()
    assert int(lay.status.item()) == 0
    assert np.array_equal(host_bits(lay.out), want_out)
    assert np.array_equal(host_bits(lay.cwin), want_comb)
    return lay, inp


def test_no_alloc_layer_equals_workspace_layer_on_two_calls():
    require_gpu()
    torch.cuda.set_device(0)
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    pol = pacing(X.XS_POLICY_INTERLEAVE, lead=2, claim=X.XS_CLAIM_DYNAMIC)
    big = synth.EPConfig("t", T=1100, H=512, E=16, k=4, I=512, W=4, n_src=2, rank=1)
    _run_both(big, X.XS_PREC_MXFP8, pol)
    lay, inp = _run_both(synth.EP_TINY, X.XS_PREC_BF16, pol)
    # the second, smaller call still matches the oracle (nothing stale from the first)
    cfg = synth.EP_TINY
    ref = oep.ep_layer(inp["x"], inp["logits"], inp["w1"], inp["w2"], cfg.k, cfg.E, cfg.W, cap=cfg.T * cfg.k)
    assert_close(host_bits(lay.out), ref["out64"], "tiny layer through the no-alloc entry point")


def test_no_alloc_rejects_layers_beyond_the_scratch():
    require_gpu()
    X = xs()
    L = X.xs_ep_layer()
    L.n_src, L.T, L.H, L.E, L.k, L.I, L.W = 1, 8192, 8192, 8, 2, 512, 4
    L.e_begin, L.n_experts, L.cap, L.precision = 0, 8, 8192 * 2, X.XS_PREC_MXFP8
    nb = C.c_int64()
    X.check(X.xs_ep_layer_workspace_bytes(C.byref(L), C.byref(nb)))
    assert nb.value > X.XS_STATIC_SCRATCH_BYTES
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    assert X.xs_fused_ep_layer_noalloc(C.byref(L), None, None, st.data_ptr(), None) == X.XS_EWORKSPACE
    torch.cuda.synchronize()
    assert int(st.item()) == 0
