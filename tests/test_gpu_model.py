"""The library's Burst-Gap model (C++) against the oracle's, and the remote-store
microbenchmark kernel on an HBM window and a host-coherent sink."""
import ctypes as C

import numpy as np
import pytest
import torch

from oracle import xstage_model as oxm
from gpu_helpers import require_gpu, xs

pytestmark = pytest.mark.gpu


def _arr(v):
    v = np.ascontiguousarray(v, dtype=np.float64)
    return v, v.ctypes.data_as(C.POINTER(C.c_double))


def test_model_predict_matches_oracle():
    X = xs()
    g = np.random.default_rng(0)
    for trial in range(50):
        n = int(g.integers(1, 60))
        V = g.uniform(0, 8e6, n)
        T0 = g.uniform(0.2, 3.0, n)
        G = g.uniform(0, 10, n) * (g.random(n) < 0.7)
        R, Q, q0 = float(g.uniform(100, 2000)), float(g.uniform(1e5, 6e6)), float(g.uniform(0, 1e6) * (trial % 2))
        bursts = (X.xs_burst * n)(*[X.xs_burst(V[i], T0[i], G[i]) for i in range(n)])
        out = (X.xs_burst_pred * n)()
        m = X.xs_model(0.0, 0.0, R, Q, 148, 0)
        X.check(X.xs_model_predict(C.byref(m), bursts, n, q0, out))
        ref = oxm.predict(V, T0, G, R, Q, q0)
        for o, r in zip(out, ref):
            for f in ("rho", "delta_b", "q_before", "b_iso", "stall"):
                a = getattr(o, "stall_us" if f == "stall" else f)
                assert a == pytest.approx(getattr(r, f), rel=1e-12, abs=1e-9)
            assert o.T_iss_us == pytest.approx(r.T_iss, rel=1e-12)
            assert bool(o.guard_ok) == r.guard_ok


def test_model_fit_matches_oracle():
    X = xs()
    a, b, R, Q = 0.7, 2e-7, 4000.0, 3.0e6
    Vr = np.linspace(1e5, 2e6, 12)
    Tr = a + b * Vr + np.random.default_rng(1).normal(0, 0.01, 12)
    Vz = np.linspace(5e5, 8e6, 10)
    Tz = Vz / R * (1 + np.random.default_rng(2).normal(0, 0.01, 10))
    Vi = np.linspace(2e5, 1.2e7, 60)
    Ti = np.maximum(a + b * Vi, (Vi - Q) / R)
    ref = oxm.fit(Vr, Tr, Vz, Tz, Vi, Ti, K=64)
    keep = [_arr(v) for v in (Vr, Tr, Vz, Tz, Vi, Ti)]
    c = X.xs_calib(keep[0][1], keep[1][1], 12, keep[2][1], keep[3][1], 10, keep[4][1], keep[5][1], 60, 64, 0.10)
    m = X.xs_model()
    X.check(X.xs_model_fit(C.byref(c), C.byref(m)))
    assert m.t0_a_us == pytest.approx(ref.t0_a, rel=1e-9)
    assert m.t0_b_us_per_byte == pytest.approx(ref.t0_b, rel=1e-9)
    assert m.R_bytes_per_us == pytest.approx(ref.R, rel=1e-12)
    assert m.Q_bytes == pytest.approx(ref.Q, rel=1e-9)


def _microbench(target_ptr, target_bytes, K, B, n_bursts, gap_ns, mode):
    X = xs()
    require_gpu()
    buf = torch.zeros((K * n_bursts, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
    tr = X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr())
    args = X.xs_microbench_args(target_ptr, target_bytes, K, B, n_bursts, gap_ns, mode, 1)
    X.check(X.xs_xstage_microbench(C.byref(args), C.byref(tr), torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert int(cnt.item()) == K * n_bursts
    r = buf.cpu().numpy()
    assert np.all(r[:, 2] >= r[:, 1]) and np.all(r[:, 3] >= r[:, 2])
    return r


def test_microbench_hbm_and_gap():
    require_gpu()
    X = xs()
    K, B, nb = 64, 16384, 8
    tgt = torch.zeros((K * nb * B // 2,), dtype=torch.int16, device="cuda")
    r = _microbench(tgt.data_ptr(), tgt.numel() * 2, K, B, nb, 0, X.XS_MB_PERIODIC)
    # every producer wrote its bursts: the pattern word 2 of each 16-byte piece is set
    v = tgt.view(torch.int32).view(-1, 4).cpu().numpy()
    assert np.all(v[:, 2] == 0x58535447)
    rate = X.xs_clock_rate_hz()
    assert rate > 0
    gap_ns = 20000
    r2 = _microbench(tgt.data_ptr(), tgt.numel() * 2, K, B, 2, gap_ns, X.XS_MB_PERIODIC)
    gaps = (r2[:, 3] - r2[:, 2]) / rate * 1e9
    assert np.all(gaps >= gap_ns * 0.99)


def test_microbench_host_coherent_sink_completion_mode():
    require_gpu()
    X = xs()
    from paper_2607_23264_amd.layer import HostCoherent
    K, B, nb = 16, 8192, 4
    h = HostCoherent(K * nb * B)
    try:
        _microbench(h.ptr, h.nbytes, K, B, nb, 0, X.XS_MB_COMPLETION)
        v = h.view.view(torch.int32).view(-1, 4).numpy()
        assert np.all(v[:, 2] == 0x58535447)
    finally:
        h.free()
