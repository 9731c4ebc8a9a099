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
        cover = g.uniform(0, 4, n)
        bursts = (X.xs_burst * n)(*[X.xs_burst(V[i], T0[i], G[i], cover[i]) for i in range(n)])
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
        # App. A.2's MMA-side stall with the predicted issue time as the remote-store span
        for i, o in enumerate(out):
            assert o.mma_stall_us == pytest.approx(float(oxm.mma_stall(ref[i].T_iss, cover[i])), rel=1e-12, abs=1e-12)


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


def _layer_struct(n_src, T, H, E, k, I, W, n_experts, precision=0):
    X = xs()
    L = X.xs_ep_layer()
    L.n_src, L.T, L.H, L.E, L.k, L.I, L.W = n_src, T, H, E, k, I, W
    L.e_begin, L.n_experts, L.precision = 0, n_experts, precision
    return L


AUDIT_CASES = [
    # (shape n_src, T, H, E, k, I, W, n_experts), producers, lead, wave_tiles, share, rows, model (t0_a, t0_b, R, Q)
    ((8, 4096, 7168, 256, 8, 2048, 8, 32), 256, 0, 0, 0.25, None, (1.06, 0.023e-6, 56000.0, 16.7e6)),
    ((8, 4096, 7168, 256, 8, 2048, 8, 32), 256, 64, 0, 0.25, "zipf", (1.06, 0.023e-6, 56000.0, 16.7e6)),
    ((8, 4096, 7168, 256, 8, 2048, 8, 32), 128, 0, 512, 1.0, None, (0.56, 0.169e-6, 5.6e6, 1e18)),
    ((1, 256, 512, 8, 2, 1024, 4, 8), 16, 0, 0, 1.0, None, (1.0, 0.02e-6, 3000.0, 2e5)),
    ((1, 2048, 2048, 8, 2, 256, 4, 8), 8, 1, 0, 1.0, [600, 0, 37, 512, 1, 300, 900, 700], (1.0, 0.01e-6, 9000.0, 1e6)),
]


@pytest.mark.parametrize("case", range(len(AUDIT_CASES)))
@pytest.mark.parametrize("prec", [0, 1])
def test_pacing_audit_matches_oracle(case, prec):
    """The library's audit of each order (and AUTO's choice) against the oracle's independent
    construction: producer 0's stream from the schedule oracle, bursts under full alignment,
    the recurrence of xstage_model.predict."""
    from oracle import schedule as osc
    from paper_2607_23264_amd.layer import pacing
    X = xs()
    shape, G, lead, wave_tiles, share, rows, (a, b, R, Q) = AUDIT_CASES[case]
    n_src, T, H, E, k, I, W, ne = shape
    if rows == "zipf":
        g = np.random.default_rng(3)
        pz = np.arange(1, ne + 1, dtype=np.float64) ** -1.2
        rows = list(g.multinomial(n_src * T * k * ne // E, pz / pz.sum()))
    L = _layer_struct(n_src, T, H, E, k, I, W, ne, prec)
    m = X.xs_model(a, b, R, Q, G, 0)
    exp_rows = rows if rows is not None else [n_src * T * k // E] * ne
    P1, P2 = I // 128, H // 256
    D = lead if lead > 0 else -(-G // P1)
    names = {X.XS_POLICY_BURST: "wave", X.XS_POLICY_INTERLEAVE: "interleave", X.XS_POLICY_CHUNK: "chunk"}
    tl1, tl2 = 210.0, 64.0
    for pol, chunk in [(X.XS_POLICY_AUTO, 0), (X.XS_POLICY_BURST, 0), (X.XS_POLICY_INTERLEAVE, 0),
                       (X.XS_POLICY_CHUNK, 2)]:
        p = pacing(pol, lead=lead, chunk=chunk, max_producers=G, wave_tiles=wave_tiles, model=m, t_l1_us=tl1,
                   t_l2_us=tl2, expert_rows=rows, sink_share=share)
        au = X.xs_pacing_audit()
        X.check(X.xs_pacing_audit_run(C.byref(L), C.byref(p), C.byref(au)))
        assert au.producers == G and au.lead_rows == D
        ref_choice, ref = osc.pacing_audit(exp_rows, prec == 0, P1, P2, G, D, wave_tiles or G, share or 1.0, tl1,
                                           tl2, a, b, R, Q,
                                           policy="auto" if pol == X.XS_POLICY_AUTO else names[pol],
                                           chunk=chunk if pol == X.XS_POLICY_CHUNK else None)
        assert au.n_cand == len(ref)
        for i, (key, (stall, nb, fails, comp)) in enumerate(ref.items()):
            assert names[au.cand_policy[i]] == key[0] and (au.cand_chunk[i] or None) == key[1]
            assert au.cand_bursts[i] == nb and au.cand_guard_fail[i] == fails
            assert au.cand_stall_us[i] == pytest.approx(stall, rel=1e-9, abs=1e-6)
            assert au.cand_compute_us[i] == pytest.approx(comp, rel=1e-12)
        assert (names[au.policy], au.chunk or None) == ref_choice


def test_trace_tile_times_are_medians():
    X = xs()
    g = np.random.default_rng(5)
    n = 301
    recs = np.zeros((n, 4), np.uint64)
    ext = np.zeros((n, 4), np.uint64)
    kind = g.integers(1, 3, n)
    start = g.integers(1000, 10 ** 6, n)
    dep = start + (kind == 2) * g.integers(0, 500, n)
    ml = dep + g.integers(100, 20000, n)
    iss = ml + g.integers(10, 900, n)
    rows = g.integers(1, 257, n)
    recs[:, 0] = (kind.astype(np.uint64) << np.uint64(56))
    recs[:, 1], recs[:, 2], recs[:, 3] = start, ml, iss
    ext[:, 0], ext[:, 3] = dep, rows
    us = 1e6 / X.xs_clock_rate_hz()
    t1, t2, t3 = C.c_double(), C.c_double(), C.c_double()
    X.check(X.xs_trace_tile_times(recs.ctypes.data, ext.ctypes.data, n, 64, C.byref(t1), C.byref(t2), C.byref(t3)))
    keep = rows >= 64
    assert t1.value == pytest.approx(np.median((ml - start)[(kind == 1) & keep]) * us)
    assert t2.value == pytest.approx(np.median((ml - dep)[(kind == 2) & keep]) * us)
    assert t3.value == pytest.approx(np.median((iss - ml)[(kind == 2) & keep]) * us)


def test_calibration_calls_match_oracle():
    """Drain rate, knee, capacity bracket, Eq. 1 and the recovery audit through the C ABI against
    the oracle's functions."""
    X = xs()
    g = np.random.default_rng(7)
    for trial in range(20):
        a, b, R = g.uniform(0.3, 2), g.uniform(0, 5e-7), g.uniform(1e3, 1e5)
        Q = g.uniform(1e6, 5e7)
        Vi = np.sort(g.uniform(1e4, 2e8, 14))
        Ti = np.maximum(a + b * Vi, (Vi - Q) / R) * (1 + g.normal(0, 0.01, 14))
        Vz = np.linspace(1e6, 1e8, 6)
        Tz = Vz / R * (1 + g.normal(0, 0.01, 6))
        Vr = np.linspace(1e5, 2e6, 5)
        Tr = a + b * Vr
        ref = oxm.fit(Vr, Tr, Vz, Tz, Vi, Ti, K=256, knee_excess=0.5)
        keep = [_arr(v) for v in (Vr, Tr, Vz, Tz, Vi, Ti)]
        Rg = C.c_double()
        X.check(X.xs_drain_rate(keep[2][0].ctypes.data, keep[3][0].ctypes.data, 6, C.byref(Rg)))
        assert Rg.value == pytest.approx(ref.R, rel=1e-12)
        c = X.xs_calib(keep[0][1], keep[1][1], 5, keep[2][1], keep[3][1], 6, keep[4][1], keep[5][1], 14, 256, 0.5)
        sm = X.xs_calib_summary()
        X.check(X.xs_model_calibrate(C.byref(c), C.byref(sm)))
        k = oxm.knee_index(Vi, Ti, 0.5)
        assert sm.knee == k
        lo, hi = oxm.capacity_bracket(Vi, k, ref)
        for got, want in ((sm.Q_bracket_lo, lo), (sm.Q_bracket_hi, hi)):
            assert (np.isinf(got) and np.isinf(want)) or got == pytest.approx(want, rel=1e-9)
        m = sm.model
        for V, G in ((1e6, 0.0), (5e7, 30.0), (3e5, 500.0)):
            tp, ti = C.c_double(), C.c_double()
            X.check(X.xs_burst_gap(C.byref(m), V, G, C.byref(tp), C.byref(ti)))
            rp, ri = oxm.burst_gap(m.t0_a_us + m.t0_b_us_per_byte * V, G, V, m.R_bytes_per_us)
            assert tp.value == pytest.approx(float(rp), rel=1e-12) and ti.value == pytest.approx(float(ri), rel=1e-12)
        # recovery audit of n aligned bursts with a gap each
        V, n, G, sigma, b_n = g.uniform(1e6, 4e7), int(g.integers(1, 6)), g.uniform(0, 900), g.uniform(0.5, 3), 64
        mq = X.xs_model(m.t0_a_us, m.t0_b_us_per_byte, m.R_bytes_per_us, Q, 256, 0)
        rec = X.xs_recovery()
        X.check(X.xs_recovery_audit(C.byref(mq), V, n, G, sigma, b_n, C.byref(rec)))
        T0 = m.t0_a_us + m.t0_b_us_per_byte * V
        pred = oxm.predict([V] * n, [T0] * n, [G] * n, m.R_bytes_per_us, Q)
        assert rec.G_star_us == pytest.approx(float(oxm.recovery_gap(V, m.R_bytes_per_us, T0)), rel=1e-12, abs=1e-12)
        assert rec.M_ub_star == oxm.fa_recovery_threshold(b_n, rec.G_star_us, sigma)
        assert rec.stall_us == pytest.approx(sum(p.stall for p in pred), rel=1e-12, abs=1e-9)
        assert bool(rec.guard_ok) == all(p.guard_ok for p in pred)
        assert rec.rho == pytest.approx(pred[0].rho, rel=1e-12)
        assert rec.coupled_us == pytest.approx(n * float(oxm.completion_coupled_period(T0, 0.0, V, m.R_bytes_per_us)),
                                               rel=1e-12)
