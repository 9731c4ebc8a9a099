"""Pins of the Burst-Gap model oracle: the worked numbers the paper prints, the
closed-form branches of Eq. 1, the equivalences of Sec. 3.4, and the algebraic
link between Eqs. 1, 7 and 8."""
import json
import math
import os

import numpy as np
import pytest

from oracle import xstage_model as xm

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "xstage_worked_numbers.json")))
KiB, MiB, GB = 2 ** 10, 2 ** 20, 1e9


def test_worked_capacity_calibration():
    c = GOLD["capacity_calibration"]
    R = c["R_GB_per_s"] * GB / 1e6        # bytes per microsecond
    Q = xm.capacity_from_knee(c["K"], c["knee_KiB_per_producer"] * KiB, R, c["T0_us"])
    assert round(Q / MiB, c["printed_digits_Q"]) == c["Q_MiB"]


def test_worked_fa4_capacity_and_recovery():
    f = GOLD["fa4_capacity_check"]
    R = GOLD["capacity_calibration"]["R_GB_per_s"] * GB / 1e6
    T0 = GOLD["capacity_calibration"]["T0_us"]
    B = f["b_m"] * f["d"] * f["bytes_per_element"]
    assert B == f["B_KiB_per_producer"] * KiB
    V = f["K"] * B
    assert round(V / MiB, 1) == f["V_MiB"]
    bi = float(xm.b_iso(V, T0, R))
    assert round(bi / MiB, 1) == f["b_iso_MiB"]
    assert xm.capacity_guard(0.0, V, T0, R, f["Q_MiB"] * MiB)
    G_star = float(xm.recovery_gap(V, R, T0))
    assert round(G_star, 1) == f["G_star_us"]
    # with the measured Q-loop gap the pressure is below one and the backlog clears
    P, rho = xm.pressure(V, T0, f["Qloop_gap_us_at_M8192"], R)
    assert rho < 1 and xm.delta_b(V, T0, f["Qloop_gap_us_at_M8192"], R) < 0
    q = xm.backlog_recurrence([V], [T0], [f["Qloop_gap_us_at_M8192"]], R)
    assert q[-1] == 0.0


def test_worked_fa_sequence_threshold():
    s = GOLD["fa_sequence_bound"]
    R = GOLD["capacity_calibration"]["R_GB_per_s"] * GB / 1e6
    T0 = GOLD["capacity_calibration"]["T0_us"]
    f = GOLD["fa4_capacity_check"]
    G_star = float(xm.recovery_gap(f["K"] * f["b_m"] * f["d"] * 2, R, T0))
    M = xm.fa_recovery_threshold(s["b_n"], G_star, s["sigma_us_per_kv_tile"])
    assert M == 1024 and round(M / 1000, 1) * 1000 == s["M_ub_tokens_approx"]
    assert xm.fa_qloop_lower_bound(s["sigma_us_per_kv_tile"], M, s["b_n"]) >= G_star
    assert xm.fa_work(128, 128, 128, 8192) == 4 * 128 * 128 * 128 * 64


@pytest.mark.parametrize("table", ["fa4_table", "gemm_a2a_table", "gemm_ar_table"])
def test_printed_speedups_and_residuals(table):
    t = GOLD[table]
    sp = xm.speedup(np.array(t["serial_us"]), np.array(t["fused_us"]))
    assert np.allclose(sp, t["speedup"], atol=1.5e-3)
    if "E_res_us" in t:
        er = xm.residual(np.array(t["fused_us"]), np.array(t["fa_only_us"]))
        assert np.allclose(er, t["E_res_us"], atol=0.051)


def test_eq1_branches_and_one_for_one_trade():
    T0, V, R = 0.8, 100.0, 10.0          # V/R = 10
    G_star = float(xm.recovery_gap(V, R, T0))
    assert G_star == pytest.approx(9.2)
    for G in np.linspace(0, G_star, 7):
        Tp, Ti = xm.burst_gap(T0, G, V, R)
        assert Tp == pytest.approx(V / R)            # drain-limited plateau
        assert Ti == pytest.approx(V / R - G)        # each unit of gap removes one unit of issue
    for G in [G_star, G_star + 1, 50]:
        Tp, Ti = xm.burst_gap(T0, G, V, R)
        assert Ti == pytest.approx(T0) and Tp == pytest.approx(T0 + G)
    # the completion-coupled counterfactual adds the gap to the transfer time instead
    assert xm.completion_coupled_period(T0, 5.0, V, R) == pytest.approx(15.0)


def test_rho_le_one_everywhere_gives_no_backlog():
    g = np.random.default_rng(0)
    for _ in range(200):
        n = 30
        T0 = g.uniform(0.1, 2, n)
        G = g.uniform(0, 5, n)
        R = 3.0
        rho = g.uniform(0, 1, n)
        V = rho * R * (T0 + G)
        assert np.all(xm.backlog_recurrence(V, T0, G, R) == 0.0)


def test_overloaded_period_recovered_by_later_ones():
    # rho > 1 then rho < 1: backlog appears, then drains (Eq. 5 keeps history)
    R = 1.0
    q = xm.backlog_recurrence([5, 1, 1], [1, 1, 1], [1, 3, 3], R)
    assert q.tolist() == [0, 3, 0, 0]


def test_homogeneous_equivalences():
    g = np.random.default_rng(1)
    for _ in range(500):
        T0, R = g.uniform(0.1, 2), g.uniform(0.5, 5)
        V, G = g.uniform(0, 30), g.uniform(0, 10)
        _, rho = xm.pressure(V, T0, G, R)
        db = xm.delta_b(V, T0, G, R)
        Gs = xm.recovery_gap(V, R, T0)
        assert (rho <= 1) == (db <= 0) == (G >= Gs)


def test_predict_steady_state_is_eq1_and_guard_holds_reduces_to_eq5():
    T0, G, V, R, Q = 1.0, 2.0, 60.0, 10.0, 25.0      # rho = 2, R G = 20 < Q
    preds = xm.predict([V] * 200, [T0] * 200, [G] * 200, R, Q)
    _, Ti = xm.burst_gap(T0, G, V, R)
    assert preds[-1].T_iss == pytest.approx(Ti)
    assert preds[-1].q_before == pytest.approx(Q - R * G)
    # light load: guard always holds and q follows Eq. 5 exactly
    Vs, T0s, Gs = [5, 15, 3, 9], [1, 1, 1, 1], [0.2, 0.1, 2, 1]
    pr = xm.predict(Vs, T0s, Gs, R, 1e9)
    q5 = xm.backlog_recurrence(Vs, T0s, Gs, R)
    assert [p.q_before for p in pr] == pytest.approx(list(q5[:-1]))
    assert all(p.stall == 0 for p in pr)


def test_capacity_guard_locates_isolated_knee():
    R, Q = 10.0, 50.0
    T0 = 1.0
    # from a recovered state the guard fails exactly when V > Q + R T0
    assert xm.capacity_guard(0, 59.9, T0, R, Q)
    assert not xm.capacity_guard(0, 60.1, T0, R, Q)
    p = xm.predict([80.0], [T0], [0.0], R, Q)[0]
    assert not p.guard_ok and p.T_iss == pytest.approx((80 - Q) / R)


def test_eq8_is_eq1_with_eq7_substituted():
    g = np.random.default_rng(2)
    for _ in range(500):
        T0, R, V = g.uniform(0.1, 1), g.uniform(1, 5), g.uniform(10, 50)
        TL2, TL1 = g.uniform(0, 3), g.uniform(0, 5)
        n1, n2 = g.integers(1, 8), g.integers(1, 8)
        over_wave = xm.burst_gap(T0, TL2, V, R)[1] - T0
        G_int = xm.interleaved_gap(TL2, TL1, n1, n2)
        over_int = xm.burst_gap(T0, G_int, V, R)[1] - T0
        assert over_int == pytest.approx(xm.interleaved_overhead(over_wave, TL1, n1, n2), abs=1e-12)


def test_eq9_average_rate_bound():
    # necessary: if interleaving fully recovers every period then the average rate <= R
    assert xm.average_rate_feasible(V=10, T0=1, T_L2=1, T_L1=3, n1=1, n2=1, R=2.5)
    assert not xm.average_rate_feasible(V=10, T0=1, T_L2=1, T_L1=1, n1=1, n2=1, R=2.5)


def test_knee_and_stall_closed_forms():
    assert xm.d_knee(b_n=128, K_sm=148, h_inter=2048) == math.ceil(128 * 148 / 4096)
    assert xm.mma_stall(5.0, 3.0) == 2.0 and xm.mma_stall(1.0, 3.0) == 0.0


def test_fit_recovers_generating_parameters():
    a, b, R, Q = 0.7, 0.002, 40.0, 3000.0
    Vr = np.linspace(100, 2000, 12)
    Tr = a + b * Vr
    Vz = np.linspace(500, 8000, 10)
    Tz = xm.burst_gap(a + b * Vz, 0.0, Vz, R)[0]
    Vi = np.linspace(200, 12000, 60)
    Ti = np.maximum(a + b * Vi, (Vi - Q) / R)
    m = xm.fit(Vr, Tr, Vz, Tz, Vi, Ti, K=64)
    assert m.t0_a == pytest.approx(a) and m.t0_b == pytest.approx(b)
    assert m.R == pytest.approx(R)
    assert m.Q == pytest.approx(Q, rel=1e-9)
    # a path with no knee reports unbounded capacity
    assert math.isinf(xm.fit(Vr, Tr, Vz, Tz, Vi, a + b * Vi, K=64).Q)
