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


def _fluid_queue(bursts, R, Q, dt, q0=0.0, completion_coupled=False):
    """Brute-force time-stepped simulation of the post-issue stage as a fluid queue (a model
    written independently of the oracle's closed forms): a burst of V bytes is offered at its
    floor rate V / T0; the queue accepts bytes only while it holds less than Q and drains at R.
    A completion-coupled issuer also waits until the queue is empty before its gap.
    Returns per burst (issue time, backlog before, period)."""
    q = q0
    out = []
    for V, T0, G in bursts:
        q_before, left, t = q, V, 0.0
        rate = V / T0
        while left > 1e-9:
            step = min(rate * dt, left)
            room = max(0.0, Q - q) + R * dt        # what the queue can take in this step
            step = min(step, room)
            q = max(0.0, q + step - R * dt)
            left -= step
            t += dt
        t_iss = t
        if completion_coupled:
            while q > 1e-9:
                q = max(0.0, q - R * dt)
                t += dt
        for _ in range(int(round(G / dt))):
            q = max(0.0, q - R * dt)
        out.append((t_iss, q_before, t + G))
    return out


def test_predict_stalled_branch_matches_fluid_queue_simulation():
    # overloaded bursts that fill the queue: the issue time stretches to (q + V - Q) / R and
    # the backlog left behind is Q drained over the gap (the reading of the stalled branch)
    R, Q, dt = 2.0, 40.0, 1e-3
    bursts = [(60.0, 1.0, 2.0), (60.0, 1.0, 2.0), (30.0, 0.5, 0.0), (90.0, 2.0, 30.0), (10.0, 1.0, 1.0),
              (45.0, 1.0, 5.0), (45.0, 1.0, 5.0)]
    sim = _fluid_queue(bursts, R, Q, dt)
    pred = xm.predict([b[0] for b in bursts], [b[1] for b in bursts], [b[2] for b in bursts], R, Q)
    assert any(not p.guard_ok for p in pred) and any(p.guard_ok for p in pred)
    for (t_iss, q_before, _), p, b in zip(sim, pred, bursts):
        assert p.q_before == pytest.approx(q_before, abs=R * dt * 3)
        assert p.T_iss == pytest.approx(t_iss, abs=dt * 3)
        assert p.stall == pytest.approx(t_iss - b[1], abs=dt * 3)


def test_completion_coupled_period_matches_simulation():
    # an issuer that waits for visibility before its gap: period max(T0, V/R) + G
    R, dt = 2.0, 1e-3
    for V, T0, G in [(10.0, 1.0, 3.0), (1.0, 1.0, 3.0), (40.0, 2.0, 0.0), (3.0, 2.0, 7.0)]:
        _, _, period = _fluid_queue([(V, T0, G)], R, math.inf, dt, completion_coupled=True)[0]
        assert xm.completion_coupled_period(T0, G, V, R) == pytest.approx(period, abs=dt * 3)


def _staging_pipeline(t_mma, t_rs, slots=2):
    """Discrete-event simulation of a producer and an epilogue role sharing `slots` local
    staging slots: tile n's mainloop takes t_mma[n] and needs a free slot; the epilogue of
    tile n starts when the mainloop ends and the epilogue role is free, takes t_rs[n] and
    frees the slot. Returns the producer's wait before each tile's mainloop."""
    free_at = [0.0] * slots         # when each slot is released
    epi_free, t, waits = 0.0, 0.0, []
    for n, (m, r) in enumerate(zip(t_mma, t_rs)):
        s = n % slots
        start = max(t, free_at[s])
        waits.append(start - t)
        end = start + m
        e0 = max(end, epi_free)
        epi_free = e0 + r
        free_at[s] = epi_free
        t = end
    return waits


def test_mma_stall_matches_two_slot_pipeline():
    # steady state of a double-buffered accumulator: the producer waits for the slot of the
    # tile before last, i.e. the part of the epilogue span its successor's mainloop does not
    # cover (App. A.2)
    for t_rs, t_cover in [(5.0, 3.0), (1.0, 3.0), (4.0, 4.0), (9.5, 2.25)]:
        w = _staging_pipeline([t_cover] * 40, [t_rs] * 40)
        assert w[-1] == pytest.approx(float(xm.mma_stall(t_rs, t_cover)))


def test_knee_is_rows_of_one_linear1_round():
    # reading of App. A.2's knee: the rows spanned by one round of Linear-1 tiles over all
    # K_SM producers, with P1 = 2 h_inter / b_n tiles per row (counted by brute force); the
    # paper calls the knee approximate, so its scheduling meaning is not pinned here
    for b_n, K, h in [(128, 148, 2048), (256, 256, 2048), (256, 8, 1024), (256, 100, 512), (128, 1, 7168)]:
        P1 = 2 * h // b_n
        rows = len({e // P1 for e in range(K)})
        assert xm.d_knee(b_n, K, h) == rows


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


def test_knee_bracket_contains_the_generating_capacity():
    # isolated bursts on the fluid law T = max(T0(V), (V - Q) / R): the knee bracket holds Q
    a, b, R = 1.0, 2e-7, 56000.0
    for Q in (3e6, 16.7e6, 40e6):
        V = np.array([2 ** k * 65536.0 for k in range(12)])
        T = np.maximum(a + b * V, (V - Q) / R)
        m = xm.fit(V[:3], a + b * V[:3], V, V / R, V, T, K=256, knee_excess=0.5)
        k = xm.knee_index(V, T, 0.5)
        assert 0 < k < len(V)
        lo, hi = xm.capacity_bracket(V, k, m)
        assert lo <= Q < hi
        # every burst before the knee is on the floor, the knee burst is off it
        assert np.all(T[:k] <= (1.5) * (a + b * V[:k])) and T[k] > a + b * V[k]
    # no stall anywhere: no knee, unbounded bracket
    V = np.linspace(1e5, 1e7, 8)
    assert xm.knee_index(V, 1.0 + 2e-7 * V, 0.5) == len(V)
