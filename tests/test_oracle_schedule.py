"""Pins of the tile-order oracle: a hand-traced run of the interleave rule, exact
coverage, phase order at large lead, and deadlock freedom under lock-step
simulation."""
import itertools

import numpy as np
import pytest

from oracle import schedule as sc


def test_interleave_hand_traced():
    # G=1, P=2 rows, P1=2, P2=1, D=1, traced by hand from the rule
    s = sc.interleave_stream(0, 1, P=2, P1=2, P2=1, D=1)
    assert s == [(1, 0, 0), (1, 0, 1), (2, 0, 0), (1, 1, 2), (1, 1, 3), (2, 1, 1)]


def test_interleave_two_instances_hand_traced():
    # G=2, P=2, P1=2, P2=2, D=1: instance 0 owns L1 tiles 0,2 and L2 tiles 0,2.
    # After L1 tile 0 its L1 cursor sits at tile 2 (row 1), one row ahead of L2 row 0.
    s0 = sc.interleave_stream(0, 2, P=2, P1=2, P2=2, D=1)
    assert s0 == [(1, 0, 0), (2, 0, 0), (1, 1, 2), (2, 1, 2)]
    s1 = sc.interleave_stream(1, 2, P=2, P1=2, P2=2, D=1)
    assert s1 == [(1, 0, 1), (2, 0, 1), (1, 1, 3), (2, 1, 3)]


@pytest.mark.parametrize("policy", ["interleave", "chunk", "wave"])
def test_every_tile_exactly_once(policy):
    for G, P, P1, P2 in itertools.product([1, 3, 8], [1, 4, 9], [1, 4], [2, 7]):
        waves = [(r, min(P, r + 2)) for r in range(0, P, 2)]
        st = sc.all_streams(policy, G, P, P1, P2, D=2, chunk=2, waves=waves)
        l1 = sorted(k for s in st for (kind, _, k) in s if kind == 1)
        l2 = sorted(k for s in st for (kind, _, k) in s if kind == 2)
        assert l1 == list(range(P * P1)) and l2 == list(range(P * P2))
        for s in st:
            for kind, row, k in s:
                assert row == k // (P1 if kind == 1 else P2)


def test_large_lead_gives_phase_order():
    for g in range(4):
        s = sc.interleave_stream(g, 4, P=6, P1=3, P2=5, D=6)
        kinds = [t[0] for t in s]
        assert kinds == sorted(kinds)


def test_chunk_caps_consecutive_l2():
    s = sc.interleave_stream(0, 1, P=8, P1=1, P2=6, D=1, chunk=2)
    run = 0
    l1_left = 8
    for kind, _, _ in s:
        if kind == 2:
            run += 1
            assert run <= 2 or l1_left == 0
        else:
            run = 0
            l1_left -= 1


def test_no_deadlock_with_positive_lead():
    rng = np.random.default_rng(0)
    for _ in range(150):
        G = int(rng.integers(1, 12))
        P = int(rng.integers(1, 12))
        P1, P2 = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        D = int(rng.integers(1, 4))
        for policy in ("interleave", "chunk"):
            sc.simulate(sc.all_streams(policy, G, P, P1, P2, D=D, chunk=1), P, P1)
        waves = sc.waves_by_tiles(list(range(P)), P1, int(rng.integers(1, 8)))
        sc.simulate(sc.all_streams("wave", G, P, P1, P2, waves=waves), P, P1)


def test_zero_lead_can_deadlock():
    with pytest.raises(RuntimeError):
        sc.simulate(sc.all_streams("interleave", 1, 2, 2, 1, D=0), 2, 2)


def test_waves_by_tiles_whole_experts():
    row_expert = [0, 0, 1, 2, 2, 2, 3]
    assert sc.waves_by_tiles(row_expert, P1=2, min_tiles=4) == [(0, 2), (2, 6), (6, 7)]


def test_expert_blocks_hand_counted():
    # 600 rows: 3 equal blocks of ceil(600 / 3) = 200 -> 224 rows (multiple of 32), the last 152
    assert sc.expert_blocks([600, 0, 1, 256], True) == ([224, 224, 152, 1, 256], [0, 0, 0, 2, 3])
    assert sc.expert_blocks([600, 257], False) == ([256, 256, 88, 256, 1], [0, 0, 0, 1, 1])


def test_audit_bursts_hand_traced():
    # G = 1, two rows, P1 = 1, P2 = 2, D = 1: row 1's Linear-1 tile releases row 0's two
    # Linear-2 tiles, and row 1's follow once Linear-1 is used up: L1 L2 L2 L1 L2 L2
    tiles = sc.interleave_stream(0, 1, P=2, P1=1, P2=2, D=1)
    assert [t[0] for t in tiles] == [1, 2, 2, 1, 2, 2]
    V, gaps, comp = sc.audit_bursts([tiles], [100, 50], sink_share=0.5, T_L1=10.0, T_L2=3.0)
    assert V == [100 * 256 * 2 * 0.5, 100 * 256 * 2 * 0.5, 50 * 256 * 2 * 0.5, 50 * 256 * 2 * 0.5]
    # after burst 0: the next Linear-2 mainloop; after burst 1: L1 + L2; then L2; last: nothing
    assert gaps == [3.0, 13.0, 3.0, 0.0]
    assert comp == 2 * 10.0 + 4 * 3.0


def test_audit_unbounded_capacity_and_fast_drain_predict_no_stall():
    for rows in ([1039] * 32, [30466, 128, 175, 9344] + [200] * 28):
        ch, res = sc.pacing_audit(rows, True, 16, 28, 256, 16, 256, 1.0, 210.0, 64.0, 1.0, 1e-8, 5.6e6, np.inf)
        assert ch == ("interleave", None)   # every order ties at zero: the preference decides
        assert all(v[0] == 0 and v[2] == 0 for v in res.values())


def test_audit_rate_infeasible_stalls_every_order():
    # offered rate far above R (Eq. 9 fails): no order can recover, every candidate stalls
    ch, res = sc.pacing_audit([1039] * 32, True, 16, 28, 256, 16, 256, 1.0, 210.0, 64.0, 1.0, 1e-8, 1000.0, 1e6)
    assert all(v[0] > 0 for v in res.values())
    # and the stall is at least the drain time the compute cannot cover, V_total / R - compute,
    # for producer 0's bursts (issue alone cannot drain faster than R)
    sizes, owner = sc.expert_blocks([1039] * 32, True)
    streams = [sc.interleave_stream(g, 256, len(sizes), 16, 28, 16) for g in range(256)]
    V, gaps, comp = sc.audit_bursts(streams, sizes, 1.0, 210.0, 64.0)
    stall = res[("interleave", None)][0]
    assert stall >= sum(V) / 1000.0 - comp - 1e-6 - (1e6 / 1000.0)


def test_aligned_volume_counts_only_producers_with_that_burst():
    # 3 producers, 4 rows of 2 Linear-2 tiles: producer g owns entries g, g + 3, g + 6 < 8, so
    # all three take part in the first two bursts and producers 0, 1 in the third
    streams = [sc.interleave_stream(g, 3, P=4, P1=1, P2=2, D=1) for g in range(3)]
    V, _, _ = sc.audit_bursts(streams, [10, 20, 30, 40], 1.0, 1.0, 1.0)
    unit = 256 * 2
    # burst 0: entries 0, 1, 2 -> rows 0, 0, 1; burst 1: entries 3, 4, 5 -> rows 1, 2, 2;
    # burst 2: entries 6, 7 -> rows 3, 3 (producer 2 owns only 2 + 3 = 5 < 8 and 8 >= 8)
    assert V == [(10 + 10 + 20) * unit, (20 + 30 + 30) * unit, (40 + 40) * unit]


def test_audit_prefers_interleave_and_takes_wave_only_when_it_stalls_less():
    # a skewed 8-expert layer (rows per expert from Zipf routing), 8 producers, P1 = 4, P2 = 8
    rows = [210, 177, 292, 820, 224, 497, 383, 1493]
    args = (True, 4, 8, 8)
    # stalls within 1 % of the compute: interleave
    ch, res = sc.pacing_audit(rows, *args, 1, 8, 1.0, 20.0, 10.0, 1.0, 1e-7, 30000.0, 1e6)
    assert ch == ("interleave", None)
    # with a longer lead Expert-Wave's bursts stall clearly less than every other order's
    ch, res = sc.pacing_audit(rows, *args, 4, 8, 1.0, 20.0, 10.0, 1.0, 1e-7, 30000.0, 3e6)
    tol = 0.01 * res[("wave", None)][3]
    assert all(res[("wave", None)][0] < v[0] - tol for k, v in res.items() if k != ("wave", None))
    assert ch == ("wave", None)
