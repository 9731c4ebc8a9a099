"""Pins of the ring-dispatch oracle: its windows against the plain dispatch definition, its
entries against brute-force counts of (token, destination) pairs, and the special cases in
which dedup changes nothing or everything."""
import numpy as np
import pytest

import synth
from oracle import ep, ring


def _routing(T, k, E, seed):
    g = np.random.default_rng(seed)
    return np.argsort(g.random((T, E)), axis=1)[:, :k].astype(np.int32)


@pytest.mark.parametrize("slots", [1, 2, 3, 7, 64, 10_000])
@pytest.mark.parametrize("dedup", [False, True])
def test_windows_equal_the_plain_dispatch(slots, dedup):
    T, H, E, k, W = 97, 48, 16, 4, 4
    idx = _routing(T, k, E, slots)
    lay = ep.dispatch_layout(idx[None], E, W)
    x = synth.normal_bf16(0, 3, (T, H))
    want, st = ep.dispatch(x[None], idx[None], lay["slot_row"], E, W, T * k)
    got, st2, stats = ring.ring_dispatch(x, idx, lay["slot_row"][0], E, W, T * k, slots, dedup)
    assert st == st2 == ep.STATUS_OK
    assert np.array_equal(got, want)
    assert stats["copies"] == T * k
    if slots == 1:
        # every production after a destination's first waits for the previous entry's release
        assert stats["stalls"] == [max(0, n - 1) for n in stats["entries"]]
    if slots >= T * k:
        assert stats["stalls"] == [0] * W


def test_entries_against_brute_force():
    T, E, k, W = 200, 32, 6, 8
    idx = _routing(T, k, E, 5)
    lay = ep.dispatch_layout(idx[None], E, W)
    sr = lay["slot_row"][0]
    epw = E // W
    plain = ring.ring_entries(idx, sr, E, W, dedup=False)
    dd = ring.ring_entries(idx, sr, E, W, dedup=True)
    assert sum(len(e) for e in plain) == T * k
    pairs = {(t, int(idx[t, j]) // epw) for t in range(T) for j in range(k)}
    assert sum(len(e) for e in dd) == len(pairs)
    # every (token, k) slot appears in exactly one dedup entry, with its own window row
    seen = {}
    for d in range(W):
        for t, rows in dd[d]:
            assert (t, d) in pairs
            for r in rows:
                seen[(d, r)] = t
    want = {(int(idx[t, j]) // epw, int(sr[t, j])): t for t in range(T) for j in range(k)}
    assert seen == want
    # entries of a destination come in token order
    for d in range(W):
        ts = [t for t, _ in dd[d]]
        assert ts == sorted(ts)


def test_dedup_special_cases():
    T, H = 40, 16
    x = synth.normal_bf16(0, 4, (T, H))
    # one expert per destination: a token's k experts are on k distinct destinations
    idx = _routing(T, 3, 8, 6)
    lay = ep.dispatch_layout(idx[None], 8, 8)
    a = ring.ring_entries(idx, lay["slot_row"][0], 8, 8, True)
    b = ring.ring_entries(idx, lay["slot_row"][0], 8, 8, False)
    assert a == b
    # one destination: one entry per token, listing all k rows
    lay1 = ep.dispatch_layout(idx[None], 8, 1)
    e1 = ring.ring_entries(idx, lay1["slot_row"][0], 8, 1, True)
    assert [t for t, _ in e1[0]] == list(range(T))
    assert all(len(rows) == 3 for _, rows in e1[0])
    w, st, stats = ring.ring_dispatch(x, idx, lay1["slot_row"][0], 8, 1, T * 3, 2, True)
    assert np.array_equal(w, ep.dispatch(x[None], idx[None], lay1["slot_row"], 8, 1, T * 3)[0])
    assert stats["entries"] == [T] and stats["copies"] == 3 * T


def test_capacity_overflow_matches_the_plain_dispatch():
    T, H, E, k, W = 64, 16, 4, 2, 2
    idx = _routing(T, k, E, 9)
    lay = ep.dispatch_layout(idx[None], E, W)
    x = synth.normal_bf16(0, 5, (T, H))
    want, st = ep.dispatch(x[None], idx[None], lay["slot_row"], E, W, 20)
    got, st2, _ = ring.ring_dispatch(x, idx, lay["slot_row"][0], E, W, 20, 3, True)
    assert st == st2 == ep.STATUS_CAPACITY
    assert np.array_equal(got, want)
