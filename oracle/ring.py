"""Oracle for dispatch through bounded destination rings (test infrastructure only).

Reading of the paper's ring-slot readiness condition (an eligible Linear-1 tile needs ready
dispatch input and a free destination ring slot, Sec. 4.3; the scheduler checks ring-slot
readiness before emitting a tile, App. A.2): each destination d owns a ring of S slots. An
entry carries one token row and the rows of d's dispatch window it is to be copied into. The
producer of entry n may fill slot n mod S only once entry n - S has been consumed and its slot
released (the lifetime protocol); the consumer copies the entry's row into every listed window
row and then releases the slot. Entries of one destination are numbered in the order producers
claim them; the windows that result do not depend on that order.

Per-destination token dedup (optional): a token routed to several experts of the same
destination is sent once, its entry listing all of its window rows there (k slots ascending);
without dedup every (token, k) slot is an entry of its own.

The final windows must equal those of the plain dispatch (oracle/ep.dispatch): the ring only
changes how rows travel, not where they land.
"""
from __future__ import annotations

import numpy as np

from . import ep

__all__ = ["ring_entries", "ring_dispatch", "entry_header_ints"]


def entry_header_ints(k: int, dedup: bool) -> int:
    """Header ints of an entry: the number of window rows, then up to k (dedup) or 1 rows."""
    return 1 + (k if dedup else 1)


def ring_entries(idx, slot_row, E: int, W: int, dedup: bool):
    """Entries of one source per destination: a list over d of lists of (token, [window rows])
    in token order, window rows in ascending k slot order."""
    idx = np.asarray(idx)
    slot_row = np.asarray(slot_row)
    T, k = idx.shape
    epw = E // W
    out = [[] for _ in range(W)]
    for t in range(T):
        if dedup:
            rows = {}
            for j in range(k):
                rows.setdefault(int(idx[t, j]) // epw, []).append(int(slot_row[t, j]))
            for d in sorted(rows):
                out[d].append((t, rows[d]))
        else:
            for j in range(k):
                out[int(idx[t, j]) // epw].append((t, [int(slot_row[t, j])]))
    return out


def ring_dispatch(x_bits, idx, slot_row, E: int, W: int, cap: int, slots: int, dedup: bool,
                  windows=None):
    """Dispatch one source's token rows x_bits [T][H] through rings of ``slots`` slots per
    destination: one producer and one consumer per ring, the producer stalling (the consumer
    draining the oldest entry) whenever its next slot is still occupied. Window rows at or
    beyond ``cap`` are skipped with STATUS_CAPACITY, as in the plain dispatch.

    Returns (windows [W][cap][H], status, stats) with stats = {"entries": [W], "stalls": [W]
    (productions that had to wait for a release), "copies": window rows written}."""
    if slots < 1:
        raise ValueError("a ring needs at least one slot")
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    T, H = x_bits.shape
    if windows is None:
        windows = np.full((W, cap, H), ep.SENTINEL_BF16, dtype=np.uint16)
    status = ep.STATUS_OK
    stats = {"entries": [0] * W, "stalls": [0] * W, "copies": 0}
    entries = ring_entries(idx, slot_row, E, W, dedup)
    for d in range(W):
        ring_rows = np.zeros((slots, H), dtype=np.uint16)
        ring_hdr = [None] * slots
        released = [0] * slots          # completed uses of each slot
        produced = consumed = 0

        def consume_one():
            nonlocal consumed, status
            s = consumed % slots
            t_rows = ring_hdr[s]
            assert t_rows is not None, "consumer read an empty slot"
            for r in t_rows:
                if r >= cap:
                    status = ep.STATUS_CAPACITY
                    continue
                windows[d, r] = ring_rows[s]
                stats["copies"] += 1
            ring_hdr[s] = None
            released[s] += 1
            consumed += 1

        for t, rows in entries[d]:
            s = produced % slots
            if released[s] != produced // slots:       # slot still holds entry produced - S
                stats["stalls"][d] += 1
                while released[s] != produced // slots:
                    consume_one()
            ring_rows[s] = x_bits[t]
            ring_hdr[s] = list(rows)
            produced += 1
        while consumed < produced:
            consume_one()
        stats["entries"][d] = produced
    return windows, status, stats
