"""Oracle of the persistent-kernel tile orders (test infrastructure only).

Rows are (expert, M-block) pairs in expert-major order; row p has P1 Linear-1
tiles and P2 Linear-2 tiles. Linear-1 tile k1 is (row k1 // P1, column block
k1 % P1), Linear-2 tile k2 likewise with P2. A Linear-2 tile of row p reads the
whole Linear-1 output row, so it depends on all P1 Linear-1 tiles of row p.

* Expert-Wave (Sec. 4.3): rows are grouped into waves of consecutive experts; the
  global order is [L1 tiles of wave 0, L2 tiles of wave 0, L1 of wave 1, ...] and
  scheduler instance g of G takes every G-th entry starting at g.
* Cross-wave interleaving (App. A.2, Alg. 1): instance g of G owns every G-th entry
  of each tile stream, starting at its own index, and a Linear-2 entry may run before
  the instance's next Linear-1 entry only when Linear-1 leads it by at least D rows
  (``interleave_stream`` writes this as a merge of the two owned lists). The
  paired-CTA role r of the paper has no counterpart here and is dropped. "P P_1" in
  the paper is read as the product rows x tiles-per-row.
* Chunked pacing (a generalisation, not in the paper): the interleave rule, but
  after ``chunk`` consecutive Linear-2 tiles a Linear-1 tile is forced if any is
  left.

Tiles are returned as (kind, row, index) with kind 1 = Linear-1, 2 = Linear-2.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

__all__ = ["interleave_stream", "expert_wave_list", "expert_wave_stream", "all_streams",
           "simulate", "waves_by_tiles"]

Tile = Tuple[int, int, int]


def interleave_stream(g: int, G: int, P: int, P1: int, P2: int, D: int,
                      chunk: int | None = None) -> List[Tile]:
    """The tiles scheduler instance g runs, in order, under cross-wave interleaving.

    Instance g owns every G-th entry of each stream starting at g: Linear-1 entries
    g, g + G, ... and Linear-2 entries g, g + G, ... It runs its own entries in stream
    order. A Linear-2 entry of row r may run ahead of the instance's next Linear-1 entry
    only when that Linear-1 entry is at least D rows further on (row >= r + D); the lead
    is what keeps a Linear-2 tile from reaching a row whose Linear-1 tiles may not all be
    done. So the order is a merge of the two owned lists: before each owned Linear-1 entry
    come the not yet run Linear-2 entries that this entry's row already releases (at most
    ``chunk`` of them when a cap is given; the rest wait for the next Linear-1 entry, whose
    row releases at least as much), and once the Linear-1 entries are used up every
    remaining Linear-2 entry follows.
    """
    own1 = list(range(g, P * P1, G))
    own2 = list(range(g, P * P2, G))
    out: List[Tile] = []
    nxt = 0   # first owned Linear-2 entry not yet placed
    for e1 in own1:
        r1 = e1 // P1
        placed = 0
        while (nxt < len(own2) and own2[nxt] // P2 + D <= r1
               and (chunk is None or placed < chunk)):
            out.append((2, own2[nxt] // P2, own2[nxt]))
            nxt += 1
            placed += 1
        out.append((1, r1, e1))
    out.extend((2, e2 // P2, e2) for e2 in own2[nxt:])
    return out


def waves_by_tiles(row_expert: Sequence[int], P1: int, min_tiles: int) -> List[Tuple[int, int]]:
    """Split rows into waves of whole experts, each wave the smallest run of
    consecutive experts whose Linear-1 tile count reaches ``min_tiles`` (the last
    wave takes what is left). Returns [row_begin, row_end) ranges."""
    waves = []
    P = len(row_expert)
    r0 = 0
    r = 0
    while r < P:
        e = row_expert[r]
        while r < P and row_expert[r] == e:
            r += 1
        if (r - r0) * P1 >= min_tiles or r == P:
            waves.append((r0, r))
            r0 = r
    return waves


def expert_wave_list(P: int, P1: int, P2: int, waves: Sequence[Tuple[int, int]]) -> List[Tile]:
    out: List[Tile] = []
    for r0, r1 in waves:
        out.extend((1, k // P1, k) for k in range(r0 * P1, r1 * P1))
        out.extend((2, k // P2, k) for k in range(r0 * P2, r1 * P2))
    if len(out) != P * (P1 + P2):
        raise ValueError("waves must cover rows [0, P) exactly")
    return out


def expert_wave_stream(g: int, G: int, P: int, P1: int, P2: int,
                       waves: Sequence[Tuple[int, int]]) -> List[Tile]:
    return expert_wave_list(P, P1, P2, waves)[g::G]


def all_streams(policy: str, G: int, P: int, P1: int, P2: int, D: int = 1,
                chunk: int | None = None, waves=None) -> List[List[Tile]]:
    if policy == "interleave":
        return [interleave_stream(g, G, P, P1, P2, D) for g in range(G)]
    if policy == "chunk":
        return [interleave_stream(g, G, P, P1, P2, D, chunk=chunk) for g in range(G)]
    if policy == "wave":
        return [expert_wave_stream(g, G, P, P1, P2, waves) for g in range(G)]
    raise ValueError(policy)


def simulate(streams: Sequence[Sequence[Tile]], P: int, P1: int) -> int:
    """Lock-step execution: every round each instance runs its next tile if that
    tile's dependencies finished in an earlier round. Returns the number of rounds;
    raises RuntimeError on deadlock (no instance can move while tiles remain)."""
    done_l1 = [0] * P
    pos = [0] * len(streams)
    rounds = 0
    remaining = sum(len(s) for s in streams)
    while remaining:
        finished = []
        for i, s in enumerate(streams):
            if pos[i] == len(s):
                continue
            kind, row, _ = s[pos[i]]
            if kind == 2 and done_l1[row] < P1:
                continue
            finished.append((i, kind, row))
        if not finished:
            raise RuntimeError("deadlock")
        for i, kind, row in finished:
            pos[i] += 1
            if kind == 1:
                done_l1[row] += 1
        remaining -= len(finished)
        rounds += 1
    return rounds


# ----------------------------------------------------------------------------- pacing audit
def expert_blocks(rows_per_expert: Sequence[int], equal: bool) -> Tuple[List[int], List[int]]:
    """Row blocks of the persistent kernel's scheduler rows, expert by expert: an expert's m
    rows give ceil(m / 256) blocks; equal blocks hold ceil(m / blocks) rows rounded up to a
    multiple of 32 (at most 256), the last block what is left; otherwise 256 rows each with
    a ragged last block. Returns (rows of each block, expert of each block)."""
    sizes, owner = [], []
    for x, m in enumerate(rows_per_expert):
        nb = -(-int(m) // 256)
        if nb == 0:
            continue
        bm = min(256, -(-(-(-int(m) // nb)) // 32) * 32) if equal else 256
        left = int(m)
        for _ in range(nb):
            sizes.append(min(bm, left))
            owner.append(x)
            left -= bm
    return sizes, owner


def audit_bursts(streams: Sequence[Sequence[Tile]], block_rows: Sequence[int], sink_share: float,
                 T_L1: float, T_L2: float):
    """The burst sequence of producer 0 (streams[0]) under full alignment of all the producers'
    streams (Sec. 4.2): its n-th Linear-2 tile is issued together with the n-th Linear-2 tile
    of every producer that has one, so V_n is the sum of those tiles' bytes (rows x 256 columns
    x 2 bytes x sink_share each); the gap after it is producer 0's mainloop time up to and
    including its next Linear-2 tile (T_L1 or T_L2 per tile). Returns (V list, gap list,
    producer 0's mainloop time)."""
    V, gaps = [], []
    tiles = streams[0]
    compute = sum(T_L1 if kind == 1 else T_L2 for kind, _, _ in tiles)
    l2_rows = [[row for kind, row, _ in s if kind == 2] for s in streams]
    l2_at = [i for i, t in enumerate(tiles) if t[0] == 2]
    for n, i in enumerate(l2_at):
        V.append(sum(block_rows[r[n]] * 256 * 2 * sink_share for r in l2_rows if len(r) > n))
        stop = l2_at[n + 1] + 1 if n + 1 < len(l2_at) else len(tiles)
        gaps.append(sum(T_L1 if tiles[j][0] == 1 else T_L2 for j in range(i + 1, stop)))
    return V, gaps, compute


def pacing_audit(rows_per_expert, equal_blocks: bool, P1: int, P2: int, G: int, D: int,
                 wave_tiles: int, sink_share: float, T_L1: float, T_L2: float,
                 t0_a: float, t0_b: float, R: float, Q: float, policy: str = "auto",
                 chunk: int | None = None):
    """Audit of producer 0's tile order (Sec. 4.1 with Eqs. 3-6 via xstage_model.predict) and
    the automatic choice among "wave" (Expert-Wave), "interleave" and "chunk" c in 1, 2, 4,
    ..., 32: the least predicted stall, and among the candidates within 1 % of the Expert-Wave
    order's mainloop time of it, the plain interleave first, then the larger chunk, then
    Expert-Wave (a reading: the paper weighs X-Stage pressure against the rest of the
    schedule, Sec. 5.3, and Expert-Wave's Linear-2 tiles wait for their whole wave's Linear-1
    tiles, a cost the audit does not price). Returns (choice (policy, chunk), {candidate:
    (stall, bursts, guard failures, mainloop time)})."""
    from . import xstage_model as xm
    sizes, owner = expert_blocks(rows_per_expert, equal_blocks)
    P = len(sizes)
    if policy == "auto":
        cands = [("wave", None), ("interleave", None)] + [("chunk", c) for c in (1, 2, 4, 8, 16, 32)]
    else:
        cands = [(policy, chunk)]
    res = {}
    for pol, c in cands:
        if pol == "wave":
            streams = all_streams("wave", G, P, P1, P2, waves=waves_by_tiles(owner, P1, wave_tiles))
        else:
            streams = [interleave_stream(g, G, P, P1, P2, D, chunk=c) for g in range(G)]
        V, gaps, compute = audit_bursts(streams, sizes, sink_share, T_L1, T_L2)
        T0 = [t0_a + t0_b * v for v in V]
        pred = xm.predict(V, T0, gaps, R, Q)
        res[(pol, c)] = (sum(p.stall for p in pred), len(pred), sum(not p.guard_ok for p in pred), compute)
    if policy != "auto":
        return cands[0], res
    tol = 0.01 * res[("wave", None)][3]
    best = min(v[0] for v in res.values())
    near = [key for key in cands if res[key][0] <= best + tol]
    if ("interleave", None) in near:
        return ("interleave", None), res
    chunks = [key for key in near if key[0] == "chunk"]
    if chunks:
        return max(chunks, key=lambda key: key[1]), res
    return ("wave", None), res
