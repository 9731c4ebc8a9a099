"""Oracle of the persistent-kernel tile orders (test infrastructure only).

Rows are (expert, M-block) pairs in expert-major order; row p has P1 Linear-1
tiles and P2 Linear-2 tiles. Linear-1 tile k1 is (row k1 // P1, column block
k1 % P1), Linear-2 tile k2 likewise with P2. A Linear-2 tile of row p reads the
whole Linear-1 output row, so it depends on all P1 Linear-1 tiles of row p.

* Expert-Wave (Sec. 4.3): rows are grouped into waves of consecutive experts; the
  global order is [L1 tiles of wave 0, L2 tiles of wave 0, L1 of wave 1, ...] and
  scheduler instance g of G takes every G-th entry starting at g.
* Cross-wave interleaving (App. A.2, Alg. 1): instance g keeps one cursor per tile
  stream, both starting at g and advancing by G. It emits the next Linear-2 tile
  when one remains and its row trails the Linear-1 cursor's row by at least the
  lead D (the Linear-1 row counts as infinitely far ahead once Linear-1 is done);
  otherwise it emits the next Linear-1 tile. The paired-CTA role r of the paper
  has no counterpart here and is dropped. "P P_1" in the paper is read as the
  product rows x tiles-per-row.
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
    n1, n2 = P * P1, P * P2
    k1 = k2 = g
    run = 0   # consecutive Linear-2 tiles since the last Linear-1 tile
    out: List[Tile] = []
    while k1 < n1 or k2 < n2:
        p1 = k1 // P1 if k1 < n1 else math.inf
        p2 = k2 // P2
        take_l2 = k2 < n2 and p2 + D <= p1
        if take_l2 and chunk is not None and run >= chunk and k1 < n1:
            take_l2 = False
        if take_l2:
            out.append((2, p2, k2))
            k2 += G
            run += 1
        else:
            out.append((1, int(p1), k1))
            k1 += G
            run = 0
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
