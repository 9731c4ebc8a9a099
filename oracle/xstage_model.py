"""Oracle of the Burst-Gap model of the post-issue stage (test infrastructure only).

Platform model M_X = (T0(K, V), R, Q) (Sec. 3.3): recovered issue floor T0, effective
aggregate drain rate R, effective outstanding capacity Q. Units are the caller's,
as long as they are consistent (bytes, microseconds, bytes per microsecond); the
worked numbers in the paper use GB = 1e9 B and KiB/MiB = 2**10 / 2**20 B.

Functions follow the equations in order:
  Eq. 1  period / issue max law           burst_gap
  Eq. 2  recovery gap                     recovery_gap
  Eq. 3  floor period and pressure        pressure
  Eq. 4  byte-level change                delta_b
  Eq. 5  backlog recurrence               backlog_recurrence
  Eq. 6  capacity guard                   b_iso, capacity_guard
  Sec. 3.5 worked calibration             capacity_from_knee
  Eq. 7  interleaved MegaMoE gap          interleaved_gap
  Eq. 8  issue-overhead exchange          interleaved_overhead
  Eq. 9  average-rate feasibility         average_rate_feasible
  App. A.2 lead knee, MMA-side stall      d_knee, mma_stall
  App. C.2 FlashAttention recovery bound  fa_work, fa_qloop_lower_bound, fa_recovery_threshold

``predict`` extends Eq. 5 past the capacity guard (the paper only says issue must
stretch until enough volume drains, Sec. 3.5). The reading used here: a fluid
queue capped at Q drains at R, so a burst whose guard fails is issued in
max(T0, (q + V - Q) / R) and leaves the queue at Q; with the guard holding this is
exactly Eq. 5, and its homogeneous steady state is Eq. 1. The stalled branch is pinned
against a brute-force time-stepped fluid-queue simulation (tests), which derives the same
issue time and backlog from the queue's rules rather than from this formula.

``fit`` reads the calibration procedure of Sec. 3.3/3.5: T0 from recovered
(large-gap) points, R from the zero-gap steady state T_period = V / R, Q from the
isolated-burst knee. The knee threshold is a reading.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Sequence

import numpy as np

__all__ = [
    "pos", "burst_gap", "recovery_gap", "pressure", "delta_b", "backlog_recurrence", "b_iso",
    "capacity_guard", "capacity_from_knee", "predict", "BurstPrediction", "fit", "Model",
    "interleaved_gap", "interleaved_overhead", "average_rate_feasible", "d_knee",
    "mma_stall", "fa_work", "fa_qloop_lower_bound", "fa_recovery_threshold",
    "completion_coupled_period", "residual", "speedup", "knee_index", "capacity_bracket",
]


def pos(x):
    """[x]_+ = max(x, 0)."""
    return np.maximum(x, 0.0)


# Eq. 1
def burst_gap(T0, G, V, R):
    """Periodic bursts of volume V separated by a non-injecting gap G.

    Returns (T_period, T_iss) = (max(T0 + G, V/R), max(T0, V/R - G)).
    """
    return np.maximum(np.add(T0, G), np.divide(V, R)), np.maximum(T0, np.divide(V, R) - G)


# Eq. 2
def recovery_gap(V, R, T0):
    """Smallest gap that returns issue to its floor: [V/R - T0]_+."""
    return pos(np.divide(V, R) - T0)


# Eq. 3
def pressure(V, T0, G, R):
    """(P_n, rho_n) = (T0 + G, V / (R P_n))."""
    P = np.add(T0, G)
    return P, np.divide(V, np.multiply(R, P))


# Eq. 4
def delta_b(V, T0, G, R):
    """Bytes carried into later periods: V - R P_n."""
    return np.subtract(V, np.multiply(R, np.add(T0, G)))


# Eq. 5
def backlog_recurrence(V: Sequence[float], T0: Sequence[float], G: Sequence[float], R: float,
                       q0: float = 0.0) -> np.ndarray:
    """q_{n+1} = [q_n + V_n - R (T0_n + G_n)]_+ in the floor-issue counterfactual.

    Returns q before each burst and after the last one (length n + 1).
    """
    q = [float(q0)]
    for v, t0, g in zip(V, T0, G):
        q.append(max(0.0, q[-1] + float(v) - R * (float(t0) + float(g))))
    return np.asarray(q)


# Eq. 6
def b_iso(V, T0, R):
    """Peak occupancy increment of one recovered burst: [V - R T0]_+."""
    return pos(np.subtract(V, np.multiply(R, T0)))


def capacity_guard(q, V, T0, R, Q) -> bool:
    return bool(q + b_iso(V, T0, R) <= Q)


# Sec. 3.5 worked calibration
def capacity_from_knee(K, B_knee, R, T0):
    """Q = K * B_knee - R * T0: the isolated-burst knee volume minus what drains
    while that burst is issued at its floor."""
    return K * B_knee - R * T0


@dataclass
class BurstPrediction:
    rho: float
    delta_b: float
    q_before: float
    b_iso: float
    guard_ok: bool
    T_iss: float
    stall: float


def predict(V, T0, G, R: float, Q: float, q0: float = 0.0):
    """Per-burst audit of a burst sequence (Sec. 4.1 procedure with Eqs. 3-6).

    Issue takes the floor while the capacity guard holds; otherwise it stretches to
    (q + V - Q) / R (fluid queue capped at Q). The backlog carried into the next
    burst is [q + V - R (T_iss + G)]_+, which is Eq. 5 whenever the guard holds.
    """
    out = []
    q = float(q0)
    for v, t0, g in zip(V, T0, G):
        v, t0, g = float(v), float(t0), float(g)
        P = t0 + g
        bi = max(0.0, v - R * t0)
        ok = q + bi <= Q
        t_iss = t0 if ok else max(t0, (q + v - Q) / R)
        out.append(BurstPrediction(rho=v / (R * P) if P > 0 else math.inf, delta_b=v - R * P,
                                   q_before=q, b_iso=bi, guard_ok=ok, T_iss=t_iss,
                                   stall=t_iss - t0))
        q = max(0.0, q + v - R * (t_iss + g))
    return out


def completion_coupled_period(T0, G, V, R):
    """Counterfactual of Sec. 3.2: an issuer blocked until remote visibility adds the
    gap to the communication time, period = max(T0, V/R) + G (a reading; pinned against
    a simulated issuer that waits for its queue to empty before the gap)."""
    return np.maximum(T0, np.divide(V, R)) + G


# ----------------------------------------------------------------------------- fit
@dataclass
class Model:
    t0_a: float        # T0(V) = t0_a + t0_b * V (fixed K)
    t0_b: float
    R: float
    Q: float
    K: int

    def T0(self, V):
        return self.t0_a + self.t0_b * np.asarray(V, dtype=np.float64)


def fit(recovered_V, recovered_Tiss, zero_gap_V, zero_gap_period, isolated_V, isolated_Tiss,
        K: int, knee_excess: float = 0.10) -> Model:
    """Calibrate (T0, R, Q) from disjoint experiment regions.

    * T0(V): least-squares line through the recovered (large-gap) issue times;
    * R: least-squares slope through the origin of zero-gap periods, T = V / R;
    * Q: the isolated-burst knee is where the floor T0(V) meets the stalled branch
      T_iss = (V - Q) / R; every isolated burst whose issue time exceeds T0(V) by
      more than ``knee_excess`` (relative) lies on that branch and gives
      Q = V - R T_iss, which equals V_knee - R T0(V_knee) at the knee (Sec. 3.5).
      The median over those bursts is returned; Q = +inf if no burst stalls.
    """
    rv = np.asarray(recovered_V, dtype=np.float64)
    rt = np.asarray(recovered_Tiss, dtype=np.float64)
    if rv.size >= 2 and np.ptp(rv) > 0:
        b, a = np.polyfit(rv, rt, 1)
    else:
        a, b = float(rt.mean()), 0.0
    zv = np.asarray(zero_gap_V, dtype=np.float64)
    zt = np.asarray(zero_gap_period, dtype=np.float64)
    R = float((zv * zv).sum() / (zv * zt).sum())
    iv = np.asarray(isolated_V, dtype=np.float64)
    it = np.asarray(isolated_Tiss, dtype=np.float64)
    stalled = it > (a + b * iv) * (1.0 + knee_excess)
    Q = float(np.median(iv[stalled] - R * it[stalled])) if stalled.any() else math.inf
    return Model(t0_a=float(a), t0_b=float(b), R=R, Q=Q, K=int(K))


def knee_index(iso_V, iso_T, knee_excess: float) -> int:
    """Sec. 3.5's isolated-burst knee (a reading of how to locate it): the first burst, from
    the third on, whose issue time exceeds (1 + knee_excess) times the straight line through
    the first burst and the one before it; len(iso_V) when none does. iso_V ascending."""
    for i in range(2, len(iso_V)):
        v0, t0, v1, t1 = iso_V[0], iso_T[0], iso_V[i - 1], iso_T[i - 1]
        slope = (t1 - t0) / (v1 - v0) if v1 > v0 else 0.0
        if iso_T[i] > (1.0 + knee_excess) * (t0 + slope * (iso_V[i] - v0)):
            return i
    return len(iso_V)


def capacity_bracket(iso_V, knee: int, model: Model):
    """Q lies between V - R T0(V) at the last isolated burst on the floor and at the first one
    past the knee (Sec. 3.5: the knee is where the floor meets the stalled branch); (inf, inf)
    without a knee."""
    if not (0 < knee < len(iso_V)):
        return math.inf, math.inf
    q = lambda V: V - model.R * float(model.T0(V))
    return q(iso_V[knee - 1]), q(iso_V[knee])


# ----------------------------------------------------------------------------- App. A
def interleaved_gap(T_L2, T_L1, n1, n2):
    """Eq. 7: G_int = T_L2 + (n1 / n2) T_L1."""
    return T_L2 + (n1 / n2) * T_L1


def interleaved_overhead(dT_wave, T_L1, n1, n2):
    """Eq. 8: [dT_wave - (n1 / n2) T_L1]_+."""
    return pos(dT_wave - (n1 / n2) * T_L1)


def average_rate_feasible(V, T0, T_L2, T_L1, n1, n2, R) -> bool:
    """Eq. 9: n2 V / (n2 (T0 + T_L2) + n1 T_L1) <= R."""
    return bool(n2 * V / (n2 * (T0 + T_L2) + n1 * T_L1) <= R)


def d_knee(b_n, K_sm, h_inter):
    """App. A.2 anti-starvation lead: ceil(b_n K_SM / (2 h_inter)), the rows spanned by one
    round of Linear-1 tiles over all K_SM producers (P1 = 2 h_inter / b_n tiles per row).
    The rows-per-round reading is pinned by counting; the paper calls the knee approximate,
    and a lock-step simulation shows the wait-free lead varies around it with the tile mix,
    so its scheduling meaning is parity unpinned."""
    return int(math.ceil(b_n * K_sm / (2.0 * h_inter)))


def mma_stall(T_RS, T_cover):
    """App. A.2: [T_RS - T_cover]_+, the part of a tile's remote-store span that the mainloop
    before its staging slot's reuse does not cover (pinned against a discrete-event
    simulation of a producer and an epilogue sharing two staging slots)."""
    return pos(np.subtract(T_RS, T_cover))


# ----------------------------------------------------------------------------- App. C
def fa_work(b_m, b_n, d, M):
    """C_FA = 4 b_m b_n d ceil(M / b_n)."""
    return 4 * b_m * b_n * d * math.ceil(M / b_n)


def fa_qloop_lower_bound(sigma, M, b_n):
    """G_Qloop(M) >= sigma ceil(M / b_n)."""
    return sigma * math.ceil(M / b_n)


def fa_recovery_threshold(b_n, G_star, sigma):
    """M_ub* = b_n ceil(G* / sigma)."""
    return b_n * math.ceil(G_star / sigma)


# ----------------------------------------------------------------------------- reporting
def residual(T_fused, T_base):
    """Sender-visible residual over the compute-only run, E_res = T_fused - T_base (Sec. 5.4)."""
    return np.subtract(T_fused, T_base)


def speedup(T_serial, T_fused):
    """Speedup of a fused operation over its serial counterpart, T_serial / T_fused
    (Tables 4-6)."""
    return np.divide(T_serial, T_fused)
