"""Calibration of the Burst-Gap model on this GPU's store paths (Sec. 3.1, Sec. 3.3, Sec. 3.5).

Runs the library's remote-store microbenchmark (xs_xstage_microbench) against a target
window (an HBM buffer, or fine-grained host-coherent memory for a slow sink), turns the
per-burst wall-clock records into sender-visible issue times and periods, and fits
(T0(V), R, Q) with the library's xs_model_fit:
  * recovered issue floor T0: bursts separated by a gap long enough to drain (large-gap
    plateau), issue time of every burst after the first;
  * drain rate R: zero-gap periodic bursts, steady-state period T_period = V / R;
  * capacity Q: isolated bursts from a recovered state, the knee where issue time leaves
    the floor.
A burst's aggregate volume is V = K * B. Issue times and periods are taken per producer
(producers drift apart over many bursts); an isolated burst, which every producer starts
at the launch, is timed from the first start to the last issued store. This module only
marshals calls and takes medians of the timestamps: every store is issued by the library's
kernel, and the model arithmetic (drain rate, knee, fit, capacity bracket, Eq. 1, G*) runs in
the library's host calls.
"""
from __future__ import annotations

import ctypes as C
import json
import math
from dataclasses import asdict, dataclass

import numpy as np
import torch

from . import xstage as X


@dataclass
class BurstRun:
    K: int
    B: int
    gap_ns: int
    mode: int
    n_bursts: int
    iss_us: np.ndarray          # [K, n_bursts] per producer: burst start -> last store issued
    period_us: np.ndarray       # [K, n_bursts - 1] per producer: start[n+1] - start[n]
    aligned_iss_us: np.ndarray  # per burst: first producer's start -> last producer's last store
    total_span_us: float        # first start of the run -> last issued store of the run

    def steady(self, a: np.ndarray) -> float:
        """Median over producers of the second half of the bursts (the steady state)."""
        return float(np.median(a[:, a.shape[1] // 2:]))


def run_bursts(target_ptr: int, target_bytes: int, K: int, B: int, n_bursts: int, gap_ns: int,
               mode: int = X.XS_MB_PERIODIC, store_waves: int = 1) -> BurstRun:
    buf = torch.zeros((K * n_bursts, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
    tr = X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr())
    args = X.xs_microbench_args(target_ptr, target_bytes, K, B, n_bursts, gap_ns, mode, store_waves)
    X.check(X.xs_xstage_microbench(C.byref(args), C.byref(tr), torch.cuda.current_stream().cuda_stream),
            "microbench")
    torch.cuda.synchronize()
    r = buf.cpu().numpy().astype(np.int64)
    us = 1e6 / X.xs_clock_rate_hz()
    prod = r[:, 0] >> 32
    burst = r[:, 0] & 0xFFFFFFFF
    start = np.zeros((K, n_bursts), np.int64)
    issued = np.zeros((K, n_bursts), np.int64)
    start[prod, burst] = r[:, 1]
    issued[prod, burst] = r[:, 2]
    aligned = (issued.max(axis=0) - start.min(axis=0)) * us
    span = float((issued.max() - start.min()) * us)
    return BurstRun(K, B, gap_ns, mode, n_bursts, (issued - start) * us, np.diff(start, axis=1) * us, aligned,
                    span)


def _f64(v):
    return np.ascontiguousarray(np.asarray(v, dtype=np.float64))


@dataclass
class Calibration:
    sink: str
    K: int
    model: dict
    recovered: list
    zero_gap: list
    isolated: list
    gap_sweep: list


def calibrate(target_ptr: int, target_bytes: int, sink: str, K: int, Bs, knee_excess: float = 0.5,
              gap_sweep_B: int | None = None, store_waves: int = 1, log=print) -> Calibration:
    """Calibrate (T0, R, Q) at K producers over per-producer burst sizes Bs (bytes, ascending).

    * isolated bursts (one burst per launch, so every producer starts recovered and aligned):
      issue time = first start to last issued store;
    * R from zero-gap periodic runs: aggregate volume over the whole run divided by the span of
      the run (producers desynchronise under arbitration, so per-producer periods would
      overstate the rate); enough bursts that the capacity absorbed at the start is small;
    * the knee: the first isolated burst whose issue time exceeds (1 + knee_excess) times the
      floor line through the smaller bursts; T0(V) is fitted on recovered (large-gap) bursts
      below the knee only, and Q on the isolated bursts past it (xs_model_fit)."""
    iso = []
    for B in Bs:
        vals = [float(run_bursts(target_ptr, target_bytes, K, B, 1, 0, store_waves=store_waves).aligned_iss_us[0])
                for _ in range(3)]
        iso.append((K * B, float(np.median(vals))))
    # every byte of a run lands at a fresh address (no wrap): rewrites of lines still in
    # flight are merged by the memory path and would overstate the drain rate
    def n_fit(B, want):
        return int(max(1, min(want, target_bytes // (K * B))))

    zg = []
    for B in Bs:
        n = n_fit(B, 64)
        if n < 4:
            continue
        run = run_bursts(target_ptr, target_bytes, K, B, n, 0, store_waves=store_waves)
        zg.append((K * B, run.total_span_us / n))
    zv, zt = _f64([v for v, _ in zg]), _f64([t for _, t in zg])
    R_est = C.c_double()
    X.check(X.xs_drain_rate(zv.ctypes.data, zt.ctypes.data, len(zg), C.byref(R_est)), "drain_rate")
    R_est = R_est.value                                      # bytes per us
    iv, it = _f64([v for v, _ in iso]), _f64([t for _, t in iso])
    knee = C.c_int32()
    X.check(X.xs_calib_knee(iv.ctypes.data, it.ctypes.data, len(iso), knee_excess, C.byref(knee)), "knee")
    knee = knee.value
    # recovered floor: large-gap bursts below the knee that actually returned to the floor
    # (issue within 3x of the isolated burst of the same volume)
    rec = []
    for i, B in enumerate(Bs[:max(2, knee)]):
        gap_us = min(20000.0, max(20.0, 4.0 * K * B / R_est))
        run = run_bursts(target_ptr, target_bytes, K, B, max(2, n_fit(B, 4)), int(gap_us * 1e3),
                         store_waves=store_waves)
        t = float(np.median(run.aligned_iss_us[1:]))
        if t <= 3.0 * iso[i][1]:
            rec.append((K * B, t))
    if len(rec) < 2:
        rec = list(iso[:max(2, knee)])
    keep = [np.ascontiguousarray(np.array(a, dtype=np.float64)) for a in
            ([v for v, _ in rec], [t for _, t in rec], [v for v, _ in zg], [t for _, t in zg],
             [v for v, _ in iso], [t for _, t in iso])]
    P = C.POINTER(C.c_double)
    c = X.xs_calib(keep[0].ctypes.data_as(P), keep[1].ctypes.data_as(P), len(rec),
                   keep[2].ctypes.data_as(P), keep[3].ctypes.data_as(P), len(zg),
                   keep[4].ctypes.data_as(P), keep[5].ctypes.data_as(P), len(iso), K, knee_excess)
    sm = X.xs_calib_summary()
    X.check(X.xs_model_calibrate(C.byref(c), C.byref(sm)), "model_calibrate")
    m = sm.model
    # Q two ways: the fluid fit (stalled isolated bursts on T = (V - Q) / R) and the knee
    # bracket between the last isolated burst on the floor and the first one off it
    bracket = [sm.Q_bracket_lo, sm.Q_bracket_hi] if math.isfinite(sm.Q_bracket_lo) else None
    model = {"t0_a_us": m.t0_a_us, "t0_b_us_per_byte": m.t0_b_us_per_byte, "R_bytes_per_us": m.R_bytes_per_us,
             "Q_bytes": m.Q_bytes if math.isfinite(m.Q_bytes) else None, "K": m.K,
             "knee_V_bytes": iso[knee][0] if knee < len(iso) else None, "Q_knee_bracket_bytes": bracket}
    # gap sweep at one burst size: aggregate issue time and period vs the gap (Eq. 1)
    sweep = []
    B = gap_sweep_B or Bs[len(Bs) // 2]
    V = K * B
    rec1 = X.xs_recovery()
    X.check(X.xs_recovery_audit(C.byref(m), V, 1, 0.0, 0.0, 1, C.byref(rec1)), "recovery_audit")
    g_star = rec1.G_star_us
    n = n_fit(B, 32)
    for frac in (0.0, 0.25, 0.5, 0.75, 1.0, 1.5, 2.0, 3.0):
        gap_us = frac * max(g_star, 1.0)
        run = run_bursts(target_ptr, target_bytes, K, B, n, int(gap_us * 1e3), store_waves=store_waves)
        tp, ti = C.c_double(), C.c_double()
        X.check(X.xs_burst_gap(C.byref(m), V, gap_us, C.byref(tp), C.byref(ti)), "burst_gap")
        sweep.append({"V": V, "G_us": gap_us, "T_iss_us": run.steady(run.iss_us),
                      "period_us": run.total_span_us / n, "pred_T_iss_us": ti.value, "pred_period_us": tp.value})
    log(f"[calibrate] {sink} K={K}: T0 = {m.t0_a_us:.3f} us + {m.t0_b_us_per_byte * 1e6:.3f} us/MB, "
        f"R = {m.R_bytes_per_us / 1e3:.1f} GB/s, Q = {model['Q_bytes']}, knee V = {model['knee_V_bytes']}")
    return Calibration(sink, K, model, rec, zg, iso, sweep)


def producer_sweep(target_ptr: int, target_bytes: int, Ks, B: int, store_waves: int = 1,
                   run_bytes: int = 240 << 20):
    """The store path against the producer count K at B bytes per producer and burst (Sec. 3.1:
    the microbenchmark's K axis): per K, the isolated burst's issue time (first start to last
    issued store), the aggregate zero-gap drain rate K B / period, and the steady per-producer
    period when each producer waits for its stores to complete before the next burst
    (XS_MB_COMPLETION, the completion-coupled schedule of Sec. 3.2). Each zero-gap run stores
    about run_bytes in all (at fresh addresses), several times what the sink absorbs before it
    pushes back, so the period is the drain's and not the capacity's: with few producers the
    bytes per producer and burst grow (powers of two from B) to keep a run within the
    microbenchmark's 256 bursts."""
    out = []
    for K0 in Ks:
        K, Bk = int(K0), int(B)
        while K * Bk * 256 < run_bytes and target_bytes % (2 * Bk) == 0:
            Bk *= 2
        n = int(max(2, min(256, -(-run_bytes // (K * Bk)), target_bytes // (K * Bk))))
        B_ = Bk
        iso = float(np.median([run_bursts(target_ptr, target_bytes, K, B_, 1, 0, store_waves=store_waves)
                               .aligned_iss_us[0] for _ in range(3)]))
        zg = run_bursts(target_ptr, target_bytes, K, B_, n, 0, store_waves=store_waves)
        cp = run_bursts(target_ptr, target_bytes, K, B_, n, 0, mode=X.XS_MB_COMPLETION, store_waves=store_waves)
        period = zg.total_span_us / n
        out.append({"K": K, "B": B_, "V": K * B_, "bursts": n, "isolated_issue_us": iso, "zero_gap_period_us": period,
                    "drain_GBps": K * B_ / period / 1e3, "completion_period_us": cp.steady(cp.period_us),
                    "completion_GBps": K * B_ / (cp.total_span_us / n) / 1e3})
    return out


def to_model(cal: Calibration, capacity: str = "fluid") -> X.xs_model:
    """xs_model from a calibration; capacity "fluid" takes the xs_model_fit Q, "knee" the lower
    end of the knee bracket (the largest volume seen absorbed without stalling)."""
    m = cal.model
    Q = m["Q_bytes"] if m["Q_bytes"] is not None else math.inf
    if capacity == "knee" and m.get("Q_knee_bracket_bytes"):
        Q = m["Q_knee_bracket_bytes"][0]
    return X.xs_model(m["t0_a_us"], m["t0_b_us_per_byte"], m["R_bytes_per_us"], Q, m["K"], 0)


def save(cals, path: str) -> None:
    with open(path, "w") as f:
        json.dump([asdict(c) for c in cals], f, indent=1)
