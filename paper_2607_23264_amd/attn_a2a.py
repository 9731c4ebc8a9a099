"""Attention with the post-attention Ulysses All-to-All on one GPU's share (Sec. 4.4; Sec. 5.4,
Table 4 and Fig. 7; App. B).

For each sequence length M (8 local heads, head_dim 128, 8 destination windows) and each sink
(windows in HBM, or in fine-grained host-coherent memory, whose stores cross the host link):
  * FA-only  xs_attention(XS_ATTN_LOCAL): attention into a local output;
  * Serial   FA-only followed by xs_ulysses_copy (the unfused exchange);
  * Fused    xs_attention(XS_ATTN_WINDOWS): the output owner stores each finished tile into its
             destination window and goes on with its next Q-loop;
  * Coupled  xs_attention(XS_ATTN_WINDOWS_COUPLED): the same, but the producer waits for its
             stores to become visible at system scope before the next Q-loop (the
             completion-coupled issuer, measured rather than only predicted).
Reported per cell: medians of interleaved rounds, E_res = Fused - FA-only, the speedup over
Serial, Coupled - FA-only, and from the device trace of a fused run the per-tile Q-loop and
the per-K/V-tile slope sigma.
The recovery audit of App. B then uses the sink's calibrated Burst-Gap model (calibrate.py,
K = the attention grid): burst per producer B_t = 128 x 128 x 2 bytes, aggregate V = K B_t,
recovery gap G* = [V / R - T0(V)]_+ (Eq. 2), the recurrence over a producer's output
boundaries with the measured Q-loop as gap (Eqs. 3-6, xs_model_predict), the tile-aligned
threshold M_ub* = b_n ceil(G* / sigma), and the completion-coupled residual predicted as one
full drain of V per output boundary of a producer.
Usage: python -m paper_2607_23264_amd.attn_a2a [--M 8192 16384 32768] [--out FILE]
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import math
import sys

import numpy as np
import torch

from . import xstage as X
from .calibrate import calibrate, to_model
from .layer import HostCoherent

B_M, B_N, HEAD_DIM = 128, 64, 128          # output tile rows, K/V tile rows, head_dim


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _timed(fns, reps, rounds=3):
    """Median per call of each function over interleaved rounds."""
    for fn in fns:
        fn()
    torch.cuda.synchronize()
    out = [[] for _ in fns]
    for _ in range(rounds):
        for i, fn in enumerate(fns):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            out[i].append(e0.elapsed_time(e1) / reps * 1e3)
    return [float(np.median(x)) for x in out]


def default_grid() -> int:
    return 3 * torch.cuda.get_device_properties(0).multi_processor_count


class Share:
    """Device inputs and outputs of one M; windows are attached per sink."""

    def __init__(self, cfg, seed=0):
        import synth
        inp = synth.attn_inputs(cfg, seed)
        dev = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int16)).cuda()
        self.cfg = cfg
        self.q, self.k, self.v = dev(inp["q"]), dev(inp["k"]), dev(inp["v"])
        self.o = torch.empty_like(self.q)
        self.out_bytes = cfg.heads * cfg.M * cfg.head_dim * 2

    def windows(self, base_ptr: int):
        c = self.cfg
        rows = c.M // c.W
        row_bytes = c.heads * c.head_dim * 2
        return X.windows([X.window((base_ptr + g * rows * row_bytes, rows, row_bytes)) for g in range(c.W)])

    def desc(self, wins=None, max_producers=0):
        c = self.cfg
        return X.xs_attn(c.heads, c.M, c.head_dim, c.W if wins is not None else 0, 0.0, max_producers,
                         self.q.data_ptr(), self.k.data_ptr(), self.v.data_ptr(),
                         0 if wins is not None else self.o.data_ptr(), wins)


def measure(share: Share, base_ptr: int, reps: int, rate: float, max_producers=0):
    st = torch.cuda.current_stream().cuda_stream
    c = share.cfg
    wins = share.windows(base_ptr)
    aL, aW = share.desc(None, max_producers), share.desc(wins, max_producers)
    fa = lambda: X.check(X.xs_attention(aL, X.XS_ATTN_LOCAL, None, st))
    cp = lambda: X.check(X.xs_ulysses_copy(share.o.data_ptr(), c.heads, c.M, c.head_dim, wins, c.W, st))
    fu = lambda: X.check(X.xs_attention(aW, X.XS_ATTN_WINDOWS, None, st))
    cc = lambda: X.check(X.xs_attention(aW, X.XS_ATTN_WINDOWS_COUPLED, None, st))

    def serial():
        fa()
        cp()

    t_fa, t_ser, t_fu, t_cc, t_cp = _timed([fa, serial, fu, cc, cp], reps)
    # one traced fused run: per tile [start, end of Q-loop, stores issued]
    tiles = c.heads * (c.M // B_M)
    buf = torch.zeros((tiles, 4), dtype=torch.int64, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    X.check(X.xs_attention(aW, X.XS_ATTN_WINDOWS, X.trace(buf, cnt), st))
    torch.cuda.synchronize()
    r = buf[:min(int(cnt.item()), tiles)].cpu().numpy().astype(np.int64)
    us = 1e6 / rate
    qloop = (r[:, 2] - r[:, 1]) * us
    issue = (r[:, 3] - r[:, 2]) * us
    flops = 4.0 * c.heads * c.M * c.M * c.head_dim
    grid = max_producers or default_grid()
    return {"M": c.M, "grid": min(grid, tiles), "tiles": tiles,
            "fa_us": t_fa, "serial_us": t_ser, "fused_us": t_fu, "coupled_us": t_cc, "a2a_copy_us": t_cp,
            "E_res_us": t_fu - t_fa, "coupled_residual_us": t_cc - t_fa,
            "speedup_vs_serial": t_ser / t_fu,
            "fa_TFLOPs": flops / (t_fa * 1e-6) / 1e12, "fused_TFLOPs": flops / (t_fu * 1e-6) / 1e12,
            "qloop_us_median": float(np.median(qloop)),
            "sigma_us_per_kv_tile": float(np.median(qloop)) / (c.M // B_N),
            "store_issue_us_median": float(np.median(issue)), "store_issue_us_max": float(issue.max()),
            "out_bytes": share.out_bytes}


def audit(model: X.xs_model, cell: dict) -> dict:
    """App. B recovery audit of one cell with a calibrated sink model (xs_recovery_audit): every
    producer's output bursts of one 128 x 128 bf16 tile, all K producers aligned, the median
    Q-loop as the gap."""
    K = cell["grid"]
    Bt = B_M * HEAD_DIM * 2
    V = K * Bt
    boundaries = math.ceil(cell["tiles"] / K)          # output bursts per producer
    G = cell["qloop_us_median"]
    sigma = cell["sigma_us_per_kv_tile"]
    rec = X.xs_recovery()
    X.check(X.xs_recovery_audit(C.byref(model), V, boundaries, G, sigma, B_N, C.byref(rec)), "recovery_audit")
    return {"B_t_bytes": Bt, "K": K, "V_bytes": V, "T0_us": rec.T0_us, "R_GBps": model.R_bytes_per_us / 1e3,
            "Q_bytes": model.Q_bytes if math.isfinite(model.Q_bytes) else None,
            "G_star_us": rec.G_star_us, "qloop_gap_us": G, "rho": rec.rho, "delta_b_bytes": rec.delta_b,
            "guard_ok": bool(rec.guard_ok), "b_iso_bytes": rec.b_iso,
            # the last burst has no Q-loop after it: with every producer aligned, what it and any
            # carried backlog leave undrained shows up after the compute (a conservative bound)
            "E_res_bound_us": rec.tail_us, "predicted_stall_us": rec.stall_us,
            "M_ub_star": rec.M_ub_star if sigma > 0 else None,
            "output_boundaries_per_producer": boundaries, "coupled_residual_predicted_us": rec.coupled_us}


def run(Ms=(8192, 16384, 32768), sinks=("hbm", "host"), reps=None, calibrate_models=True, seed=0):
    import synth
    torch.cuda.set_device(0)
    rate = X.xs_clock_rate_hz()
    grid = default_grid()
    report = {"workload": "Ulysses share: 8 local heads, head_dim 128, 8 windows, bf16 output",
              "grid": grid, "cells": [], "models": {}}
    max_out = max(Ms) * 8 * HEAD_DIM * 2
    host = HostCoherent(max_out) if "host" in sinks else None
    hbm = torch.empty(max_out // 2, dtype=torch.int16, device="cuda") if "hbm" in sinks else None
    try:
        models = {}
        if calibrate_models:
            Bs = [4096, 16384, 32768, 65536, 131072]
            if host is not None:
                tgt = HostCoherent(128 << 20)
                try:
                    ch = calibrate(tgt.ptr, tgt.nbytes, "host-coherent", grid, Bs, store_waves=4, log=log)
                finally:
                    tgt.free()
                models["host"] = to_model(ch, capacity="knee")
                report["models"]["host"] = ch.model
            if hbm is not None:
                tgt = torch.empty(256 << 20, dtype=torch.int16, device="cuda")
                cd = calibrate(tgt.data_ptr(), tgt.numel() * 2, "hbm", grid, Bs, store_waves=4, log=log)
                del tgt
                models["hbm"] = to_model(cd, capacity="knee")
                report["models"]["hbm"] = cd.model
        for M in Ms:
            cfg = synth.AttnConfig(f"attn_up_M{M}_h8_d128_W8", M=M, heads=8, head_dim=HEAD_DIM, W=8)
            share = Share(cfg, seed)
            n = reps or max(2, int(round(12 * 8192 / M)))
            for sink in sinks:
                base = host.ptr if sink == "host" else hbm.data_ptr()
                cell = measure(share, base, n, rate)
                cell["sink"] = sink
                if sink in models:
                    cell["audit"] = audit(models[sink], cell)
                log(f"[attn] {sink} M={M}: FA {cell['fa_us']:.1f} serial {cell['serial_us']:.1f} "
                    f"fused {cell['fused_us']:.1f} coupled {cell['coupled_us']:.1f} us; E_res "
                    f"{cell['E_res_us']:+.1f}, x{cell['speedup_vs_serial']:.3f} over serial")
                report["cells"].append(cell)
            del share
            torch.cuda.empty_cache()
    finally:
        if host is not None:
            host.free()
    report["summary"] = summarize(report["cells"])
    return report


def summarize(cells):
    """Per sink: E_res and speedup per M, and the completion-coupled residual's slope per output
    boundary of a producer (least squares through the cells) beside the model's V / R."""
    out = {}
    for sink in sorted({c["sink"] for c in cells}):
        cs = [c for c in cells if c["sink"] == sink]
        s = {"M": [c["M"] for c in cs], "E_res_us": [c["E_res_us"] for c in cs],
             "speedup_vs_serial": [c["speedup_vs_serial"] for c in cs],
             "coupled_residual_us": [c["coupled_residual_us"] for c in cs]}
        if len(cs) >= 2 and all("audit" in c for c in cs):
            n = np.array([c["audit"]["output_boundaries_per_producer"] for c in cs], dtype=np.float64)
            r = np.array(s["coupled_residual_us"])
            if np.ptp(n) > 0:
                s["coupled_slope_us_per_boundary"] = float(np.polyfit(n, r, 1)[0])
            a = cs[0]["audit"]
            s["model_drain_us_per_boundary"] = a["V_bytes"] / (a["R_GBps"] * 1e3)
            s["G_star_us"] = a["G_star_us"]
            s["M_ub_star"] = [c["audit"]["M_ub_star"] for c in cs]
            s["rho"] = [c["audit"]["rho"] for c in cs]
        out[sink] = s
    return out


def launches(M: int, mode: str, n: int, seed=0):
    """n back-to-back launches of one mode at one M and nothing else (for kernel statistics
    and counter passes): fa = XS_ATTN_LOCAL, fused = XS_ATTN_WINDOWS into HBM windows."""
    import synth
    torch.cuda.set_device(0)
    cfg = synth.AttnConfig(f"attn_up_M{M}_h8_d128_W8", M=M, heads=8, head_dim=HEAD_DIM, W=8)
    share = Share(cfg, seed)
    st = torch.cuda.current_stream().cuda_stream
    win = torch.empty(share.out_bytes // 2, dtype=torch.int16, device="cuda")
    wins = share.windows(win.data_ptr())
    a = share.desc(wins if mode == "fused" else None)
    md = X.XS_ATTN_WINDOWS if mode == "fused" else X.XS_ATTN_LOCAL
    torch.cuda.synchronize()
    for _ in range(n):
        X.check(X.xs_attention(a, md, None, st))
    torch.cuda.synchronize()
    log(f"[attn] {n} {mode} launches at M={M} done")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--M", type=int, nargs="+", default=[8192, 16384, 32768])
    ap.add_argument("--launches", choices=["fa", "fused"], default=None,
                    help="only launch this mode --reps times at the first M (for rocprofv3)")
    ap.add_argument("--sinks", nargs="+", default=["hbm", "host"])
    ap.add_argument("--reps", type=int, default=None)
    ap.add_argument("--no-calibration", action="store_true")
    ap.add_argument("--out", default=None)
    a = ap.parse_args()
    if a.launches:
        launches(a.M[0], a.launches, a.reps or 20)
        return
    rep = run(tuple(a.M), tuple(a.sinks), a.reps, not a.no_calibration)
    if a.out:
        with open(a.out, "w") as f:
            json.dump(rep, f, indent=1, default=float)
    print(json.dumps(rep, default=float), flush=True)


if __name__ == "__main__":
    main()
