"""Slow-sink pacing sweep (post-issue backpressure on a real slow path).

The EP layer's combine windows are placed in fine-grained host-coherent memory
(hipHostMalloc coherent), so the Linear-2 epilogue stores (the bursts of Sec. 4.3) drain
across the host link; the same layer with HBM combine windows is the local-memory control
(Sec. 3.1). Layers:
  * tiny: T=256, H=512, 8 experts, top-2, I=1024, 4 windows (512 KiB of combine stores);
  * tiny_T32768: the same dimensions at 32768 tokens (64 MiB of combine stores), enough to
    exceed the sink's post-issue capacity.
First both sinks are calibrated with the remote-store microbenchmark (calibrate.py). Then, for
each policy (Expert-Wave burst issue, Alg. 1 interleave at the anti-starvation lead,
chunked bursts, the model-driven AUTO) and producer cap, the fused layer is timed with HIP
events around the persistent kernel and its device trace gives every Linear-2 tile's issue
span (mainloop end -> last store issued):
  (interleave_dyn: the same rule with tiles claimed from shared counters, XS_CLAIM_DYNAMIC)
  * measured stall = sum over tiles of [span - median span of the HBM control]_+, and its
    share of the producers' time (stall / (producers x kernel time));
  * predicted stall = xs_model_predict (Eqs. 3-6) on the burst sequence reconstructed from
    the trace (epilogues with overlapping issue intervals form one burst of their bytes; G
    is the gap to the next burst) with the calibrated host-sink (T0, R) and the capacity at
    the lower end of the measured knee bracket, weighted by the tiles in each burst.
Usage: python -m paper_2607_23264_amd.slow_sink [--out FILE] [--quick]
"""
from __future__ import annotations

import argparse
import ctypes as C
import dataclasses
import json
import sys

import numpy as np
import torch

from . import xstage as X
from .calibrate import calibrate, to_model
from .layer import EPLayer, HostCoherent, Shape, pacing


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def trace_l2(buf, cnt, rate):
    n = min(int(cnt.item()), buf.shape[0])
    r = buf[:n].cpu().numpy().astype(np.int64)
    l2 = r[(r[:, 0] >> 56) == 2]
    us = 1e6 / rate
    t_origin = r[:, 1].min()
    return (l2[:, 2] - t_origin) * us, (l2[:, 3] - l2[:, 2]) * us, (r[:, 3].max() - t_origin) * us


def bursts_from_trace(start, span, bytes_per_tile):
    """Epilogues whose issue intervals overlap form one burst: (V, issue span, gap after)."""
    order = np.argsort(start)
    s, e = start[order], start[order] + span[order]
    groups = []
    g0, gend, n = s[0], e[0], 1
    for i in range(1, len(s)):
        if s[i] <= gend:
            gend = max(gend, e[i])
            n += 1
        else:
            groups.append((g0, gend, n))
            g0, gend, n = s[i], e[i], 1
    groups.append((g0, gend, n))
    out = []
    for i, (a, b, n) in enumerate(groups):
        nxt = groups[i + 1][0] if i + 1 < len(groups) else b
        out.append((n * bytes_per_tile, b - a, max(0.0, nxt - b)))
    return out


def predicted_stall(model: X.xs_model, bursts, bytes_per_tile) -> float:
    """Producer-time stall: each burst's predicted excess issue time (Eqs. 3-6 and the stalled
    reading) times the number of tiles (producers) that issued it."""
    n = len(bursts)
    arr = (X.xs_burst * n)(*[X.xs_burst(V, model.t0_a_us + model.t0_b_us_per_byte * V, G) for V, _, G in bursts])
    out = (X.xs_burst_pred * n)()
    X.check(X.xs_model_predict(C.byref(model), arr, n, 0.0, out), "model_predict")
    return float(sum(o.stall_us * (b[0] / bytes_per_tile) for o, b in zip(out, bursts)))


def calibrate_sinks(K, Bs, store_waves, target_bytes=1 << 30):
    host = HostCoherent(target_bytes)
    hbm = torch.empty(target_bytes // 2, dtype=torch.int16, device="cuda")
    try:
        ch = calibrate(host.ptr, host.nbytes, "host-coherent", K, Bs, store_waves=store_waves, log=log)
        cd = calibrate(hbm.data_ptr(), hbm.numel() * 2, "hbm", K, Bs, store_waves=store_waves, log=log)
    finally:
        host.free()
    return ch, cd


def sweep_layer(cfg, host_model, caps, chunks, reps, rate):
    import synth
    inp = synth.ep_inputs(cfg, 0)
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, 0, cfg.E)
    tile_bytes = (cfg.T * cfg.k // cfg.E) * 256 * 2   # rows of an expert's M-block x 256 columns
    tile_bytes = min(tile_bytes, 256 * 256 * 2)
    P1 = cfg.I // 128
    configs = [("burst", X.XS_POLICY_BURST, 0, 0, 0)]
    configs += [(f"chunk{c}", X.XS_POLICY_CHUNK, c, 0, 0) for c in chunks]
    configs += [("interleave", X.XS_POLICY_INTERLEAVE, 0, 0, 0), ("interleave_4xlead", X.XS_POLICY_INTERLEAVE, 0, 4, 0),
                ("auto", X.XS_POLICY_AUTO, 0, 0, 0), ("interleave_dyn", X.XS_POLICY_INTERLEAVE, 0, 0, 1)]
    results, control = [], {}
    for where in ("hbm", "host"):
        lay = EPLayer(s, combine_host=(where == "host"))
        lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
        buf = torch.zeros((16384, 4), dtype=torch.int64, device="cuda")
        cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
        e0, e1 = X.HipEvents(1), X.HipEvents(1)
        for cap in caps:
            for name, pol, chunk, lead_mult, claim in configs:
                knee = -(-(cap or 256) // P1)          # App. A.2 anti-starvation lead
                p = pacing(pol, lead=lead_mult * knee, chunk=chunk, max_producers=cap,
                           model=host_model if pol == X.XS_POLICY_AUTO else None, claim=claim)
                times = []
                for _ in range(reps):
                    cnt.zero_()
                    lay.L.events[X.XS_EV_FFN], lay.L.events[X.XS_EV_FFN_END] = e0.ev[0], e1.ev[0]
                    lay.fused(p, X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr()))
                    torch.cuda.synchronize()
                    times.append(X.HipEvents.elapsed_ms_pair(e0.ev[0], e1.ev[0]) * 1e3)
                lay.L.events[X.XS_EV_FFN], lay.L.events[X.XS_EV_FFN_END] = None, None
                if int(lay.status.item()):
                    raise RuntimeError(f"device status {int(lay.status.item())}")
                start, span, kern_us = trace_l2(buf, cnt, rate)
                if where == "hbm":
                    control[(cap, name)] = float(np.median(span))
                meas = float(np.maximum(0.0, span - control[(cap, name)]).sum())
                pred = predicted_stall(host_model, bursts_from_trace(start, span, tile_bytes), tile_bytes) \
                    if where == "host" else None
                row = {"layer": cfg.name, "sink": where, "policy": name, "chunk": chunk,
                       "max_producers": cap or 256, "kernel_us_median": float(np.median(times)),
                       "kernel_us_p10": float(np.percentile(times, 10)),
                       "kernel_us_p90": float(np.percentile(times, 90)),
                       "l2_span_us_median": float(np.median(span)), "l2_span_us_p90": float(np.percentile(span, 90)),
                       # share of the producers' kernel time spent in issue beyond the control
                       "stall_measured_us": meas, "stall_fraction": meas / max((cap or 256) * kern_us, 1e-9),
                       "stall_predicted_us": pred}
                results.append(row)
                log(f"[slow-sink] {cfg.name} {where} cap={cap or 256} {name}: {row['kernel_us_median']:.1f} us, "
                    f"span med {row['l2_span_us_median']:.2f} p90 {row['l2_span_us_p90']:.2f} us, "
                    f"stall {meas:.1f} us, pred {pred}")
        del lay
        torch.cuda.empty_cache()
    return results


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--reps", type=int, default=5)
    a = ap.parse_args()
    import synth
    torch.cuda.set_device(0)
    rate = X.xs_clock_rate_hz()
    K = 256
    Bs = [4096, 8192, 16384, 32768, 65536, 131072, 262144]
    ch, cd = calibrate_sinks(K, Bs, store_waves=8)
    host_model = to_model(ch, capacity="knee")
    report = {"calibration": [dataclasses.asdict(ch), dataclasses.asdict(cd)], "sweeps": []}
    layers = [synth.EP_TINY, dataclasses.replace(synth.EP_TINY, name="ep_tiny_dims_T32768", T=32768)]
    caps = [16, 0] if a.quick else [16, 64, 0]
    chunks = [1, 8] if a.quick else [1, 2, 4, 8, 16, 32, 64]
    for cfg in layers:
        report["sweeps"] += sweep_layer(cfg, host_model, caps, chunks, a.reps, rate)
    speed = {}
    for cfg in layers:
        for cap in caps:
            rows = [r for r in report["sweeps"] if r["layer"] == cfg.name and r["sink"] == "host"
                    and r["max_producers"] == (cap or 256)]
            burst = next(r for r in rows if r["policy"] == "burst")
            best = min((r for r in rows if r["policy"] != "burst"), key=lambda r: r["kernel_us_median"])
            speed[f"{cfg.name}/cap{cap or 256}"] = {
                "burst_us": burst["kernel_us_median"], "best_policy": best["policy"],
                "best_us": best["kernel_us_median"], "speedup_over_burst": burst["kernel_us_median"] / best["kernel_us_median"],
                "burst_stall_measured_us": burst["stall_measured_us"], "burst_stall_predicted_us": burst["stall_predicted_us"],
                "best_stall_measured_us": best["stall_measured_us"], "best_stall_predicted_us": best["stall_predicted_us"]}
    report["pacing_speedup_host"] = speed
    if a.out:
        with open(a.out, "w") as f:
            json.dump(report, f, indent=1, default=float)
    print(json.dumps(speed), flush=True)


if __name__ == "__main__":
    main()
