"""Store pacing against a slow sink: the EP layer with combine windows in host-coherent memory.

The Linear-2 epilogue stores (the bursts of Sec. 4.3) of the combine windows placed in
fine-grained host-coherent memory (hipHostMalloc coherent) drain across the host link; the same
layer with every window in HBM is the local-memory control (Sec. 3.1). Two layers:
  * tiny (the c1 dimensions: T=256, H=512, 8 experts, top-2, I=1024, 4 windows), every combine
    window on the sink: 512 KiB of combine stores per layer, swept over chunk sizes and producer
    caps;
  * the DeepSeek-V3-like share with two of its eight source windows on the sink (a quarter of
    the combine bytes), uniform and Zipf(1.2) routing: Eq. 9 holds at the sink's drain rate, and
    the skewed routing gives the long runs of aligned Linear-2 epilogues the paper describes.
Per policy (Expert-Wave burst, cross-wave interleave at the anti-starvation lead, chunked, and
AUTO with the calibrated model):
  * kernel time (HIP events around the persistent kernel, median of repetitions), on the sink
    and on the HBM control;
  * measured issue stall: from one traced run (ext records), the sum over Linear-2 tiles of the
    epilogue issue span beyond the HBM control's median span, per producer; the staging wait
    (App. A.2's MMA-side wait on this design: the first wave's wait before the next mainloop for
    its previous stores); the dependency waits and the mainloop time against the control;
  * predicted stall: the library's audit of the same order (xs_pacing_audit_run: the schedule's
    aligned bursts through the backlog recurrence and capacity guard) with the calibrated sink
    model and the mainloop times of the HBM control's trace (xs_trace_tile_times).
This module only allocates, launches and takes sums and medians of trace timestamps; the model
arithmetic runs in the library.
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
from .calibrate import calibrate, producer_sweep, to_model
from .layer import EPLayer, HostCoherent, Shape, pacing


def log(*a):
    print(*a, file=sys.stderr, flush=True)


SWEEP_KS = (1, 2, 4, 8, 16, 32, 64, 128, 256)


def calibrate_sinks(K, Bs, store_waves, target_bytes=1 << 30, sweep_B=None):
    """Burst-Gap calibration of the host-coherent sink and the HBM control at K producers; with
    sweep_B also the producer-count sweep of both at sweep_B bytes per producer (returned as the
    third value, {sink: rows})."""
    host = HostCoherent(target_bytes)
    hbm = torch.empty(target_bytes // 2, dtype=torch.int16, device="cuda")
    sweeps = {}
    try:
        ch = calibrate(host.ptr, host.nbytes, "host-coherent", K, Bs, store_waves=store_waves, log=log)
        cd = calibrate(hbm.data_ptr(), hbm.numel() * 2, "hbm", K, Bs, store_waves=store_waves, log=log)
        if sweep_B:
            sweeps["host-coherent"] = producer_sweep(host.ptr, host.nbytes, SWEEP_KS, sweep_B, store_waves)
            sweeps["hbm"] = producer_sweep(hbm.data_ptr(), hbm.numel() * 2, SWEEP_KS, sweep_B, store_waves)
            for k, rows in sweeps.items():
                log(f"[calibrate] {k} producer sweep at B = {sweep_B}: " + ", ".join(
                    f"K={r['K']} {r['drain_GBps']:.1f} GB/s (iso {r['isolated_issue_us']:.1f} us)" for r in rows))
    finally:
        host.free()
    return (ch, cd, sweeps) if sweep_B else (ch, cd)


class Traced:
    """A traced run's records (with ext records) on the host."""

    def __init__(self, lay: EPLayer, pol: X.xs_pacing, cap_records: int = 65536):
        buf = torch.zeros((cap_records, 4), dtype=torch.int64, device="cuda")
        ext = torch.zeros((cap_records, 4), dtype=torch.int64, device="cuda")
        cnt = torch.zeros((1,), dtype=torch.int32, device="cuda")
        lay.fused(pol, X.xs_trace(buf.data_ptr(), buf.shape[0], cnt.data_ptr(), ext.data_ptr()))
        torch.cuda.synchronize()
        n = min(int(cnt.item()), cap_records)
        self.r = np.ascontiguousarray(buf[:n].cpu().numpy().astype(np.uint64))
        self.x = np.ascontiguousarray(ext[:n].cpu().numpy().astype(np.uint64))
        self.n = n
        us = 1e6 / X.xs_clock_rate_hz()
        r = self.r.astype(np.int64)
        x = self.x.astype(np.int64)
        self.kind = r[:, 0] >> 56
        self.issue_us = (r[:, 3] - r[:, 2]) * us
        self.stage_us = x[:, 1] * us
        self.dep_us = (x[:, 0] - r[:, 1]) * us
        self.main_us = (r[:, 2] - x[:, 0]) * us

    def tile_times(self, min_rows: int = 0):
        t1, t2, t3 = C.c_double(), C.c_double(), C.c_double()
        X.check(X.xs_trace_tile_times(self.r.ctypes.data, self.x.ctypes.data, self.n, min_rows, C.byref(t1),
                                      C.byref(t2), C.byref(t3)), "trace_tile_times")
        return t1.value, t2.value, t3.value


def rotated_us(lay: EPLayer, pols: list, reps: int, clocks: list | None = None) -> list:
    """Kernel times of every pacing in pols, reps launches each, the order rotated from one
    repetition to the next (round r starts at policy r mod n), so that clock drift and the
    first-run boost fall on every policy alike. Returns one list of times per pacing; with
    clocks, also appends per pacing the driver's shader clock sampled during its launches."""
    import time
    from .profiling import ClockSampler
    ev = X.HipEvents(2)
    lay.L.events[X.XS_EV_FFN], lay.L.events[X.XS_EV_FFN_END] = ev.ev[0], ev.ev[1]
    out = [[] for _ in pols]
    windows = [[] for _ in pols]
    n = len(pols)
    with ClockSampler() as sclk:
        for r in range(reps):
            for q in range(n):
                j = (r + q) % n
                t0 = time.perf_counter()
                lay.fused(pols[j])
                torch.cuda.synchronize()
                windows[j].append((t0, time.perf_counter()))
                out[j].append(X.HipEvents.elapsed_ms_pair(ev.ev[0], ev.ev[1]) * 1e3)
    if clocks is not None:
        clocks.extend(sclk.summary(w) for w in windows)
    lay.L.events[X.XS_EV_FFN], lay.L.events[X.XS_EV_FFN_END] = None, None
    if int(lay.status.item()):
        raise RuntimeError(f"device status {int(lay.status.item())}: {X.xs_strerror(int(lay.status.item())).decode()}")
    return out


def audit(lay: EPLayer, pol: X.xs_pacing) -> X.xs_pacing_audit:
    au = X.xs_pacing_audit()
    X.check(X.xs_pacing_audit_run(C.byref(lay.L), C.byref(pol), C.byref(au)), "pacing_audit")
    return au


POLICY_NAMES = {X.XS_POLICY_BURST: "burst", X.XS_POLICY_INTERLEAVE: "interleave", X.XS_POLICY_CHUNK: "chunk"}


def evaluate(name: str, make_layer, policies: dict, model: X.xs_model, sink_share: float, reps: int,
             claim: int = X.XS_CLAIM_DYNAMIC) -> dict:
    """Every policy on the HBM control and on the sink layer: kernel time, measured and predicted
    stall. make_layer(on_sink) returns an uploaded EPLayer; policies maps a name to
    (policy, lead, chunk, max_producers)."""
    out = {"layer": name, "sink_share": sink_share, "policies": {}}
    control = {}                 # (policy, lead, chunk, producers) -> kernel time and trace
    ctrl = make_layer(False)
    counts = None
    try:
        s = ctrl.s
        c = ctrl.expert_counts.sum(0).cpu().numpy()
        counts = [int(v) for v in c[s.e_begin:s.e_begin + s.n_experts]]   # the layout's rows per local expert
        keys, pols = [], []
        for pname, (pol, lead, chunk, cap) in policies.items():
            if pol == X.XS_POLICY_AUTO or (pol, lead, chunk, cap) in keys:
                continue
            keys.append((pol, lead, chunk, cap))
            pols.append(pacing(pol, lead=lead, chunk=chunk, max_producers=cap, claim=claim))
        for key, p, times in zip(keys, pols, rotated_us(ctrl, pols, reps)):
            control[key] = {"kernel_us": float(np.median(times)), "trace": Traced(ctrl, p)}
        ref = next(v for k, v in control.items() if k[0] == X.XS_POLICY_INTERLEAVE)
        tl1, tl2, _ = ref["trace"].tile_times(min_rows=0)
        out["control_tile_times_us"] = {"T_L1": tl1, "T_L2": tl2}
    finally:
        ctrl.close()
        del ctrl
        torch.cuda.empty_cache()
    lay = make_layer(True)
    try:
        names = list(policies)
        pols = [pacing(pol, lead=lead, chunk=chunk, max_producers=cap, claim=claim, model=model, t_l1_us=tl1,
                       t_l2_us=tl2, expert_rows=counts, sink_share=sink_share)
                for (pol, lead, chunk, cap) in policies.values()]
        clocks = []
        all_times = rotated_us(lay, pols, reps, clocks)
        for pname, p, times, clk in zip(names, pols, all_times, clocks):
            pol, lead, chunk, cap = policies[pname]
            au = audit(lay, p)
            chosen = au.policy
            tr = Traced(lay, p)
            G = au.producers
            base = control.get((chosen, lead, au.chunk, cap))
            ctr = base["trace"] if base else None
            l2 = tr.kind == 2
            if ctr is not None:
                excess = np.maximum(0.0, tr.issue_us[l2] - float(np.median(ctr.issue_us[ctr.kind == 2])))
                stage = np.maximum(0.0, tr.stage_us - float(np.median(ctr.stage_us)))
                main_excess = float(tr.main_us.sum() - ctr.main_us.sum()) / G
                dep_excess = float(tr.dep_us.sum() - ctr.dep_us.sum()) / G
            else:
                excess, stage, main_excess, dep_excess = tr.issue_us[l2] * 0, tr.stage_us * 0, 0.0, 0.0
            k_us = float(np.median(times))
            i = next(j for j in range(au.n_cand) if au.cand_policy[j] == chosen and au.cand_chunk[j] == au.chunk)
            row = {"policy": POLICY_NAMES[chosen], "chunk": au.chunk, "lead_rows": au.lead_rows, "producers": G,
                   "kernel_us": k_us, "kernel_us_p10": float(np.percentile(times, 10)),
                   "kernel_us_p90": float(np.percentile(times, 90)),
                   "control_kernel_us": base["kernel_us"] if base else None,
                   "stall_measured_us_per_producer": float(excess.sum()) / G,
                   # all the time the producers lose on the sink: kernel time beyond the control's
                   "time_lost_us": k_us - base["kernel_us"] if base else None,
                   "stall_predicted_us_per_producer": au.cand_stall_us[i],
                   "mma_stall_predicted_us_per_producer": au.cand_mma_stall_us[i],
                   "staging_wait_measured_us_per_producer": float(stage.sum()) / G,
                   "stall_fraction_measured": float(excess.sum()) / G / k_us,
                   "stall_fraction_predicted": au.cand_stall_us[i] / k_us,
                   "l2_issue_us_median": float(np.median(tr.issue_us[l2])),
                   "l2_issue_us_p90": float(np.percentile(tr.issue_us[l2], 90)),
                   "mainloop_excess_us_per_producer": main_excess,
                   "dependency_wait_excess_us_per_producer": dep_excess,
                   "guard_failures_predicted": au.cand_guard_fail[i], "bursts_predicted": au.cand_bursts[i],
                   "rate_feasible_eq9": bool(au.rate_feasible),
                   "sclk_MHz_median": clk["median"] if clk else None}
            if pol == X.XS_POLICY_AUTO:
                row["auto_candidates"] = [{"policy": POLICY_NAMES[au.cand_policy[j]], "chunk": au.cand_chunk[j],
                                           "stall_predicted_us": au.cand_stall_us[j]} for j in range(au.n_cand)]
            out["policies"][pname] = row
            log(f"[slow-sink] {name} {pname}: {k_us:.1f} us (control {row['control_kernel_us']}), stall measured "
                f"{row['stall_measured_us_per_producer']:.1f} / predicted {row['stall_predicted_us_per_producer']:.1f} "
                f"us per producer, staging {row['staging_wait_measured_us_per_producer']:.1f}")
    finally:
        lay.close()
        del lay
        torch.cuda.empty_cache()
    burst = out["policies"].get("burst")
    if burst:
        for row in out["policies"].values():
            row["speedup_over_burst"] = burst["kernel_us"] / row["kernel_us"]
    return out


def tiny_layer(cfg, inp):
    def make(on_sink: bool) -> EPLayer:
        s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, 0, cfg.E)
        lay = EPLayer(s, combine_host=on_sink)
        lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
        lay.route()
        lay.layout()
        torch.cuda.synchronize()
        return lay
    return make


def share_layer(cfg, inp, host_sources, precision=X.XS_PREC_BF16):
    def make(on_sink: bool) -> EPLayer:
        experts = list(range(cfg.rank * cfg.E_local, (cfg.rank + 1) * cfg.E_local))
        s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=cfg.rank)
        lay = EPLayer(s, sentinel=False, host_combine_sources=host_sources if on_sink else None,
                      precision=precision)
        lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
        lay.prefill_other_sources(inp["fill"])
        return lay
    return make


def tiny_policies(caps, chunks):
    pol = {}
    for cap in caps:
        suffix = f"_p{cap}" if cap else ""
        pol[f"burst{suffix}"] = (X.XS_POLICY_BURST, 0, 0, cap)
        pol[f"interleave{suffix}"] = (X.XS_POLICY_INTERLEAVE, 0, 0, cap)
        for c in chunks:
            pol[f"chunk{c}{suffix}"] = (X.XS_POLICY_CHUNK, 0, c, cap)
        pol[f"auto{suffix}"] = (X.XS_POLICY_AUTO, 0, 0, cap)
    return pol


SHARE_POLICIES = {"burst": (X.XS_POLICY_BURST, 0, 0, 0), "interleave": (X.XS_POLICY_INTERLEAVE, 0, 0, 0),
                  "chunk2": (X.XS_POLICY_CHUNK, 0, 2, 0), "auto": (X.XS_POLICY_AUTO, 0, 0, 0)}


def most_loaded_rank(logits: np.ndarray, k: int, E: int, W: int) -> int:
    """The destination window receiving the most rows, from the library's routing and layout of
    every source (n_src x T tokens)."""
    n_src, T, _ = logits.shape
    st = torch.cuda.current_stream().cuda_stream
    i32 = dict(dtype=torch.int32, device="cuda")
    lg = torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)).cuda()
    idx = torch.empty((n_src, T, k), **i32)
    w = torch.empty((n_src, T, k), dtype=torch.float32, device="cuda")
    X.check(X.xs_route_topk_softmax(lg.data_ptr(), n_src * T, E, k, 0, idx.data_ptr(), w.data_ptr(), st), "route")
    cap = 1                     # only the counts are wanted: rows past capacity are not recorded
    ec, sb, eo = torch.empty((n_src, E), **i32), torch.empty((n_src, E), **i32), torch.empty((E,), **i32)
    dc, sr, rs = torch.empty((W,), **i32), torch.empty((n_src, T, k), **i32), torch.empty((W, cap), **i32)
    status = torch.zeros((1,), **i32)
    nb = C.c_int64()
    X.check(X.xs_dispatch_layout_workspace_bytes(n_src, T, E, C.byref(nb)), "layout workspace")
    ws = torch.empty((max(1, nb.value),), dtype=torch.uint8, device="cuda")
    X.check(X.xs_dispatch_layout(idx.data_ptr(), n_src, T, k, E, W, cap, ec.data_ptr(), sb.data_ptr(), eo.data_ptr(),
                                 dc.data_ptr(), sr.data_ptr(), rs.data_ptr(), ws.data_ptr(), ws.numel(),
                                 status.data_ptr(), st), "layout")
    torch.cuda.synchronize()
    return int(dc.cpu().numpy().argmax())


def share_inputs(routing: str, seed: int = 0):
    """Inputs of the DeepSeek-V3-like share; Zipf routing puts this GPU on the most loaded rank,
    taken from the library's own routing and layout of every source."""
    import synth
    cfg = dataclasses.replace(synth.EP_DSV3_SHARE, routing=routing)
    inp = {"logits": synth.ep_logits(cfg, seed), "x": synth.ep_x(cfg, seed)}
    rank = most_loaded_rank(inp["logits"], cfg.k, cfg.E, cfg.W) if routing == "zipf" else 0
    cfg = dataclasses.replace(cfg, rank=rank)
    experts = list(range(rank * cfg.E_local, (rank + 1) * cfg.E_local))
    inp["w1"], inp["w2"] = synth.ep_weights(cfg, experts, seed)
    inp["fill"] = synth.ep_remote_combine_fill(cfg, seed)
    return cfg, inp


def run(quick=False, reps=5, routings=("zipf", "uniform"), sink_windows=(1, 2), seed=0,
        mx_routings=("uniform",)):
    """Calibrate the sink, then evaluate the tiny layer and the share layers: bf16 for every
    routing in routings, and MXFP8 (W8A8, the precision of the paper's EP measurements) for
    every routing in mx_routings, each with sink_windows of its source windows on the sink."""
    import synth
    torch.cuda.set_device(0)
    # five burst sizes (1 to 64 MiB aggregate): enough below the knee for the floor line and
    # past it for the capacity bracket
    ch, cd, sweeps = calibrate_sinks(256, [4096, 16384, 65536, 131072, 262144], store_waves=8,
                                     target_bytes=256 << 20, sweep_B=65536)
    model = to_model(ch, capacity="knee")
    report = {"sink_model": {k: ch.model[k] for k in ("t0_a_us", "t0_b_us_per_byte", "R_bytes_per_us",
                                                        "Q_knee_bracket_bytes", "Q_bytes")},
              "hbm_R_bytes_per_us": cd.model["R_bytes_per_us"], "gap_sweep": ch.gap_sweep,
              "producer_sweep": sweeps, "layers": []}
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, seed)
    caps = [16, 0] if quick else [8, 16, 32, 64, 0]
    chunks = [1, 8] if quick else [1, 2, 4, 8, 16, 32, 64]
    report["layers"].append(evaluate(cfg.name + " (every combine window on the sink)", tiny_layer(cfg, inp),
                                     tiny_policies(caps, chunks), model, 1.0, reps))
    for routing in dict.fromkeys(tuple(routings) + tuple(mx_routings)):
        scfg, sinp = share_inputs(routing, seed)
        others = [q for q in range(scfg.n_src) if q != scfg.rank]
        precs = ([("", X.XS_PREC_BF16)] if routing in routings else []) + \
                ([("MXFP8, ", X.XS_PREC_MXFP8)] if routing in mx_routings else [])
        # one source window on the sink: the average rate leaves the sink half idle (Eq. 9 holds
        # with room), yet aligned Linear-2 bursts can still exceed the capacity; two windows:
        # the sink close to saturation. At MXFP8 the expert GEMMs take about 0.6 of the bf16
        # time for the same combine bytes, so the same windows load the sink more.
        for tag, prec in precs:
            for n_host in sink_windows:
                hosts = others[:n_host]
                report["layers"].append(evaluate(f"{scfg.name} ({tag}{routing}, rank {scfg.rank}; combine windows of "
                                                 f"sources {hosts} on the sink)", share_layer(scfg, sinp, hosts, prec),
                                                 SHARE_POLICIES, model, len(hosts) / scfg.n_src, reps))
        del sinp
    return report


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--reps", type=int, default=5)
    a = ap.parse_args()
    rep = run(quick=a.quick, reps=a.reps)
    if a.out:
        with open(a.out, "w") as f:
            json.dump(rep, f, indent=1, default=float)
    print(json.dumps({L["layer"]: {k: (v["kernel_us"], v.get("speedup_over_burst")) for k, v in L["policies"].items()}
                      for L in rep["layers"]}), flush=True)


if __name__ == "__main__":
    main()
