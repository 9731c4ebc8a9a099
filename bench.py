"""Benchmark of the fused expert-parallel layer share on one MI355X.

One step = one pass of the whole hot path over one batch: route (all sources) -> dispatch
layout -> dispatch stores of this rank's tokens -> persistent Linear-1 / Linear-2 kernel with
the combine-send epilogue -> combine-reduce. Workload: one rank's share of a
DeepSeek-V3-like layer (8 ranks x 4096 tokens, H=7168, 256 experts / 32 local, top-8,
SwiGLU I=2048, 8 destination windows in HBM), synthetic seeded inputs, bf16 with fp32
accumulation. Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
METRIC = "fused EP layer µs + GEMM MFMA util % + dispatch/combine store GB/s, 1 MI355X"
MFMA_PEAK_BF16 = 2.5e15      # dense bf16 FLOP/s
MFMA_PEAK_FP8 = 5.0e15       # dense fp8 FLOP/s
HBM_PEAK = 8.0e12            # B/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--routing", choices=["uniform", "zipf"], default="uniform")
    p.add_argument("--policy", choices=["burst", "interleave", "chunk"], default="interleave")
    p.add_argument("--lead", type=int, default=64,
                   help="lead D in rows (0 = the anti-starvation knee, ceil(grid / P1) = 16 here); "
                        "64 = four knees, the fastest interleave measured on this share")
    p.add_argument("--chunk", type=int, default=2)
    p.add_argument("--claim", choices=["static", "dynamic"], default="dynamic",
                   help="how producers take tiles (dynamic: shared counters, same tile rule)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-phases", action="store_true")
    p.add_argument("--no-scatter", action="store_true", help="skip the TP / SP scatter GEMM lines")
    p.add_argument("--no-slow-sink", action="store_true",
                   help="skip the store-pacing lines against the host-coherent sink (the tiny layer with "
                        "every combine window on the sink; the DeepSeek-V3 share with two of eight)")
    p.add_argument("--no-zipf", action="store_true", help="skip the Zipf(1.2)-routed share line")
    p.add_argument("--no-tiny", action="store_true", help="skip the tiny-layer line (eager and HIP graph)")
    p.add_argument("--no-attn", action="store_true",
                   help="skip the attention + Ulysses exchange line (HBM and host-coherent windows)")
    p.add_argument("--policies", action="store_true",
                   help="also time the fused layer under every pacing policy (phases)")
    p.add_argument("--no-mx", action="store_true", help="skip the MXFP8 (W8A8) and W4A8 layer lines")
    p.add_argument("--no-ring", action="store_true", help="skip the bounded-ring dispatch line")
    p.add_argument("--seed", type=int, default=0)
    return p.parse_args()


def cpu_baseline(cfg, inp, rank, seed, ffn_budget_s=12.0, comb_budget_s=3.0):
    """The oracle, untuned, on a bounded sample of the same layer share: route and layout of
    every source's tokens, dispatch of this rank's tokens, the SwiGLU FFN of local experts on
    as many rows as the layout gives each (synthetic rows of the dispatched distribution) and
    the combine-reduce of this rank's tokens. BLAS threads = the host cores it may use."""
    from oracle import ep as oep
    threads = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    idx = np.empty((cfg.n_src, cfg.T, cfg.k), np.int32)
    w = np.empty((cfg.n_src, cfg.T, cfg.k), np.float32)
    for s in range(cfg.n_src):
        idx[s], w[s] = oep.route_topk_softmax(inp["logits"][s], cfg.k)
    lay = oep.dispatch_layout(idx, cfg.E, cfg.W)
    t_route_layout = time.perf_counter() - t0
    t1 = time.perf_counter()
    sub = idx[rank:rank + 1]
    lay_s = oep.dispatch_layout(sub, cfg.E, cfg.W)
    oep.dispatch(inp["x"][rank:rank + 1], sub, lay_s["slot_row"], cfg.E, cfg.W,
                 int(lay_s["dest_counts"].max()))
    t_disp = time.perf_counter() - t1
    experts = list(range(rank * cfg.E_local, (rank + 1) * cfg.E_local))
    total = lay["expert_counts"].sum(0)
    # the FFN and the combine-reduce run until a time budget is spent; their times are then
    # scaled by the share of the work done (rows, tokens)
    rows_all = int(sum(total[e] for e in experts))
    t2 = time.perf_counter()
    g = np.random.default_rng(seed)
    rows_done, n_exp = 0, 0
    for i, e in enumerate(experts):
        m = int(total[e])
        oep.expert_ffn(synth_rows(g, m, cfg.H), inp["w1"][i], inp["w2"][i])
        rows_done += m
        n_exp += 1
        if time.perf_counter() - t2 > ffn_budget_s:
            break
    t_ffn = (time.perf_counter() - t2) * rows_all / max(1, rows_done)
    t3 = time.perf_counter()
    tok, chunk = 0, 256
    while tok < cfg.T:
        oep.combine_reduce(inp["fill"][tok * cfg.k:(tok + chunk) * cfg.k], w[rank, tok:tok + chunk])
        tok += chunk
        if time.perf_counter() - t3 > comb_budget_s:
            break
    t_comb = (time.perf_counter() - t3) * cfg.T / tok
    wall = time.perf_counter() - t0
    total_s = t_route_layout + t_disp + t_ffn + t_comb
    return {"value": total_s * 1e6, "unit": "us", "cores": threads, "kind": "oracle",
            "sample": (f"route+layout of all {cfg.n_src}x{cfg.T} tokens and dispatch of rank {rank}'s "
                       f"{cfg.T} tokens in full; SwiGLU FFN of {n_exp} of {cfg.E_local} local experts "
                       f"({rows_done} of {rows_all} rows, synthetic rows) scaled by rows; combine-reduce "
                       f"of {tok} of {cfg.T} tokens scaled by tokens; {wall:.1f} s of CPU time"),
            "cpu": cpu_model(),
            "phases_us": {"route_layout": t_route_layout * 1e6, "dispatch": t_disp * 1e6,
                          "expert_ffn": t_ffn * 1e6, "combine_reduce": t_comb * 1e6}}


def cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), else the machine type."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def tiny_line(X, torch, synth, steps=20, warmup=3):
    """The tiny layer (c1: T=256, H=512, 8 experts, top-2, I=1024, 4 windows, one source): one
    step = the whole fused layer, timed eagerly and as a HIP graph replay (the step captured
    once), since it is launch-bound."""
    from paper_2607_23264_amd.layer import EPLayer, Shape, pacing
    cfg = synth.EP_TINY
    inp = synth.ep_inputs(cfg, 0)
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, 0, cfg.E)
    lay = EPLayer(s, sentinel=False)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    pol = pacing(X.XS_POLICY_INTERLEAVE, lead=0, claim=X.XS_CLAIM_DYNAMIC)
    for _ in range(warmup):
        lay.fused(pol)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        lay.fused(pol)
    e1.record()
    torch.cuda.synchronize()
    eager = e0.elapsed_time(e1) * 1e3 / steps
    graph = graph_steps(torch, lay, pol, steps)
    status = int(lay.status.item())
    del lay
    torch.cuda.empty_cache()
    if status:
        raise RuntimeError(f"tiny layer: device status {status}")
    flops = 6.0 * cfg.H * cfg.I * cfg.T * cfg.k
    return {"workload": cfg.name, "us_per_step_eager": eager, "us_per_step_graph": graph["us_per_step"],
            "graph": graph, "flops_per_step": flops}


def zipf_line(X, torch, synth, pol, steps, warmup):
    """The same share with Zipf(1.2) routing, this GPU the most loaded rank: step time and the
    expert-FFN kernel's rate (FLOPs scale with the rows this rank computes)."""
    from paper_2607_23264_amd import slow_sink as ss
    from paper_2607_23264_amd.layer import EPLayer, Shape
    cfg, inp = ss.share_inputs("zipf", 0)
    experts = list(range(cfg.rank * cfg.E_local, (cfg.rank + 1) * cfg.E_local))
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=cfg.rank)
    lay = EPLayer(s, sentinel=False)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(inp["fill"])
    for _ in range(warmup):
        lay.fused(pol)
    torch.cuda.synchronize()
    ev = X.HipEvents(2 * steps)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        lay.L.events[X.XS_EV_FFN] = ev.ev[2 * i]
        lay.L.events[X.XS_EV_FFN_END] = ev.ev[2 * i + 1]
        lay.fused(pol)
    e1.record()
    torch.cuda.synchronize()
    step_us = e0.elapsed_time(e1) * 1e3 / steps
    ffn_us = float(np.mean([ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(steps)])) * 1e3
    rows = int(lay.dest_counts[cfg.rank].item())
    status = int(lay.status.item())
    del lay
    torch.cuda.empty_cache()
    if status:
        raise RuntimeError(f"zipf share: device status {status}")
    flops = 6.0 * cfg.H * cfg.I * rows
    return {"workload": f"{cfg.name} (zipf routing, rank {cfg.rank}, the most loaded)", "us_per_step": step_us,
            "ffn_us": ffn_us, "rows_computed": rows, "ffn_TFLOPs": flops / (ffn_us * 1e-6) / 1e12,
            "mfma_frac": flops / (ffn_us * 1e-6) / MFMA_PEAK_BF16}


def scatter_lines(X, torch, synth, reps=20):
    """TP row-block and Ulysses head-group scatter GEMMs: fused epilogue vs the plain GEMM
    (residual E_res = fused - plain, Sec. 5.4) vs the serial GEMM + permutation copy."""
    import ctypes as C
    st = torch.cuda.current_stream().cuda_stream
    out = {}

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()

    def timed(*fns, rounds=5):
        """Median per call of each function, timed in interleaved rounds (clock drift and
        the first-run boost then fall on every variant alike)."""
        for fn in fns:
            fn()
        torch.cuda.synchronize()
        t = [[] for _ in fns]
        for _ in range(rounds):
            for i, fn in enumerate(fns):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps // rounds):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                t[i].append(e0.elapsed_time(e1) / (reps // rounds) * 1e3)
        return [float(np.median(x)) for x in t]

    tp = synth.TP_ROWBLOCK
    inp = synth.tp_inputs(tp, 0)
    a, bt = dev(inp["a"]), dev(np.ascontiguousarray(inp["b"].T))
    rpd = tp.M // tp.W
    win = torch.empty((tp.W, rpd, tp.N), dtype=torch.int16, device="cuda")
    wins = X.windows([X.window(win[d]) for d in range(tp.W)])
    desc = X.xs_scatter_desc(X.XS_SCATTER_ROW_BLOCK, rpd, 0, 0, 0, 0)
    c = torch.empty((tp.M, tp.N), dtype=torch.int16, device="cuda")
    M, N, K = tp.M, tp.N, tp.K
    f = lambda: X.check(X.xs_gemm_scatter(a.data_ptr(), K, bt.data_ptr(), K, M, N, K, desc, wins, tp.W, None, None, st))
    g = lambda: X.check(X.xs_gemm(a.data_ptr(), K, bt.data_ptr(), K, c.data_ptr(), N, M, N, K, None, st))
    sc = lambda: X.check(X.xs_scatter_copy(c.data_ptr(), N, M, N, desc, wins, tp.W, st))
    out["tp_rowblock"] = _scatter_result(tp.name, 2.0 * M * N * K, 2.0 * M * N,
                                         *timed(f, g, lambda: (g(), sc())))
    del a, bt, win, c
    sp = synth.SP_QKV
    inp = synth.sp_inputs(sp, 0)
    x, wt = dev(inp["x"]), dev(np.ascontiguousarray(inp["w"].T))
    S, Dm = sp.S, sp.Dm
    N = 3 * sp.n_heads * sp.head_dim
    G = sp.n_heads // sp.heads_per_group
    win = torch.empty((G, 3, sp.heads_per_group, S, sp.head_dim), dtype=torch.int16, device="cuda")
    wins = X.windows([X.xs_window(win[q].data_ptr(), 3 * sp.heads_per_group * S, sp.head_dim * 2, None)
                      for q in range(G)])
    desc = X.xs_scatter_desc(X.XS_SCATTER_HEAD_GROUP, 0, 3, sp.n_heads, sp.head_dim, sp.heads_per_group)
    c = torch.empty((S, N), dtype=torch.int16, device="cuda")
    f = lambda: X.check(X.xs_gemm_scatter(x.data_ptr(), Dm, wt.data_ptr(), Dm, S, N, Dm, desc, wins, G, None, None, st))
    g = lambda: X.check(X.xs_gemm(x.data_ptr(), Dm, wt.data_ptr(), Dm, c.data_ptr(), N, S, N, Dm, None, st))
    sc = lambda: X.check(X.xs_scatter_copy(c.data_ptr(), N, S, N, desc, wins, G, st))
    out["sp_qkv"] = _scatter_result(sp.name, 2.0 * S * N * Dm, 2.0 * S * N, *timed(f, g, lambda: (g(), sc())))
    del x, wt, win, c
    torch.cuda.empty_cache()
    return out


def _scatter_result(name, flops, store_bytes, t_fused, t_plain, t_serial):
    return {"workload": name, "fused_us": t_fused, "plain_gemm_us": t_plain, "serial_us": t_serial,
            "fused_TFLOPs": flops / (t_fused * 1e-6) / 1e12,
            "mfma_frac": flops / (t_fused * 1e-6) / MFMA_PEAK_BF16,
            "residual_us": t_fused - t_plain, "speedup_vs_serial": t_serial / t_fused,
            "stored_bytes": store_bytes}


def store_ceiling(X, torch):
    """Plain store stream into HBM: 256 producers x 8 waves of 128-bit stores, zero gap, 1 GiB
    at fresh addresses (the remote-store microbenchmark)."""
    from paper_2607_23264_amd.calibrate import run_bursts
    nb = 1 << 30
    buf = torch.empty(nb // 2, dtype=torch.int16, device="cuda")
    K, B = 256, 256 << 10
    n = nb // (K * B)
    run_bursts(buf.data_ptr(), nb, K, B, n, 0, store_waves=8)
    spans = [run_bursts(buf.data_ptr(), nb, K, B, n, 0, store_waves=8).total_span_us for _ in range(3)]
    del buf
    torch.cuda.empty_cache()
    span = float(np.median(spans))
    return {"bytes": nb, "span_us": span, "GBps": nb / (span * 1e-6) / 1e9,
            "frac_of_hbm_peak": nb / (span * 1e-6) / HBM_PEAK}


def slow_sink_line(reps=10):
    """Store pacing against the host-coherent sink (paper_2607_23264_amd.slow_sink, quick sweep):
    the tiny layer with every combine window on the sink (c5) and the DeepSeek-V3 share with one
    and with two of its eight source windows there, uniform and Zipf at bf16 and uniform at
    MXFP8; per policy the kernel time on the sink
    and on the HBM control, the speedup over Expert-Wave burst issue, and the stall per producer
    measured (issue spans and staging waits beyond the control) against the audit's prediction."""
    from paper_2607_23264_amd import slow_sink as ss
    rep = ss.run(quick=True, reps=reps)
    keep = ("policy", "chunk", "kernel_us", "control_kernel_us", "speedup_over_burst",
            "stall_measured_us_per_producer", "stall_predicted_us_per_producer", "time_lost_us",
            "staging_wait_measured_us_per_producer", "mma_stall_predicted_us_per_producer",
            "stall_fraction_measured", "stall_fraction_predicted", "mainloop_excess_us_per_producer",
            "dependency_wait_excess_us_per_producer", "l2_issue_us_median", "l2_issue_us_p90", "rate_feasible_eq9",
            "sclk_MHz_median")
    return {"sink_model": rep["sink_model"], "hbm_R_bytes_per_us": rep["hbm_R_bytes_per_us"],
            "gap_sweep": rep["gap_sweep"], "producer_sweep": rep["producer_sweep"],
            "layers": [{"layer": L["layer"], "sink_share": L["sink_share"],
                        "control_tile_times_us": L.get("control_tile_times_us"),
                        "policies": {k: {f: v.get(f) for f in keep} for k, v in L["policies"].items()}}
                       for L in rep["layers"]]}


def synth_rows(g, m, H):
    import synth
    return synth.to_bf16_bits(g.standard_normal((m, H), dtype=np.float32))


def mx_line(X, torch, cfg, inp, rank, experts, pol, steps, warmup, bf16_step_us, prec="MXFP8"):
    """The same layer share at MXFP8 (W8A8) or W4A8 (E2M1 weights): token rows quantized in the
    dispatch phase, both expert GEMMs on the scaled MFMA. Step time, FFN kernel rate against
    the dense fp8 peak (an fp8 x fp4 MFMA issues at the fp8 rate) and the in-step phases."""
    from paper_2607_23264_amd.layer import EPLayer, Shape
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=rank)
    lay = EPLayer(s, sentinel=False, precision=getattr(X, f"XS_PREC_{prec}"))
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(inp["fill"])
    for i in range(8):
        lay.L.events[i] = None
    for _ in range(warmup):
        lay.fused(pol)
    torch.cuda.synchronize()
    ev = X.HipEvents(2 * steps)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        lay.L.events[X.XS_EV_FFN] = ev.ev[2 * i]
        lay.L.events[X.XS_EV_FFN_END] = ev.ev[2 * i + 1]
        lay.fused(pol)
    stop.record()
    torch.cuda.synchronize()
    step_us = start.elapsed_time(stop) / steps * 1e3
    ffn_us = float(np.mean([ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(steps)])) * 1e3
    n_ph = 10
    pev = X.HipEvents(8 * n_ph)
    for i in range(n_ph):
        for e in range(8):
            lay.L.events[e] = pev.ev[8 * i + e]
        lay.fused(pol)
    torch.cuda.synchronize()
    for e in range(8):
        lay.L.events[e] = None
    names = ["route", "layout", "dispatch", "plan", "expert_ffn", "signal", "combine_reduce"]
    in_step = {n: float(np.median([pev.elapsed_ms(8 * i + j, 8 * i + j + 1) * 1e3 for i in range(n_ph)]))
               for j, n in enumerate(names)}
    status = int(lay.status.item())
    rows = int(lay.dest_counts[rank].item())
    del lay
    torch.cuda.empty_cache()
    if status:
        raise RuntimeError(f"{prec} layer: device status {status}: {X.xs_strerror(status).decode()}")
    flops = 6.0 * cfg.H * cfg.I * rows
    tflops = flops / (ffn_us * 1e-6) / 1e12
    # algorithmic HBM bytes of one launch: dispatched MXFP8 rows read once, codes (1 byte, or
    # half a byte for E2M1) and scales of both weight matrices of every local expert read
    # once, MXFP8 h written and read back once, bf16 output rows stored once
    hb = cfg.I + cfg.I // 32
    wbytes = (0.5 if prec == "W4A8" else 1.0) + 1 / 32
    alg_bytes = (rows * (cfg.H + cfg.H // 32) + len(experts) * 3 * cfg.H * cfg.I * wbytes + 2 * rows * hb
                 + rows * cfg.H * 2)
    kname = "ep_ffn_w4a8_kernel" if prec == "W4A8" else "ep_ffn_mx_kernel"
    from paper_2607_23264_amd.profiling import read_traffic
    tr = read_traffic(os.path.join(HERE, "profiles", f"{kname}_dsv3_share_traffic.md"))
    # dispatch phase: bf16 rows read, MXFP8 rows staged, then read and stored k times
    rb = cfg.H + cfg.H // 32
    disp_moved = cfg.T * cfg.H * 2 + cfg.T * rb * 2 + cfg.T * cfg.k * rb
    fmt = "E2M1 weights, E4M3 activations" if prec == "W4A8" else "E4M3 codes"
    return {"workload": f"{cfg.name} at {prec} ({fmt}, E8M0 scales per 32), rank {rank}",
            "dtype": f"{prec.lower()} (fp32 accumulation)", "us_per_step": step_us, "bf16_us_per_step": bf16_step_us,
            "speedup_vs_bf16": bf16_step_us / step_us, "rows_computed": rows,
            "phases_in_step_us": in_step,
            "dispatch_moved_GBps": disp_moved / (in_step["dispatch"] * 1e-6) / 1e9,
            "roofline": {"bound": "mfma", "kernel": f"{kname}<3> (persistent fused MX Linear-1 + Linear-2)",
                         "achieved": tflops, "peak": MFMA_PEAK_FP8 / 1e12, "unit": "TFLOP/s",
                         "frac": tflops * 1e12 / MFMA_PEAK_FP8, "traffic": tr["traffic_bytes"] if tr else None,
                         "flops_per_launch": flops, "algorithmic_bytes_per_launch": alg_bytes,
                         "avg_launch_us": ffn_us, "hbm_GBps_algorithmic": alg_bytes / (ffn_us * 1e-6) / 1e9}}


def gpu_route_layout(X, torch, logits, k, E, W):
    """Top-k route and dispatch layout of one source on the GPU (the library's own calls).
    Returns device (topk_idx [T][k], slot_row [T][k]) and the host dest_counts [W]."""
    import ctypes as C
    T = logits.shape[0]
    stream = torch.cuda.current_stream().cuda_stream
    lg = torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)).cuda()
    idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    X.check(X.xs_route_topk_softmax(lg.data_ptr(), T, E, k, 0, idx.data_ptr(), w.data_ptr(), stream))
    cap = T * k
    i32 = dict(dtype=torch.int32, device="cuda")
    ec, sb, eo = torch.empty((1, E), **i32), torch.empty((1, E), **i32), torch.empty((E,), **i32)
    dc, sr, rs = torch.empty((W,), **i32), torch.empty((T, k), **i32), torch.empty((W, cap), **i32)
    st = torch.zeros((1,), **i32)
    nb = C.c_int64()
    X.check(X.xs_dispatch_layout_workspace_bytes(1, T, E, C.byref(nb)))
    ws = torch.empty((max(1, nb.value),), dtype=torch.uint8, device="cuda")
    X.check(X.xs_dispatch_layout(idx.data_ptr(), 1, T, k, E, W, cap, ec.data_ptr(), sb.data_ptr(), eo.data_ptr(),
                                 dc.data_ptr(), sr.data_ptr(), rs.data_ptr(), ws.data_ptr(), ws.numel(),
                                 st.data_ptr(), stream))
    torch.cuda.synchronize()
    if int(st.item()):
        raise RuntimeError(f"layout status {int(st.item())}")
    return idx, sr, dc.cpu().numpy()


def ring_line(X, torch, synth, reps=5):
    """Dispatch of one source of the share through bounded destination rings: time, entries,
    producer stalls and ring bytes for ring sizes S and per-destination dedup, rings in HBM
    and (a slow sink) in host-coherent memory, against the plain dispatch."""
    import ctypes as C
    from paper_2607_23264_amd.layer import HostCoherent
    cfg = synth.EP_DSV3_SHARE
    T, H, k, E, W = cfg.T, cfg.H, cfg.k, cfg.E, cfg.W
    di, ds, dest_counts = gpu_route_layout(X, torch, synth.ep_logits(cfg, 0)[0], k, E, W)
    cap = int(dest_counts.max())
    dx = torch.from_numpy(np.ascontiguousarray(synth.ep_x(cfg, 0)[0]).view(np.int16)).cuda()
    win = torch.empty((W, cap, H), dtype=torch.int16, device="cuda")
    wins = X.windows([X.window(win[d]) for d in range(W)])
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    nb = C.c_int64()
    X.check(X.xs_ring_slot_bytes(H, k, C.byref(nb)))
    slot_bytes = nb.value

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    plain_us = timed(lambda: X.check(X.xs_dispatch(dx.data_ptr(), T, H, di.data_ptr(), ds.data_ptr(), k, E, wins,
                                                   W, st.data_ptr(), stream)))
    window_bytes = T * k * H * 2
    cells = []
    for sink in ("hbm", "host"):
        for S in ((4, 16, 64, 256, 4096) if sink == "hbm" else (16, 256)):
            ring_mem = HostCoherent(W * S * slot_bytes) if sink == "host" else \
                torch.empty((W * S * slot_bytes,), dtype=torch.uint8, device="cuda")
            base = ring_mem.ptr if sink == "host" else ring_mem.data_ptr()
            rings = X.windows([X.window((base + d * S * slot_bytes, S, slot_bytes)) for d in range(W)])
            X.check(X.xs_dispatch_ring_workspace_bytes(T, k, W, S, C.byref(nb)))
            ws = torch.zeros((nb.value,), dtype=torch.uint8, device="cuda")
            stats = torch.zeros((2 * W,), dtype=torch.int32, device="cuda")
            for dedup in (0, 1):
                us = timed(lambda: X.check(X.xs_dispatch_ring(
                    dx.data_ptr(), T, H, di.data_ptr(), ds.data_ptr(), k, E, wins, W, rings, dedup, 0, 0,
                    ws.data_ptr(), ws.numel(), stats.data_ptr(), st.data_ptr(), stream)))
                sv = stats.cpu().numpy()
                entries = int(sv[:W].sum())
                cells.append({"sink": sink, "slots": S, "dedup": dedup, "us": us, "entries": entries,
                              "stalls": int(sv[W:].sum()), "ring_bytes": entries * slot_bytes,
                              "window_GBps": window_bytes / (us * 1e-6) / 1e9})
            torch.cuda.synchronize()
            if sink == "host":
                ring_mem.free()
            else:
                del ring_mem
    status = int(st.item())
    if status:
        raise RuntimeError(f"ring dispatch: device status {status}: {X.xs_strerror(status).decode()}")
    no_dd = next(c["entries"] for c in cells if c["dedup"] == 0)
    dd = next(c["entries"] for c in cells if c["dedup"] == 1)
    return {"workload": f"one source of {cfg.name}: {T} tokens, top-{k} of {E} experts, {W} destinations",
            "plain_dispatch_us": plain_us, "slot_bytes": slot_bytes, "entries_without_dedup": no_dd,
            "entries_with_dedup": dd, "dedup_ratio": no_dd / dd, "cells": cells}


def graph_steps(torch, lay, pol, steps):
    """The same step captured once in a HIP graph (torch's graph API over the library's launches
    on the capture stream) and replayed `steps` times: the launch gaps between the step's
    kernels go away, the work is identical (the layer's kernels only; no memset, copy or host
    synchronisation inside a step). Reported beside the eager step, not instead of it."""
    try:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            lay.fused(pol)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            lay.fused(pol)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return {"us_per_step": e0.elapsed_time(e1) * 1e3 / steps, "steps": steps}
    except RuntimeError as err:   # capture refused: report it, keep the eager figures
        torch.cuda.synchronize()
        return {"us_per_step": None, "error": str(err)[:200]}


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {a.gpus}); the library has no multi-GPU path",
              file=sys.stderr)
        sys.exit(2)
    import dataclasses
    import torch
    import synth
    from paper_2607_23264_amd import xstage as X
    from paper_2607_23264_amd.layer import EPLayer, Shape, pacing

    torch.cuda.set_device(0)
    cfg = dataclasses.replace(synth.EP_DSV3_SHARE, routing=a.routing)
    t0 = time.time()
    log(f"[bench] generating inputs for {cfg.name} ({a.routing})")
    inp = {"logits": synth.ep_logits(cfg, a.seed), "x": synth.ep_x(cfg, a.seed)}
    rank = 0
    if a.routing == "zipf":
        # the most loaded destination, from the library's own routing of every source
        loads = np.zeros(cfg.W, np.int64)
        for s in range(cfg.n_src):
            loads += gpu_route_layout(X, torch, inp["logits"][s], cfg.k, cfg.E, cfg.W)[2]
        rank = int(loads.argmax())
    cfg = dataclasses.replace(cfg, rank=rank)
    experts = synth.computed_experts(cfg)
    inp["w1"], inp["w2"] = synth.ep_weights(cfg, experts, a.seed)
    inp["fill"] = synth.ep_remote_combine_fill(cfg, a.seed)
    log(f"[bench] inputs ready in {time.time() - t0:.1f} s; uploading")
    s = Shape(cfg.n_src, cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.W, experts[0], len(experts), src=rank)
    lay = EPLayer(s, sentinel=False)
    lay.upload(inp["logits"], inp["x"], inp["w1"], inp["w2"])
    lay.prefill_other_sources(inp["fill"])
    claim = X.XS_CLAIM_DYNAMIC if a.claim == "dynamic" else X.XS_CLAIM_STATIC
    pol = {"burst": pacing(X.XS_POLICY_BURST, claim=claim),
           "interleave": pacing(X.XS_POLICY_INTERLEAVE, lead=a.lead, claim=claim),
           "chunk": pacing(X.XS_POLICY_CHUNK, lead=a.lead, chunk=a.chunk, claim=claim)}
    ev = X.HipEvents(2 * a.steps + 2)
    for i in range(8):
        lay.L.events[i] = None
    for _ in range(a.warmup):
        lay.fused(pol[a.policy])
    torch.cuda.synchronize()
    log(f"[bench] warmup done; timing {a.steps} steps ({a.policy})")
    stream = torch.cuda.current_stream().cuda_stream
    # one event per step boundary (the first and last bracket the timed region)
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    torch.cuda.synchronize()
    from paper_2607_23264_amd.profiling import ClockSampler
    with ClockSampler() as sclk:
        bounds[0].record()
        for i in range(a.steps):
            lay.L.events[X.XS_EV_FFN] = ev.ev[2 * i]
            lay.L.events[X.XS_EV_FFN_END] = ev.ev[2 * i + 1]
            lay.fused(pol[a.policy])
            bounds[i + 1].record()
        torch.cuda.synchronize()
    total_ms = bounds[0].elapsed_time(bounds[-1])
    step_us = [bounds[i].elapsed_time(bounds[i + 1]) * 1e3 for i in range(a.steps)]
    ffn_ms = [ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(a.steps)]
    lay.L.events[X.XS_EV_FFN] = None
    lay.L.events[X.XS_EV_FFN_END] = None
    # phases inside the step: every phase boundary recorded, after the timed region
    n_ph = 10
    pev = X.HipEvents(8 * n_ph)
    for i in range(n_ph):
        for e in range(8):
            lay.L.events[e] = pev.ev[8 * i + e]
        lay.fused(pol[a.policy])
    torch.cuda.synchronize()
    for e in range(8):
        lay.L.events[e] = None
    names = ["route", "layout", "dispatch", "plan", "expert_ffn", "signal", "combine_reduce"]
    in_step = {n: float(np.median([pev.elapsed_ms(8 * i + j, 8 * i + j + 1) * 1e3 for i in range(n_ph)]))
               for j, n in enumerate(names)}
    graph = graph_steps(torch, lay, pol[a.policy], a.steps)
    status = int(lay.status.item())
    if status:
        log(f"[bench] device status {status}: {X.xs_strerror(status).decode()}")
        sys.exit(1)
    ms_per_step = total_ms / a.steps
    rows = int(lay.dest_counts[rank].item())
    flops = 6.0 * cfg.H * cfg.I * rows
    ffn_avg = float(np.mean(ffn_ms))
    achieved_tflops = flops / (ffn_avg * 1e-3) / 1e12
    log(f"[bench] {ms_per_step * 1e3:.1f} us/step, FFN kernel {ffn_avg * 1e3:.1f} us "
        f"({achieved_tflops:.1f} TFLOP/s, {rows} rows)")

    res = {"metric": METRIC, "value": ms_per_step * 1e3, "unit": "us", "n_gpus": 1, "steps": a.steps,
           "warmup": a.warmup, "ms_per_step": ms_per_step, "higher_is_better": False, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": f"{cfg.name} ({a.routing} routing, rank {rank}; one rank's EP share)",
                      "policy": a.policy, "claim": a.claim, "lead_rows": a.lead, "rows_computed": rows,
                      "global_tokens": cfg.n_src * cfg.T, "seq_len": cfg.T}}
    # algorithmic HBM bytes of one launch: dispatched rows read once, both weight matrices of
    # every local expert read once, h written and read back once, output rows stored once
    alg_bytes = 2.0 * (rows * cfg.H + len(experts) * 3 * cfg.H * cfg.I + 2 * rows * cfg.I + rows * cfg.H)
    from paper_2607_23264_amd.profiling import read_traffic
    tr = read_traffic(os.path.join(HERE, "profiles", "ep_ffn_kernel_dsv3_share_traffic.md"))
    disp_bytes = cfg.T * cfg.k * cfg.H * 2          # stored rows (plus T * H * 2 read)
    red_bytes = cfg.T * cfg.k * cfg.H * 2 + cfg.T * cfg.H * 2
    res["graph_replay"] = graph
    # the shader clock during the timed steps (clock state differs between boxes and runs)
    res["sclk_MHz"] = sclk.summary()
    if res["sclk_MHz"]:
        log(f"[bench] shader clock during the timed steps (driver's figure): median "
            f"{res['sclk_MHz']['median']:.0f} MHz over {res['sclk_MHz']['samples']} samples")
    res["step_us_dist"] = {"median": float(np.median(step_us)), "p10": float(np.percentile(step_us, 10)),
                           "p90": float(np.percentile(step_us, 90)), "min": float(np.min(step_us)),
                           "max": float(np.max(step_us))}
    res["ffn_us_dist"] = {"median": float(np.median(ffn_ms)) * 1e3, "p10": float(np.percentile(ffn_ms, 10)) * 1e3,
                          "p90": float(np.percentile(ffn_ms, 90)) * 1e3}
    res["phases_in_step_us"] = in_step
    res["store_GBps"] = {
        "dispatch_stored": disp_bytes / (in_step["dispatch"] * 1e-6) / 1e9,
        "dispatch_moved": (disp_bytes + cfg.T * cfg.H * 2) / (in_step["dispatch"] * 1e-6) / 1e9,
        "combine_reduce_moved": red_bytes / (in_step["combine_reduce"] * 1e-6) / 1e9}
    res["store_GBps"]["dispatch_frac_of_hbm_peak"] = res["store_GBps"]["dispatch_moved"] * 1e9 / HBM_PEAK
    res["store_GBps"]["combine_reduce_frac_of_hbm_peak"] = res["store_GBps"]["combine_reduce_moved"] * 1e9 / HBM_PEAK
    log("[bench] in-step phases (us): " + ", ".join(f"{k}={v:.1f}" for k, v in in_step.items()))
    res["mfma_util_pct"] = 100.0 * achieved_tflops * 1e12 / MFMA_PEAK_BF16
    res["roofline"] = {"bound": "mfma", "kernel": "ep_ffn_kernel<3> (persistent fused Linear-1 + Linear-2)",
                       "achieved": achieved_tflops, "peak": MFMA_PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                       "frac": achieved_tflops * 1e12 / MFMA_PEAK_BF16,
                       "traffic": tr["traffic_bytes"] if tr else None,
                       "flops_per_launch": flops, "algorithmic_bytes_per_launch": alg_bytes,
                       "avg_launch_us": ffn_avg * 1e3,
                       "hbm_GBps_algorithmic": alg_bytes / (ffn_avg * 1e-3) / 1e9}

    if not a.no_phases:
        log("[bench] phase breakdown (each call timed alone, back to back)")
        ph = {}
        reps = 5

        def timed(fn):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            fn()
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps * 1e3

        ph["route_us"] = timed(lay.route)
        ph["layout_us"] = timed(lay.layout)
        ph["dispatch_us"] = timed(lambda: lay.dispatch(rank))
        ph["expert_ffn_unfused_us"] = timed(lay.expert_ffn)
        ph["combine_send_us"] = timed(lay.combine_send)
        ph["combine_reduce_us"] = timed(lay.combine_reduce)
        disp_bytes = cfg.T * cfg.k * cfg.H * 2
        comb_bytes = rows * cfg.H * 2
        ph["dispatch_store_GBps"] = disp_bytes / (ph["dispatch_us"] * 1e-6) / 1e9
        ph["combine_send_store_GBps"] = comb_bytes / (ph["combine_send_us"] * 1e-6) / 1e9
        # combine-send reads every y row and stores it once: against a plain device copy of
        # the same bytes
        ph["combine_send_moved_GBps"] = 2 * ph["combine_send_store_GBps"]
        cp_src = torch.empty(comb_bytes, dtype=torch.uint8, device="cuda")
        cp_dst = torch.empty_like(cp_src)
        ph["device_copy_same_bytes_us"] = timed(lambda: cp_dst.copy_(cp_src))
        ph["combine_send_frac_of_device_copy"] = ph["device_copy_same_bytes_us"] / ph["combine_send_us"]
        del cp_src, cp_dst
        # the same expert FFN as two standalone grouped GEMMs (xs_grouped_gemm): Linear-1 with
        # the SwiGLU epilogue, then Linear-2, each local expert one segment of this rank's
        # dispatch window; the MFMA utilisation of the GEMM phase on its own
        e0, ne = experts[0], len(experts)
        seg_off = lay.expert_offsets[e0:e0 + ne].contiguous()
        seg_rows = torch.minimum(lay.expert_counts[:, e0:e0 + ne].sum(0).to(torch.int32),
                                 lay.cap - seg_off).to(torch.int32).contiguous()
        a_win = lay.dwin[e0 // (cfg.E // cfg.W)]
        h_g = torch.empty((lay.cap, cfg.I), dtype=torch.int16, device="cuda")
        y_g = torch.empty((lay.cap, cfg.H), dtype=torch.int16, device="cuda")
        gg1 = lambda: X.check(X.xs_grouped_gemm(a_win.data_ptr(), cfg.H, lay.cap, seg_off.data_ptr(), seg_rows.data_ptr(),
                                                ne, lay.w1.data_ptr(), 2 * cfg.I, cfg.H, h_g.data_ptr(), cfg.I,
                                                X.XS_EPI_SWIGLU, lay.status.data_ptr(), lay.stream), "grouped_gemm")
        gg2 = lambda: X.check(X.xs_grouped_gemm(h_g.data_ptr(), cfg.I, lay.cap, seg_off.data_ptr(), seg_rows.data_ptr(),
                                                ne, lay.w2.data_ptr(), cfg.H, cfg.I, y_g.data_ptr(), cfg.H,
                                                X.XS_EPI_STORE, lay.status.data_ptr(), lay.stream), "grouped_gemm")
        ph["grouped_gemm_l1_swiglu_us"] = timed(gg1)
        ph["grouped_gemm_l2_us"] = timed(gg2)
        gg_us = ph["grouped_gemm_l1_swiglu_us"] + ph["grouped_gemm_l2_us"]
        ph["grouped_gemm_TFLOPs"] = flops / (gg_us * 1e-6) / 1e12
        ph["grouped_gemm_mfma_frac"] = flops / (gg_us * 1e-6) / MFMA_PEAK_BF16
        del h_g, y_g
        ph["combine_reduce_GBps"] = (cfg.T * cfg.k * cfg.H * 2 + cfg.T * cfg.H * 2) / (ph["combine_reduce_us"] * 1e-6) / 1e9
        for name, p in pol.items():
            if a.policies or name == a.policy:
                ph[f"fused_{name}_us"] = timed(lambda p=p: lay.fused(p))
        res["phases_isolated"] = ph
        log("[bench] " + ", ".join(f"{k}={v:.1f}" for k, v in ph.items()))
    if int(lay.status.item()):
        log("[bench] device status set during phases")
        sys.exit(1)
    del lay
    torch.cuda.empty_cache()
    if not a.no_mx:
        for prec in ("MXFP8", "W4A8"):
            log(f"[bench] the same layer share at {prec}")
            res[f"ep_{prec.lower()}"] = m = mx_line(X, torch, cfg, inp, rank, experts, pol[a.policy], a.steps,
                                                    a.warmup, ms_per_step * 1e3, prec)
            log(f"[bench] {prec}: {m['us_per_step']:.1f} us/step ({m['speedup_vs_bf16']:.2f}x bf16), FFN kernel "
                f"{m['roofline']['avg_launch_us']:.1f} us ({m['roofline']['achieved']:.1f} TFLOP/s)")
    if not a.no_ring:
        log("[bench] dispatch through bounded destination rings")
        res["dispatch_ring"] = ring_line(X, torch, synth)
        r = res["dispatch_ring"]
        log(f"[bench] ring dispatch: plain {r['plain_dispatch_us']:.1f} us; dedup ratio {r['dedup_ratio']:.2f}; " +
            ", ".join(f"{c['sink']} S={c['slots']} dd={c['dedup']}: {c['us']:.0f} us" for c in r["cells"]))
    if not a.no_phases:
        log("[bench] store ceiling")
        res["store_ceiling"] = store_ceiling(X, torch)
    if not a.no_scatter:
        log("[bench] TP / SP scatter GEMMs")
        res["scatter"] = scatter_lines(X, torch, synth)
        log("[bench] " + json.dumps(res["scatter"]))
    if not a.no_attn:
        log("[bench] attention + post-attention Ulysses exchange (FA-only / serial / fused / coupled)")
        from paper_2607_23264_amd import attn_a2a
        rep = attn_a2a.run()
        res["attention_a2a"] = {"workload": rep["workload"], "grid": rep["grid"], "summary": rep["summary"],
                                "cells": rep["cells"]}
        from paper_2607_23264_amd.profiling import ATTN_KERNEL_SOURCES, sources_hash
        ref = next((c for c in rep["cells"] if c["sink"] == "hbm" and c["M"] == 16384), None)
        if ref is not None:
            atr = read_traffic(os.path.join(HERE, "profiles", "attn_kernel_M16384_h8_d128_traffic.md"),
                               sources_hash(ATTN_KERNEL_SOURCES))
            res["attention_a2a"]["roofline"] = {
                "bound": "mfma", "kernel": "attn_kernel (FA-only launch, M=16384, 8 heads, d=128)",
                "achieved": ref["fa_TFLOPs"], "peak": MFMA_PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                "frac": ref["fa_TFLOPs"] * 1e12 / MFMA_PEAK_BF16,
                "traffic": atr["traffic_bytes"] if atr else None,
                "flops_per_launch": 4.0 * 8 * 16384 ** 2 * 128,
                "algorithmic_bytes_per_launch": 4.0 * 8 * 16384 * 128 * 2}
        torch.cuda.empty_cache()
    if not a.no_tiny:
        log("[bench] tiny layer (eager and HIP graph replay)")
        res["tiny_layer"] = tiny_line(X, torch, synth)
        log(f"[bench] tiny layer: {res['tiny_layer']['us_per_step_eager']:.1f} us eager, "
            f"{res['tiny_layer']['us_per_step_graph']} us graph")
    if not a.no_zipf:
        log("[bench] the share with Zipf(1.2) routing")
        res["zipf_share"] = zipf_line(X, torch, synth, pol[a.policy], min(a.steps, 10), a.warmup)
        log(f"[bench] zipf: {res['zipf_share']['us_per_step']:.1f} us/step, FFN {res['zipf_share']['ffn_us']:.1f} us")
    if not a.no_slow_sink:
        log("[bench] store pacing against the host-coherent sink")
        res["slow_sink"] = slow_sink_line()
        for L in res["slow_sink"]["layers"]:
            log("[bench] " + L["layer"] + ": " + ", ".join(f"{k} {v['kernel_us']:.0f} us" for k, v in L["policies"].items()))
    if not a.no_cpu_baseline:
        log("[bench] oracle on the host (bounded sample)")
        res["cpu_baseline"] = cpu_baseline(cfg, inp, rank, a.seed)
        log(f"[bench] oracle sample: {res['cpu_baseline']['value']:.0f} us/layer equivalent")
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
