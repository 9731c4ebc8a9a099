"""rocprofv3 helpers: a plain copy of known size (the counter calibration) and summaries.

  python -m paper_2607_23264_amd.profiling copy [--mib N] [--reps R]
      R device-to-device copies of N MiB (torch's copy kernel). Under
      `rocprofv3 --pmc FETCH_SIZE` / `--pmc WRITE_SIZE` the counters of these dispatches
      against their known bytes give the scale factor of each counter.
  python -m paper_2607_23264_amd.profiling stats --csv K.csv --command CMD --out F.md
      Markdown summary of a `--kernel-trace --stats` kernel_stats.csv.
  python -m paper_2607_23264_amd.profiling traffic --kernel NAME --fetch F.csv --write W.csv
      --copy-fetch CF.csv --copy-write CW.csv --copy-bytes B --commands CMDS --out F.md
      Per-dispatch HBM bytes of one kernel from two counter passes, each scaled by what the
      same counter reads for the copy; writes a markdown summary whose `traffic-json:` line
      the benchmark reads, keyed by the hash of the kernel's sources.
  python -m paper_2607_23264_amd.profiling mfma --csv C.csv --kernel NAME=FLOPS [...]
      --command CMD --out F.md
      MFMA busy fraction, shader clock and executed MFMA flops per dispatch from one counter
      pass (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE, SQ_INSTS_VALU_MFMA_MOPS_*), beside
      each kernel's algorithmic flops.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
# sources that define a kernel's code; they and the compiler flags key a stored traffic
# measurement (a change to either makes it stale)
FFN_KERNEL_SOURCES = ("csrc/xs_ep_ffn.hip", "csrc/xs_gemm.hpp", "csrc/xs_gemm_mx.hpp", "csrc/xs_common.hpp")
ATTN_KERNEL_SOURCES = ("csrc/xs_attn.hip", "csrc/xs_common.hpp")
EP_KERNEL_SOURCES = ("csrc/xs_ep.hip", "csrc/xs_common.hpp")
KERNEL_SOURCES = {"ffn": FFN_KERNEL_SOURCES, "attn": ATTN_KERNEL_SOURCES, "ep": EP_KERNEL_SOURCES}


def sources_hash(paths=FFN_KERNEL_SOURCES) -> str:
    if os.path.dirname(HERE) not in sys.path:        # also when run as a script
        sys.path.insert(0, os.path.dirname(HERE))
    from paper_2607_23264_amd.build import FLAGS, HIPCC, ROOT
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(HERE, p), "rb") as f:
            h.update(f.read())
    # include paths relative to the repository, which sits at different absolute paths on
    # different machines
    flags = [f.replace(ROOT, "<root>") for f in FLAGS]
    h.update(" ".join([os.path.basename(HIPCC)] + flags).encode())
    return h.hexdigest()[:16]


class ClockSampler:
    """The shader clock the driver reports (the current entry of pp_dpm_sclk in sysfs), sampled
    every 2 ms on a host thread while a region runs, as (host time, MHz) pairs. It is the
    driver's running figure, not a count of the kernel's own cycles (the counter summaries give
    that one). Without the sysfs file it samples nothing."""

    def __init__(self, period_s: float = 0.002):
        import glob
        paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = paths[0] if paths else None
        self.period = period_s
        self.samples = []
        self._stop = None
        self._thread = None

    def read(self):
        import re
        try:
            with open(self.path) as f:
                for line in f:
                    if "*" in line:
                        m = re.search(r"(\d+)\s*mhz", line, re.I)
                        return int(m.group(1)) if m else None
        except (OSError, TypeError):
            return None
        return None

    def __enter__(self):
        import threading
        import time
        if self.path is None:
            return self
        self._stop = threading.Event()

        def run():
            while not self._stop.is_set():
                v = self.read()
                if v is not None:
                    self.samples.append((time.perf_counter(), v))
                self._stop.wait(self.period)
        self._thread = threading.Thread(target=run, daemon=True)
        self._thread.start()
        return self

    def __exit__(self, *exc):
        if self._thread is not None:
            self._stop.set()
            self._thread.join()
        return False

    def summary(self, windows=None):
        """Median, p10, p90, min and max of the samples, or of those inside the given
        (start, end) host-time windows; None without samples."""
        import numpy as np
        v = [m for (t, m) in self.samples if windows is None or any(a <= t <= b for a, b in windows)]
        if not v:
            return None
        v = np.array(v, dtype=np.float64)
        return {"samples": int(v.size), "median": float(np.median(v)), "p10": float(np.percentile(v, 10)),
                "p90": float(np.percentile(v, 90)), "min": float(v.min()), "max": float(v.max())}


def read_traffic(md_path: str, kernel_hash: str | None = None):
    """The `traffic-json:` record of a traffic summary, or None if absent or stale."""
    try:
        with open(md_path) as f:
            for line in f:
                if line.startswith("traffic-json:"):
                    rec = json.loads(line[len("traffic-json:"):])
                    if rec.get("sources_sha") != (kernel_hash or sources_hash()):
                        return None
                    return rec
    except OSError:
        return None
    return None


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _short(name: str) -> str:
    m = re.match(r"(?:void )?([^(]*)", name)
    return (m.group(1) if m else name).strip()


def cmd_copy(a):
    import torch
    torch.cuda.set_device(0)
    n = a.mib << 20
    src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(a.reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copy: {a.reps} x {n} bytes", flush=True)


def cmd_stats(a):
    rows = _rows(a.csv)
    key = lambda r, *ks: next((r[k] for k in ks if k in r), None)
    out = ["# rocprofv3 kernel statistics", "", "Command (run from the repository root):", "",
           "```", a.command, "```", "", "| kernel | calls | average µs | min µs | max µs | total % |",
           "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        name = _short(key(r, "Name", "KernelName", "Kernel_Name") or "?")
        calls = key(r, "Calls")
        avg = float(key(r, "AverageNs") or 0) / 1e3
        mn = float(key(r, "MinNs") or 0) / 1e3
        mx = float(key(r, "MaxNs") or 0) / 1e3
        pct = float(key(r, "Percentage") or 0)
        out.append(f"| `{name}` | {calls} | {avg:.1f} | {mn:.1f} | {mx:.1f} | {pct:.2f} |")
    if a.note:
        out += ["", a.note]
    with open(a.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def _per_dispatch(path, kernel, counter):
    vals = [float(r["Counter_Value"]) for r in _rows(path)
            if r["Counter_Name"] == counter and _short(r["Kernel_Name"]).startswith(kernel)]
    return vals


def cmd_traffic(a):
    fetch = _per_dispatch(a.fetch, a.kernel, "FETCH_SIZE")
    write = _per_dispatch(a.write, a.kernel, "WRITE_SIZE")
    cf = max(_per_dispatch(a.copy_fetch, a.copy_kernel, "FETCH_SIZE"))
    cw = max(_per_dispatch(a.copy_write, a.copy_kernel, "WRITE_SIZE"))
    kf = a.copy_bytes / (cf * 1024.0)      # true bytes per counted byte
    kw = a.copy_bytes / (cw * 1024.0)
    if not fetch or not write:
        sys.exit(f"no {a.kernel} dispatches in the counter files")
    mean = lambda v: sum(v) / len(v)
    fb, wb = mean(fetch) * 1024.0 * kf, mean(write) * 1024.0 * kw
    rec = {"kernel": a.kernel, "sources_sha": sources_hash(KERNEL_SOURCES[a.sources]), "fetch_bytes": fb, "write_bytes": wb,
           "traffic_bytes": fb + wb, "fetch_scale": kf, "write_scale": kw,
           "dispatches": [len(fetch), len(write)], "algorithmic_bytes": a.algorithmic_bytes}
    out = ["# HBM traffic per dispatch (rocprofv3 counters)", "",
           f"Kernel: `{a.kernel}`", "", "Commands (run from the repository root, one counter pass each):", "",
           "```", *a.commands.split(";;"), "```", "",
           "FETCH_SIZE and WRITE_SIZE are read in KiB per dispatch and scaled by what the same counter",
           f"reads for a plain copy of {a.copy_bytes} bytes (`{a.copy_kernel}`): "
           f"FETCH_SIZE x {kf:.3f}, WRITE_SIZE x {kw:.3f}.", "",
           "| quantity | value |", "|---|---:|",
           f"| dispatches (fetch pass, write pass) | {len(fetch)}, {len(write)} |",
           f"| FETCH_SIZE raw, KiB/dispatch (mean) | {mean(fetch):.0f} |",
           f"| WRITE_SIZE raw, KiB/dispatch (mean) | {mean(write):.0f} |",
           f"| copy FETCH_SIZE / WRITE_SIZE, KiB | {cf:.0f} / {cw:.0f} |",
           f"| fetched bytes per dispatch (scaled) | {fb / 1e9:.3f} GB |",
           f"| written bytes per dispatch (scaled) | {wb / 1e9:.3f} GB |",
           f"| total bytes per dispatch (HBM traffic as these counters see it; MALL hits included) | {(fb + wb) / 1e9:.3f} GB |"]
    if a.algorithmic_bytes:
        out.append(f"| algorithmic bytes per dispatch | {a.algorithmic_bytes / 1e9:.3f} GB |")
        out.append(f"| traffic / algorithmic | {(fb + wb) / a.algorithmic_bytes:.2f} |")
    out += ["", "traffic-json: " + json.dumps(rec)]
    with open(a.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


MOPS_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F8", "SQ_INSTS_VALU_MFMA_MOPS_F6F4")


def cmd_mfma(a):
    """Per kernel, averaged over its dispatches in one counter pass:
    busy = SQ_VALU_MFMA_BUSY_CYCLES (summed over every SIMD), active = GRBM_GUI_ACTIVE (summed
    over the XCDs; per XCD it counts the cycles the GPU was busy), duration from the dispatch's
    timestamps. MFMA busy fraction = busy / (active per XCD x SIMDs), the definition of the
    profiler's MfmaUtil; shader clock = active per XCD / duration; executed MFMA flops = MOPS x
    512 (the counters count 512-flop units)."""
    by = {}
    for r in _rows(a.csv):
        by.setdefault(_short(r["Kernel_Name"]), {}).setdefault(int(r["Dispatch_Id"]), {})[r["Counter_Name"]] = r
    out = ["# MFMA utilisation per dispatch (rocprofv3 counters)", "", "Command (run from the repository root):",
           "", "```", a.command, "```", "",
           f"Busy fraction = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE per XCD x {a.simds} SIMDs); "
           f"clock = GRBM_GUI_ACTIVE per XCD / dispatch duration; executed flops = MFMA MOPS x 512. "
           f"Durations are those of the counter run (kernels serialized by the profiler).", "",
           "| kernel | dispatches | µs | MFMA busy | clock GHz | executed TFLOP | algorithmic TFLOP | "
           "executed / algorithmic | algorithmic TFLOP/s |", "|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    recs = []
    for spec in a.kernel:
        name, flops = spec.rsplit("=", 1)
        flops = float(flops)
        ds = [d for k, v in by.items() if k.startswith(name) for d in v.values()]
        ds = [d for d in ds if "SQ_VALU_MFMA_BUSY_CYCLES" in d and "GRBM_GUI_ACTIVE" in d]
        if not ds:
            sys.exit(f"no {name} dispatches with the MFMA counters in {a.csv}")
        mean = lambda f: sum(f(d) for d in ds) / len(ds)
        val = lambda d, c: float(d[c]["Counter_Value"]) if c in d else 0.0
        dur = mean(lambda d: (int(d["GRBM_GUI_ACTIVE"]["End_Timestamp"]) - int(d["GRBM_GUI_ACTIVE"]["Start_Timestamp"])) * 1e-9)
        act = mean(lambda d: val(d, "GRBM_GUI_ACTIVE")) / a.xcds
        busy = mean(lambda d: val(d, "SQ_VALU_MFMA_BUSY_CYCLES"))
        ex = mean(lambda d: sum(val(d, c) for c in MOPS_COUNTERS)) * 512.0
        util = busy / (act * a.simds)
        clk = act / dur / 1e9
        rec = {"kernel": name, "dispatches": len(ds), "us": dur * 1e6, "mfma_busy": util, "clock_GHz": clk,
               "executed_flops": ex, "algorithmic_flops": flops, "algorithmic_TFLOPs": flops / dur / 1e12}
        recs.append(rec)
        out.append(f"| `{name}` | {len(ds)} | {dur * 1e6:.1f} | {util:.3f} | {clk:.2f} | {ex / 1e12:.3f} | "
                   f"{flops / 1e12:.3f} | {ex / flops:.3f} | {flops / dur / 1e12:.0f} |")
    out += ["", "mfma-json: " + json.dumps(recs)]
    with open(a.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("copy")
    c.add_argument("--mib", type=int, default=1024)
    c.add_argument("--reps", type=int, default=3)
    s = sub.add_parser("stats")
    s.add_argument("--csv", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--note", default="")
    t = sub.add_parser("traffic")
    t.add_argument("--kernel", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-bytes", type=float, required=True)
    t.add_argument("--copy-kernel", default="__amd_rocclr_copyBuffer")
    t.add_argument("--algorithmic-bytes", type=float, default=0.0)
    t.add_argument("--sources", choices=sorted(KERNEL_SOURCES), default="ffn",
                   help="which kernel's sources key the record")
    t.add_argument("--commands", required=True, help="the counter commands, separated by ';;'")
    t.add_argument("--out", required=True)
    m = sub.add_parser("mfma")
    m.add_argument("--csv", required=True)
    m.add_argument("--kernel", action="append", required=True, help="NAME=ALGORITHMIC_FLOPS, repeatable")
    m.add_argument("--simds", type=int, default=1024)
    m.add_argument("--xcds", type=int, default=8)
    m.add_argument("--command", required=True)
    m.add_argument("--out", required=True)
    a = ap.parse_args()
    {"copy": cmd_copy, "stats": cmd_stats, "traffic": cmd_traffic, "mfma": cmd_mfma}[a.cmd](a)


if __name__ == "__main__":
    main()
