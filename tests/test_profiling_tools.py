"""Host logic of the rocprofv3 summary helpers on synthetic counter files: the traffic scaling by
the copy calibration, the staleness key of a stored traffic record, the MFMA busy / clock /
executed-flops arithmetic, and the shader-clock sampler's parsing and windows."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TOOL = os.path.join(ROOT, "paper_2607_23264_amd", "profiling.py")
FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for i, (kernel, disp, counter, value, t0, t1) in enumerate(rows):
            r = {k: 0 for k in FIELDS}
            r.update(Correlation_Id=i, Dispatch_Id=disp, Kernel_Name=kernel, Counter_Name=counter,
                     Counter_Value=value, Start_Timestamp=t0, End_Timestamp=t1)
            w.writerow(r)


def _run(*args):
    return subprocess.run([sys.executable, TOOL, *args], check=True, capture_output=True, text=True).stdout


def test_traffic_scales_each_counter_by_the_copy(tmp_path):
    k = "void xs::some_kernel<3>(xs::EpArgs)"
    # the copy of 1 GiB reads FETCH_SIZE = 512 MiB (x 2.0) and WRITE_SIZE = 1 GiB (x 1.0), in KiB
    _csv(tmp_path / "cf.csv", [("__amd_rocclr_copyBuffer", 1, "FETCH_SIZE", 524288.0, 0, 1)])
    _csv(tmp_path / "cw.csv", [("__amd_rocclr_copyBuffer", 1, "WRITE_SIZE", 1048576.0, 0, 1)])
    _csv(tmp_path / "f.csv", [(k, 1, "FETCH_SIZE", 1000.0, 0, 1), (k, 2, "FETCH_SIZE", 3000.0, 0, 1),
                              ("void other()", 3, "FETCH_SIZE", 9e9, 0, 1)])
    _csv(tmp_path / "w.csv", [(k, 1, "WRITE_SIZE", 500.0, 0, 1), (k, 2, "WRITE_SIZE", 500.0, 0, 1)])
    out = tmp_path / "t.md"
    _run("traffic", "--kernel", "xs::some_kernel<3>", "--fetch", str(tmp_path / "f.csv"), "--write",
         str(tmp_path / "w.csv"), "--copy-fetch", str(tmp_path / "cf.csv"), "--copy-write", str(tmp_path / "cw.csv"),
         "--copy-bytes", str(1 << 30), "--algorithmic-bytes", "2048000", "--commands", "a;;b", "--out", str(out))
    rec = json.loads(out.read_text().split("traffic-json:")[1])
    assert rec["fetch_scale"] == pytest.approx(2.0) and rec["write_scale"] == pytest.approx(1.0)
    assert rec["fetch_bytes"] == pytest.approx(2000.0 * 1024 * 2.0)      # mean of 1000 and 3000 KiB, x 2
    assert rec["write_bytes"] == pytest.approx(500.0 * 1024)
    assert rec["dispatches"] == [2, 2]
    # the record is read back only while the kernel's sources hash to the stored key
    sys.path.insert(0, ROOT)
    from paper_2607_23264_amd import profiling
    assert profiling.read_traffic(str(out), rec["sources_sha"])["traffic_bytes"] == pytest.approx(rec["traffic_bytes"])
    assert profiling.read_traffic(str(out), "0" * 16) is None


def test_mfma_summary_arithmetic(tmp_path):
    k = "void xs::ep_ffn_kernel<3>(xs::EpArgs)"
    rows = []
    for d, (t0, t1) in enumerate(((1000, 2001000), (5000000, 7000000)), start=1):   # 2000 us each
        rows += [(k, d, "SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 0.5 * 3.4e6, t0, t1),    # busy half of the cycles
                 (k, d, "GRBM_GUI_ACTIVE", 8 * 3.4e6, t0, t1),                      # 3.4e6 cycles per XCD
                 (k, d, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 4e12 / 512, t0, t1)]
    rows.append(("void other()", 9, "GRBM_GUI_ACTIVE", 1.0, 0, 1))
    _csv(tmp_path / "m.csv", rows)
    out = tmp_path / "m.md"
    _run("mfma", "--csv", str(tmp_path / "m.csv"), "--kernel", "xs::ep_ffn_kernel<3>=3e12", "--command", "cmd",
         "--out", str(out))
    rec = json.loads(out.read_text().split("mfma-json:")[1])[0]
    assert rec["dispatches"] == 2
    assert rec["us"] == pytest.approx(2000.0)
    assert rec["mfma_busy"] == pytest.approx(0.5)
    assert rec["clock_GHz"] == pytest.approx(1.7)
    assert rec["executed_flops"] == pytest.approx(4e12)
    assert rec["algorithmic_TFLOPs"] == pytest.approx(1500.0)


def test_clock_sampler_reads_the_current_level_and_windows(tmp_path):
    # the sysfs file lists DPM levels and marks the current one; the sampler takes that one
    sys.path.insert(0, ROOT)
    from paper_2607_23264_amd.profiling import ClockSampler
    f = tmp_path / "pp_dpm_sclk"
    cs = ClockSampler()
    cs.path = str(f)
    f.write_text("0: 500Mhz\n1: 2400Mhz *\n")
    assert cs.read() == 2400
    f.write_text("S: 110Mhz *\n0: 500Mhz\n1: 2400Mhz\n")
    assert cs.read() == 110
    f.write_text("0: 500Mhz\n1: 2400Mhz\n")         # no current level marked
    assert cs.read() is None
    cs.path = str(tmp_path / "missing")
    assert cs.read() is None
    cs.samples = [(1.0, 1800), (2.0, 1900), (3.0, 2000), (4.0, 2100)]
    s = cs.summary()
    assert s["samples"] == 4 and s["median"] == 1950.0 and s["min"] == 1800 and s["max"] == 2100
    w = cs.summary([(1.5, 2.5), (3.5, 4.5)])           # samples inside either window
    assert w["samples"] == 2 and w["median"] == 2000.0
    assert cs.summary([(9.0, 10.0)]) is None


def test_clock_sampler_without_sysfs_samples_nothing(monkeypatch):
    sys.path.insert(0, ROOT)
    import glob
    from paper_2607_23264_amd.profiling import ClockSampler
    monkeypatch.setattr(glob, "glob", lambda pattern: [])
    with ClockSampler() as cs:
        pass
    assert cs.path is None and cs.summary() is None
