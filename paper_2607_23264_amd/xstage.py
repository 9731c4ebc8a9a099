"""ctypes binding of libxstage.so: the C ABI in include/xstage.h, same names, argument
marshalling only. Every step of the path runs in the library's HIP kernels; there is no
Python or CPU fallback. Importing this module fails loudly if the library is missing.

Tensors are passed as raw pointers (torch CUDA tensors via ``data_ptr()``); the stream is
``torch.cuda.current_stream().cuda_stream`` unless given.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libxstage.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_23264_amd.build`")
lib = C.CDLL(LIB_PATH)

# ----------------------------------------------------------------------------- constants
XS_OK, XS_EINVAL, XS_EUNSUPPORTED, XS_EHIP, XS_EWORKSPACE, XS_ECAPACITY, XS_ETIMEOUT, XS_EBADINPUT = range(8)
XS_MAX_WINDOWS = 64
XS_EXPERT_SWIGLU, XS_EXPERT_IDENTITY = 0, 1
XS_POLICY_BURST, XS_POLICY_INTERLEAVE, XS_POLICY_CHUNK, XS_POLICY_AUTO = 0, 1, 2, 3
XS_CLAIM_STATIC, XS_CLAIM_DYNAMIC = 0, 1
(XS_EV_ROUTE, XS_EV_LAYOUT, XS_EV_DISPATCH, XS_EV_PLAN, XS_EV_FFN, XS_EV_FFN_END, XS_EV_REDUCE,
 XS_EV_END) = range(8)
XS_SCATTER_ROW_BLOCK, XS_SCATTER_HEAD_GROUP = 0, 1
XS_MB_PERIODIC, XS_MB_COMPLETION = 0, 1
XS_ATTN_LOCAL, XS_ATTN_WINDOWS, XS_ATTN_WINDOWS_COUPLED = 0, 1, 2
XS_FMT_E4M3, XS_FMT_E2M1 = 0, 1
XS_PREC_BF16, XS_PREC_MXFP8, XS_PREC_W4A8 = 0, 1, 2
XS_EPI_STORE, XS_EPI_SWIGLU = 0, 1

vp = C.c_void_p
i32 = C.c_int32
i64 = C.c_int64
f64 = C.c_double
pi32 = C.POINTER(C.c_int32)


class xs_window(C.Structure):
    _fields_ = [("base", vp), ("capacity_rows", i64), ("row_stride_bytes", i64), ("ready_flag", vp)]


class xs_model(C.Structure):
    _fields_ = [("t0_a_us", f64), ("t0_b_us_per_byte", f64), ("R_bytes_per_us", f64),
                ("Q_bytes", f64), ("K", i32), ("_pad", i32)]


class xs_pacing(C.Structure):
    _fields_ = [("policy", i32), ("lead_rows", i32), ("chunk_tiles", i32), ("max_producers", i32),
                ("wave_tiles", i32), ("gap_ns", i32), ("spin_timeout_us", i32), ("withhold_row", i32),
                ("claim", i32), ("reserved", i32),
                ("t_l1_us", f64), ("t_l2_us", f64), ("model", C.POINTER(xs_model)),
                ("expert_rows", C.POINTER(i32)), ("sink_share", f64)]


class xs_trace(C.Structure):
    _fields_ = [("buf", vp), ("capacity", i64), ("count", vp), ("ext", vp)]


class xs_ep_layer(C.Structure):
    _fields_ = [("n_src", i32), ("T", i32), ("H", i32), ("E", i32), ("k", i32), ("I", i32), ("W", i32),
                ("e_begin", i32), ("n_experts", i32), ("src", i32), ("renormalize", i32),
                ("expert_mode", i32), ("cap", i32),
                ("logits", vp), ("x", vp), ("w1", vp), ("w2", vp), ("topk_idx", vp), ("topk_w", vp),
                ("expert_counts", vp), ("src_base", vp), ("expert_offsets", vp), ("dest_counts", vp),
                ("slot_row", vp), ("row_src", vp), ("dispatch_win", C.POINTER(xs_window)),
                ("combine_win", C.POINTER(xs_window)), ("h_ws", vp), ("h_rows", i64), ("y_ws", vp),
                ("out", vp), ("events", vp * 8), ("precision", i32), ("reserved", i32),
                ("w1_scale", vp), ("w2_scale", vp)]


class xs_attn(C.Structure):
    _fields_ = [("heads", i32), ("M", i32), ("head_dim", i32), ("W", i32), ("scale", C.c_float),
                ("max_producers", i32), ("q", vp), ("k", vp), ("v", vp), ("o", vp),
                ("win", C.POINTER(xs_window))]


class xs_scatter_desc(C.Structure):
    _fields_ = [("kind", i32), ("rows_per_dest", i32), ("n_proj", i32), ("n_heads", i32),
                ("head_dim", i32), ("heads_per_group", i32)]


class xs_burst(C.Structure):
    _fields_ = [("V_bytes", f64), ("T0_us", f64), ("G_us", f64), ("cover_us", f64)]


class xs_burst_pred(C.Structure):
    _fields_ = [("rho", f64), ("delta_b", f64), ("q_before", f64), ("b_iso", f64), ("T_iss_us", f64),
                ("stall_us", f64), ("mma_stall_us", f64), ("guard_ok", i32), ("_pad", i32)]


class xs_calib_summary(C.Structure):
    _fields_ = [("model", xs_model), ("knee", i32), ("_pad", i32), ("Q_bracket_lo", f64), ("Q_bracket_hi", f64)]


class xs_recovery(C.Structure):
    _fields_ = [("T0_us", f64), ("G_star_us", f64), ("rho", f64), ("delta_b", f64), ("b_iso", f64),
                ("stall_us", f64), ("tail_us", f64), ("coupled_us", f64), ("guard_ok", i32), ("M_ub_star", i32)]


XS_AUDIT_MAX = 16


class xs_pacing_audit(C.Structure):
    _fields_ = [("policy", i32), ("chunk", i32), ("lead_rows", i32), ("producers", i32), ("rows", i32),
                ("rate_feasible", i32), ("n_cand", i32), ("_pad", i32), ("t_l1_us", f64), ("t_l2_us", f64),
                ("V_full_bytes", f64), ("cand_policy", i32 * XS_AUDIT_MAX), ("cand_chunk", i32 * XS_AUDIT_MAX),
                ("cand_bursts", i32 * XS_AUDIT_MAX), ("cand_guard_fail", i32 * XS_AUDIT_MAX),
                ("cand_stall_us", f64 * XS_AUDIT_MAX), ("cand_mma_stall_us", f64 * XS_AUDIT_MAX),
                ("cand_compute_us", f64 * XS_AUDIT_MAX)]


class xs_calib(C.Structure):
    _fields_ = [("rec_V", C.POINTER(f64)), ("rec_T", C.POINTER(f64)), ("n_rec", i32),
                ("zg_V", C.POINTER(f64)), ("zg_T", C.POINTER(f64)), ("n_zg", i32),
                ("iso_V", C.POINTER(f64)), ("iso_T", C.POINTER(f64)), ("n_iso", i32),
                ("K", i32), ("knee_excess", f64)]


class xs_microbench_args(C.Structure):
    _fields_ = [("target", vp), ("target_bytes", i64), ("K", i32), ("B_bytes", i32), ("n_bursts", i32),
                ("gap_ns", i32), ("mode", i32), ("store_waves", i32)]


def _sig(name, res, *args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = list(args)
    return f


P = C.POINTER
xs_strerror = _sig("xs_strerror", C.c_char_p, C.c_int)
xs_version = _sig("xs_version", C.c_int)
xs_route_topk_softmax = _sig("xs_route_topk_softmax", C.c_int, vp, i32, i32, i32, i32, vp, vp, vp)
xs_dispatch_layout_workspace_bytes = _sig("xs_dispatch_layout_workspace_bytes", C.c_int, i32, i32, i32, P(i64))
xs_dispatch_layout = _sig("xs_dispatch_layout", C.c_int, vp, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp,
                          vp, vp, vp, i64, vp, vp)
xs_dispatch = _sig("xs_dispatch", C.c_int, vp, i32, i32, vp, vp, i32, i32, P(xs_window), i32, vp, vp)
xs_ep_layer_workspace_bytes = _sig("xs_ep_layer_workspace_bytes", C.c_int, P(xs_ep_layer), P(i64))
xs_expert_ffn = _sig("xs_expert_ffn", C.c_int, P(xs_ep_layer), vp, i64, vp, vp)
xs_combine_send = _sig("xs_combine_send", C.c_int, P(xs_ep_layer), P(xs_pacing), vp, vp)
xs_combine_reduce = _sig("xs_combine_reduce", C.c_int, vp, i64, vp, i32, i32, i32, vp, vp)
xs_fused_ep_layer = _sig("xs_fused_ep_layer", C.c_int, P(xs_ep_layer), P(xs_pacing), P(xs_trace), vp, i64,
                         vp, vp)
xs_gemm = _sig("xs_gemm", C.c_int, vp, i64, vp, i64, vp, i64, i32, i32, i32, P(xs_trace), vp)
xs_gemm_scatter = _sig("xs_gemm_scatter", C.c_int, vp, i64, vp, i64, i32, i32, i32, P(xs_scatter_desc),
                       P(xs_window), i32, P(xs_pacing), P(xs_trace), vp)
xs_scatter_copy = _sig("xs_scatter_copy", C.c_int, vp, i64, i32, i32, P(xs_scatter_desc), P(xs_window),
                       i32, vp)
xs_attention = _sig("xs_attention", C.c_int, P(xs_attn), i32, P(xs_trace), vp)
xs_ulysses_copy = _sig("xs_ulysses_copy", C.c_int, vp, i32, i32, i32, P(xs_window), i32, vp)
xs_dispatch_rows = _sig("xs_dispatch_rows", C.c_int, vp, i64, i32, i32, vp, vp, i32, i32, P(xs_window), i32,
                        vp, vp)
xs_ring_slot_bytes = _sig("xs_ring_slot_bytes", C.c_int, i32, i32, P(i64))
xs_dispatch_ring_workspace_bytes = _sig("xs_dispatch_ring_workspace_bytes", C.c_int, i32, i32, i32, i32, P(i64))
xs_dispatch_ring = _sig("xs_dispatch_ring", C.c_int, vp, i32, i32, vp, vp, i32, i32, P(xs_window), i32,
                        P(xs_window), i32, i32, i64, vp, i64, vp, vp, vp)
xs_quantize_mx = _sig("xs_quantize_mx", C.c_int, vp, i64, i32, i64, i32, vp, i64, vp, i64, vp)
xs_quantize_mx_grouped = _sig("xs_quantize_mx_grouped", C.c_int, vp, i64, i32, i64, i32, vp, i64, vp, vp)
xs_gemm_mx = _sig("xs_gemm_mx", C.c_int, vp, i64, vp, i64, vp, i64, vp, i64, i32, vp, i64, i32, i32, i32,
                  P(xs_trace), vp)
xs_model_predict = _sig("xs_model_predict", C.c_int, P(xs_model), P(xs_burst), i32, f64, P(xs_burst_pred))
xs_model_fit = _sig("xs_model_fit", C.c_int, P(xs_calib), P(xs_model))
xs_xstage_microbench = _sig("xs_xstage_microbench", C.c_int, P(xs_microbench_args), P(xs_trace), vp)
xs_clock_rate_hz = _sig("xs_clock_rate_hz", C.c_double)
XS_STATIC_SCRATCH_BYTES = 48 << 20
xs_fused_ep_layer_noalloc = _sig("xs_fused_ep_layer_noalloc", C.c_int, P(xs_ep_layer), P(xs_pacing), P(xs_trace),
                                 vp, vp)
xs_grouped_gemm = _sig("xs_grouped_gemm", C.c_int, vp, i64, i32, vp, vp, i32, vp, i32, i32, vp, i64, i32, vp, vp)
xs_drain_rate = _sig("xs_drain_rate", C.c_int, vp, vp, i32, P(f64))
xs_calib_knee = _sig("xs_calib_knee", C.c_int, vp, vp, i32, f64, P(i32))
xs_model_calibrate = _sig("xs_model_calibrate", C.c_int, P(xs_calib), P(xs_calib_summary))
xs_burst_gap = _sig("xs_burst_gap", C.c_int, P(xs_model), f64, f64, P(f64), P(f64))
xs_recovery_audit = _sig("xs_recovery_audit", C.c_int, P(xs_model), f64, i32, f64, f64, i32, P(xs_recovery))
xs_pacing_audit_run = _sig("xs_pacing_audit_run", C.c_int, P(xs_ep_layer), P(xs_pacing), P(xs_pacing_audit))
xs_trace_tile_times = _sig("xs_trace_tile_times", C.c_int, vp, vp, i64, i32, P(f64), P(f64), P(f64))

EXPORTED = ["xs_strerror", "xs_version", "xs_route_topk_softmax", "xs_dispatch_layout_workspace_bytes",
            "xs_dispatch_layout", "xs_dispatch", "xs_ep_layer_workspace_bytes", "xs_expert_ffn",
            "xs_combine_send", "xs_combine_reduce", "xs_fused_ep_layer", "xs_gemm", "xs_gemm_scatter",
            "xs_scatter_copy", "xs_attention", "xs_ulysses_copy", "xs_quantize_mx", "xs_quantize_mx_grouped", "xs_gemm_mx", "xs_dispatch_rows",
            "xs_ring_slot_bytes", "xs_dispatch_ring_workspace_bytes", "xs_dispatch_ring",
            "xs_model_predict", "xs_model_fit", "xs_pacing_audit_run", "xs_trace_tile_times",
            "xs_grouped_gemm", "xs_fused_ep_layer_noalloc", "xs_drain_rate", "xs_calib_knee", "xs_model_calibrate", "xs_burst_gap", "xs_recovery_audit",
            "xs_xstage_microbench", "xs_clock_rate_hz"]


class XStageError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where}: {xs_strerror(code).decode()} ({code})")
        self.code = code


def check(code: int, where: str = "xstage") -> None:
    if code != XS_OK:
        raise XStageError(code, where)


# ----------------------------------------------------------------------------- marshalling
def ptr(t) -> int | None:
    """Device pointer of a tensor (or None)."""
    return None if t is None else t.data_ptr()


def stream_handle(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def window(t, capacity_rows: int | None = None, row_bytes: int | None = None, flag=None) -> xs_window:
    """Window over a 2-D (rows, cols) tensor, or over raw memory given (ptr, rows, row_bytes)."""
    if isinstance(t, tuple):
        base, rows, stride = t
        return xs_window(base, rows, stride, flag if isinstance(flag, int) else ptr(flag))
    rows = t.shape[0] if capacity_rows is None else capacity_rows
    stride = t.stride(0) * t.element_size() if row_bytes is None else row_bytes
    return xs_window(t.data_ptr(), rows, stride, flag if isinstance(flag, int) else ptr(flag))


def windows(ws) -> C.Array:
    arr = (xs_window * len(ws))()
    for i, w in enumerate(ws):
        arr[i] = w
    return arr


def trace(buf, count) -> xs_trace:
    return xs_trace(buf.data_ptr(), buf.numel() // 4, count.data_ptr())


class HipEvents:
    """Raw hipEvent_t handles (created with timing enabled) for the library to record
    around a kernel on the caller's stream."""

    _hip = None

    def __init__(self, n: int):
        if HipEvents._hip is None:
            h = C.CDLL("libamdhip64.so")
            h.hipEventCreate.argtypes = [C.POINTER(vp)]
            h.hipEventDestroy.argtypes = [vp]
            h.hipEventSynchronize.argtypes = [vp]
            h.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), vp, vp]
            h.hipEventRecord.argtypes = [vp, vp]
            HipEvents._hip = h
        self.ev = []
        for _ in range(n):
            e = vp()
            if HipEvents._hip.hipEventCreate(C.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.ev.append(e.value)

    def record(self, i: int, stream) -> None:
        if HipEvents._hip.hipEventRecord(self.ev[i], stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, i: int, j: int) -> float:
        HipEvents._hip.hipEventSynchronize(self.ev[j])
        ms = C.c_float()
        if HipEvents._hip.hipEventElapsedTime(C.byref(ms), self.ev[i], self.ev[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    @staticmethod
    def elapsed_ms_pair(a, b) -> float:
        HipEvents._hip.hipEventSynchronize(b)
        ms = C.c_float()
        if HipEvents._hip.hipEventElapsedTime(C.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def destroy(self):
        for e in self.ev:
            HipEvents._hip.hipEventDestroy(e)
        self.ev = []
