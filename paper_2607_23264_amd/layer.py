"""Buffers and calls of one rank's expert-parallel layer share, through the C ABI.

This module only allocates torch device memory, uploads inputs and marshals arguments to
libxstage.so; all arithmetic and data movement of the layer happen in the HIP kernels.
bf16 tensors are held as int16 storage of the bf16 bit patterns.
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import numpy as np
import torch

from . import xstage as X


def _dev_bits(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


@dataclass
class Shape:
    n_src: int
    T: int
    H: int
    E: int
    k: int
    I: int
    W: int
    e_begin: int
    n_experts: int
    src: int = 0
    renormalize: int = 0
    expert_mode: int = X.XS_EXPERT_SWIGLU
    cap: int | None = None

    @property
    def epw(self) -> int:
        return self.E // self.W

    @property
    def n_cwin(self) -> int:
        return self.n_experts // self.epw


class EPLayer:
    """Owns every device buffer of one EP layer call (inputs, layout, windows, outputs)."""

    def __init__(self, s: Shape, device="cuda", combine_host: bool = False, sentinel: bool = True,
                 precision: int = X.XS_PREC_BF16, ready_flags: bool = False,
                 host_combine_sources=None):
        self.s = s
        self.precision = precision
        mxp = precision in (X.XS_PREC_MXFP8, X.XS_PREC_W4A8)
        self.mx = mxp
        # weight code bytes per element: E4M3 one, packed E2M1 a half
        self.w_fmt = X.XS_FMT_E2M1 if precision == X.XS_PREC_W4A8 else X.XS_FMT_E4M3
        wdiv = 2 if precision == X.XS_PREC_W4A8 else 1
        # bytes per dispatched token row (MXFP8: codes, then one scale per 32) and per h row;
        # MX token rows sit at a pitch of whole 128-byte lines in the dispatch windows, so that
        # each 128-byte K step of a GEMM activation load reads one line, not two (MX h is
        # h_rows code rows of I bytes followed by the scale groups)
        self.row_bytes = s.H + s.H // 32 if mxp else 2 * s.H
        self.row_pitch = -(-self.row_bytes // 128) * 128 if mxp else self.row_bytes
        self.h_bytes = s.I + s.I // 32 if mxp else 2 * s.I
        self.dev = torch.device(device)
        cap = s.cap if s.cap is not None else s.n_src * s.T * min(s.k, s.epw)
        self.cap = cap
        d = self.dev
        i32 = torch.int32
        self.logits = torch.zeros((s.n_src, s.T, s.E), dtype=torch.float32, device=d)
        self.x_all = torch.zeros((s.n_src, s.T, s.H), dtype=torch.int16, device=d)
        self.w1 = torch.zeros((s.n_experts, 2 * s.I, s.H), dtype=torch.int16, device=d) \
            if s.expert_mode == X.XS_EXPERT_SWIGLU else None
        self.w2 = torch.zeros((s.n_experts, s.H, s.I), dtype=torch.int16, device=d) \
            if s.expert_mode == X.XS_EXPERT_SWIGLU else None
        self.topk_idx = torch.zeros((s.n_src, s.T, s.k), dtype=i32, device=d)
        self.topk_w = torch.zeros((s.n_src, s.T, s.k), dtype=torch.float32, device=d)
        self.expert_counts = torch.zeros((s.n_src, s.E), dtype=i32, device=d)
        self.src_base = torch.zeros((s.n_src, s.E), dtype=i32, device=d)
        self.expert_offsets = torch.zeros((s.E,), dtype=i32, device=d)
        self.dest_counts = torch.zeros((s.W,), dtype=i32, device=d)
        self.slot_row = torch.zeros((s.n_src, s.T, s.k), dtype=i32, device=d)
        self.row_src = torch.full((s.W, cap), -1, dtype=i32, device=d)
        fill = -1 if sentinel else 0
        if mxp:
            self.dwin = torch.full((s.W, cap, self.row_pitch), 0xFF if sentinel else 0, dtype=torch.uint8, device=d)
            self.xq = torch.zeros((s.T, self.row_bytes), dtype=torch.uint8, device=d)
        else:
            self.dwin = torch.full((s.W, cap, s.H), fill, dtype=torch.int16, device=d) if sentinel \
                else torch.empty((s.W, cap, s.H), dtype=torch.int16, device=d)
        self.combine_host = combine_host
        # combine windows of the sources listed in host_combine_sources (all of them with
        # combine_host) live in host-coherent memory: slow sinks beside HBM windows
        host_src = list(range(s.n_src)) if combine_host else list(host_combine_sources or [])
        self.host_sources = host_src
        if host_src and len(host_src) == s.n_src:
            self._host = HostCoherent(s.n_src * s.T * s.k * s.H * 2)
            self.cwin = self._host.view.view(s.n_src, s.T * s.k, s.H)
            self.cwin.fill_(fill)
            self._cw = [self.cwin[i] for i in range(s.n_src)]
        else:
            self.cwin = torch.full((s.n_src, s.T * s.k, s.H), fill, dtype=torch.int16, device=d) if sentinel \
                else torch.empty((s.n_src, s.T * s.k, s.H), dtype=torch.int16, device=d)
            self._cw = [self.cwin[i] for i in range(s.n_src)]
            self._hosts = {}
            for i in host_src:
                h = HostCoherent(s.T * s.k * s.H * 2)
                self._hosts[i] = h
                self._cw[i] = h.view.view(s.T * s.k, s.H)
                self._cw[i].fill_(fill)
        # readiness words: dispatch windows [0, W), combine windows [W, W + n_src)
        self.flags = torch.zeros((s.W + s.n_src,), dtype=i32, device=d) if ready_flags else None
        h_rows = s.n_cwin * cap
        if mxp:
            self.h_ws = torch.zeros((h_rows, self.h_bytes), dtype=torch.uint8, device=d)
            E_, I_, H_ = s.n_experts, s.I, s.H
            self.w1q = torch.zeros((E_, 2 * I_, H_ // wdiv), dtype=torch.uint8, device=d)
            self.w1s = torch.zeros((H_ // 512, E_ * 2 * I_, 16), dtype=torch.uint8, device=d)   # scale groups
            self.w2q = torch.zeros((E_, H_, I_ // wdiv), dtype=torch.uint8, device=d)
            self.w2s = torch.zeros((I_ // 512, E_ * H_, 16), dtype=torch.uint8, device=d)
        else:
            self.h_ws = torch.zeros((h_rows, s.I if s.I else 1), dtype=torch.int16, device=d)
        self.y_ws = torch.zeros((h_rows, s.H), dtype=torch.int16, device=d)
        self.out = torch.zeros((s.T, s.H), dtype=torch.int16, device=d)
        self.status = torch.zeros((1,), dtype=i32, device=d)
        fl = (lambda i: self.flags[i].data_ptr()) if ready_flags else (lambda i: None)
        self._dwins = X.windows([X.window(self.dwin[w], flag=fl(w)) for w in range(s.W)])
        self._cflag = [fl(s.W + i) for i in range(s.n_src)]
        self._cwins = X.windows([self._cwin_desc(i) for i in range(s.n_src)])
        self.L = self._layer_struct()
        nb = C.c_int64()
        X.check(X.xs_ep_layer_workspace_bytes(C.byref(self.L), C.byref(nb)), "workspace")
        self.workspace = torch.zeros((max(1, nb.value),), dtype=torch.uint8, device=d)

    def close(self):
        """Releases the host-coherent sinks (device buffers go with the object)."""
        torch.cuda.synchronize(self.dev)
        for h in list(getattr(self, "_hosts", {}).values()) + ([self._host] if hasattr(self, "_host") else []):
            h.free()

    def _cwin_desc(self, i):
        t = self._cw[i]
        return X.xs_window(t.data_ptr(), t.shape[0], t.stride(0) * 2, self._cflag[i])

    def combine_rows(self, src: int) -> torch.Tensor:
        """Combine window of source src ([T * k][H] int16; a CPU view for host-coherent ones)."""
        return self._cw[src]

    def _layer_struct(self) -> X.xs_ep_layer:
        s = self.s
        L = X.xs_ep_layer()
        for f in ("n_src", "T", "H", "E", "k", "I", "W", "e_begin", "n_experts", "src", "renormalize",
                  "expert_mode"):
            setattr(L, f, getattr(s, f))
        L.cap = self.cap
        L.logits = self.logits.data_ptr()
        L.x = self.x_all[s.src].data_ptr()
        L.precision = self.precision
        if self.mx:
            L.w1, L.w2 = self.w1q.data_ptr(), self.w2q.data_ptr()
            L.w1_scale, L.w2_scale = self.w1s.data_ptr(), self.w2s.data_ptr()
        else:
            L.w1 = X.ptr(self.w1)
            L.w2 = X.ptr(self.w2)
        L.topk_idx = self.topk_idx.data_ptr()
        L.topk_w = self.topk_w.data_ptr()
        L.expert_counts = self.expert_counts.data_ptr()
        L.src_base = self.src_base.data_ptr()
        L.expert_offsets = self.expert_offsets.data_ptr()
        L.dest_counts = self.dest_counts.data_ptr()
        L.slot_row = self.slot_row.data_ptr()
        L.row_src = self.row_src.data_ptr()
        L.dispatch_win = C.cast(self._dwins, C.POINTER(X.xs_window))
        L.combine_win = C.cast(self._cwins, C.POINTER(X.xs_window))
        L.h_ws = self.h_ws.data_ptr()
        L.h_rows = self.h_ws.shape[0]
        L.y_ws = self.y_ws.data_ptr()
        L.out = self.out.data_ptr()
        return L

    # -------------------------------------------------------------------------- inputs
    def upload(self, logits: np.ndarray, x_bits: np.ndarray, w1_bits=None, w2_bits=None):
        self.logits.copy_(torch.from_numpy(np.ascontiguousarray(logits, dtype=np.float32)))
        self.x_all.copy_(_dev_bits(x_bits, "cpu"))
        if w1_bits is not None:
            for i in range(w1_bits.shape[0]):   # expert by expert to bound host staging
                self.w1[i].copy_(_dev_bits(w1_bits[i], "cpu"))
                self.w2[i].copy_(_dev_bits(w2_bits[i], "cpu"))
            if self.mx:
                self.quantize_weights()
        torch.cuda.synchronize(self.dev)

    def quantize_weights(self):
        """MX codes (E4M3, or packed E2M1 for W4A8) and scales of W1 (along H) and W2 (along I),
        on the GPU; the scales grouped by 512 K elements over all weight rows."""
        s = self.s
        st = self.stream
        X.check(X.xs_quantize_mx_grouped(self.w1.data_ptr(), s.n_experts * 2 * s.I, s.H, s.H, self.w_fmt,
                                         self.w1q.data_ptr(), self.w1q.shape[2], self.w1s.data_ptr(), st),
                "quantize w1")
        X.check(X.xs_quantize_mx_grouped(self.w2.data_ptr(), s.n_experts * s.H, s.I, s.I, self.w_fmt,
                                         self.w2q.data_ptr(), self.w2q.shape[2], self.w2s.data_ptr(), st),
                "quantize w2")

    @property
    def stream(self):
        return torch.cuda.current_stream(self.dev).cuda_stream

    # -------------------------------------------------------------------------- steps
    def route(self):
        s = self.s
        X.check(X.xs_route_topk_softmax(self.logits.data_ptr(), s.n_src * s.T, s.E, s.k, s.renormalize,
                                        self.topk_idx.data_ptr(), self.topk_w.data_ptr(), self.stream),
                "route")

    def layout(self):
        s = self.s
        ws = self.workspace
        X.check(X.xs_dispatch_layout(self.topk_idx.data_ptr(), s.n_src, s.T, s.k, s.E, s.W, self.cap,
                                     self.expert_counts.data_ptr(), self.src_base.data_ptr(),
                                     self.expert_offsets.data_ptr(), self.dest_counts.data_ptr(),
                                     self.slot_row.data_ptr(), self.row_src.data_ptr(), ws.data_ptr(),
                                     ws.numel(), self.status.data_ptr(), self.stream), "layout")

    def dispatch(self, src: int):
        s = self.s
        if self.mx:
            rb = self.row_bytes
            X.check(X.xs_quantize_mx(self.x_all[src].data_ptr(), s.T, s.H, s.H, X.XS_FMT_E4M3, self.xq.data_ptr(),
                                     rb, self.xq.data_ptr() + s.H, rb, self.stream), "quantize x")
            X.check(X.xs_dispatch_rows(self.xq.data_ptr(), rb, rb, s.T, self.topk_idx[src].data_ptr(),
                                       self.slot_row[src].data_ptr(), s.k, s.E, self._dwins, s.W,
                                       self.status.data_ptr(), self.stream), "dispatch rows")
            return
        X.check(X.xs_dispatch(self.x_all[src].data_ptr(), s.T, s.H, self.topk_idx[src].data_ptr(),
                              self.slot_row[src].data_ptr(), s.k, s.E, self._dwins, s.W,
                              self.status.data_ptr(), self.stream), "dispatch")

    def expert_ffn(self):
        ws = self.workspace
        X.check(X.xs_expert_ffn(C.byref(self.L), ws.data_ptr(), ws.numel(), self.status.data_ptr(),
                                self.stream), "expert_ffn")

    def combine_send(self, pacing: X.xs_pacing | None = None):
        X.check(X.xs_combine_send(C.byref(self.L), C.byref(pacing) if pacing is not None else None,
                                  self.status.data_ptr(), self.stream), "combine_send")

    def combine_reduce(self):
        s = self.s
        c = self._cw[s.src]
        X.check(X.xs_combine_reduce(c.data_ptr(), c.stride(0) * 2, self.topk_w[s.src].data_ptr(), s.T, s.k,
                                    s.H, self.out.data_ptr(), self.stream), "combine_reduce")

    def prefill_other_sources(self, remote_combine_bits: np.ndarray | None = None):
        """Untimed set-up standing in for the other ranks: route + layout of every source,
        dispatch of every source other than ``src`` and, optionally, the rows of this rank's
        combine buffer that other ranks' experts would write."""
        self.route()
        self.layout()
        for s in range(self.s.n_src):
            if s != self.s.src:
                self.dispatch(s)
        if remote_combine_bits is not None:
            self._cw[self.s.src].copy_(_dev_bits(remote_combine_bits, "cpu"))
        torch.cuda.synchronize(self.dev)

    def fused(self, pacing: X.xs_pacing | None = None, trace: X.xs_trace | None = None):
        ws = self.workspace
        X.check(X.xs_fused_ep_layer(C.byref(self.L), C.byref(pacing) if pacing is not None else None,
                                    C.byref(trace) if trace is not None else None, ws.data_ptr(),
                                    ws.numel(), self.status.data_ptr(), self.stream), "fused_ep_layer")

    def unfused(self):
        self.route()
        self.layout()
        self.dispatch(self.s.src)
        self.expert_ffn()
        self.combine_send()
        self.combine_reduce()


def pacing(policy=X.XS_POLICY_INTERLEAVE, lead=1, chunk=0, max_producers=0, wave_tiles=0, gap_ns=0,
           spin_timeout_us=0, withhold_row=-1, t_l1_us=0.0, t_l2_us=0.0, model=None,
           claim=0, expert_rows=None, sink_share=0.0) -> X.xs_pacing:
    p = X.xs_pacing(policy, lead, chunk, max_producers, wave_tiles, gap_ns, spin_timeout_us, withhold_row,
                    claim, 0, t_l1_us, t_l2_us, None, None, sink_share)
    if model is not None:
        p._model_ref = model
        p.model = C.pointer(model)
    if expert_rows is not None:
        arr = (C.c_int32 * len(expert_rows))(*[int(v) for v in expert_rows])
        p._rows_ref = arr
        p.expert_rows = C.cast(arr, C.POINTER(C.c_int32))
    return p


class HostCoherent:
    """Fine-grained host-coherent memory (hipHostMalloc with hipHostMallocCoherent): a slow
    store sink whose writes cross the fabric to host memory. ``view`` is a CPU tensor over it;
    ``ptr`` is the address kernels store to."""

    _hip = None
    COHERENT = 0x40000000

    def __init__(self, nbytes: int):
        if HostCoherent._hip is None:
            HostCoherent._hip = C.CDLL("libamdhip64.so")
            HostCoherent._hip.hipHostMalloc.argtypes = [C.POINTER(C.c_void_p), C.c_size_t, C.c_uint]
            HostCoherent._hip.hipHostFree.argtypes = [C.c_void_p]
        p = C.c_void_p()
        rc = HostCoherent._hip.hipHostMalloc(C.byref(p), C.c_size_t(nbytes), C.c_uint(self.COHERENT))
        if rc != 0 or not p.value:
            raise RuntimeError(f"hipHostMalloc({nbytes}) failed: {rc}")
        self.ptr = p.value
        self.nbytes = nbytes
        arr = np.ctypeslib.as_array(C.cast(p, C.POINTER(C.c_int16)), shape=(nbytes // 2,))
        self.view = torch.from_numpy(arr)

    def free(self):
        if self.ptr:
            HostCoherent._hip.hipHostFree(C.c_void_p(self.ptr))
            self.ptr = 0
