"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

# bf16-input / fp32-accumulate outputs against the oracle's fp64 value before its final
# rounding: per element |gpu - ref| / max(1, |ref|) <= 2e-2 and relative L2 <= 1e-2.
ELEM_TOL = 2e-2
L2_TOL = 1e-2


def require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def xs():
    from paper_2607_23264_amd import xstage
    return xstage


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint16)


def dev_bits(a: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)


def bits_f64(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_close(gpu_bits: np.ndarray, ref64: np.ndarray, what: str):
    g = bits_f64(gpu_bits)
    r = np.asarray(ref64, dtype=np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite values"
    err = np.abs(g - r) / np.maximum(1.0, np.abs(r))
    worst = float(err.max()) if err.size else 0.0
    rl2 = float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-300)) if r.size else 0.0
    assert worst <= ELEM_TOL, f"{what}: max scaled error {worst:.3e} at {np.unravel_index(err.argmax(), err.shape)}"
    assert rl2 <= L2_TOL, f"{what}: relative L2 {rl2:.3e}"
    return worst, rl2
