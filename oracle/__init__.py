"""CPU oracle for the fused store path (test infrastructure only).

This package is the correctness reference for the HIP library. It is plain,
slow, obviously correct numpy written from the X-Stage paper ("X-Stage: Modeling
Post-Issue Backpressure in GPU Communication-Computation Fusion") and the stated
workloads. Only the test-suite, the smoke check and the benchmark's CPU-baseline
leg may import it; the product path never calls into it and shares no code with
it (the two meet only through the seeded input generators in ``synth``).

Arithmetic is fp64 unless a storage format forces a rounding: bf16 tensors are
rounded to nearest-even at the points where the data is stored in bf16 (token
rows, the SwiGLU activation h, expert outputs y, the combined output).

Modules:
  ep              routing, dispatch layout, dispatch, expert SwiGLU FFN,
                  combine-send, combine-reduce, dense brute-force cross-check
  scatter         TP row-block and Ulysses head-group GEMM scatter epilogues
  xstage_model    Burst-Gap model (Eqs. 1-9), calibration fit, audit helpers
  schedule        tile orders: Expert-Wave, cross-wave interleave (Alg. 1), chunked
  attention       softmax attention and the post-attention Ulysses exchange
  ep_mx           the quantized EP layer (W8A8 MXFP8, W4A8 with E2M1 weights)
  ring            dispatch through bounded destination rings, with optional per-destination
                  token dedup
  mx              microscaled formats (E4M3 / E2M1 elements, E8M0 block scales) of the
                  quantized EP path: encode, decode, block quantizer, dequantized GEMM

Parity status: every function here is pinned by tests under ``tests/`` against
closed forms, worked numbers the paper prints, brute force or library routines,
except where a function's docstring says "parity unpinned".
"""
from . import attention, ep, ep_mx, mx, ring, scatter, xstage_model, schedule  # noqa: F401
