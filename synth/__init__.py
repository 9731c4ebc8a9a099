"""Seeded synthetic inputs for the fused store-path workloads.

This module only draws random numbers and rounds the draws to bf16 storage; it
holds none of the arithmetic of routing, dispatch, expert compute, combine or the
scatter GEMMs. Both the CPU oracle and the HIP path are fed from here.

Every array comes from ``numpy.random.default_rng(SeedSequence([seed, stream]))``
with a fixed stream number per tensor, so the same (seed, config) always yields
the same bytes. Floating-point tensors are drawn in fp32 and rounded to bf16 with
round-to-nearest-even; they are returned as ``uint16`` bit patterns.

Stream numbers: 1 x, 2 logits, 3 W1, 4 W2, 5 A (TP), 6 B (TP), 7 X (SP),
8 Wqkv (SP), 10+s per-source x, 50+s per-source logits, 100 Zipf popularity
permutation, 101+s per-source Gumbel noise, 200 pre-filled remote combine rows,
300+e per-expert W1, 600+e per-expert W2.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = [
    "rng", "to_bf16_bits", "bf16_bits_to_f32", "normal_bf16", "EPConfig", "TPConfig",
    "SPConfig", "EP_TINY", "EP_DSV3_SHARE", "TP_ROWBLOCK", "SP_QKV", "ep_inputs",
    "tp_inputs", "sp_inputs", "zipf_logits", "uniform_logits", "int_valued_bf16",
]


def rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(stream)]))


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(seed: int, stream: int, shape, std: float = 1.0, chunk_rows: int = 1024) -> np.ndarray:
    """N(0, std^2) draws rounded to bf16 bits; generated in row chunks to bound memory."""
    shape = tuple(int(s) for s in shape)
    g = rng(seed, stream)
    out = np.empty(shape, dtype=np.uint16)
    flat = out.reshape(shape[0], -1) if len(shape) > 1 else out.reshape(-1, 1)
    for r0 in range(0, flat.shape[0], chunk_rows):
        r1 = min(flat.shape[0], r0 + chunk_rows)
        d = g.standard_normal((r1 - r0, flat.shape[1]), dtype=np.float32)
        if std != 1.0:
            d *= np.float32(std)
        flat[r0:r1] = to_bf16_bits(d)
    return out


def int_valued_bf16(seed: int, stream: int, shape, lo: int = -2, hi: int = 2) -> np.ndarray:
    """Small integers in [lo, hi] as bf16 bits (exactly representable)."""
    g = rng(seed, stream)
    v = g.integers(lo, hi + 1, size=tuple(shape)).astype(np.float32)
    return to_bf16_bits(v)


def uniform_logits(seed: int, stream: int, T: int, E: int) -> np.ndarray:
    """Router logits drawn N(0,1) in fp32."""
    return rng(seed, stream).standard_normal((T, E), dtype=np.float32)


def zipf_logits(seed: int, src: int, T: int, E: int, s: float = 1.2) -> np.ndarray:
    """Zipf(s)-skewed router logits.

    Expert popularity is p_r proportional to r^-s for ranks r = 1..E, assigned to experts
    by one seeded permutation shared by every source; per-token logits are
    log p + Gumbel(0,1) noise, so taking the top k samples experts without
    replacement with probability proportional to p.
    """
    perm = rng(seed, 100).permutation(E)
    r = np.arange(1, E + 1, dtype=np.float64)
    p = r ** (-s)
    p /= p.sum()
    logp = np.empty(E, dtype=np.float64)
    logp[perm] = np.log(p)
    gum = rng(seed, 101 + src).gumbel(size=(T, E))
    return (logp[None, :] + gum).astype(np.float32)


@dataclass(frozen=True)
class EPConfig:
    """One rank's share of an expert-parallel MoE layer."""
    name: str
    T: int                # tokens per source rank
    H: int                # hidden size
    E: int                # experts in total
    k: int                # experts per token
    I: int                # SwiGLU intermediate size
    W: int                # destination windows (ranks)
    n_src: int            # source ranks whose tokens reach this rank
    rank: int = 0         # which destination window is "this GPU"
    compute_all: bool = False  # compute every expert here (single-source layer)
    routing: str = "uniform"   # "uniform" | "zipf"
    w_std: float = 0.02

    @property
    def E_local(self) -> int:
        return self.E // self.W


# Tiny layer: T=256, H=512, 8 experts, top-2, I=1024, 4 windows, one source.
EP_TINY = EPConfig("ep_tiny_T256_H512_E8_k2_I1024_W4", T=256, H=512, E=8, k=2, I=1024, W=4,
                   n_src=1, rank=0, compute_all=True)
# One rank's EP share of a DeepSeek-V3-like layer: 8 ranks x 4096 tokens, H=7168,
# 256 experts (32 per rank), top-8, I=2048.
EP_DSV3_SHARE = EPConfig("ep_dsv3_share_T4096_H7168_E256_k8_I2048_W8", T=4096, H=7168, E=256, k=8,
                         I=2048, W=8, n_src=8, rank=0)


@dataclass(frozen=True)
class TPConfig:
    name: str
    M: int
    K: int
    N: int
    W: int
    b_std: float = 0.02


TP_ROWBLOCK = TPConfig("tp_rowblock_M8192_K1024_N8192_W8", M=8192, K=1024, N=8192, W=8)


@dataclass(frozen=True)
class SPConfig:
    name: str
    S: int          # local sequence tokens
    Dm: int         # model dim
    n_heads: int
    head_dim: int
    heads_per_group: int
    w_std: float = 0.02

    @property
    def W(self) -> int:
        return self.n_heads // self.heads_per_group


SP_QKV = SPConfig("sp_qkv_S4096_D4096_h32x128_g4", S=4096, Dm=4096, n_heads=32, head_dim=128,
                  heads_per_group=4)


def ep_logits(cfg: EPConfig, seed: int = 0) -> np.ndarray:
    """Router logits for every source, fp32 [n_src, T, E]."""
    out = np.empty((cfg.n_src, cfg.T, cfg.E), dtype=np.float32)
    for s in range(cfg.n_src):
        if cfg.routing == "zipf":
            out[s] = zipf_logits(seed, s, cfg.T, cfg.E)
        elif cfg.n_src == 1:
            out[s] = uniform_logits(seed, 2, cfg.T, cfg.E)
        else:
            out[s] = uniform_logits(seed, 50 + s, cfg.T, cfg.E)
    return out


def ep_x(cfg: EPConfig, seed: int = 0) -> np.ndarray:
    """Token activations for every source, bf16 bits [n_src, T, H]."""
    if cfg.n_src == 1:
        return normal_bf16(seed, 1, (cfg.T, cfg.H))[None]
    out = np.empty((cfg.n_src, cfg.T, cfg.H), dtype=np.uint16)

    def one(s):
        out[s] = normal_bf16(seed, 10 + s, (cfg.T, cfg.H))

    with cf.ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0))))) as ex:
        list(ex.map(one, range(cfg.n_src)))
    return out


def ep_weights(cfg: EPConfig, experts, seed: int = 0):
    """Expert weights for the listed global expert ids, bf16 bits.

    W1 is [n][2I][H] (rows [0,I) gate, [I,2I) up), W2 is [n][H][I]; both are
    output-major (the reduction dimension is contiguous).
    """
    experts = list(experts)
    w1 = np.empty((len(experts), 2 * cfg.I, cfg.H), dtype=np.uint16)
    w2 = np.empty((len(experts), cfg.H, cfg.I), dtype=np.uint16)

    def one(i):   # every expert has its own streams, so experts are drawn concurrently
        e = experts[i]
        w1[i] = normal_bf16(seed, 300 + e, (2 * cfg.I, cfg.H), std=cfg.w_std)
        w2[i] = normal_bf16(seed, 600 + e, (cfg.H, cfg.I), std=cfg.w_std)

    with cf.ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0))))) as ex:
        list(ex.map(one, range(len(experts))))
    return w1, w2


def ep_remote_combine_fill(cfg: EPConfig, seed: int = 0) -> np.ndarray:
    """bf16 N(0,1) rows standing in for expert outputs computed by other ranks,
    [T*k, H] for this rank's own combine buffer."""
    return normal_bf16(seed, 200, (cfg.T * cfg.k, cfg.H))


def computed_experts(cfg: EPConfig):
    if cfg.compute_all:
        return list(range(cfg.E))
    return list(range(cfg.rank * cfg.E_local, (cfg.rank + 1) * cfg.E_local))


def ep_inputs(cfg: EPConfig, seed: int = 0, with_weights: bool = True):
    d = {"logits": ep_logits(cfg, seed), "x": ep_x(cfg, seed)}
    if with_weights:
        d["w1"], d["w2"] = ep_weights(cfg, computed_experts(cfg), seed)
    return d


def tp_inputs(cfg: TPConfig, seed: int = 0):
    """A [M,K] ~ N(0,1) and B logically [K,N] ~ N(0, b_std^2), both bf16 bits."""
    return {"a": normal_bf16(seed, 5, (cfg.M, cfg.K)),
            "b": normal_bf16(seed, 6, (cfg.K, cfg.N), std=cfg.b_std)}


def sp_inputs(cfg: SPConfig, seed: int = 0):
    """X [S,Dm] ~ N(0,1) and Wqkv logically [Dm, 3*Dm] ~ N(0, w_std^2), bf16 bits."""
    return {"x": normal_bf16(seed, 7, (cfg.S, cfg.Dm)),
            "w": normal_bf16(seed, 8, (cfg.Dm, 3 * cfg.n_heads * cfg.head_dim), std=cfg.w_std)}


@dataclass(frozen=True)
class AttnConfig:
    """One rank's Ulysses attention share: all M tokens of its local heads."""
    name: str
    M: int                # sequence length (all tokens, after the pre-attention exchange)
    heads: int            # local heads
    head_dim: int
    W: int                # sequence chunks = destination windows of the post-attention exchange


ATTN_UP_8K = AttnConfig("attn_up_M8192_h8_d128_W8", M=8192, heads=8, head_dim=128, W=8)
ATTN_UP_16K = AttnConfig("attn_up_M16384_h8_d128_W8", M=16384, heads=8, head_dim=128, W=8)
ATTN_UP_32K = AttnConfig("attn_up_M32768_h8_d128_W8", M=32768, heads=8, head_dim=128, W=8)


def attn_inputs(cfg: AttnConfig, seed: int = 0):
    """Q, K, V [heads][M][head_dim] ~ N(0, 1), bf16 bits."""
    sh = (cfg.heads, cfg.M, cfg.head_dim)
    return {"q": normal_bf16(seed, 900, sh), "k": normal_bf16(seed, 901, sh), "v": normal_bf16(seed, 902, sh)}
