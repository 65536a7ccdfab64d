"""Seeded synthetic inputs for the BSQ codec: weights, activations, LoRA
adapters and decoder parameters.

This module is shared by the tests, the benchmark and the smoke check. It holds
random draws and shapes only, none of the codec's arithmetic, so that both the
CPU oracle and the HIP library can consume the very same bytes.

Workload recipe (stand-ins for the Qwen3 checkpoints the paper evaluates on,
Section IV-A; only the projection shapes are taken from those models):

* weights ~ N(0, 0.02), drawn in fp32 and rounded to bf16 (fp32 for the tiny
  case); exactly ceil(d_in/100) input columns, chosen by a seeded shuffle, are
  multiplied by 10 after sampling (the 1% outlier channels that the protected
  8-bit path is meant for, Section III-E);
* activations ~ N(0, 1) in bf16 (fp32 for the tiny case);
* LoRA adapters A (r x d_in) and B (d_out x r) ~ N(0, 0.01) in bf16, rank 16;
* decoder parameters ~ U(-1/sqrt(fan_in), +1/sqrt(fan_in)) from a
  counter-based SplitMix64 stream keyed by (seed, category, stage, tensor), so
  a decoder is the same on every machine and needs no torch generator.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

MASK64 = (1 << 64) - 1
BASE_SEED = 2607_08643

# Decoder kinds, numbered as in include/bsq.h.
DEC_IDENTITY = 0
DEC_LINEAR = 1
DEC_MLP = 2
DEC_MLP_RES1 = 3


# --------------------------------------------------------------------------
# Counter-based generator (SplitMix64, Steele, Lea & Flood 2014).
# --------------------------------------------------------------------------
def _splitmix64_np(x: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser applied elementwise to uint64 counters."""
    with np.errstate(over="ignore"):
        z = (x + np.uint64(0x9E3779B97F4A7C15)).astype(np.uint64)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def splitmix64(x: int) -> int:
    """Scalar SplitMix64 (used to derive stream keys)."""
    z = (x + 0x9E3779B97F4A7C15) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def stream_key(*parts: int) -> int:
    """Fold a tuple of small integers into one 64-bit stream key."""
    k = 0
    for p in parts:
        k = splitmix64((k ^ (int(p) & MASK64)) & MASK64)
    return k


def uniform01(key: int, n: int) -> np.ndarray:
    """n doubles in [0, 1): the top 53 bits of SplitMix64(key + i)."""
    ctr = (np.arange(n, dtype=np.uint64) + np.uint64(key & MASK64)).astype(np.uint64)
    bits = _splitmix64_np(ctr) >> np.uint64(11)
    return bits.astype(np.float64) * (1.0 / (1 << 53))


def uniform_sym(key: int, n: int, bound: float) -> np.ndarray:
    """n fp32 values ~ U(-bound, +bound), rounded from fp64 to nearest fp32."""
    u = uniform01(key, n)
    return ((2.0 * u - 1.0) * bound).astype(np.float32)


# --------------------------------------------------------------------------
# Decoder parameters.
# --------------------------------------------------------------------------
@dataclass
class StageDecoder:
    """Parameters of one stage's decoder, all fp32, row-major.

    MLP:      W1 [h, b], b1 [h], W2 [d, h], b2 [d]
    MLP_RES1: the MLP's tensors plus the residual block's R [h, h], c [h]
    LINEAR:   W1 = M [d, b], b1 = beta [d]   (W2, b2 unused)
    IDENTITY: no parameters.
    E [b, d]: the stage's linear encoder z = E r, when the codec has one.
    """
    W1: np.ndarray | None = None
    b1: np.ndarray | None = None
    W2: np.ndarray | None = None
    b2: np.ndarray | None = None
    R: np.ndarray | None = None
    c: np.ndarray | None = None
    E: np.ndarray | None = None


def decoder_params(kind: int, d: int, b: int, hidden: int, stages: int,
                   seed: int = BASE_SEED, category: int = 0, encoder: bool = False) -> list[StageDecoder]:
    """Seeded stage codecs; with encoder=True each also gets a linear encoder
    E [b, d] ~ U(-1/sqrt(d), 1/sqrt(d)) (an untrained stand-in for the
    learned one)."""
    out = []
    for s in range(stages):
        def draw(tensor: int, n: int, fan_in: int) -> np.ndarray:
            key = stream_key(seed, category, s, tensor)
            return uniform_sym(key, n, 1.0 / math.sqrt(fan_in))
        if kind == DEC_IDENTITY:
            out.append(StageDecoder())
        elif kind == DEC_LINEAR:
            out.append(StageDecoder(W1=draw(0, d * b, b).reshape(d, b),
                                    b1=draw(1, d, b)))
        elif kind in (DEC_MLP, DEC_MLP_RES1):
            h = hidden
            dec = StageDecoder(W1=draw(0, h * b, b).reshape(h, b),
                               b1=draw(1, h, b),
                               W2=draw(2, d * h, h).reshape(d, h),
                               b2=draw(3, d, h))
            if kind == DEC_MLP_RES1:
                dec.R = draw(4, h * h, h).reshape(h, h)
                dec.c = draw(5, h, h)
            out.append(dec)
        else:
            raise ValueError(f"unknown decoder kind {kind}")
        if encoder:
            out[-1].E = draw(6, b * d, d).reshape(b, d)
    return out


# --------------------------------------------------------------------------
# Weights, activations, adapters (torch tensors on the requested device).
# --------------------------------------------------------------------------
def n_outliers(d_in: int, num: int = 1, den: int = 100) -> int:
    """ceil(d_in * num / den) in integer arithmetic."""
    return (d_in * num + den - 1) // den


def outlier_columns(d_in: int, k: int, seed: int) -> np.ndarray:
    """k distinct input columns from a seeded shuffle, ascending."""
    if k == 0:
        return np.zeros(0, dtype=np.int64)
    u = uniform01(stream_key(seed, 0xC01, d_in), d_in)
    perm = np.argsort(u, kind="stable")
    return np.sort(perm[:k]).astype(np.int64)


def weight(d_out: int, d_in: int, seed: int, k_outliers: int = 0,
           dtype=None, device="cpu", std: float = 0.02, outlier_scale: float = 10.0,
           n_mats: int = 1):
    """Weight tensor [n_mats, d_out, d_in] (or [d_out, d_in] if n_mats == 1)."""
    import torch
    dtype = dtype or torch.bfloat16
    g = torch.Generator(device=device)
    g.manual_seed(stream_key(seed, d_out, d_in) & 0x7FFFFFFFFFFFFFFF)
    w = torch.randn((n_mats, d_out, d_in), generator=g, device=device,
                    dtype=torch.float32).mul_(std)
    cols = None
    if k_outliers:
        cols = []
        for m in range(n_mats):
            c = outlier_columns(d_in, k_outliers, stream_key(seed, m))
            w[m][:, torch.as_tensor(c, device=device)] *= outlier_scale
            cols.append(c)
    w = w.to(dtype)
    if n_mats == 1:
        w = w[0]
        cols = None if cols is None else cols[0]
    return w, cols


def activation(n: int, seed: int, dtype=None, device="cpu", batch: int | None = None):
    """Activations ~ N(0, 1): [n] for batch None, else [batch, n]."""
    import torch
    dtype = dtype or torch.bfloat16
    g = torch.Generator(device=device)
    g.manual_seed(stream_key(seed, 0xA, n, batch or 0) & 0x7FFFFFFFFFFFFFFF)
    shape = (n,) if batch is None else (batch, n)
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(dtype)


def lora(d_out: int, d_in: int, rank: int, seed: int, dtype=None, device="cpu",
         std: float = 0.01):
    """LoRA adapters A [rank, d_in] and B [d_out, rank] ~ N(0, std)."""
    import torch
    dtype = dtype or torch.bfloat16
    g = torch.Generator(device=device)
    g.manual_seed(stream_key(seed, 0x10A, d_out, d_in, rank) & 0x7FFFFFFFFFFFFFFF)
    A = torch.randn((rank, d_in), generator=g, device=device, dtype=torch.float32).mul_(std)
    B = torch.randn((d_out, rank), generator=g, device=device, dtype=torch.float32).mul_(std)
    return A.to(dtype), B.to(dtype)


# --------------------------------------------------------------------------
# Workload shapes (Qwen3-8B and Qwen3-32B linear projections).
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Proj:
    name: str
    d_out: int
    d_in: int
    group: str  # projections in one group read the same activation


def qwen3_8b_block() -> list[Proj]:
    return [Proj("q", 4096, 4096, "qkv"), Proj("k", 1024, 4096, "qkv"),
            Proj("v", 1024, 4096, "qkv"), Proj("o", 4096, 4096, "o"),
            Proj("gate", 12288, 4096, "gateup"), Proj("up", 12288, 4096, "gateup"),
            Proj("down", 4096, 12288, "down")]


def qwen3_32b_block() -> list[Proj]:
    return [Proj("q", 8192, 5120, "qkv"), Proj("k", 1024, 5120, "qkv"),
            Proj("v", 1024, 5120, "qkv"), Proj("o", 5120, 8192, "o"),
            Proj("gate", 25600, 5120, "gateup"), Proj("up", 25600, 5120, "gateup"),
            Proj("down", 5120, 25600, "down")]


CATEGORIES = ("q", "k", "v", "o", "gate", "up", "down")


@dataclass(frozen=True)
class Workload:
    name: str
    projs: tuple = field(default_factory=tuple)
    layers: int = 1
    d: tuple = (8,)
    lora_rank: int = 0
    protect: bool = True
    batch: tuple = (1,)
    fp32: bool = False


WORKLOADS = {
    "tiny": Workload("tiny: one 256x256 fp32 layer, d=8, 2 stages, MLP decoder, no protection",
                     (Proj("tiny", 256, 256, "tiny"),), 1, (8,), 0, False, (1,), True),
    "qwen3-8b-block": Workload("Qwen3-8B-shaped block, bf16, 1% int8-protected input columns",
                               tuple(qwen3_8b_block()), 1, (8, 16), 0, True, (1,)),
    "qwen3-8b-stack": Workload("36-layer Qwen3-8B-shaped stack + rank-16 LoRA, batch-1 decode",
                               tuple(qwen3_8b_block()), 36, (8, 16), 16, True, (1,)),
    "qwen3-8b-batched": Workload("Qwen3-8B-shaped projections, M in {16,64,256}",
                                 tuple(qwen3_8b_block()), 1, (8, 16), 16, True, (16, 64, 256)),
    "qwen3-32b-stack": Workload("64-layer Qwen3-32B-shaped stack, encode + batch-1 decode",
                                tuple(qwen3_32b_block()), 64, (8, 16), 0, True, (1,)),
}
