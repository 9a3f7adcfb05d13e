"""Seeded synthetic Q/K/V for the fused-attention workloads.

This module is shared by the tests, the benchmark and the smoke check.  It
holds none of the attention arithmetic: it draws N(0,1) float32 values from a
fixed numpy PCG64 stream (order Q, K, V, each in C order with shape
[B, H, L, d]), optionally multiplies K by a constant in float32, and rounds
every value once, to nearest-even, to the storage type (bfloat16 or float16).
The GPU path and the oracle both consume exactly these rounded values.

The paper measures single-head, d=128 attention over synthetic shapes
(Section 6, Tables 2 and 3); the named workloads below keep those shapes and
add the batched / causal cases used for parity.
"""
from __future__ import annotations

import dataclasses

import numpy as np

DTYPES = ("bf16", "f16")


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    L: int
    d: int
    dtype: str
    causal: bool
    k_scale: float
    seed: int

    @property
    def scale(self) -> float:
        return softmax_scale(self.d)


# Five workloads: a tiny fp16 case, an 8-head bf16 case, a batched causal
# case with K scaled by 3 (forces frequent running-max rescaling), the
# paper's headline single-head shape L=16384, d=128, and a full-occupancy
# batched causal case at the same sequence length.
WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny_f16_l128_d64", 1, 1, 128, 64, "f16", False, 1.0, 1001),
        Workload("h8_l1024_d128", 1, 8, 1024, 128, "bf16", False, 1.0, 1002),
        Workload("causal_b2h16_l4096_d128_kx3", 2, 16, 4096, 128, "bf16", True, 3.0, 1003),
        Workload("single_head_l16384_d128", 1, 1, 16384, 128, "bf16", False, 1.0, 1004),
        Workload("causal_b4h32_l16384_d128", 4, 32, 16384, 128, "bf16", True, 1.0, 1005),
    )
}


# The sequence-length sweep of the paper's Table 3 (single head, d=128,
# non-causal); L=16384 is the headline workload itself.
SWEEP = (
    Workload("sweep_l4096_d128", 1, 1, 4096, 128, "bf16", False, 1.0, 1101),
    Workload("sweep_l8192_d128", 1, 1, 8192, 128, "bf16", False, 1.0, 1102),
    WORKLOADS["single_head_l16384_d128"],
    Workload("sweep_l32768_d128", 1, 1, 32768, 128, "bf16", False, 1.0, 1104),
)
WORKLOADS.update({w.name: w for w in SWEEP})

# Head dimension 256 (t_kv = 32, 16 rows per wave): one long head and a
# batched causal case of the same flop count as the H=32, d=128 one.
HEAD_DIM_256 = (
    Workload("single_head_l16384_d256", 1, 1, 16384, 256, "bf16", False, 1.0, 1201),
    Workload("causal_b4h16_l16384_d256", 4, 16, 16384, 256, "bf16", True, 1.0, 1202),
)
WORKLOADS.update({w.name: w for w in HEAD_DIM_256})

# Head dimension 96 (t_kv = 64, 48 rows per wave): the same two shapes as the
# d = 128 headline and batched causal workloads.
HEAD_DIM_96 = (
    Workload("single_head_l16384_d96", 1, 1, 16384, 96, "bf16", False, 1.0, 1211),
    Workload("causal_b4h32_l16384_d96", 4, 32, 16384, 96, "bf16", True, 1.0, 1212),
)
WORKLOADS.update({w.name: w for w in HEAD_DIM_96})

# Head dimension 64 (t_kv = 128, 32 rows per wave): the same two shapes.
HEAD_DIM_64 = (
    Workload("single_head_l16384_d64", 1, 1, 16384, 64, "bf16", False, 1.0, 1221),
    Workload("causal_b4h32_l16384_d64", 4, 32, 16384, 64, "bf16", True, 1.0, 1222),
)
WORKLOADS.update({w.name: w for w in HEAD_DIM_64})

# Causal attention with few heads, whose key split runs as pieces of each query
# tile's own key range: one head and two heads at L = 16384.
CAUSAL_FEW_HEADS = (
    Workload("causal_single_head_l16384_d128", 1, 1, 16384, 128, "bf16", True, 1.0, 1231),
    Workload("causal_h2_l16384_d128", 1, 2, 16384, 128, "bf16", True, 1.0, 1232),
)
WORKLOADS.update({w.name: w for w in CAUSAL_FEW_HEADS})

# Many heads of short sequences (the fused kernel's persistent launch).
SHORT_SEQUENCES = (
    Workload("heads1024_l512_d128", 1, 1024, 512, 128, "bf16", False, 1.0, 1241),
    Workload("heads512_l1024_d64", 1, 512, 1024, 64, "bf16", False, 1.0, 1242),
    Workload("causal_heads512_l1024_d128", 1, 512, 1024, 128, "bf16", True, 1.0, 1243),
)
WORKLOADS.update({w.name: w for w in SHORT_SEQUENCES})


def softmax_scale(d: int) -> float:
    """1/sqrt(d) evaluated in float32, returned as the Python float of that value."""
    return float(np.float32(1.0) / np.sqrt(np.float32(d)))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to IEEE binary16 (numpy's cast is round-to-nearest-even)."""
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def bits_to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored bf16/f16 bit patterns to float64."""
    if dtype == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def bits_to_f32(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored bf16/f16 bit patterns to float32."""
    if dtype == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def round_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    if dtype == "f16":
        return f32_to_f16_bits(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def make_qkv(B: int, H: int, L: int, d: int, dtype: str, seed: int, k_scale: float = 1.0):
    """Draw Q, K, V (in that order) and return their storage bit patterns as uint16 [B,H,L,d]."""
    if dtype not in DTYPES:
        raise ValueError(f"unknown dtype {dtype!r}")
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = (B, H, L, d)
    out = []
    for name in ("q", "k", "v"):
        x = rng.standard_normal(shape, dtype=np.float32)
        if name == "k" and k_scale != 1.0:
            x *= np.float32(k_scale)
        out.append(round_bits(x, dtype))
        del x
    return out[0], out[1], out[2]


def make_matrix(rows: int, n: int, dtype: str, seed: int, spread: float = 1.0):
    """A rows x n matrix of N(0,1) float32 values times `spread` (in float32),
    rounded once to the storage type; returns the uint16 bit patterns."""
    if dtype not in DTYPES:
        raise ValueError(f"unknown dtype {dtype!r}")
    x = np.random.Generator(np.random.PCG64(seed)).standard_normal((rows, n), dtype=np.float32)
    if spread != 1.0:
        x *= np.float32(spread)
    return round_bits(x, dtype)


def make_matrix_f32(rows: int, n: int, seed: int, spread: float = 1.0):
    """A rows x n float32 matrix of N(0,1) values times `spread`."""
    x = np.random.Generator(np.random.PCG64(seed)).standard_normal((rows, n), dtype=np.float32)
    if spread != 1.0:
        x *= np.float32(spread)
    return x


def workload_inputs(w: Workload):
    return make_qkv(w.B, w.H, w.L, w.d, w.dtype, w.seed, w.k_scale)
