"""Seeded synthetic inputs shared by the tests, the bench and the smoke check.

This module holds no arithmetic of the quantization method: it only draws
weights and activations of the shapes and distributions of the workloads the
paper evaluates (OPT / LLaMA linear layers, Section 4), and defines those
workloads.  Both sides of every parity test (the CPU oracle and the HIP
library) receive the arrays produced here.

Random numbers come from a counter-based generator so that any element can be
regenerated on its own (the HIP library carries an independent twin of the
same definition for stacks too large to generate on the host):

* hash: the SplitMix64 output function (Steele, Lea and Flood, "Fast
  splittable pseudorandom number generators", OOPSLA 2014), applied to the
  counter ``base + (i + 1) * GAMMA`` (mod 2**64);
* normal deviate: Irwin-Hall sum of eight 16-bit uniforms taken from two
  hashes, centred and scaled with one fp64 multiply, then rounded once to
  fp32.  It has mean 0, the requested variance, kurtosis 2.85 and support
  +-4.9 sigma.  Every step is an exact integer or a single correctly rounded
  IEEE operation, so the host and device twins agree bit for bit;
* outliers: a third hash below ``OUTLIER_THRESHOLD`` (probability 1e-3) marks
  an entry that is multiplied by 10 in fp32.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
# Var of a discrete uniform on 0..65535 is (65536**2 - 1) / 12; eight of them.
IH_TERMS = 8
IH_CENTER2 = IH_TERMS * 65535            # 2*S - IH_CENTER2 is the centred sum, doubled
IH_STD = math.sqrt(IH_TERMS * (65536.0 ** 2 - 1.0) / 12.0)
OUTLIER_PROB = 1e-3
OUTLIER_THRESHOLD = int(OUTLIER_PROB * 2.0 ** 64)
OUTLIER_GAIN = np.float32(10.0)


def _mix64_int(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def stream_base(seed: int, stream: int) -> int:
    """Key of one independent stream: a hash of (seed, stream)."""
    return _mix64_int(((seed & MASK64) * GAMMA + (stream & MASK64)) & MASK64)


def _mix64(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.uint64, copy=False)
    z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX2)
    return z ^ (z >> np.uint64(31))


def hashes(base: int, counters: np.ndarray) -> np.ndarray:
    """SplitMix64 output for counters i: mix(base + (i + 1) * GAMMA)."""
    c = counters.astype(np.uint64, copy=False)
    with np.errstate(over="ignore"):
        z = np.uint64(base) + (c + np.uint64(1)) * np.uint64(GAMMA)
        return _mix64(z)


def _halves_sum(h: np.ndarray) -> np.ndarray:
    m = np.uint64(0xFFFF)
    return ((h & m) + ((h >> np.uint64(16)) & m) + ((h >> np.uint64(32)) & m)
            + (h >> np.uint64(48))).astype(np.int64)


def normal_f32(base: int, counters: np.ndarray, sigma: float) -> np.ndarray:
    """fp32 deviates ~N(0, sigma^2) (Irwin-Hall 8) for the given element counters.

    Element e uses hashes at counters 3e and 3e+1; 3e+2 is its outlier draw.
    """
    e = counters.astype(np.uint64, copy=False)
    with np.errstate(over="ignore"):
        h1 = hashes(base, e * np.uint64(3))
        h2 = hashes(base, e * np.uint64(3) + np.uint64(1))
    s = _halves_sum(h1) + _halves_sum(h2)            # 0 .. 8*65535
    centred2 = (2 * s - IH_CENTER2).astype(np.float64)  # exact integer
    factor = np.float64(sigma / (2.0 * IH_STD))
    return (centred2 * factor).astype(np.float32)


def outlier_mask(base: int, counters: np.ndarray) -> np.ndarray:
    e = counters.astype(np.uint64, copy=False)
    with np.errstate(over="ignore"):
        h3 = hashes(base, e * np.uint64(3) + np.uint64(2))
    return h3 < np.uint64(OUTLIER_THRESHOLD)


def normal_factor(sigma: float) -> float:
    """The fp64 constant multiplying the doubled centred Irwin-Hall sum."""
    return float(np.float64(sigma / (2.0 * IH_STD)))


def weight_rows(seed: int, linear_id: int, n: int, k: int, sigma: float,
                outliers: bool, rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Rows of a synthetic fp32 weight W (n x k, row-major element counter r*k + c).

    ``rows`` selects a subset of rows (all rows when None); any row can be
    regenerated alone.
    """
    base = stream_base(seed, 2 * linear_id)
    rows = np.arange(n, dtype=np.int64) if rows is None else np.asarray(rows, np.int64)
    out = np.empty((rows.size, k), dtype=np.float32)
    step = max(1, (1 << 22) // max(k, 1))
    cols = np.arange(k, dtype=np.uint64)
    for i0 in range(0, rows.size, step):
        rr = rows[i0:i0 + step].astype(np.uint64)
        cnt = (rr[:, None] * np.uint64(k) + cols[None, :]).reshape(-1)
        w = normal_f32(base, cnt, sigma)
        if outliers:
            msk = outlier_mask(base, cnt)
            w = np.where(msk, w * OUTLIER_GAIN, w).astype(np.float32)
        out[i0:i0 + rr.size] = w.reshape(rr.size, k)
    return out


def activations_f32(seed: int, stream: int, m: int, k: int) -> np.ndarray:
    """Activation matrix x (m x k) ~N(0, 1) in fp32, before the storage cast."""
    base = stream_base(seed, 2 * stream + 1)
    cnt = np.arange(m * k, dtype=np.uint64)
    return normal_f32(base, cnt, 1.0).reshape(m, k)


def hadamard_signs(seed: int, block: int) -> np.ndarray:
    """``block`` random signs (int8, +-1) for the sign-randomised Hadamard: sign
    t is -1 when the top bit of hash t of stream (seed, 2**31) is set."""
    h = hashes(stream_base(seed, 1 << 31), np.arange(block, dtype=np.uint64))
    return np.where((h >> np.uint64(63)) == np.uint64(1), -1, 1).astype(np.int8)


def to_f16(x32: np.ndarray) -> np.ndarray:
    return x32.astype(np.float16)


def to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round fp32 to bfloat16 (nearest, ties to even); returns the uint16 bit patterns."""
    b = x32.astype(np.float32).view(np.uint32).astype(np.uint64)
    rnd = ((b >> np.uint64(16)) & np.uint64(1)) + np.uint64(0x7FFF)
    return ((b + rnd) >> np.uint64(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def log_uniform_variance(seed: int, linear_id: int, lo: float, hi: float) -> float:
    """Per-linear variance drawn log-uniformly over [lo, hi] (host-side fp64)."""
    h = int(hashes(stream_base(seed, 1_000_000 + linear_id), np.zeros(1, np.uint64))[0])
    u = (h >> 11) * (1.0 / (1 << 53))
    return float(math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo))))


# --------------------------------------------------------------------------
# Workloads: synthetic OPT / LLaMA-shaped linear layers (paper Section 4.1).
# Shapes are (n_out, k_in) = (N, K).
# --------------------------------------------------------------------------


@dataclass
class Linear:
    name: str
    n: int
    k: int
    sigma: float
    layer: int = 0
    linear_id: int = 0


@dataclass
class Workload:
    index: int
    name: str
    linears: List[Linear]
    levels: int
    osr: Optional[float]              # fixed OSR, or None when MultiOSR assigns it
    batches: Tuple[int, ...]
    x_dtype: str                      # "f16" or "bf16"
    outliers: bool
    seed: int
    multiosr: Optional[Tuple[float, float, float]] = None   # (target, lo, hi)
    notes: str = ""
    prefill: Tuple[int, ...] = field(default_factory=tuple)


def _llama7b_layer(layer: int, first_id: int, sigmas: List[float]) -> List[Linear]:
    shapes = [("q_proj", 4096, 4096), ("k_proj", 4096, 4096), ("v_proj", 4096, 4096),
              ("o_proj", 4096, 4096), ("gate_proj", 11008, 4096), ("up_proj", 11008, 4096),
              ("down_proj", 4096, 11008)]
    return [Linear(nm, n, k, sigmas[i], layer, first_id + i) for i, (nm, n, k) in enumerate(shapes)]


def _llama70b_layer(layer: int, first_id: int, sigma: float) -> List[Linear]:
    shapes = [("q_proj", 8192, 8192), ("k_proj", 1024, 8192), ("v_proj", 1024, 8192),
              ("o_proj", 8192, 8192), ("gate_proj", 28672, 8192), ("up_proj", 28672, 8192),
              ("down_proj", 8192, 28672)]
    return [Linear(nm, n, k, sigma, layer, first_id + i) for i, (nm, n, k) in enumerate(shapes)]


def workload(index: int) -> Workload:
    """The five synthetic workloads (1-based index)."""
    seed = 2510 + index
    if index == 1:
        return Workload(1, "opt125m_q_proj_768x768", [Linear("q_proj", 768, 768, 0.02)],
                        levels=3, osr=2.0, batches=(1, 8), x_dtype="f16", outliers=True, seed=seed)
    if index == 2:
        return Workload(2, "llama7b_down_proj_4096x11008",
                        [Linear("down_proj", 4096, 11008, 0.015)],
                        levels=2, osr=1.5, batches=(1,), x_dtype="f16", outliers=True, seed=seed)
    if index == 3:
        sig = [math.sqrt(log_uniform_variance(seed, i, 1e-4, 1e-3)) for i in range(7)]
        return Workload(3, "llama7b_layer_7_linears", _llama7b_layer(0, 0, sig), levels=3,
                        osr=None, batches=(1, 4, 16), x_dtype="f16", outliers=False, seed=seed,
                        multiosr=(2.5, 1.5, 3.0))
    if index == 4:
        lins = [Linear("sq_8192x8192", 8192, 8192, 0.01, 0, 0),
                Linear("up_28672x8192", 28672, 8192, 0.01, 0, 1),
                Linear("down_8192x28672", 8192, 28672, 0.01, 0, 2)]
        return Workload(4, "llama70b_linears", lins, levels=3, osr=2.0, batches=(1,),
                        x_dtype="bf16", outliers=True, seed=seed, prefill=(2048,))
    if index == 5:
        lins: List[Linear] = []
        for layer in range(80):
            var = 5e-5 + 1.5e-4 * layer / 79.0
            lins += _llama70b_layer(layer, 7 * layer, math.sqrt(var))
        return Workload(5, "llama70b_stack_80x7", lins, levels=3, osr=None, batches=(1, 8),
                        x_dtype="f16", outliers=False, seed=seed, multiosr=(2.5, 1.5, 3.0))
    raise ValueError(f"no workload {index}")
