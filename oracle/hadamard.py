"""Hadamard matrices and the block transform used for weight smoothing.

Section 3.3 defines a Hadamard matrix by H H^T = n I and builds it with the
Sylvester recursion H_2k = [[H_k, H_k], [H_k, -H_k]] (Eq. 13).  Algorithm 1
(line 6) multiplies each B-column weight block by ``Had`` before Sigma-Delta
quantization and by ``Had^T`` afterwards, so ``Had`` must be orthogonal: this
oracle uses the normalised Sylvester matrix Had = H_B / sqrt(B).
"""
from __future__ import annotations

import numpy as np


def sylvester(n: int) -> np.ndarray:
    """Sylvester Hadamard matrix H_n (int64) by the Eq. 13 recursion, n a power of two."""
    if n < 1 or (n & (n - 1)):
        raise ValueError("Hadamard order must be a power of two")
    h = np.ones((1, 1), dtype=np.int64)
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def fwht_f32(v: np.ndarray) -> np.ndarray:
    """Unnormalised fast Walsh-Hadamard transform along the last axis, in fp32.

    Computes H_n v with the natural (Sylvester) ordering.  Stages run with the
    butterfly span h = 1, 2, 4, ..., n/2; each butterfly replaces (a, b) by
    (a + b, a - b), every add rounded to fp32.  Butterflies of one stage are
    independent, so evaluating them together changes no rounding.
    """
    x = np.array(v, dtype=np.float32, copy=True)
    n = x.shape[-1]
    if n & (n - 1):
        raise ValueError("transform length must be a power of two")
    h = 1
    while h < n:
        y = x.reshape(x.shape[:-1] + (n // (2 * h), 2, h))
        a = y[..., 0, :].copy()
        b = y[..., 1, :].copy()
        y[..., 0, :] = a + b
        y[..., 1, :] = a - b
        h *= 2
    return x


def inv_sqrt_f32(n: int) -> np.float32:
    """fp32 rounding of 1/sqrt(n) (exact for n = 64 and 256)."""
    return np.float32(1.0 / np.sqrt(np.float64(n)))


def rotate_blocks_f32(w_blocks: np.ndarray) -> np.ndarray:
    """w * Had for each length-B row block, in fp32: FWHT then one rounded scaling.

    Had = H_B / sqrt(B) is symmetric, so the row vector w Had equals (H_B w)/sqrt(B).
    """
    n = w_blocks.shape[-1]
    y = fwht_f32(w_blocks)
    return (y * inv_sqrt_f32(n)).astype(np.float32)


def had_fp64(n: int) -> np.ndarray:
    """Normalised Had = H_n / sqrt(n) in fp64 (orthogonal and symmetric)."""
    return sylvester(n).astype(np.float64) / np.sqrt(np.float64(n))
