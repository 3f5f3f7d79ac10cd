"""Hadamard matrices and the block transform used for weight smoothing.

Section 3.3 defines a Hadamard matrix by H H^T = n I and builds it with the
Sylvester recursion H_2k = [[H_k, H_k], [H_k, -H_k]] (Eq. 13).  Algorithm 1
multiplies each B-column weight block by ``Had`` before Sigma-Delta
quantization and by ``Had^T`` afterwards, so ``Had`` must be orthogonal.
Three choices of ``Had`` (one B x B matrix shared by every block, as
Algorithm 1's input list has it):

* HAD_SYLVESTER: the normalised Sylvester matrix Had = H_B / sqrt(B);
* HAD_SIGNED: Algorithm 1 calls its input a *random* Hadamard matrix without
  saying how it is randomised; read here as Had = diag(s) H_B / sqrt(B) with
  a vector s of B signs (+-1) drawn by the caller, which keeps Had orthogonal
  and makes w Had the transform of the sign-flipped block w * s;
* HAD_NONE: Had = I, the "without Hadamard" rows of the ablation (Table 2).
"""
from __future__ import annotations

import numpy as np

HAD_NONE, HAD_SYLVESTER, HAD_SIGNED = 0, 1, 2


def check_mode(mode: int, signs, block: int) -> np.ndarray | None:
    """Validate (mode, signs) for blocks of length ``block``; returns the signs as int8."""
    if mode not in (HAD_NONE, HAD_SYLVESTER, HAD_SIGNED):
        raise ValueError("hadamard mode must be 0 (none), 1 (Sylvester) or 2 (signed)")
    if mode != HAD_SIGNED:
        return None
    s = np.asarray(signs)
    if s.shape != (block,) or not np.all((s == 1) | (s == -1)):
        raise ValueError("signed Hadamard needs `block` signs in {-1, +1}")
    return s.astype(np.int8)


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


def rotate_blocks_f32(w_blocks: np.ndarray, mode: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """w * Had for each length-B row block, in fp32.

    Sylvester: Had = H_B / sqrt(B) is symmetric, so the row vector w Had equals
    (H_B w) / sqrt(B): FWHT then one rounded scaling.  Signed: w diag(s) is
    w with the signs of its entries flipped where s = -1 (exact), then as
    Sylvester.  None: w unchanged.
    """
    n = w_blocks.shape[-1]
    s = check_mode(mode, signs, n)
    if mode == HAD_NONE:
        return np.array(w_blocks, dtype=np.float32, copy=True)
    x = np.asarray(w_blocks, dtype=np.float32)
    if mode == HAD_SIGNED:
        x = np.where(s < 0, -x, x).astype(np.float32)
    y = fwht_f32(x)
    return (y * inv_sqrt_f32(n)).astype(np.float32)


def had_fp64(n: int, mode: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """Had in fp64 (orthogonal): H_n / sqrt(n), diag(s) H_n / sqrt(n) or I."""
    s = check_mode(mode, signs, n)
    if mode == HAD_NONE:
        return np.eye(n)
    h = sylvester(n).astype(np.float64) / np.sqrt(np.float64(n))
    if mode == HAD_SIGNED:
        h = s.astype(np.float64)[:, None] * h
    return h
