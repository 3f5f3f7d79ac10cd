"""Weight encoder: Algorithm 1 without the block compensation, in fp32.

For every row r of W (N x K) and every block b of B consecutive columns
(Algorithm 1, the loop over i = 0, B, 2B, ...):

1. smoothing: v = W[r, bB:(b+1)B] * Had (Section 3.3; ``hadamard.rotate_blocks_f32``;
   Had is the Sylvester matrix, its sign-randomised form or the identity);
2. ``SDQuant`` first resamples the block to M = round(OSR * B) samples
   (Algorithm 1, ``Resample(W, n * d_col)``), evaluated here in its closed form
   as a plain sum in fp32: x_up[m] = sum_t fl(v[t] * g32[p(t, m)]), added in
   the order t = 0, 1, ..., B-1 starting from +0.0, every product and every
   partial sum rounded (no fused multiply-add);
3. the scale of row r is s_r = max |x_up| over all its blocks (one scale per
   row), with threshold theta = s_r / 2;
4. the Sigma-Delta recursion (Eq. 7-8, ``sigma_delta.scan_f32``) runs over the
   M samples of each (row, block) from a zero state, giving codes in {-1, +1}
   (binary, Eq. 4) or {-1, 0, +1} (ternary, Eq. 6);
5. codes are placed block-major: C[r, b*M + m] (Algorithm 1 writes block
   i of Q_out to columns i*osr ... (i+B)*osr).

The GPTQ-style compensation of Algorithm 1 (its column updates) is not applied: the
raw weights are encoded.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .hadamard import HAD_SYLVESTER, rotate_blocks_f32
from .resample import g_table_f32, phase_index
from .sigma_delta import scan_f32


@dataclass
class EncodeResult:
    codes: np.ndarray      # int8 (N, nb * M), values in {-1, 0, +1}
    scales: np.ndarray     # fp32 (N,)
    m_up: int              # M, samples per block after upsampling
    block: int


def m_up_for(osr: float, block: int) -> int:
    """Upsampled block length M = round(OSR * B)."""
    return int(round(float(osr) * block))


def upsample_f32(v: np.ndarray, block: int, m_up: int) -> np.ndarray:
    """Closed-form Resample(v, M) of length-B fp32 rows, in fp32, sequential over t."""
    g32 = g_table_f32(block, m_up)
    coef = g32[phase_index(block, m_up)]            # [t, m], fp32
    acc = np.zeros(v.shape[:-1] + (m_up,), dtype=np.float32)
    for t in range(block):                          # reduction index stays sequential
        prod = (v[..., t:t + 1] * coef[t]).astype(np.float32)
        acc = (acc + prod).astype(np.float32)
    return acc


def encode(w: np.ndarray, osr: float, levels: int, block: int = 256,
           hadamard: int = HAD_SYLVESTER, signs=None) -> EncodeResult:
    """Encode fp32 weights W (N x K) into Sigma-Delta codes and per-row scales.

    ``hadamard`` and ``signs`` select Had (``hadamard.rotate_blocks_f32``)."""
    w = np.asarray(w, dtype=np.float32)
    if w.ndim != 2:
        raise ValueError("W must be 2-D")
    if levels not in (2, 3):
        raise ValueError("levels must be 2 (binary) or 3 (ternary)")
    n, k = w.shape
    if block < 1 or (block & (block - 1)) or k % block:
        raise ValueError("K must be a multiple of a power-of-two block size")
    if not np.all(np.isfinite(w)):
        raise ValueError("non-finite weight")
    m_up = m_up_for(osr, block)
    if m_up < block:
        raise ValueError("OSR below 1")
    nb = k // block
    v = rotate_blocks_f32(w.reshape(n, nb, block), hadamard, signs)   # step 1
    x_up = upsample_f32(v, block, m_up)                      # step 2, (n, nb, M)
    s = np.max(np.abs(x_up).reshape(n, -1), axis=1).astype(np.float32) if n else \
        np.zeros(0, np.float32)                              # step 3
    codes = scan_f32(x_up, s[:, None], levels)               # step 4
    return EncodeResult(codes.reshape(n, nb * m_up), s, m_up, block)   # step 5


def upsampled_rows_f32(w: np.ndarray, osr: float, block: int = 256,
                       hadamard: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """Steps 1-2 only: the fp32 upsampled rotated rows (N, nb*M), for tests."""
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    m_up = m_up_for(osr, block)
    v = rotate_blocks_f32(w.reshape(n, k // block, block), hadamard, signs)
    return upsample_f32(v, block, m_up).reshape(n, -1)
