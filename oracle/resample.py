"""The ``Resample`` function of Algorithm 1 and its matrix forms.

Algorithm 1 resamples each row with an FFT: transform, zero-pad (upsampling)
or truncate (downsampling) the spectrum to the new length, weight the bin at
half the original length by 1/2 when upsampling or by 2 when downsampling,
inverse transform, and scale by N_new / d_col.

Reading taken here (the listing leaves the padding position and the Nyquist
index implicit): the spectrum is kept one-sided (real FFT), padded or cut at
its high-frequency end, and the weighted bin is the Nyquist bin of the
*shorter* of the two lengths, when that length is even.  With a one-sided
spectrum, halving that bin on upsampling splits the Nyquist component evenly
between its two mirror frequencies, and doubling it on downsampling folds both
mirror bins into one; the result is real and Resample(Resample(v, M), B) = v.

Closed forms (derived from the band-limited periodic interpolation that these
steps implement, pinned against the FFT form in the tests):

* upsampling B -> M: out[m] = sum_t v[t] * g(p), p = (m*B - t*M) mod (B*M),
  g = 1 at p = 0, g = 0 at other multiples of M, otherwise
  g = sin(pi*tau) / (B * tan(pi*tau/B)) with tau = p / M;
* downsampling M -> B: out[t] = sum_m y[m] * D[m, t] with
  D[m, t] = (sin(pi*tau) * cot(pi*tau/B) + cos(pi*tau)) / M,
  tau = (m*B - t*M) / M, whose value at an integer tau = k is
  (B * [k = 0 mod B] + (-1)**k) / M.  This holds for M > B; at M = B no bin
  is cut or folded and D is the identity.
"""
from __future__ import annotations

import math

import numpy as np


def resample_fft(w: np.ndarray, n_new: int) -> np.ndarray:
    """Algorithm 1 ``Resample(W, N_new)`` along the last axis, fp64.

    At N_new = d_col no bin is padded, cut or weighted and the scale is 1, so
    the steps compose to IFFT(FFT(w)) = w: the block is returned as it is
    (exactly, without the round trip's fp64 rounding)."""
    w = np.asarray(w, dtype=np.float64)
    d = w.shape[-1]
    if n_new == d:
        return w.copy()
    x = np.fft.rfft(w, axis=-1)                       # FFT(w), one-sided
    y = np.zeros(w.shape[:-1] + (n_new // 2 + 1,), dtype=np.complex128)
    keep = min(d, n_new) // 2 + 1                     # ZeroPadOrTruncate
    y[..., :keep] = x[..., :keep]
    short = min(d, n_new)
    if n_new != d and short % 2 == 0:
        nyq = short // 2
        if n_new > d:
            y[..., nyq] *= 0.5                        # upsample: split Nyquist
        else:
            y[..., nyq] *= 2.0                        # downsample: fold mirrors
    out = np.fft.irfft(y, n=n_new, axis=-1)           # IFFT(Y)
    return out * (n_new / d)                          # scale by N_new / d_col


def _g_value(p: int, block: int, m_up: int) -> float:
    if p == 0:
        return 1.0
    if p % m_up == 0:
        return 0.0
    tau = p / m_up
    return math.sin(math.pi * tau) / (block * math.tan(math.pi * tau / block))


def g_table_fp64(block: int, m_up: int) -> np.ndarray:
    """Interpolation kernel g(p) for p in [0, B*M), fp64."""
    return np.array([_g_value(p, block, m_up) for p in range(block * m_up)], dtype=np.float64)


def g_table_f32(block: int, m_up: int) -> np.ndarray:
    """The same kernel rounded once to fp32: the coefficients the fp32 encoder uses."""
    return g_table_fp64(block, m_up).astype(np.float32)


def phase_index(block: int, m_up: int) -> np.ndarray:
    """p(t, m) = (m*B - t*M) mod (B*M) as an int64 matrix indexed [t, m]."""
    t = np.arange(block, dtype=np.int64)[:, None]
    m = np.arange(m_up, dtype=np.int64)[None, :]
    return (m * block - t * m_up) % (block * m_up)


def up_matrix_fp64(block: int, m_up: int) -> np.ndarray:
    """U[t, m] with Resample(v, M) = v @ U (closed form)."""
    return g_table_fp64(block, m_up)[phase_index(block, m_up)]


def down_matrix_fp64(block: int, m_up: int) -> np.ndarray:
    """D[m, t] with Resample(y, B) = y @ D (closed form), y of length M."""
    if m_up == block:
        return np.eye(block)
    d = np.empty((m_up, block), dtype=np.float64)
    for m in range(m_up):
        for t in range(block):
            num = m * block - t * m_up
            if num % m_up == 0:
                k = num // m_up
                val = (block if k % block == 0 else 0) + (1 if k % 2 == 0 else -1)
            else:
                tau = num / m_up
                val = (math.sin(math.pi * tau) / math.tan(math.pi * tau / block)
                       + math.cos(math.pi * tau))
            d[m, t] = val / m_up
    return d
