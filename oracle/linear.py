"""The dequantized linear layer in fp64.

Plain definition.  Algorithm 1 defines the dequantized block as
Q[:, block b] = Resample(Y_b, B) * Had^T, where Y_b are the block's
Sigma-Delta outputs (codes times the row scale) and ``Resample`` brings the M
upsampled samples back to B.  The layer output is the plain product
y = x * W_hat^T with W_hat the concatenation of these blocks
(``reconstruct_fp64`` then ``linear_fp64``).

Expansion identity.  Fig. 5 has the activations brought to the upsampled
length so that they meet the codes directly.  The exact way to do so is the
transpose of the decimation: with D the M x B matrix of Resample(., B)
(y @ D = Resample(y, B) for a row vector y), row r's block is
w_hat_b = (s_r c_b) D Had^T, so x_b . w_hat_b = s_r (x_b Had D^T) . c_b.
Hence x_tilde_b = (x_b Had) D^T and y_r = s_r * sum_j C[r, j] * x_tilde[j]
(``expand_activations_fp64``, ``linear_via_expansion_fp64``).  By Parseval's
identity (Eq. 12) this inner product sees the codes only through the band the
activations occupy, which is where Sigma-Delta pushes little noise.  Note this
D^T is not the upsampler used for the weights: it equals (B/M) U plus a
Nyquist term (tested).
"""
from __future__ import annotations

import numpy as np

from .hadamard import HAD_SYLVESTER, had_fp64
from .resample import resample_fft, down_matrix_fp64


def reconstruct_fp64(codes: np.ndarray, scales: np.ndarray, block: int, m_up: int,
                     hadamard: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """W_hat (N x K) in fp64 from int8 codes (N x nb*M) and fp32 row scales."""
    codes = np.asarray(codes)
    n = codes.shape[0]
    nb = codes.shape[1] // m_up
    y = codes.astype(np.float64).reshape(n, nb, m_up) * np.asarray(scales, np.float64)[:, None, None]
    z = resample_fft(y, block)                       # Resample(Y, d_col), (n, nb, B)
    q = z @ had_fp64(block, hadamard, signs).T       # * Had^T
    return q.reshape(n, nb * block)


def linear_fp64(x: np.ndarray, codes: np.ndarray, scales: np.ndarray, block: int,
                m_up: int, hadamard: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """y = x W_hat^T in fp64; x (m x K) in any float type (converted exactly)."""
    w_hat = reconstruct_fp64(codes, scales, block, m_up, hadamard, signs)
    return np.asarray(x, dtype=np.float64) @ w_hat.T


def expand_activations_fp64(x: np.ndarray, block: int, m_up: int,
                            hadamard: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """x_tilde (m x nb*M): per block, (x_b Had) D^T, fp64."""
    x = np.asarray(x, dtype=np.float64)
    m, k = x.shape
    nb = k // block
    h = x.reshape(m, nb, block) @ had_fp64(block, hadamard, signs)   # x_b Had
    d = down_matrix_fp64(block, m_up)                # (M, B)
    return (h @ d.T).reshape(m, nb * m_up)


def linear_via_expansion_fp64(x: np.ndarray, codes: np.ndarray, scales: np.ndarray,
                              block: int, m_up: int, hadamard: int = HAD_SYLVESTER,
                              signs=None) -> np.ndarray:
    """y[i, r] = s_r * sum_j C[r, j] x_tilde[i, j], fp64."""
    xt = expand_activations_fp64(x, block, m_up, hadamard, signs)
    return (xt @ np.asarray(codes, np.float64).T) * np.asarray(scales, np.float64)[None, :]


def rel_err_rows(y: np.ndarray, y_ref: np.ndarray) -> np.ndarray:
    """Per activation row: max_r |y - y_ref| / max_r |y_ref| (the parity metric)."""
    y = np.asarray(y, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    den = np.max(np.abs(y_ref), axis=1)
    num = np.max(np.abs(y - y_ref), axis=1)
    return num / np.where(den > 0, den, 1.0)
