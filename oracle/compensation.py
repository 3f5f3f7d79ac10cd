"""Block compensation of Algorithm 1 (the GPTQ-style loop), fp64 with fp32 codes.

Algorithm 1 takes the inverse Hessian H^-1 = (2 X X^T + lambda I)^-1 of the
layer's calibration inputs X, replaces it by its upper Cholesky factor U
(H^-1 = U^T U), and walks the weight in blocks of B columns: the
block is quantized (Had, SDQuant, Had^T), its error E is
formed, and the columns after it are corrected so that the layer output on
X loses as little as possible.

Readings:

* the update.  The text keeps GPTQ's block-wise compensation and drops its
  column-wise one (Section 3.5), and the listing prepares the factor exactly
  as GPTQ does (U = Cholesky(H^-1)^T).  GPTQ's block-wise step divides each
  column's error by that column's diagonal entry of U before propagating it
  past the block; the printed correction W_F -= E U[Q, F] (Q the block's
  columns, F the later ones) writes the error without that division.  The
  default update here is GPTQ's block step with the column-wise part removed:
  W_F -= E diag(U_QQ)^-1 U_QF (``COMP_GPTQ``).  Because SDQ quantizes the
  block's columns jointly, the optional ``COMP_JOINT`` applies the
  optimal-brain-surgeon correction of the whole block instead,
  W_F -= E U_QQ^-1 U_QF, which minimises ||(W - W_hat) X|| over W_F; the two
  agree whenever U_QQ is diagonal.
* the row scale.  The stored format has one scale per row; it is taken from
  the uncompensated W (the scale the plain encoder would use), and every block
  of the row is scanned with it.
* precision.  W is carried in fp64 and every compensation step runs in fp64;
  a block is rounded to fp32 once, when it is handed to the (bit-exact fp32)
  block encoder.

Functions:

* ``hessian_fp64``            -- 2 X^T X for calibration rows X (m x K);
* ``inverse_cholesky_upper``  -- U with U^T U = (H + lambda I)^-1, upper (numpy
                                 inverse and Cholesky as library steps);
* ``encode_block_with_scale`` -- Had, Resample up and the Sigma-Delta scan of
                                 one block column with a given row scale;
* ``encode_compensated``      -- the loop.
"""
from __future__ import annotations

import numpy as np
from scipy.linalg import solve_triangular

from .encoder import EncodeResult, encode, m_up_for, upsample_f32
from .hadamard import HAD_SYLVESTER, rotate_blocks_f32
from .linear import reconstruct_fp64
from .sigma_delta import scan_f32

COMP_GPTQ, COMP_JOINT = 0, 1      # the block update (see the module docstring)


def hessian_fp64(x: np.ndarray) -> np.ndarray:
    """H = 2 X^T X (K x K) for calibration activations X (m x K), fp64."""
    x = np.asarray(x, dtype=np.float64)
    return 2.0 * (x.T @ x)


def inverse_cholesky_upper(h: np.ndarray, lam: float) -> np.ndarray:
    """Algorithm 1, factor step: U = Cholesky((H + lambda I)^-1)^T, so U^T U = (H + lambda I)^-1."""
    h = np.asarray(h, dtype=np.float64)
    hinv = np.linalg.inv(h + lam * np.eye(h.shape[0]))
    hinv = 0.5 * (hinv + hinv.T)
    return np.ascontiguousarray(np.linalg.cholesky(hinv).T)


def encode_block_with_scale(wb: np.ndarray, osr: float, levels: int, block: int, s: np.ndarray,
                            hadamard: int = HAD_SYLVESTER, signs=None) -> np.ndarray:
    """Codes (n x M) of one fp32 block column (n x B) scanned with row scales s."""
    wb = np.asarray(wb, dtype=np.float32)
    v = rotate_blocks_f32(wb[:, None, :], hadamard, signs)
    x_up = upsample_f32(v, block, m_up_for(osr, block))
    return scan_f32(x_up, np.asarray(s, np.float32)[:, None], levels).reshape(wb.shape[0], -1)


def encode_compensated(w: np.ndarray, osr: float, levels: int, block: int, u: np.ndarray,
                       hadamard: int = HAD_SYLVESTER, signs=None,
                       update: int = COMP_GPTQ) -> EncodeResult:
    """Algorithm 1 with its block compensation: codes and row scales of W (n x K).

    ``update`` selects the correction of the columns after each block:
    ``COMP_GPTQ`` (E diag(U_QQ)^-1 U_QF) or ``COMP_JOINT`` (E U_QQ^-1 U_QF)."""
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    if u.shape != (k, k):
        raise ValueError("U must be K x K")
    if update not in (COMP_GPTQ, COMP_JOINT):
        raise ValueError("update must be COMP_GPTQ or COMP_JOINT")
    plain = encode(w, osr, levels, block, hadamard, signs)     # row scales of the raw W
    s = plain.scales
    m_up = plain.m_up
    nb = k // block
    w64 = w.astype(np.float64)
    codes = np.empty((n, nb * m_up), dtype=np.int8)
    for b in range(nb):
        q, f = slice(b * block, (b + 1) * block), slice((b + 1) * block, k)
        cb = encode_block_with_scale(w64[:, q].astype(np.float32), osr, levels, block, s,
                                     hadamard, signs)
        codes[:, b * m_up:(b + 1) * m_up] = cb
        if b == nb - 1:
            break
        q_hat = reconstruct_fp64(cb, s, block, m_up, hadamard, signs)   # Resample(Y, B) Had^T
        e = w64[:, q] - q_hat
        if update == COMP_GPTQ:
            g = e / np.diag(u[q, q])[None, :]          # each column's error over its pivot
        else:
            # G = E U_QQ^-1, i.e. U_QQ^T G^T = E^T (lower-triangular system)
            g = solve_triangular(u[q, q], e.T, trans="T", lower=False).T
        w64[:, f] -= g @ u[q, f]
    return EncodeResult(codes, s, m_up, block)
