"""Seeded inputs for the exact-arithmetic test of the block compensation.

The weights are small integers times 2^-9 (a few of them x10), and the upper
factor U has power-of-two pivots (1, 1/2, 1/4) and sparse off-diagonal
entries of +-1/8 or +-1/4.  Inside each B x B diagonal block the off-diagonal
entries sit only in rows of the block's first half and columns of its second
half, so the block's strictly upper part N satisfies N D^-1 N = 0 and
U_QQ^-1 = D^-1 - D^-1 N D^-1 holds exactly (D the pivots).  With OSR 1 the
resampling is the identity and Had = H_B / 16 has entries +-1/16, so every
value the block loop forms is a dyadic rational of a few dozen bits: fp64
carries the loop without rounding whatever the summation order (the CPU test
of the oracle certifies this step by step), and the compensated codes must
then agree bit for bit on every row.

This module only draws inputs; it holds none of the method's arithmetic.
"""
from __future__ import annotations

import numpy as np


def dyadic_case(n: int, k: int, block: int, seed: int, density: float = 0.03):
    """(w fp32 [n, k], u fp64 [k, k] upper triangular) as described above."""
    rng = np.random.default_rng(seed)
    w = rng.integers(-200, 201, size=(n, k)).astype(np.float64)
    w *= np.where(rng.random((n, k)) < 0.005, 10.0, 1.0)
    w = (w * 2.0 ** -9).astype(np.float32)
    u = np.zeros((k, k))
    np.fill_diagonal(u, 2.0 ** -rng.integers(0, 3, size=k).astype(np.float64))
    val = lambda size: rng.choice([-2.0, -1.0, 1.0, 2.0], size=size) * 2.0 ** -3
    half = block // 2
    for b in range(k // block):
        q0 = b * block
        # first half rows x second half columns of the diagonal block
        m = rng.random((half, half)) < density
        u[q0:q0 + half, q0 + half:q0 + block] = np.where(m, val((half, half)), 0.0)
        # the block's rows x every later column
        f0 = q0 + block
        if f0 < k:
            m = rng.random((block, k - f0)) < density
            u[q0:q0 + block, f0:] = np.where(m, val((block, k - f0)), 0.0)
    return w, u
