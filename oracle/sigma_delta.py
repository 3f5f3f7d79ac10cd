"""Quantizers and the first-order Sigma-Delta recursion (Section 3.1-3.2).

Eq. 4: the binary quantizer maps x >= 0 to +1 and x < 0 to -1.
Eq. 6: the ternary quantizer maps x > theta to +1, x < -theta to -1 and the
closed interval [-theta, theta] to 0.  Both outputs are multiplied by a scale
(Eq. 3, Eq. 5); here the scale is s, the row's absolute maximum after
upsampling, and theta = s / 2 (the paper's threshold is half the scale).

Eq. 7-8: the integrator i_n = i_{n-1} + x_n - y_{n-1} starts at i_0 = 0 and the
output is y_n = Q(i_n).  Writing u_n = i_n - y_n (the negated quantization
error), the recursion is v_n = u_{n-1} + x_n, y_n = Q(v_n), u_n = v_n - y_n with
u_0 = 0.  In fp32 the oracle rounds exactly two operations per step:
v = fl(u + x) and u = fl(v - c*s) (c*s is exact; for the ternary quantizer
v - s is exact as well whenever c != 0).  The listing's loop body, which sets
the integrator to the input minus the previous output without accumulating,
is read as this true integrator, as Eq. 7 and the integrator 1/(1 - z^-1) of
Fig. 1 define it.
"""
from __future__ import annotations

import numpy as np


def quant_binary(v: np.ndarray) -> np.ndarray:
    """Eq. 4: +1 where v >= 0, -1 where v < 0 (int8)."""
    return np.where(v >= 0, 1, -1).astype(np.int8)


def quant_ternary(v: np.ndarray, theta) -> np.ndarray:
    """Eq. 6: +1 where v > theta, -1 where v < -theta, 0 otherwise (int8)."""
    return np.where(v > theta, 1, np.where(v < -theta, -1, 0)).astype(np.int8)


def scan_f32(x_up: np.ndarray, s: np.ndarray, levels: int) -> np.ndarray:
    """First-order Sigma-Delta over the last axis, one independent chain per leading index.

    x_up: fp32 array (..., L); s: fp32 scale broadcastable to x_up[..., 0].
    Returns int8 codes of the same shape.  The state starts at +0.0 for every chain.
    """
    x_up = np.asarray(x_up, dtype=np.float32)
    s = np.broadcast_to(np.asarray(s, dtype=np.float32), x_up.shape[:-1])
    theta = (s * np.float32(0.5)).astype(np.float32)
    u = np.zeros(x_up.shape[:-1], dtype=np.float32)
    codes = np.empty(x_up.shape, dtype=np.int8)
    for n in range(x_up.shape[-1]):
        v = (u + x_up[..., n]).astype(np.float32)
        c = quant_ternary(v, theta) if levels == 3 else quant_binary(v)
        u = (v - c.astype(np.float32) * s).astype(np.float32)
        codes[..., n] = c
    return codes


def scan_state_f32(x_up: np.ndarray, s, levels: int):
    """Same recursion for one 1-D chain, also returning the state after every step."""
    x_up = np.asarray(x_up, dtype=np.float32)
    s = np.float32(s)
    theta = np.float32(s * np.float32(0.5))
    u = np.float32(0.0)
    codes = np.empty(x_up.shape, dtype=np.int8)
    states = np.empty(x_up.shape, dtype=np.float32)
    for n, x in enumerate(x_up):
        v = np.float32(u + x)
        if levels == 3:
            c = 1 if v > theta else (-1 if v < -theta else 0)
        else:
            c = 1 if v >= 0 else -1
        u = np.float32(v - np.float32(c) * s)
        codes[n] = c
        states[n] = u
    return codes, states
