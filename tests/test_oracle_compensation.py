"""Pins of the oracle's block compensation (Algorithm 1's block loop)."""
import numpy as np
import pytest

import synth
from oracle import compensation as C
from oracle import encoder as E
from oracle import linear as L


def _lowrank_x(m, k, seed, rank=16):
    # Correlated calibration activations: a shared low-rank part plus noise,
    # with uneven channel scales (the structure that makes compensation pay).
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((k, rank))
    ch = np.exp(0.5 * rng.standard_normal(k))
    return (rng.standard_normal((m, rank)) @ g.T * 0.9 + rng.standard_normal((m, k))) * ch


def test_hessian_is_twice_the_gram_matrix():
    x = np.random.default_rng(0).standard_normal((7, 5))
    h = C.hessian_fp64(x)
    want = np.zeros((5, 5))
    for row in x:
        want += 2.0 * np.outer(row, row)
    assert np.allclose(h, want, rtol=1e-14, atol=1e-14)


def test_inverse_cholesky_factor():
    x = _lowrank_x(300, 64, 1)
    h = C.hessian_fp64(x)
    lam = 0.01 * np.mean(np.diag(h))
    u = C.inverse_cholesky_upper(h, lam)
    assert np.array_equal(u, np.triu(u)) and np.all(np.diag(u) > 0)
    assert np.allclose(u.T @ u @ (h + lam * np.eye(64)), np.eye(64), atol=1e-9)


@pytest.mark.parametrize("levels", [2, 3])
def test_one_block_is_the_plain_encoding(levels):
    w = synth.weight_rows(1, 0, 20, 256, 0.02, True)
    u = C.inverse_cholesky_upper(C.hessian_fp64(_lowrank_x(512, 256, 2)), 1.0)
    a = C.encode_compensated(w, 2.0, levels, 256, u)
    b = E.encode(w, 2.0, levels)
    assert np.array_equal(a.codes, b.codes) and np.array_equal(a.scales, b.scales)


@pytest.mark.parametrize("levels", [2, 3])
def test_uncorrelated_hessian_changes_nothing(levels):
    # H diagonal: U is diagonal, U_QF = 0, so no block corrects another.
    w = synth.weight_rows(3, 0, 16, 768, 0.02, True)
    d = np.random.default_rng(4).uniform(0.5, 2.0, 768)
    u = C.inverse_cholesky_upper(np.diag(d), 0.0)
    a = C.encode_compensated(w, 1.5, levels, 256, u)
    assert np.array_equal(a.codes, E.encode(w, 1.5, levels).codes)


def test_block_update_is_the_obs_optimum():
    # After block 0 is fixed with error E0, the correction of the later columns
    # minimises ||[E0, -delta] X||^2 over delta: delta = E0 H_QF H_FF^-1 (from
    # the normal equations of the Hessian, not from its Cholesky factor).
    k, b = 512, 256
    x = _lowrank_x(2000, k, 5)
    h = C.hessian_fp64(x) + 5.0 * np.eye(k)
    u = C.inverse_cholesky_upper(h, 0.0)
    e0 = np.random.default_rng(6).standard_normal((3, b))
    q, f = slice(0, b), slice(b, k)
    from scipy.linalg import solve_triangular
    g = solve_triangular(u[q, q], e0.T, trans="T", lower=False).T
    via_u = g @ u[q, f]
    via_h = -e0 @ h[q, f] @ np.linalg.inv(h[f, f])
    assert np.allclose(via_u, via_h, rtol=1e-7, atol=1e-9 * np.abs(via_h).max())


def test_compensation_lowers_the_calibration_loss():
    # The point of the column updates: on correlated inputs the compensated codes fit
    # the layer output on X better than the plain ones (about 2x measured).
    w = synth.weight_rows(7, 0, 24, 768, 0.02, True)
    x = _lowrank_x(4096, 768, 8)
    h = C.hessian_fp64(x)
    u = C.inverse_cholesky_upper(h, 0.01 * np.mean(np.diag(h)))
    y = x @ w.astype(np.float64).T
    errs = []
    for r in (E.encode(w, 2.0, 3), C.encode_compensated(w, 2.0, 3, 256, u)):
        yq = x @ L.reconstruct_fp64(r.codes, r.scales, 256, r.m_up).T
        errs.append(np.linalg.norm(yq - y) / np.linalg.norm(y))
    assert errs[1] < 0.75 * errs[0], errs


def test_second_block_takes_the_normal_equation_correction():
    # Two blocks: block 0 keeps its plain codes, and block 1 is the plain
    # row-scaled encoding of W_1 + E_0 H_QF H_FF^-1 (H damped), the correction
    # computed here from the Hessian's normal equations, not from its Cholesky
    # factor.  (The two routes differ by fp64 rounding, which can move a value
    # across an fp32 rounding boundary: a tiny share of codes may differ; a
    # wrong sign, a missing U_QQ^-1 or a wrong block changes thousands.)
    n, k, b = 16, 512, 256
    w = synth.weight_rows(9, 0, n, k, 0.02, True)
    x = _lowrank_x(2000, k, 10)
    h = C.hessian_fp64(x)
    lam = 0.01 * np.mean(np.diag(h))
    u = C.inverse_cholesky_upper(h, lam)
    r = C.encode_compensated(w, 2.0, 3, b, u)
    plain = E.encode(w, 2.0, 3)
    m_up = plain.m_up
    assert np.array_equal(r.codes[:, :m_up], plain.codes[:, :m_up])
    hd = h + lam * np.eye(k)
    q, f = slice(0, b), slice(b, k)
    e0 = w[:, q].astype(np.float64) - L.reconstruct_fp64(plain.codes[:, :m_up], plain.scales, b, m_up)
    w1 = w[:, f].astype(np.float64) + e0 @ hd[q, f] @ np.linalg.inv(hd[f, f])
    want = C.encode_block_with_scale(w1.astype(np.float32), 2.0, 3, b, plain.scales)
    assert np.mean(want != r.codes[:, m_up:]) < 1e-3
    assert np.mean(want != plain.codes[:, m_up:]) > 0.05     # the correction does change codes
