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


@pytest.mark.parametrize("update", [C.COMP_GPTQ, C.COMP_JOINT])
def test_compensation_lowers_the_calibration_loss(update):
    # The point of the column updates: on correlated inputs the compensated codes fit
    # the layer output on X better than the plain ones (about 2x measured).
    w = synth.weight_rows(7, 0, 24, 768, 0.02, True)
    x = _lowrank_x(4096, 768, 8)
    h = C.hessian_fp64(x)
    u = C.inverse_cholesky_upper(h, 0.01 * np.mean(np.diag(h)))
    y = x @ w.astype(np.float64).T
    errs = []
    for r in (E.encode(w, 2.0, 3), C.encode_compensated(w, 2.0, 3, 256, u, update=update)):
        yq = x @ L.reconstruct_fp64(r.codes, r.scales, 256, r.m_up).T
        errs.append(np.linalg.norm(yq - y) / np.linalg.norm(y))
    assert errs[1] < 0.75 * errs[0], errs


def test_second_block_takes_the_normal_equation_correction():
    # Joint update.  Two blocks: block 0 keeps its plain codes, and block 1 is the plain
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
    r = C.encode_compensated(w, 2.0, 3, b, u, update=C.COMP_JOINT)
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


def _two_block_normal_equation_codes(w, h, b, plain):
    """Block 1's codes as the plain row-scaled encoding of W_1 + E_0 H_QF H_FF^-1,
    the correction taken from the normal equations of the (damped) Hessian h."""
    m_up = plain.m_up
    q, f = slice(0, b), slice(b, w.shape[1])
    e0 = w[:, q].astype(np.float64) - L.reconstruct_fp64(plain.codes[:, :m_up], plain.scales, b, m_up)
    w1 = w[:, f].astype(np.float64) + e0 @ h[q, f] @ np.linalg.inv(h[f, f])
    return C.encode_block_with_scale(w1.astype(np.float32), 2.0, 3, b, plain.scales)


def test_gptq_update_is_the_normal_equation_correction_for_diagonal_pivot_blocks():
    # GPTQ's block step divides each column's error by its pivot.  Where the
    # factor's diagonal block U_QQ is diagonal (with unequal pivots), that is
    # the whole-block optimum, so block 1 must be the plain encoding of
    # W_1 + E_0 H_QF H_FF^-1 with H = (U^T U)^-1 from the normal equations.
    # A missing division, a wrong sign or the wrong block of U fails it.
    n, k, b = 16, 512, 256
    rng = np.random.default_rng(12)
    u = np.triu(rng.standard_normal((k, k))) * 0.05
    u[:b, :b] = np.diag(rng.uniform(0.3, 3.0, b))
    u[b:, b:] += np.diag(rng.uniform(0.5, 2.0, k - b))
    h = np.linalg.inv(u.T @ u)
    w = synth.weight_rows(13, 0, n, k, 0.02, True)
    r = C.encode_compensated(w, 2.0, 3, b, u, update=C.COMP_GPTQ)
    plain = E.encode(w, 2.0, 3)
    assert np.array_equal(r.codes[:, :plain.m_up], plain.codes[:, :plain.m_up])
    want = _two_block_normal_equation_codes(w, h, b, plain)
    assert np.mean(want != r.codes[:, plain.m_up:]) < 1e-3
    assert np.mean(want != plain.codes[:, plain.m_up:]) > 0.05
    # with a diagonal U_QQ the joint update is the same correction
    j = C.encode_compensated(w, 2.0, 3, b, u, update=C.COMP_JOINT)
    assert np.mean(j.codes != r.codes) < 1e-3


def test_gptq_and_joint_updates_differ_on_a_full_factor():
    w = synth.weight_rows(14, 0, 16, 768, 0.02, True)
    h = C.hessian_fp64(_lowrank_x(3000, 768, 15))
    u = C.inverse_cholesky_upper(h, 0.01 * np.mean(np.diag(h)))
    a = C.encode_compensated(w, 2.0, 3, 256, u, update=C.COMP_GPTQ)
    j = C.encode_compensated(w, 2.0, 3, 256, u, update=C.COMP_JOINT)
    assert np.array_equal(a.codes[:, :512], j.codes[:, :512])        # block 0 is never corrected
    assert np.mean(a.codes != j.codes) > 0.01


def _gran_exp(x):
    """Exponent of the lowest set bit of each fp64 value (+inf for zeros)."""
    x = np.asarray(x, np.float64)
    f, e = np.frexp(np.abs(x))
    mant = np.ldexp(f, 53).astype(np.int64)
    low = mant & -mant
    with np.errstate(divide="ignore"):
        out = e.astype(np.float64) - 53.0 + np.log2(np.where(mant > 0, low, 1).astype(np.float64))
    return np.where(x == 0, np.inf, out)


def _certify_dot(base, a, bmat):
    """base + a @ bmat is exact in fp64 for every summation order: the sum of
    |terms| over the common granularity of the terms stays below 2^52."""
    mag = np.abs(base) + np.abs(a) @ np.abs(bmat)
    ga, gb, g0 = _gran_exp(a), _gran_exp(bmat), _gran_exp(base)
    gmin = np.array(g0, dtype=np.float64, copy=True)
    for r in range(a.shape[0]):
        gmin[r] = np.minimum(gmin[r], np.min(ga[r][:, None] + gb, axis=0))
    with np.errstate(divide="ignore", invalid="ignore"):
        bits = np.where(mag > 0, np.log2(mag) - gmin, 0.0)
    assert np.all(bits < 52), float(np.max(bits))


@pytest.mark.parametrize("update", [C.COMP_GPTQ, C.COMP_JOINT])
@pytest.mark.parametrize("levels", [2, 3])
def test_dyadic_inputs_keep_the_block_loop_exact(update, levels):
    # The inputs of the device's exact-arithmetic parity test: every fp64 step
    # of the block loop (reconstruction, error, division by the pivots or the
    # triangular solve -- and the device's product with U_QQ^-1 --, the update
    # of the later columns) is certified free of rounding, so any summation
    # order gives the same values; the loop run here step by step gives the
    # oracle's codes.
    from scipy.linalg import solve_triangular
    from oracle.hadamard import had_fp64
    from tests.dyadic_inputs import dyadic_case
    n, k, b = 70, 1024, 256
    w, u = dyadic_case(n, k, b, seed=3 + levels)
    d = np.diag(u)
    assert np.all(np.log2(d) == np.round(np.log2(d)))
    r = C.encode_compensated(w, 1.0, levels, b, u, update=update)
    s = r.scales
    had = had_fp64(b)
    w64 = w.astype(np.float64)
    codes = []
    for blk in range(k // b):
        q, f = slice(blk * b, (blk + 1) * b), slice((blk + 1) * b, k)
        cb = C.encode_block_with_scale(w64[:, q].astype(np.float32), 1.0, levels, b, s)
        codes.append(cb)
        if blk == k // b - 1:
            break
        y = cb.astype(np.float64) * s.astype(np.float64)[:, None]
        _certify_dot(np.zeros((n, b)), y, had.T)                      # Resample(Y, B) Had^T, M = B
        q_hat = L.reconstruct_fp64(cb, s, b, b)
        assert np.array_equal(q_hat, y @ had.T)
        _certify_dot(w64[:, q], -q_hat, np.eye(b))                    # E = W_Q - Q_hat
        e = w64[:, q] - q_hat
        uqq = u[q, q]
        if update == C.COMP_GPTQ:
            g = e / np.diag(uqq)[None, :]
        else:
            g = solve_triangular(uqq, e.T, trans="T", lower=False).T
            strict = np.triu(uqq, 1)
            _certify_dot(e, -g, strict)                               # forward substitution
            dq = np.diag(1.0 / np.diag(uqq))
            v = dq - dq @ strict @ dq                                  # U_QQ^-1 exactly (N D^-1 N = 0)
            assert np.array_equal(v @ uqq, np.eye(b))
            _certify_dot(np.zeros((n, b)), e, v)                       # the device's E U_QQ^-1
            assert np.array_equal(g, e @ v)
        _certify_dot(w64[:, f], -g, u[q, f])                          # W_F -= G U_QF
        w64[:, f] -= g @ u[q, f]
    assert np.array_equal(np.concatenate(codes, axis=1), r.codes)
