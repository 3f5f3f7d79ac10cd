"""Pins of the oracle's fp64 linear (Algorithm 1's reconstruction, Fig. 5)."""
import numpy as np
import pytest
from scipy import signal
import scipy.linalg

from oracle import encoder as E
from oracle import linear as L


def _codes(n, k, osr, levels, seed):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    return w, E.encode(w, osr, levels)


@pytest.mark.parametrize("osr,levels", [(1.5, 2), (2.0, 3), (2.5, 3), (1.0, 3)])
def test_expansion_identity(osr, levels):
    # y via x_tilde = (x Had) D^T against the plain definition x W_hat^T.
    w, r = _codes(24, 512, osr, levels, 1)
    x = np.random.default_rng(2).standard_normal((5, 512))
    y1 = L.linear_fp64(x, r.codes, r.scales, 256, r.m_up)
    y2 = L.linear_via_expansion_fp64(x, r.codes, r.scales, 256, r.m_up)
    assert np.max(np.abs(y1 - y2)) <= 1e-12 * np.max(np.abs(y1))


@pytest.mark.parametrize("block,m_up", [(4, 6), (4, 8), (8, 12), (8, 13)])
def test_tiny_reconstruction_against_library_routines(block, m_up):
    # Brute force on tiny shapes: each block is scipy's FFT resample of the
    # scaled codes, then multiplied by the normalised Hadamard matrix.
    rng = np.random.default_rng(block * m_up)
    n, nb = 3, 2
    codes = rng.integers(-1, 2, size=(n, nb * m_up)).astype(np.int8)
    scales = rng.uniform(0.1, 1.0, size=n).astype(np.float32)
    had = scipy.linalg.hadamard(block) / np.sqrt(block)
    want = np.zeros((n, nb * block))
    for r in range(n):
        for b in range(nb):
            z = signal.resample(codes[r, b * m_up:(b + 1) * m_up] * float(scales[r]), block)
            want[r, b * block:(b + 1) * block] = z @ had.T
    got = L.reconstruct_fp64(codes, scales, block, m_up)
    assert np.max(np.abs(got - want)) < 1e-12
    x = rng.standard_normal((2, nb * block))
    assert np.max(np.abs(L.linear_fp64(x, codes, scales, block, m_up) - x @ want.T)) < 1e-12
    assert np.max(np.abs(L.linear_via_expansion_fp64(x, codes, scales, block, m_up) - x @ want.T)) < 1e-12


def test_exact_weights_reproduce_exactly():
    # A row whose rotated blocks are constant is encoded without error
    # (all codes +1), so the linear reproduces x w^T.
    w = np.zeros((2, 512), np.float32)
    w[0, 0] = 0.32
    w[1, 256] = -0.16
    r = E.encode(w, 2.0, 3)
    x = np.random.default_rng(0).standard_normal((3, 512))
    y = L.linear_fp64(x, r.codes, r.scales, 256, r.m_up)
    assert np.max(np.abs(y - x @ w.astype(np.float64).T)) < 1e-6


def test_quantized_linear_approaches_dense_with_osr():
    w, _ = _codes(64, 512, 1.0, 3, 9)
    x = np.random.default_rng(4).standard_normal((4, 512))
    ref = x @ w.astype(np.float64).T
    errs = []
    for osr in (1.0, 2.0, 4.0):
        r = E.encode(w, osr, 3)
        errs.append(np.max(L.rel_err_rows(L.linear_fp64(x, r.codes, r.scales, 256, r.m_up), ref)))
    assert errs[0] > errs[1] > errs[2]


def test_rel_err_metric():
    y = np.array([[1.0, -2.0], [0.0, 0.0]])
    assert np.allclose(L.rel_err_rows(y + [[0.0, 0.002], [0.0, 0.0]], y), [0.001, 0.0])


@pytest.mark.parametrize("mode", [0, 2])
@pytest.mark.parametrize("osr,levels", [(1.5, 2), (2.125, 3)])
def test_expansion_identity_for_every_had(mode, osr, levels):
    # x_tilde = (x Had) D^T against x W_hat^T for Had = I and the signed Had.
    import synth
    s = synth.hadamard_signs(9, 256) if mode == 2 else None
    rng = np.random.default_rng(3)
    w = (rng.standard_normal((20, 512)) * 0.02).astype(np.float32)
    r = E.encode(w, osr, levels, 256, mode, s)
    x = rng.standard_normal((4, 512))
    y1 = L.linear_fp64(x, r.codes, r.scales, 256, r.m_up, mode, s)
    y2 = L.linear_via_expansion_fp64(x, r.codes, r.scales, 256, r.m_up, mode, s)
    assert np.max(np.abs(y1 - y2)) <= 1e-12 * np.max(np.abs(y1))


def test_tiny_signed_reconstruction_against_library_routines():
    # Brute force as above with Had = diag(s) H / sqrt(B): each block is
    # scipy's resample of the scaled codes times Had^T = H / sqrt(B) diag(s).
    block, m_up, n, nb = 8, 12, 3, 2
    rng = np.random.default_rng(8)
    s = np.array([1, -1, -1, 1, 1, 1, -1, 1])
    codes = rng.integers(-1, 2, size=(n, nb * m_up)).astype(np.int8)
    scales = rng.uniform(0.1, 1.0, size=n).astype(np.float32)
    had = np.diag(s) @ scipy.linalg.hadamard(block) / np.sqrt(block)
    want = np.zeros((n, nb * block))
    for r in range(n):
        for b in range(nb):
            z = signal.resample(codes[r, b * m_up:(b + 1) * m_up] * float(scales[r]), block)
            want[r, b * block:(b + 1) * block] = z @ had.T
    got = L.reconstruct_fp64(codes, scales, block, m_up, 2, s)
    assert np.max(np.abs(got - want)) < 1e-12


def test_hadamard_smoothing_lowers_error_on_outlier_weights():
    # The direction of the ablation (Table 2, Section 3.3): on weights with
    # sparse large outliers, the rotated encodings reconstruct the layer better
    # than the unrotated one, with either Had.
    import synth
    w = synth.weight_rows(2510, 0, 48, 1024, 0.02, True)
    x = synth.activations_f32(2510, 0, 16, 1024).astype(np.float64)
    y = x @ w.astype(np.float64).T
    s = synth.hadamard_signs(2510, 256)
    err = {}
    for mode in (0, 1, 2):
        r = E.encode(w, 2.0, 3, 256, mode, s if mode == 2 else None)
        yq = L.linear_fp64(x, r.codes, r.scales, 256, r.m_up, mode, s if mode == 2 else None)
        err[mode] = np.linalg.norm(yq - y) / np.linalg.norm(y)
    assert err[1] < 0.8 * err[0] and err[2] < 0.8 * err[0], err
