"""Pins of the oracle's Hadamard smoothing (Section 3.3, Eq. 13) to mathematics
and to an independent library routine."""
import numpy as np
import pytest
import scipy.linalg

from oracle import hadamard as H


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 32, 64, 128, 256])
def test_hht_is_n_identity(n):
    # Section 3.3: H H^T = n I.
    h = H.sylvester(n)
    assert np.array_equal(h @ h.T, n * np.eye(n, dtype=np.int64))
    assert set(np.unique(h)) <= {-1, 1}


@pytest.mark.parametrize("n", [2, 8, 64, 256])
def test_sylvester_closed_form(n):
    # Sylvester's matrix has entries (-1)^popcount(i & j).
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    pc = np.vectorize(lambda a: bin(a).count("1"))(i & j)
    assert np.array_equal(H.sylvester(n), np.where(pc % 2 == 0, 1, -1))


@pytest.mark.parametrize("n", [1, 4, 32, 256])
def test_matches_scipy_hadamard(n):
    assert np.array_equal(H.sylvester(n), scipy.linalg.hadamard(n))


@pytest.mark.parametrize("n", [2, 16, 256])
def test_fwht_exact_on_integers(n):
    rng = np.random.default_rng(n)
    x = rng.integers(-1000, 1000, size=(5, n))
    got = H.fwht_f32(x.astype(np.float32))
    want = x @ H.sylvester(n).T
    # integers below 2^24 in magnitude are exact in fp32 at every stage
    assert np.array_equal(got.astype(np.int64), want)


def test_rotation_orthonormal_round_trip():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 256)).astype(np.float32)
    y = H.rotate_blocks_f32(x)
    back = H.rotate_blocks_f32(y)
    assert np.max(np.abs(back - x)) < 1e-5
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-5)


def test_rotation_scale_is_exact_for_256():
    # 1/sqrt(256) = 1/16 is exact, so rotating H_256-transformable integers is exact.
    x = np.zeros((1, 256), np.float32)
    x[0, 0] = 16.0
    y = H.rotate_blocks_f32(x)
    assert np.all(y == 1.0)


def test_outlier_smoothing():
    # Fig. 3's observation in miniature: the rotation spreads an outlier,
    # lowering the peak-to-rms ratio of a block.
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((32, 256)) * 0.02).astype(np.float32)
    x[:, 17] = 1.0
    y = H.rotate_blocks_f32(x)
    crest = lambda a: np.max(np.abs(a), axis=1) / np.sqrt(np.mean(a.astype(np.float64) ** 2, axis=1))
    assert np.all(crest(y) < 0.5 * crest(x))


# --- choices of Had: Sylvester, sign-randomised diag(s) H / sqrt(B), none ---

def test_signed_had_worked_example_n4():
    # diag(s) H_4 / 2 with s = (+1, -1, +1, +1), written out by hand.
    want = np.array([[1, 1, 1, 1],
                     [-1, 1, -1, 1],
                     [1, 1, -1, -1],
                     [1, -1, -1, 1]], dtype=np.float64) / 2.0
    got = H.had_fp64(4, H.HAD_SIGNED, np.array([1, -1, 1, 1]))
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", [H.HAD_NONE, H.HAD_SYLVESTER, H.HAD_SIGNED])
@pytest.mark.parametrize("n", [4, 64, 256])
def test_every_had_is_orthogonal(mode, n):
    s = np.where(np.random.default_rng(n).random(n) < 0.5, -1, 1)
    h = H.had_fp64(n, mode, s if mode == H.HAD_SIGNED else None)
    assert np.max(np.abs(h @ h.T - np.eye(n))) < 1e-13


@pytest.mark.parametrize("n", [64, 256])
def test_signed_rotation_matches_library_hadamard(n):
    # w Had for Had = diag(s) H / sqrt(n), against scipy's Hadamard in fp64.
    rng = np.random.default_rng(n + 1)
    s = np.where(rng.random(n) < 0.5, -1, 1).astype(np.int8)
    w = rng.standard_normal((6, n)).astype(np.float32)
    want = (w.astype(np.float64) * s) @ scipy.linalg.hadamard(n) / np.sqrt(n)
    got = H.rotate_blocks_f32(w, H.HAD_SIGNED, s)
    assert np.max(np.abs(got - want)) < 1e-5 * np.max(np.abs(want))
    # and the flip really is on the input side: the plain rotation of w differs
    assert not np.allclose(H.rotate_blocks_f32(w), got)


def test_signed_with_all_plus_signs_is_sylvester_bit_for_bit():
    w = np.random.default_rng(5).standard_normal((4, 256)).astype(np.float32)
    a = H.rotate_blocks_f32(w, H.HAD_SIGNED, np.ones(256, np.int8))
    assert np.array_equal(a.view(np.uint32), H.rotate_blocks_f32(w).view(np.uint32))


def test_no_hadamard_is_the_identity():
    w = np.random.default_rng(6).standard_normal((3, 64)).astype(np.float32)
    assert np.array_equal(H.rotate_blocks_f32(w, H.HAD_NONE).view(np.uint32), w.view(np.uint32))


@pytest.mark.parametrize("mode,signs", [(3, None), (-1, None), (H.HAD_SIGNED, None),
                                        (H.HAD_SIGNED, np.ones(63)), (H.HAD_SIGNED, np.zeros(64))])
def test_bad_had_choices_are_rejected(mode, signs):
    with pytest.raises(ValueError):
        H.rotate_blocks_f32(np.zeros((1, 64), np.float32), mode, signs)
