"""Pins of the oracle encoder (Algorithm 1 ``SDQuant`` with Hadamard smoothing)."""
import numpy as np
import pytest

import synth
from oracle import encoder as E
from oracle import hadamard as H
from oracle import resample as R
from oracle import sigma_delta as SD


def _rows(n=16, k=512, seed=0, sigma=0.02):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((n, k)) * sigma).astype(np.float32)


@pytest.mark.parametrize("osr", [1.0, 1.5, 2.0, 2.5, 3.0])
@pytest.mark.parametrize("levels", [2, 3])
def test_decimated_codes_track_rotated_row(osr, levels):
    # Summation by parts on Eq. 11: with e_m = s c_m - x_m = u_{m-1} - u_m,
    # |Resample(s c - x_up, B)[t]| <= max|u| * TV_t, where TV_t is the total
    # variation of column t of the decimation matrix; max|u| <= step / 2.
    w = _rows(seed=int(osr * 10) + levels)
    r = E.encode(w, osr, levels)
    m = r.m_up
    v = H.rotate_blocks_f32(w.reshape(16, 2, 256)).astype(np.float64)
    z = R.resample_fft(r.codes.reshape(16, 2, m) * r.scales[:, None, None].astype(np.float64), 256)
    d = R.down_matrix_fp64(256, m)
    tv = np.abs(np.diff(d, axis=0)).sum(0) + np.abs(d[-1])
    half_step = (0.5 if levels == 3 else 1.0) * r.scales.astype(np.float64)[:, None, None]
    slack = 1e-4 * r.scales.astype(np.float64)[:, None, None]
    assert np.all(np.abs(z - v) <= half_step * tv + slack)


@pytest.mark.parametrize("levels", [2, 3])
def test_error_falls_with_osr(levels):
    w = _rows(n=32, seed=21)
    v = H.rotate_blocks_f32(w.reshape(32, 2, 256)).astype(np.float64)
    errs = []
    for osr in (1.0, 1.5, 2.0, 3.0, 4.0):
        r = E.encode(w, osr, levels)
        z = R.resample_fft(r.codes.reshape(32, 2, r.m_up) * r.scales[:, None, None].astype(np.float64), 256)
        errs.append(np.sqrt(np.mean((z - v) ** 2) / np.mean(v ** 2)))
    assert all(a > b for a, b in zip(errs, errs[1:])), errs


def test_scale_is_row_absmax_of_upsampled_rows():
    w = _rows(n=8, k=768)
    r = E.encode(w, 2.0, 3)
    up = E.upsampled_rows_f32(w, 2.0)
    assert np.array_equal(r.scales, np.max(np.abs(up), axis=1))
    # At OSR 2 the even samples are the rotated weights themselves.
    v = H.rotate_blocks_f32(w.reshape(8, 3, 256)).reshape(8, -1)
    assert np.all(r.scales >= np.max(np.abs(v), axis=1))


def test_osr_one_is_plain_sigma_delta_of_rotated_block():
    w = _rows(n=4, k=256)
    r = E.encode(w, 1.0, 3)
    v = H.rotate_blocks_f32(w)
    s = np.max(np.abs(v), axis=1)
    assert np.array_equal(r.scales, s)
    assert np.array_equal(r.codes, SD.scan_f32(v, s, 3))


def test_zero_rows_and_dc_rows():
    w = np.zeros((3, 256), np.float32)
    w[1, 0] = 0.32          # rotates to a constant block 0.02: DC interpolates to a constant
    w[2, 0] = -0.32
    for levels in (2, 3):
        r = E.encode(w, 2.0, levels)
        assert r.scales[0] == 0
        assert np.all(r.codes[0] == (0 if levels == 3 else 1))
        assert abs(float(r.scales[1]) - 0.02) < 1e-7 and np.all(r.codes[1] == 1)
        assert np.all(r.codes[2] == -1)


def test_block_state_resets_per_block():
    # Each block starts from a zero state: a block's codes depend on that block only.
    w = _rows(n=2, k=768, seed=5)
    r = E.encode(w, 2.0, 3)
    w2 = w.copy()
    w2[:, 256:512] *= -1.0     # keeps |x_up|, so the row scale is unchanged
    r2 = E.encode(w2, 2.0, 3)
    assert np.array_equal(r.scales, r2.scales)
    assert np.array_equal(r.codes[:, :512], r2.codes[:, :512])
    assert np.array_equal(r.codes[:, 1024:], r2.codes[:, 1024:])
    assert np.array_equal(r.codes[:, 512:1024], -r2.codes[:, 512:1024])


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        E.encode(np.full((2, 256), np.nan, np.float32), 2.0, 3)
    with pytest.raises(ValueError):
        E.encode(np.zeros((2, 300), np.float32), 2.0, 3)
    with pytest.raises(ValueError):
        E.encode(np.zeros((2, 256), np.float32), 2.0, 4)


def test_empty_rows():
    r = E.encode(np.zeros((0, 512), np.float32), 2.0, 3)
    assert r.codes.shape == (0, 1024) and r.scales.shape == (0,)


def test_synthetic_weights_deterministic_and_row_addressable():
    a = synth.weight_rows(7, 3, 20, 512, 0.02, True)
    b = synth.weight_rows(7, 3, 20, 512, 0.02, True, rows=np.array([4, 19]))
    assert np.array_equal(a[[4, 19]], b)
    assert abs(float(np.std(synth.weight_rows(1, 0, 64, 1024, 0.02, False))) - 0.02) < 0.001


@pytest.mark.parametrize("levels", [2, 3])
def test_signed_hadamard_is_sylvester_on_sign_flipped_columns(levels):
    # w diag(s) H / sqrt(B) = (w * s) H / sqrt(B): encoding W with the signed
    # Had equals encoding W with its columns' signs flipped by s (tiled over
    # the blocks) with the plain Sylvester Had, bit for bit.
    import synth
    from oracle import hadamard as Hd
    rng = np.random.default_rng(11)
    w = (rng.standard_normal((9, 512)) * 0.02).astype(np.float32)
    s = synth.hadamard_signs(4, 256)
    a = E.encode(w, 2.0, levels, 256, Hd.HAD_SIGNED, s)
    b = E.encode((w * np.tile(s, 2)).astype(np.float32), 2.0, levels, 256)
    assert np.array_equal(a.codes, b.codes)
    assert np.array_equal(a.scales.view(np.uint32), b.scales.view(np.uint32))


@pytest.mark.parametrize("levels", [2, 3])
def test_no_hadamard_at_osr_one_is_plain_sigma_delta_of_the_weights(levels):
    # Had = I and M = B: the resampling is the identity, so the codes are the
    # Sigma-Delta scan of the raw weight blocks with the row absmax scale.
    from oracle import hadamard as Hd
    from oracle import sigma_delta as SD
    rng = np.random.default_rng(12)
    w = (rng.standard_normal((7, 512)) * 0.02).astype(np.float32)
    r = E.encode(w, 1.0, levels, 256, Hd.HAD_NONE)
    s = np.max(np.abs(w), axis=1).astype(np.float32)
    want = SD.scan_f32(w.reshape(7, 2, 256), s[:, None], levels).reshape(7, 512)
    assert np.array_equal(r.codes, want)
    assert np.array_equal(r.scales, s)
