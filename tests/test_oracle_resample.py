"""Pins of the oracle's Resample (Algorithm 1) and its closed forms."""
import numpy as np
import pytest
from scipy import signal

from oracle import resample as R
from oracle import encoder as E

CASES = [(4, 5), (8, 12), (8, 13), (8, 16), (16, 24), (256, 384), (256, 512), (256, 640), (256, 416)]


@pytest.mark.parametrize("d,n", CASES + [(n, d) for d, n in CASES] + [(13, 7), (12, 7), (7, 12)])
def test_fft_resample_matches_scipy(d, n):
    rng = np.random.default_rng(d * 1000 + n)
    x = rng.standard_normal((3, d))
    assert np.max(np.abs(R.resample_fft(x, n) - signal.resample(x, n, axis=-1))) < 1e-12


@pytest.mark.parametrize("b,m", [(8, 12), (8, 13), (8, 16), (16, 24), (256, 384), (256, 512), (256, 640)])
def test_closed_forms_match_fft(b, m):
    up = R.up_matrix_fp64(b, m)
    down = R.down_matrix_fp64(b, m)
    assert np.max(np.abs(up - R.resample_fft(np.eye(b), m))) < 1e-12
    assert np.max(np.abs(down - R.resample_fft(np.eye(m), b))) < 1e-12
    # decimation undoes interpolation
    assert np.max(np.abs(up @ down - np.eye(b))) < 1e-12


def test_identity_when_no_oversampling():
    assert np.max(np.abs(R.up_matrix_fp64(16, 16) - np.eye(16))) < 1e-15


@pytest.mark.parametrize("b,m", [(256, 384), (256, 512), (256, 640)])
def test_in_band_tone_interpolates_exactly(b, m):
    t = np.arange(b)
    mm = np.arange(m)
    for f in (0, 1, 7, 100, b // 2 - 1):
        v = np.cos(2 * np.pi * f * t / b + 0.3)
        want = np.cos(2 * np.pi * f * mm / m + 0.3)
        assert np.max(np.abs(R.resample_fft(v, m) - want)) < 1e-11


def test_down_transpose_is_scaled_up_plus_nyquist_term():
    # D^T = (B/M) U + (1/M) cos(pi tau): the activation expansion is not U / OSR.
    b, m = 16, 24
    up = R.up_matrix_fp64(b, m)
    down = R.down_matrix_fp64(b, m)
    tau = (np.arange(m)[None, :] * b - np.arange(b)[:, None] * m) / m
    assert np.max(np.abs(down.T - ((b / m) * up + np.cos(np.pi * tau) / m))) < 1e-12
    assert np.max(np.abs(down.T - up * (b / m))) > 1e-3


@pytest.mark.parametrize("osr", [1.5, 2.0, 2.5])
def test_fp32_upsample_tracks_library_resample(osr):
    # The fp32 sequential sum reproduces scipy's resample to fp32 accuracy; a
    # wrong phase index p(t, m) or kernel sign fails this.
    rng = np.random.default_rng(11)
    v = rng.standard_normal((6, 256)).astype(np.float32)
    m = E.m_up_for(osr, 256)
    got = E.upsample_f32(v, 256, m).astype(np.float64)
    want = signal.resample(v.astype(np.float64), m, axis=-1)
    assert np.max(np.abs(got - want)) < 2e-5 * np.max(np.abs(want))


def test_g_table_special_entries():
    g = R.g_table_f32(256, 512)
    assert g[0] == 1.0
    assert np.all(g[512::512] == 0.0)
    assert np.all(g[np.arange(256 * 512) % 512 != 0] != 0.0)


def test_even_samples_copy_at_osr2():
    # M = 2B: tau is an integer for even m, so x_up[2i] = v[i] exactly.
    rng = np.random.default_rng(5)
    v = rng.standard_normal((3, 256)).astype(np.float32)
    up = E.upsample_f32(v, 256, 512)
    assert np.array_equal(up[:, 0::2], v)
