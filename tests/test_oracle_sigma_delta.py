"""Pins of the oracle's quantizers (Eq. 4, Eq. 6) and Sigma-Delta recursion (Eq. 7-11)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import sigma_delta as SD


def eq7_exact(xs, s, levels):
    """Eq. 7-8 literally, in exact rational arithmetic: i_n = i_{n-1} + x_n - y_{n-1}."""
    s = Fraction(s)
    theta = s / 2
    i_prev, y_prev = Fraction(0), Fraction(0)
    out = []
    for x in xs:
        i_n = i_prev + Fraction(x) - y_prev
        if levels == 3:
            c = 1 if i_n > theta else (-1 if i_n < -theta else 0)
        else:
            c = 1 if i_n >= 0 else -1
        y_prev = c * s
        i_prev = i_n
        out.append(c)
    return out


@pytest.mark.parametrize("levels", [2, 3])
def test_matches_exact_recursion_on_dyadic_inputs(levels):
    # Inputs on a coarse dyadic grid keep every fp32 operation exact, so the
    # fp32 scan must equal the rational transliteration of Eq. 7-8.
    rng = np.random.default_rng(levels)
    for trial in range(20):
        x = (rng.integers(-64, 65, size=200) / 64.0).astype(np.float32)
        s = np.float32(1.0)
        got = SD.scan_f32(x[None, :], s, levels)[0]
        assert list(got) == eq7_exact([float(a) for a in x], 1.0, levels)


def test_quantizer_ties():
    # Eq. 4: sign(0) = +1.  Eq. 6: |v| = theta maps to 0.
    assert SD.quant_binary(np.array([0.0, -0.0, -1e-30])).tolist() == [1, 1, -1]
    assert SD.quant_ternary(np.array([0.5, -0.5, 0.50001, -0.50001]), 0.5).tolist() == [0, 0, 1, -1]


@pytest.mark.parametrize("levels,half_step", [(3, 0.5), (2, 1.0)])
def test_state_bounded_for_in_range_input(levels, half_step):
    rng = np.random.default_rng(9)
    x = rng.uniform(-1, 1, size=(50, 400)).astype(np.float32)
    s = np.float32(np.max(np.abs(x)))
    for row in x:
        _, u = SD.scan_state_f32(row, s, levels)
        assert np.max(np.abs(u)) <= half_step * s * (1 + 1e-6)


@pytest.mark.parametrize("levels", [2, 3])
def test_prefix_tracking(levels):
    # Y = X + (1 - z^-1) E (Eq. 11): the running sum of output minus input is
    # the negated state, so the codes' prefix sums track the input's.
    rng = np.random.default_rng(4)
    x = rng.uniform(-0.9, 0.9, size=300).astype(np.float32)
    s = np.float32(1.0)
    c, u = SD.scan_state_f32(x, s, levels)
    run = np.cumsum(c.astype(np.float64) * 1.0 - x.astype(np.float64))
    assert np.max(np.abs(run + u.astype(np.float64))) < 1e-4


def test_special_inputs():
    s = np.float32(0.25)
    zeros = np.zeros((1, 64), np.float32)
    assert np.all(SD.scan_f32(zeros, s, 3) == 0)
    # binary on zero input alternates +1, -1 around the zero mean
    b = SD.scan_f32(zeros, s, 2)[0]
    assert b[0] == 1 and np.all(b[1:] == -b[:-1])
    assert np.all(SD.scan_f32(np.full((1, 64), s, np.float32), s, 3) == 1)
    assert np.all(SD.scan_f32(np.full((1, 64), -s, np.float32), s, 3) == -1)
    assert np.all(SD.scan_f32(np.full((1, 64), s, np.float32), s, 2) == 1)


@pytest.mark.parametrize("a", [0.1, 0.3, -0.45, 0.77])
@pytest.mark.parametrize("levels", [2, 3])
def test_constant_input_code_mean(a, levels):
    n = 512
    s = np.float32(1.0)
    x = np.full((1, n), np.float32(a), np.float32)
    c = SD.scan_f32(x, s, levels)[0]
    half_step = 0.5 if levels == 3 else 1.0
    assert abs(c.mean() - a) <= half_step / n + 1e-6


def test_scale_zero_row():
    x = np.zeros((1, 16), np.float32)
    assert np.all(SD.scan_f32(x, np.float32(0), 3) == 0)
    assert np.all(SD.scan_f32(x, np.float32(0), 2) == 1)


@pytest.mark.parametrize("levels", [2, 3])
def test_noise_is_high_pass(levels):
    # H_e = 1 - z^-1 (Eq. 11): the quantization error has little energy at low
    # frequencies, unlike memoryless rounding of the same signal.
    rng = np.random.default_rng(12)
    n = 4096
    t = np.arange(n)
    x = (0.5 * np.sin(2 * np.pi * 3 * t / n) + 0.2 * rng.standard_normal(n) * 0.1).astype(np.float32)
    s = np.float32(1.0)
    c = SD.scan_f32(x[None, :], s, levels)[0].astype(np.float64)
    e = c - x
    spec = np.abs(np.fft.rfft(e)) ** 2
    low = spec[1:n // 32].mean()
    high = spec[n // 4:].mean()
    assert low < 0.01 * high
    memoryless = (SD.quant_ternary(x, 0.5) if levels == 3 else SD.quant_binary(x)).astype(np.float64)
    spec_m = np.abs(np.fft.rfft(memoryless - x)) ** 2
    assert low < 0.1 * spec_m[1:n // 32].mean()
