"""Invariants of the oracle's MultiOSR reading (Section 3.4).  The paper gives the
rule in words only, so exact allocations are parity-unpinned; these tests pin
the properties the words fix and the closed form of the unclipped case."""
import numpy as np
import pytest

from oracle import multiosr as MO


def _wmean(osr, n):
    return float(np.dot(osr, n) / np.sum(n))


def test_single_linear_gets_target():
    assert MO.multiosr([3e-4], [1000], [0], 2.5, 1.5, 3.0) == [2.5]


def test_all_equal_gets_target():
    out = MO.multiosr([2e-4] * 7, [100] * 7, [0] * 7, 2.25, 1.5, 3.0)
    assert out == [2.25] * 7


def test_unclipped_closed_form():
    # One layer, bounds inactive: OSR_j = mu * n_j / var_j with the weighted mean = T.
    var = [2e-4, 4e-4, 5e-4]
    n = [1000, 1500, 1200]
    T = 2.0
    cont = MO.multiosr_continuous(var, n, [0, 0, 0], T, 0.01, 100.0)
    b = np.array(n) / np.array(var)
    mu = T * sum(n) / float(np.dot(n, b))
    assert np.allclose(cont, mu * b, rtol=1e-12)


def test_layer_level_inverse_pooled_variance():
    var = [1e-4, 1e-4, 4e-4, 4e-4]
    n = [10, 10, 10, 10]
    cont = MO.multiosr_continuous(var, n, [0, 0, 1, 1], 2.5, 0.01, 100.0)
    # layer osr proportional to 1/V_l: 4:1, weighted mean 2.5 -> 4.0 and 1.0
    assert np.allclose(cont, [4.0, 4.0, 1.0, 1.0], rtol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_invariants_random(seed):
    rng = np.random.default_rng(seed)
    cnt = int(rng.integers(1, 30))
    var = list(np.exp(rng.uniform(np.log(1e-4), np.log(1e-3), cnt)))
    n = [int(v) for v in rng.integers(1000, 100000, cnt)]
    layers = sorted(int(v) for v in rng.integers(0, 5, cnt))
    T, lo, hi, g = 2.5, 1.5, 3.0, 0.125
    out = np.array(MO.multiosr(var, n, layers, T, lo, hi, g))
    assert np.all(out >= lo) and np.all(out <= hi)
    assert np.allclose(out / g, np.round(out / g), atol=1e-12)
    mean = _wmean(out, n)
    assert mean <= T + 1e-12
    assert mean > T - g * max(n) / sum(n) - 1e-12


def test_monotone_in_variance_and_size():
    var = [2e-4, 3e-4, 4e-4, 5e-4]
    n = [1000, 1000, 1000, 1000]
    base = MO.multiosr_continuous(var, n, [0] * 4, 2.0, 1.0, 4.0)
    up_var = MO.multiosr_continuous([2e-4, 3e-4, 6e-4, 5e-4], n, [0] * 4, 2.0, 1.0, 4.0)
    assert up_var[2] < base[2]
    up_n = MO.multiosr_continuous(var, [1000, 1000, 2000, 1000], [0] * 4, 2.0, 1.0, 4.0)
    assert up_n[2] > base[2]
    # lower variance -> higher OSR inside a layer
    assert base[0] > base[1] > base[2] > base[3]


def test_nonpositive_variance_maps_to_hi():
    out = MO.multiosr([0.0, 2e-4, 3e-4], [10, 1000, 1000], [0, 0, 0], 2.0, 1.5, 3.0)
    assert out[0] == 3.0


def test_rejects_target_outside_bounds():
    with pytest.raises(ValueError):
        MO.multiosr([1e-4], [10], [0], 3.5, 1.5, 3.0)


def test_variance_two_pass():
    rng = np.random.default_rng(0)
    w = (rng.standard_normal((100, 300)) * 0.02 + 5.0).astype(np.float32)
    assert abs(MO.variance_fp64(w) - np.var(w.astype(np.float64))) < 1e-15
