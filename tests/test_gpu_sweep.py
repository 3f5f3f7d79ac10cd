"""The continuous-precision sweep of bench.py (layer-output error and weight
reconstruction SNR against OSR for each Hadamard choice) on a small layer,
against the same metrics computed from the oracle's codes on the same seeded
inputs; and the MultiOSR ablation's bookkeeping."""
import math

import numpy as np
import pytest

import bench
import oracle
import synth
from oracle import linear as OL
from tests.gpu_common import require_gpu

pytestmark = pytest.mark.gpu


def test_precision_sweep_matches_oracle_metrics():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    n, k, m, seed = 192, 512, 24, 77
    osrs = (1.0, 2.125, 3.0)
    rows = bench.precision_sweep(torch, P, synth, SG, n=n, k=k, m=m, osrs=osrs, seed=seed)
    assert len(rows) == 3 * 3 * 2
    w = synth.weight_rows(seed, 0, n, k, 0.02, True)
    x = synth.to_f16(synth.activations_f32(seed, 7, m, k)).astype(np.float64)
    y_ref = x @ w.astype(np.float64).T
    signs = synth.hadamard_signs(seed, 256)
    for r in rows:
        s = signs if r["had"] == 2 else None
        o = oracle.encode(w, r["osr"], r["levels"], 256, r["had"], s)
        y = OL.linear_fp64(x, o.codes, o.scales, 256, o.m_up, r["had"], s)
        err = np.linalg.norm(y - y_ref) / np.linalg.norm(y_ref)
        w_hat = OL.reconstruct_fp64(o.codes, o.scales, 256, o.m_up, r["had"], s)
        snr = 10 * math.log10(np.sum(w.astype(np.float64) ** 2) / np.sum((w_hat - w) ** 2))
        assert abs(r["out_rel_err"] - err) <= 1e-2 * err, (r, err)
        assert abs(r["weight_snr_db"] - snr) <= 0.05, (r, snr)
        assert r["bits_per_weight"] == (1 if r["levels"] == 2 else 2) * r["osr"]
    # more samples per weight, less error, for every choice
    for levels in (2, 3):
        for had in (0, 1, 2):
            e = [r["out_rel_err"] for r in rows if r["levels"] == levels and r["had"] == had]
            assert e[0] > e[1] > e[2], (levels, had, e)


def test_multiosr_ablation_keeps_the_budget():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    res = bench.multiosr_ablation(torch, P, synth, SG, targets=(2.0,), m=4)
    row = res["rows"][0]
    assert row["uniform"]["mean_osr"] == 2.0
    assert 2.0 - 0.125 <= row["multiosr"]["mean_osr"] <= 2.0 + 1e-12
    assert all(1.0 <= o <= 4.0 for o in row["multiosr"]["osr"])
    for name in ("uniform", "multiosr"):
        assert 0 < row[name]["weighted_mean_out_rel_err"] <= row[name]["max_out_rel_err"] < 10
