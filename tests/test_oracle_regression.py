"""The oracle still reproduces its frozen tiny encodings (see tests/golden/make_golden.py)."""
import json
import os

import numpy as np

import oracle
import synth


def test_oracle_matches_frozen_fixture():
    path = os.path.join(os.path.dirname(__file__), "golden", "oracle_regression.json")
    with open(path) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        w = synth.weight_rows(c["seed"], 0, c["n"], c["k"], c["sigma"], True)
        r = oracle.encode(w, c["osr"], c["levels"])
        assert r.m_up == c["m_up"]
        want = np.array([[int(ch) - 1 for ch in row] for row in c["codes"]], np.int8)
        assert np.array_equal(r.codes, want)
        assert [float(s).hex() for s in r.scales] == c["scales"]
