"""Writes tests/golden/oracle_regression.json from the oracle alone.

The fixture freezes tiny oracle encodings so that an unintended change of the
oracle's arithmetic shows up as a test failure.  Inputs come from the seeded
synthetic generator; outputs only from ``oracle``.  Run from the repo root:
    python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402

CASES = [
    {"seed": 11, "n": 3, "k": 512, "osr": 1.5, "levels": 2, "sigma": 0.015},
    {"seed": 12, "n": 3, "k": 512, "osr": 2.0, "levels": 3, "sigma": 0.02},
    {"seed": 13, "n": 2, "k": 256, "osr": 2.5, "levels": 3, "sigma": 0.01},
    {"seed": 14, "n": 2, "k": 256, "osr": 1.625, "levels": 3, "sigma": 0.01},
]


def main():
    out = []
    for c in CASES:
        w = synth.weight_rows(c["seed"], 0, c["n"], c["k"], c["sigma"], True)
        r = oracle.encode(w, c["osr"], c["levels"])
        packed = (r.codes + 1).astype(np.uint8)      # 0, 1, 2 for -1, 0, +1
        out.append(dict(c, m_up=r.m_up,
                        codes=["".join("012"[v] for v in row) for row in packed],
                        scales=[float(s).hex() for s in r.scales]))
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_regression.json")
    with open(path, "w") as f:
        json.dump({"generator": "tests/golden/make_golden.py (oracle only)", "cases": out}, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
