"""Pins of the oracle's packer (the library's documented format) and of Eq. 14."""
import json
import os

import numpy as np
import pytest

from oracle import layout as LY

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_compression_ratio_worked_numbers():
    # Values the paper prints for its compression ratio (Eq. 14).
    with open(os.path.join(GOLDEN, "compression_ratio.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        eta = LY.compression_ratio(c["bits_per_code"], c["osr"])
        assert round(100 * eta, 2) == c["eta_percent"], c


def test_hand_packed_binary_chunk():
    # Row 0 codes 0..3 = +1, -1, -1, +1 and code 127 = +1 (all others -1):
    # word 0 = 0b1001, word 3 has bit 31 set; rows 1..63 are padding (zero).
    codes = -np.ones((1, 128), np.int8)
    codes[0, [0, 3, 127]] = 1
    buf = LY.pack(codes, 2)
    assert buf.size == 64 * 16
    words = buf.view("<u4")
    assert words[0] == 0b1001 and words[1] == 0 and words[2] == 0 and words[3] == 1 << 31
    assert np.all(words[4:] == 0)


def test_hand_packed_ternary_panel():
    # Row 65 is row 1 of panel 1; K_up = 80 gives 2 chunks per row.
    codes = np.zeros((66, 80), np.int8)
    codes[65, 0] = 1       # field 01 at bits 0..1 of word 0, chunk 0
    codes[65, 17] = -1     # field 11 at bits 2..3 of word 1, chunk 0
    codes[65, 64] = 1      # chunk 1, word 0, bits 0..1
    buf = LY.pack(codes, 3)
    assert buf.size == 128 * 2 * 16
    words = buf.view("<u4").reshape(-1, 4)     # one row = one chunk
    chunk0 = words[(1 * 2 + 0) * 64 + 1]
    chunk1 = words[(1 * 2 + 1) * 64 + 1]
    assert chunk0.tolist() == [1, 0b1100, 0, 0]
    assert chunk1.tolist() == [1, 0, 0, 0]
    assert np.count_nonzero(words) == 3      # the three words set above


@pytest.mark.parametrize("levels", [2, 3])
@pytest.mark.parametrize("n,k_up", [(1, 1), (64, 128), (65, 129), (130, 1536), (3, 16512)])
def test_round_trip(levels, n, k_up):
    rng = np.random.default_rng(n + k_up)
    vals = [-1, 1] if levels == 2 else [-1, 0, 1]
    codes = rng.choice(vals, size=(n, k_up)).astype(np.int8)
    buf = LY.pack(codes, levels)
    assert buf.size == LY.packed_bytes(n, k_up, levels)
    assert np.array_equal(LY.unpack(buf, n, k_up, levels), codes)
