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


# --- base-3 packing of ternary codes (five codes per byte) ---

def test_base3_worked_bytes():
    # codes (+1, 0, -1, -1, +1) -> digits (2, 1, 0, 0, 2), first most significant
    # -> v = 162 + 27 + 0 + 0 + 2 = 191 -> q = ceil(256 * 191 / 243) = ceil(201.2) = 202;
    # all zeros -> v = 121 -> ceil(127.5) = 128; all +1 -> v = 242 -> ceil(254.9) = 255;
    # all -1 -> 0.
    from oracle import layout as LY
    codes = np.zeros((1, 80), np.int8)
    codes[0, :5] = [1, 0, -1, -1, 1]
    codes[0, 5:10] = 1
    codes[0, 10:15] = -1
    buf = LY.pack_base3(codes)
    assert buf.size == 64 * 16
    assert list(buf[:4]) == [202, 255, 0, 128]
    assert np.all(buf[16:] == 0)                       # padding rows


@pytest.mark.parametrize("n,k_up", [(1, 80), (5, 81), (70, 512), (130, 1088)])
def test_base3_round_trip_and_size(n, k_up):
    from oracle import layout as LY
    rng = np.random.default_rng(n + k_up)
    codes = rng.integers(-1, 2, size=(n, k_up)).astype(np.int8)
    buf = LY.pack_base3(codes)
    assert buf.size == LY.packed_bytes_base3(n, k_up) == -(-n // 64) * 64 * -(-k_up // 80) * 16
    valid = {-(-256 * v // 243) for v in range(243)}
    assert set(np.unique(buf).tolist()) <= valid
    assert np.array_equal(LY.unpack_base3(buf, n, k_up), codes)


def test_base3_digits_by_multiplication():
    # The stored byte q is v / 243 rounded up to an 8-bit fraction, so the
    # base-3 digits of v come out most significant first by repeatedly
    # multiplying by 3 and taking the integer part (r <- 3 r; d = r >> 8;
    # r <- r & 255), and the leading three and trailing two digits as
    # (27 q) >> 8 and (9 ((27 q) & 255)) >> 8.  Checked for every v in [0, 243)
    # against plain base-3 digits, and the oracle's unpack agrees.
    from oracle import layout as LY
    codes = np.array([[(v // 3 ** (4 - i)) % 3 - 1 for v in range(243) for i in range(5)]], np.int8)
    buf = LY.pack_base3(codes)                     # one row, 1215 codes: 16 chunks
    qs = buf.reshape(16, 64, 16)[:, 0, :].reshape(-1)[:243]
    for v, q in enumerate(qs.tolist()):
        r, ds = q, []
        for _ in range(5):
            r *= 3
            ds.append(r >> 8)
            r &= 255
        assert ds == [(v // 3 ** (4 - i)) % 3 for i in range(5)], v
        assert (27 * q) >> 8 == v // 9 and (9 * ((27 * q) & 255)) >> 8 == v % 9
    assert np.array_equal(LY.unpack_base3(buf, 1, 1215), codes)


def test_base3_is_smaller_than_two_bit_fields():
    from oracle import layout as LY
    # 1.6 bits per code against 2: 20 % fewer bytes for whole chunks; Eq. 14's
    # eta for OSR 2 at 1.6 bits is 20 %.
    assert LY.packed_bytes_base3(64, 16000) * 10 == LY.packed_bytes(64, 16000, 3) * 8
    assert LY.compression_ratio(1.6, 2.0) == 0.2
