"""Packed code format of the library, re-implemented from its header description,
and the compression ratio of Eq. 14.

Format (the library's C header is the normative description):

* bits per code: 1 for binary codes, 2 for ternary codes; a 16-byte chunk holds
  CPC = 128 / bits codes of one row (128 binary or 64 ternary codes);
* K_up = nb * M codes per row, n_chunks = ceil(K_up / CPC) chunks per row, rows
  padded to N_pad = ceil(N / 64) * 64;
* chunk c of row r starts at byte 16 * (((r // 64) * n_chunks + c) * 64 + r % 64),
  i.e. the 64 rows of a panel store their chunk c side by side;
* code j of a row is in chunk j // CPC at position q = j % CPC: little-endian
  32-bit word q // (32 / bits) of the chunk, field of ``bits`` bits starting at
  bit bits * (q % (32 / bits));
* binary field 1 means +1 and 0 means -1; ternary field 00 means 0, 01 means +1,
  11 means -1 (10 is never written);
* padding codes and padding rows are all-zero bits.

Base-3 packing of ternary codes (Eq. 14 counts a ternary code as log2(3) =
1.58 bits; five codes per byte, 3^5 = 243 <= 256, store 1.6 bits each):

* a 16-byte chunk holds 80 codes; the chunk and panel layout are as above;
* code j of a row is in chunk j // 80 at position q = j % 80, the (q % 5)-th
  code of byte q // 5 of the chunk; with digits d_i = code + 1 in {0, 1, 2} of
  the byte's five codes, first code most significant,
  v = 81 d_0 + 27 d_1 + 9 d_2 + 3 d_3 + d_4 in [0, 243), and the byte stores
  q = ceil(256 v / 243), v / 243 as an 8-bit fraction rounded up; it is read
  back as v = floor(243 q / 256).  Byte values up to 255 occur (v = 242 gives
  255), and 13 of the 256 byte values are never written;
* padding codes are code 0 (digit 1) and padding rows all-zero bytes.
"""
from __future__ import annotations

import numpy as np

PANEL = 64
CHUNK_BYTES = 16


def bits_for(levels: int) -> int:
    return 1 if levels == 2 else 2


def codes_per_chunk(levels: int) -> int:
    return CHUNK_BYTES * 8 // bits_for(levels)


def geometry(n: int, k_up: int, levels: int):
    cpc = codes_per_chunk(levels)
    n_chunks = -(-k_up // cpc)
    n_pad = -(-n // PANEL) * PANEL
    return n_pad, n_chunks, cpc


def packed_bytes(n: int, k_up: int, levels: int) -> int:
    n_pad, n_chunks, _ = geometry(n, k_up, levels)
    return n_pad * n_chunks * CHUNK_BYTES


def _field_values(codes: np.ndarray, levels: int) -> np.ndarray:
    if levels == 2:
        return (codes > 0).astype(np.uint32)
    f = np.zeros(codes.shape, dtype=np.uint32)
    f[codes == 1] = 1
    f[codes == -1] = 3
    return f


def pack(codes: np.ndarray, levels: int) -> np.ndarray:
    """int8 codes (N x K_up) -> uint8 packed buffer of ``packed_bytes`` bytes."""
    codes = np.asarray(codes)
    n, k_up = codes.shape
    bits = bits_for(levels)
    n_pad, n_chunks, cpc = geometry(n, k_up, levels)
    per_word = 32 // bits
    fields = np.zeros((n_pad, n_chunks * cpc), dtype=np.uint32)
    fields[:n, :k_up] = _field_values(codes, levels)
    fields = fields.reshape(n_pad, n_chunks, 4, per_word)
    shifts = (np.arange(per_word, dtype=np.uint32) * bits)
    words = np.zeros((n_pad, n_chunks, 4), dtype=np.uint32)
    for q in range(per_word):
        words |= fields[..., q] << shifts[q]
    # [panel, row-in-panel, chunk, word] -> [panel, chunk, row-in-panel, word]
    words = words.reshape(n_pad // PANEL, PANEL, n_chunks, 4).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(words).astype("<u4").view(np.uint8).reshape(-1)


def unpack(buf: np.ndarray, n: int, k_up: int, levels: int) -> np.ndarray:
    """Inverse of ``pack``: uint8 buffer -> int8 codes (N x K_up)."""
    bits = bits_for(levels)
    n_pad, n_chunks, cpc = geometry(n, k_up, levels)
    per_word = 32 // bits
    words = np.frombuffer(np.asarray(buf, dtype=np.uint8).tobytes(), dtype="<u4")
    words = words.reshape(n_pad // PANEL, n_chunks, PANEL, 4).transpose(0, 2, 1, 3)
    words = words.reshape(n_pad, n_chunks, 4)
    mask = np.uint32((1 << bits) - 1)
    fields = np.stack([(words >> np.uint32(q * bits)) & mask for q in range(per_word)], axis=-1)
    fields = fields.reshape(n_pad, n_chunks * cpc)[:n, :k_up]
    if levels == 2:
        return np.where(fields == 1, 1, -1).astype(np.int8)
    return np.where(fields == 1, 1, np.where(fields == 3, -1, 0)).astype(np.int8)


def compression_ratio(bits_per_code: float, osr: float) -> float:
    """Eq. 14: eta = N * OSR / 16 (storage of the codes relative to fp16 weights)."""
    return bits_per_code * osr / 16.0


B3_CODES_PER_CHUNK = 80


def geometry_base3(n: int, k_up: int):
    n_chunks = -(-k_up // B3_CODES_PER_CHUNK)
    n_pad = -(-n // PANEL) * PANEL
    return n_pad, n_chunks


def pack_base3(codes: np.ndarray) -> np.ndarray:
    """Ternary int8 codes (N x K_up) -> the base-3 packed buffer.

    Five codes per byte: with digits d_i = c_i + 1 of codes c_0 .. c_4 (the
    first one most significant), v = 81 d_0 + 27 d_1 + 9 d_2 + 3 d_3 + d_4 in
    [0, 243) is stored as the byte q = ceil(256 v / 243), i.e. v / 243 as an
    8-bit binary fraction rounded up.  (The rounding makes the leading digits
    readable by multiplying q by a power of 3 and keeping the high bits; the
    oracle reads it back through v = floor(243 q / 256).)"""
    codes = np.asarray(codes)
    n, k_up = codes.shape
    n_pad, n_chunks = geometry_base3(n, k_up)
    digits = np.zeros((n_pad, n_chunks * B3_CODES_PER_CHUNK), dtype=np.uint32)
    digits[:n] = 1                                   # padding codes of real rows: code 0
    digits[:n, :k_up] = codes.astype(np.int64) + 1
    digits[n:] = 0                                   # padding rows: zero bytes
    d = digits.reshape(n_pad, n_chunks, 16, 5).astype(np.int64)
    v = 81 * d[..., 0] + 27 * d[..., 1] + 9 * d[..., 2] + 3 * d[..., 3] + d[..., 4]
    q = -((-256 * v) // 243)                         # ceil(256 v / 243)
    byte = q.astype(np.uint8).reshape(n_pad // PANEL, PANEL, n_chunks, 16).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(byte).reshape(-1)


def unpack_base3(buf: np.ndarray, n: int, k_up: int) -> np.ndarray:
    """Inverse of ``pack_base3``: buffer -> ternary int8 codes (N x K_up)."""
    n_pad, n_chunks = geometry_base3(n, k_up)
    b = np.asarray(buf, dtype=np.uint8).reshape(n_pad // PANEL, n_chunks, PANEL, 16)
    b = b.transpose(0, 2, 1, 3).reshape(n_pad, n_chunks * 16).astype(np.int64)
    v = (243 * b) // 256
    digits = np.stack([(v // 3 ** (4 - i)) % 3 for i in range(5)], axis=-1).reshape(n_pad, -1)
    return (digits[:n, :k_up] - 1).astype(np.int8)


def packed_bytes_base3(n: int, k_up: int) -> int:
    n_pad, n_chunks = geometry_base3(n, k_up)
    return n_pad * n_chunks * CHUNK_BYTES
