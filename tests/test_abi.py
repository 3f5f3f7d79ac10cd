"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point of include/sdq.h, validates arguments, and its host-only
functions agree with the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2510_03275_amd as P
from paper_2510_03275_amd import binding as Bd
from oracle import layout as LY
from oracle import multiosr as MO
from oracle import resample as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "sdq.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(sdq_[a-z_0-9]+)\s*\(", text)
    return sorted(set(names))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert len(names) >= 18
    lib = ctypes.CDLL(Bd.LIB_PATH)
    for name in names:
        assert hasattr(lib, name), name


def test_layout_struct_size_matches_header():
    assert ctypes.sizeof(Bd.sdq_layout) == 112
    assert Bd.sdq_layout.hadamard.offset == 68 and Bd.sdq_layout.had_signs.offset == 72
    assert Bd.sdq_layout.packing.offset == 104


def test_layout_hadamard_choice():
    import synth
    L = P.sdq_layout_init(8, 512, 2.0, 3, 256)
    assert L.hadamard == P.SDQ_HAD_SYLVESTER and list(L.had_signs) == [0] * 8
    s = synth.hadamard_signs(1, 256)
    P.sdq_layout_set_hadamard(L, P.SDQ_HAD_SIGNED, s)
    bits = np.array([(L.had_signs[t // 32] >> (t % 32)) & 1 for t in range(256)])
    assert np.array_equal(bits == 1, s < 0)
    P.sdq_layout_set_hadamard(L, P.SDQ_HAD_NONE)
    assert L.hadamard == P.SDQ_HAD_NONE and list(L.had_signs) == [0] * 8
    Ls = P.sdq_layout_init(8, 128, 2.0, 3, 64)
    P.sdq_layout_set_hadamard(Ls, P.SDQ_HAD_SIGNED, -np.ones(64, np.int8))
    assert list(Ls.had_signs) == [0xFFFFFFFF, 0xFFFFFFFF] + [0] * 6


@pytest.mark.parametrize("mode,signs", [(3, None), (-1, None), (2, None),
                                        (2, np.zeros(256, np.int8)), (2, np.full(256, 2, np.int8))])
def test_layout_hadamard_rejects(mode, signs):
    L = P.sdq_layout_init(8, 512, 2.0, 3, 256)
    with pytest.raises(P.SdqError) as ei:
        P.sdq_layout_set_hadamard(L, mode, signs)
    assert ei.value.status == -1
    assert L.hadamard == P.SDQ_HAD_SYLVESTER


def test_tampered_hadamard_fields_are_rejected_before_gpu_work():
    L = P.sdq_layout_init(8, 128, 2.0, 3, 64)
    L.had_signs[0] = 1                       # sign bits without the signed Had
    assert P.lib().sdq_quantize_workspace_bytes(ctypes.byref(L)) == 0
    L2 = P.sdq_layout_init(8, 128, 2.0, 3, 64)
    P.sdq_layout_set_hadamard(L2, P.SDQ_HAD_SIGNED, np.ones(64, np.int8))
    L2.had_signs[2] = 1                      # a sign beyond the block of 64
    assert P.lib().sdq_quantize_workspace_bytes(ctypes.byref(L2)) == 0
    L3 = P.sdq_layout_init(8, 128, 2.0, 3, 64)
    L3.hadamard = 5
    assert P.lib().sdq_linear_workspace_bytes(ctypes.byref(L3), 1) == 0


@pytest.mark.parametrize("n,k,osr,levels,block,m_up,cpc", [
    (768, 768, 2.0, 3, 256, 512, 64),
    (4096, 11008, 1.5, 2, 256, 384, 128),
    (8192, 28672, 2.0, 3, 256, 512, 64),
    (1, 256, 1.0, 3, 0, 256, 64),
    (5, 512, 1.625, 3, 256, 416, 64),
    (70, 512, 1.5, 2, 64, 96, 128),
])
def test_layout_geometry(n, k, osr, levels, block, m_up, cpc):
    L = P.sdq_layout_init(n, k, osr, levels, block)
    assert L.m_up == m_up and L.codes_per_chunk == cpc
    assert L.k_up == (k // L.block) * m_up
    assert P.sdq_codes_bytes(L) == LY.packed_bytes(n, L.k_up, levels)


def test_codes_bytes_of_the_down_proj_workload():
    L = P.sdq_layout_init(4096, 11008, 1.5, 2)
    assert P.sdq_codes_bytes(L) == 8_454_144


@pytest.mark.parametrize("args,status", [
    ((10, 300, 2.0, 3, 256), -2),     # K not a multiple of B
    ((10, 256, 2.0, 3, 100), -2),     # unsupported block
    ((10, 256, 2.0, 4, 256), -4),     # levels
    ((10, 256, 0.5, 3, 256), -3),     # OSR < 1
    ((10, 256, 1.55, 3, 256), -3),    # M not a multiple of 32
    ((10, 256, float("nan"), 3, 256), -3),
    ((-1, 256, 2.0, 3, 256), -1),
    ((10, 0, 2.0, 3, 256), -1),
])
def test_layout_rejects(args, status):
    with pytest.raises(P.SdqError) as ei:
        P.sdq_layout_init(*args)
    assert ei.value.status == status


def test_quantize_and_linear_reject_bad_arguments_without_gpu_work():
    L = P.sdq_layout_init(64, 256, 2.0, 3)
    lib = P.lib()
    need = lib.sdq_quantize_workspace_bytes(ctypes.byref(L))
    assert need > 0
    # workspace too small / missing: rejected before anything is enqueued
    assert lib.sdq_quantize(ctypes.c_void_p(16), ctypes.byref(L), ctypes.c_void_p(16),
                            ctypes.c_void_p(16), ctypes.c_void_p(16), need - 1, None) == -6
    assert lib.sdq_quantize(None, ctypes.byref(L), None, None, ctypes.c_void_p(16), need, None) == -1
    assert lib.sdq_quantize(None, None, None, None, None, 0, None) == -1
    bad = Bd.sdq_layout()
    bad.n, bad.k, bad.block = 64, 256, 256
    assert lib.sdq_quantize(None, ctypes.byref(bad), None, None, None, 0, None) == -1
    assert lib.sdq_linear(None, 0, -1, None, None, ctypes.byref(L), None, 0, None, 0, None) == -1
    assert lib.sdq_linear(None, 7, 1, None, None, ctypes.byref(L), None, 0, None, 0, None) == -1
    assert lib.sdq_linear(ctypes.c_void_p(16), 0, 1, ctypes.c_void_p(16), ctypes.c_void_p(16),
                          ctypes.byref(L), ctypes.c_void_p(16), 0, None, 0, None) == -6
    assert lib.sdq_linear_expanded(1, ctypes.c_void_p(16), ctypes.c_void_p(16), ctypes.byref(L),
                                   ctypes.c_void_p(16), 1, None, 0, None) == -6
    # misaligned weights, activations, codes or workspace: rejected before anything is enqueued
    lneed = lib.sdq_linear_workspace_bytes(ctypes.byref(L), 1)
    assert lib.sdq_quantize(ctypes.c_void_p(24), ctypes.byref(L), ctypes.c_void_p(16),
                            ctypes.c_void_p(16), ctypes.c_void_p(16), need, None) == -1
    assert lib.sdq_quantize(ctypes.c_void_p(16), ctypes.byref(L), ctypes.c_void_p(20),
                            ctypes.c_void_p(16), ctypes.c_void_p(16), need, None) == -1
    assert lib.sdq_quantize(ctypes.c_void_p(16), ctypes.byref(L), ctypes.c_void_p(16),
                            ctypes.c_void_p(16), ctypes.c_void_p(40), need, None) == -1
    assert lib.sdq_linear(ctypes.c_void_p(18), 0, 1, ctypes.c_void_p(16), ctypes.c_void_p(16),
                          ctypes.byref(L), ctypes.c_void_p(16), 0, ctypes.c_void_p(16), lneed, None) == -1
    assert lib.sdq_linear(ctypes.c_void_p(16), 0, 1, ctypes.c_void_p(24), ctypes.c_void_p(16),
                          ctypes.byref(L), ctypes.c_void_p(16), 0, ctypes.c_void_p(16), lneed, None) == -1
    assert lib.sdq_linear(ctypes.c_void_p(16), 0, 1, ctypes.c_void_p(16), ctypes.c_void_p(16),
                          ctypes.byref(L), ctypes.c_void_p(16), 0, ctypes.c_void_p(8), lneed, None) == -1
    assert lib.sdq_linear_expanded(1, ctypes.c_void_p(16), ctypes.c_void_p(16), ctypes.byref(L),
                                   ctypes.c_void_p(16), 1, ctypes.c_void_p(4), lneed, None) == -1
    # m == 0 is a successful no-op
    assert lib.sdq_linear(None, 0, 0, None, None, ctypes.byref(L), None, 0, None, 0, None) == 0
    assert lib.sdq_linear(None, 0, 0, None, None, ctypes.byref(L), None, 1, None, 0, None) == 0
    assert lib.sdq_linear_workspace_bytes(ctypes.byref(L), 0) == 0
    assert lib.sdq_linear_workspace_bytes(ctypes.byref(L), 1) > 0
    assert lib.sdq_linear_workspace_bytes(ctypes.byref(L), 2048) >= 2048 * 512 * 2
    assert P.sdq_version() >= 100
    assert lib.sdq_status_string(-5) == b"non-finite weight"


@pytest.mark.parametrize("block,m_up", [(256, 384), (256, 512), (256, 640), (256, 416), (256, 768),
                                         (128, 192), (128, 256), (64, 96)])
def test_upsample_table_bit_identical_to_oracle(block, m_up):
    got = P.sdq_upsample_table(block, m_up)
    want = R.g_table_f32(block, m_up)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("levels", [2, 3])
@pytest.mark.parametrize("n,k,osr", [(1, 256, 2.0), (65, 512, 1.5), (130, 768, 2.5), (3, 512, 1.625)])
def test_unpack_matches_oracle_packer(levels, n, k, osr):
    L = P.sdq_layout_init(n, k, osr, levels)
    rng = np.random.default_rng(n * 7 + levels)
    vals = [-1, 1] if levels == 2 else [-1, 0, 1]
    codes = rng.choice(vals, size=(n, L.k_up)).astype(np.int8)
    buf = LY.pack(codes, levels)
    assert np.array_equal(P.sdq_unpack_codes(L, buf), codes)


@pytest.mark.parametrize("n,k,osr", [(1, 256, 2.0), (65, 512, 1.5), (130, 768, 2.5), (3, 512, 1.625),
                                     (64, 1024, 2.0)])
def test_unpack_base3_matches_oracle_packer(n, k, osr):
    L = P.sdq_layout_set_packing(P.sdq_layout_init(n, k, osr, 3), P.SDQ_PACK_BASE3)
    n_pad, n_chunks = LY.geometry_base3(n, L.k_up)
    assert (L.packing, L.codes_per_chunk, L.n_chunks, L.n_pad) == (1, 80, n_chunks, n_pad)
    assert P.sdq_codes_bytes(L) == LY.packed_bytes_base3(n, L.k_up)
    rng = np.random.default_rng(n * 11 + k)
    codes = rng.choice([-1, 0, 1], size=(n, L.k_up)).astype(np.int8)
    assert np.array_equal(P.sdq_unpack_codes(L, LY.pack_base3(codes)), codes)


def test_layout_packing_choice_and_rejects():
    L = P.sdq_layout_init(8, 512, 2.0, 3)
    assert (L.packing, L.codes_per_chunk, L.n_chunks) == (0, 64, 16)
    P.sdq_layout_set_packing(L, P.SDQ_PACK_BASE3)
    assert (L.packing, L.codes_per_chunk, L.n_chunks) == (1, 80, 13)
    assert abs(P.sdq_compression_ratio(L) - 1.6 * 2.0 / 16) < 1e-15
    P.sdq_layout_set_packing(L, P.SDQ_PACK_FIELDS)
    assert (L.packing, L.codes_per_chunk, L.n_chunks) == (0, 64, 16)
    Lb = P.sdq_layout_init(8, 512, 2.0, 2)
    with pytest.raises(P.SdqError) as ei:
        P.sdq_layout_set_packing(Lb, P.SDQ_PACK_BASE3)      # base-3 holds ternary codes only
    assert ei.value.status == -4 and Lb.packing == 0
    with pytest.raises(P.SdqError):
        P.sdq_layout_set_packing(L, 7)
    Lt = P.sdq_layout_init(8, 512, 2.0, 3)
    Lt.packing = 1                                          # tampered: chunk geometry still 2-bit
    assert P.lib().sdq_quantize_workspace_bytes(ctypes.byref(Lt)) == 0
    assert P.lib().sdq_linear_workspace_bytes(ctypes.byref(Lt), 1) == 0


@pytest.mark.parametrize("seed", range(8))
def test_multiosr_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    cnt = int(rng.integers(1, 40))
    var = np.exp(rng.uniform(np.log(5e-5), np.log(1e-3), cnt))
    n = rng.integers(1000, 10_000_000, cnt)
    layers = np.sort(rng.integers(0, 6, cnt))
    T, lo, hi = [(2.5, 1.5, 3.0), (2.0, 1.0, 4.0), (1.75, 1.5, 2.5)][seed % 3]
    got = P.sdq_multiosr(var, n, layers, T, lo, hi, 0.125)
    want = MO.multiosr(list(var), list(int(v) for v in n), list(int(v) for v in layers), T, lo, hi, 0.125)
    assert np.array_equal(got, np.array(want))


def test_multiosr_llama7b_layer_and_70b_stack():
    import synth
    for idx in (3, 5):
        wl = synth.workload(idx)
        var = [lin.sigma ** 2 for lin in wl.linears]
        n = [lin.n * lin.k for lin in wl.linears]
        lay = [lin.layer for lin in wl.linears]
        T, lo, hi = wl.multiosr
        got = P.sdq_multiosr(var, n, lay, T, lo, hi)
        want = MO.multiosr(var, n, lay, T, lo, hi)
        assert np.array_equal(got, np.array(want))
        mean = float(np.dot(got, n) / np.sum(n))
        assert T - 0.125 < mean <= T


def test_multiosr_rejects():
    with pytest.raises(P.SdqError):
        P.sdq_multiosr([1e-4], [10], [0], 3.5, 1.5, 3.0)
    with pytest.raises(P.SdqError):
        P.sdq_multiosr([1e-4], [0], [0], 2.0, 1.5, 3.0)


def test_compression_ratio_of_layout():
    assert abs(P.sdq_compression_ratio(P.sdq_layout_init(8, 512, 2.0, 3)) - 2 * 2.0 / 16) < 1e-15
    assert abs(P.sdq_compression_ratio(P.sdq_layout_init(8, 512, 1.5, 2)) - 1.5 / 16) < 1e-15


def test_single_hip_runtime_in_process():
    # libsdq must bind to PyTorch's HIP runtime: device pointers and streams
    # handed over by torch belong to that runtime.
    import torch  # noqa: F401
    from synth import gpu  # noqa: F401
    assert len(Bd.hip_runtimes_loaded()) == 1


def test_compensation_entry_points_validate_before_gpu_work():
    lib = P.lib()
    assert lib.sdq_hessian_factor_workspace_bytes(100) == 0
    assert lib.sdq_hessian_factor_workspace_bytes(128) >= 2 * 128 * 128 * 8
    fake = ctypes.c_void_p(0x1000)
    assert lib.sdq_hessian_factor(fake, 100, 0.1, fake, fake, 1 << 30, None) == -2
    assert lib.sdq_hessian_factor(None, 128, 0.1, fake, fake, 1 << 30, None) == -1
    assert lib.sdq_hessian_factor(fake, 128, -1.0, fake, fake, 1 << 30, None) == -1
    assert lib.sdq_hessian_factor(fake, 128, float("nan"), fake, fake, 1 << 30, None) == -1
    assert lib.sdq_hessian_factor(fake, 128, 0.1, fake, fake, 16, None) == -6
    assert lib.sdq_hessian_accumulate(fake, -1, 64, fake, None) == -1
    assert lib.sdq_hessian_accumulate(None, 0, 64, fake, None) == 0          # m = 0: nothing to do
    L = P.sdq_layout_init(64, 512, 2.0, 3)
    need = lib.sdq_quantize_compensated_workspace_bytes(ctypes.byref(L))
    assert need > lib.sdq_quantize_workspace_bytes(ctypes.byref(L)) + 64 * 512 * 8
    assert lib.sdq_quantize_compensated(fake, ctypes.byref(L), None, 0, fake, fake, fake, need, None) == -1
    assert lib.sdq_quantize_compensated(fake, ctypes.byref(L), fake, 0, fake, fake, fake, need - 1, None) == -6
    assert lib.sdq_quantize_compensated(fake, ctypes.byref(L), fake, 2, fake, fake, fake, need, None) == -1
    assert lib.sdq_status_string(-10) == b"matrix not positive definite"


def test_noalloc_scratch_covers_every_decode_call_of_the_header():
    # sdq.h: the fixed scratch of sdq_linear_noalloc fits every 1..16-row call
    # on 2-bit fields up to k = 28672 at OSR 8 (every block and OSR step).
    limit = P.SDQ_NOALLOC_SCRATCH_BYTES
    assert limit == 32 << 20
    lib = P.lib()
    worst = 0
    for block in (64, 128, 256):
        for m_up in range(block, 8 * block + 1, 32):
            for levels in (2, 3):
                L = P.sdq_layout_init(64, 28672, m_up / block, levels, block)
                for m in range(1, 17):
                    worst = max(worst, lib.sdq_linear_workspace_bytes(ctypes.byref(L), m))
    assert 0 < worst <= limit, worst


def test_noalloc_entry_point_validates_before_gpu_work():
    lib = P.lib()
    fake = ctypes.c_void_p(0x1000)
    L = P.sdq_layout_init(64, 28672, 2.0, 3)
    # a prefill call beyond the fixed scratch is refused before anything else
    assert lib.sdq_linear_noalloc(fake, 0, 2048, fake, fake, ctypes.byref(L), fake, 0, None) == -6
    assert lib.sdq_linear_noalloc(fake, 0, 0, fake, fake, ctypes.byref(L), fake, 0, None) in (0, -7)


def test_group_entry_point_validates_before_gpu_work():
    lib = P.lib()
    fake = ctypes.c_void_p(0x1000)
    a = P.sdq_layout_init(64, 512, 2.0, 3)
    b = P.sdq_layout_init(128, 512, 2.5, 3)
    c = P.sdq_layout_init(128, 512, 2.0, 3)
    ptrs = (ctypes.c_void_p * 2)(fake, fake)
    assert P.sdq_linear_group_workspace_bytes([a, c], 1) >= P.sdq_linear_workspace_bytes(a, 1)
    assert P.sdq_linear_group_workspace_bytes([a, b], 1) == 0           # M differs
    assert P.sdq_linear_group_workspace_bytes([a] * 5, 1) == 0          # more than four
    arr = (P.sdq_layout * 2)(a, b)
    assert lib.sdq_linear_group(fake, 0, 1, 2, ptrs, ptrs, arr, ptrs, 0, fake, 1 << 30, None) == -1
    arr = (P.sdq_layout * 2)(a, c)
    assert lib.sdq_linear_group(fake, 0, 1, 0, ptrs, ptrs, arr, ptrs, 0, fake, 1 << 30, None) == -1
    assert lib.sdq_linear_group(fake, 0, 1, 2, ptrs, ptrs, arr, ptrs, 0, fake, 16, None) == -6
    assert lib.sdq_linear_group(fake, 0, 0, 2, ptrs, ptrs, arr, ptrs, 0, None, 0, None) == 0   # m = 0
