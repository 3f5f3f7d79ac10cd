"""GPU parity of sdq_linear (decode GEMV for m <= 16, prefill MFMA GEMM above)
against the fp64 oracle: per activation row, max_r |y - y*| / max_r |y*| <= 1e-3."""
import numpy as np
import pytest

import oracle
import synth
from oracle import layout as LY
from oracle import hadamard as OH
from oracle import linear as OL
from tests.gpu_common import TOL, gpu_encode, host_bytes, require_gpu, to_device_x

pytestmark = pytest.mark.gpu


def _oracle_codes_on_device(torch, n, k, osr, levels, seed, block=256):
    """Codes from the oracle encoder, packed by the oracle packer, uploaded."""
    import paper_2510_03275_amd as P
    w = synth.weight_rows(seed, 2, n, k, 0.02, True)
    r = oracle.encode(w, osr, levels, block)
    L = P.sdq_layout_init(n, k, osr, levels, block)
    enc = P.Encoded(L, torch.from_numpy(LY.pack(r.codes, levels)).cuda(), torch.from_numpy(r.scales).cuda())
    return enc, r


def _run_linear(torch, enc, x_dev):
    import paper_2510_03275_amd as P
    y = P.linear(x_dev, enc)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


SHAPES = [(130, 768, 2.0, 3), (64, 512, 1.5, 2), (100, 512, 1.625, 3), (200, 1024, 2.5, 3),
          (65, 512, 3.0, 2)]


@pytest.mark.parametrize("m", [1, 2, 3, 8, 16, 17, 64, 130])
@pytest.mark.parametrize("n,k,osr,levels", SHAPES)
def test_linear_small_f16(n, k, osr, levels, m):
    torch = require_gpu()
    enc, r = _oracle_codes_on_device(torch, n, k, osr, levels, seed=n + m)
    x_dev, x64 = to_device_x(synth.activations_f32(m, 0, m, k), "f16", torch)
    y = _run_linear(torch, enc, x_dev)
    y_ref = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up)
    err = OL.rel_err_rows(y, y_ref)
    assert np.all(err <= TOL), err.max()


@pytest.mark.parametrize("lds", ["0", "1"])
@pytest.mark.parametrize("m", [5, 8, 12])
@pytest.mark.parametrize("n,k,osr,levels", SHAPES)
def test_linear_mfma_planes_from_lds_or_l2(n, k, osr, levels, m, lds, monkeypatch):
    # The 5-12-row contraction has two kernels: planes read per panel from L2,
    # or staged in LDS once per four panels (chosen by launch size; forced
    # here so that both run on every shape).
    torch = require_gpu()
    monkeypatch.setenv("SDQ_MFMA_LDS", lds)
    enc, r = _oracle_codes_on_device(torch, n, k, osr, levels, seed=3 * n + m)
    x_dev, x64 = to_device_x(synth.activations_f32(m + 1, 0, m, k), "f16", torch)
    y = _run_linear(torch, enc, x_dev)
    y_ref = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up)
    err = OL.rel_err_rows(y, y_ref)
    assert np.all(err <= TOL), err.max()


@pytest.mark.parametrize("path", ["lut", "mfma"])
@pytest.mark.parametrize("m", [1, 2, 7])
@pytest.mark.parametrize("n,k,osr,levels", SHAPES)
def test_linear_decode_both_paths(n, k, osr, levels, m, path, monkeypatch):
    # Both decode contractions on every shape and row count (the choice by
    # row count and code kind forced here): the addition-only table GEMV and
    # the integer-MFMA one (compact planes at one row).
    torch = require_gpu()
    monkeypatch.setenv("SDQ_DECODE_PATH", path)
    enc, r = _oracle_codes_on_device(torch, n, k, osr, levels, seed=5 * n + m)
    x_dev, x64 = to_device_x(synth.activations_f32(m + 3, 0, m, k), "f16", torch)
    y = _run_linear(torch, enc, x_dev)
    y_ref = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up)
    err = OL.rel_err_rows(y, y_ref)
    assert np.all(err <= TOL), err.max()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m", [1, 5, 16, 40])
def test_linear_small_other_dtypes(dtype, m):
    torch = require_gpu()
    enc, r = _oracle_codes_on_device(torch, 96, 768, 2.0, 3, seed=7)
    x_dev, x64 = to_device_x(synth.activations_f32(11, 0, m, 768), dtype, torch)
    y = _run_linear(torch, enc, x_dev)
    err = OL.rel_err_rows(y, OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
    assert np.all(err <= TOL), err.max()


def test_linear_block_sizes():
    torch = require_gpu()
    for block, osr in ((128, 2.0), (64, 1.5)):
        enc, r = _oracle_codes_on_device(torch, 70, 512, osr, 3, seed=block, block=block)
        for m in (1, 5, 24):
            x_dev, x64 = to_device_x(synth.activations_f32(3, 0, m, 512), "f16", torch)
            y = _run_linear(torch, enc, x_dev)
            err = OL.rel_err_rows(y, OL.linear_fp64(x64, r.codes, r.scales, block, r.m_up))
            assert np.all(err <= TOL), (block, m, err.max())


@pytest.mark.parametrize("block,osr,levels", [(64, 1.5, 2), (64, 2.5, 3), (128, 1.25, 2),
                                               (256, 2.125, 3), (256, 1.875, 2)])
def test_linear_decode_blocks_inside_chunks(block, osr, levels):
    # M = OSR * block not a multiple of the code chunk (64 ternary, 128 binary
    # codes): blocks start and end inside chunks, and at block 64 binary a
    # block is shorter than one chunk.
    torch = require_gpu()
    k = 8 * block
    enc, r = _oracle_codes_on_device(torch, 130, k, osr, levels, seed=block + levels, block=block)
    assert r.m_up % (128 if levels == 2 else 64) != 0
    for m in (1, 2, 4, 9, 16):
        x_dev, x64 = to_device_x(synth.activations_f32(17, 0, m, k), "f16", torch)
        y = _run_linear(torch, enc, x_dev)
        err = OL.rel_err_rows(y, OL.linear_fp64(x64, r.codes, r.scales, block, r.m_up))
        assert np.all(err <= TOL), (block, osr, levels, m, err.max())


def test_linear_decode_repeatable():
    # Split-K decode adds partials with fp32 atomics: repeat calls agree to
    # rounding; a layer with a single K segment is bitwise repeatable.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    enc, _ = _oracle_codes_on_device(torch, 4096, 2048, 2.0, 3, seed=1)
    x_dev, _ = to_device_x(synth.activations_f32(1, 0, 1, 2048), "f16", torch)
    ws = torch.zeros(P.sdq_linear_workspace_bytes(enc.layout, 1), dtype=torch.uint8, device="cuda")
    y1 = P.linear(x_dev, enc, workspace=ws)
    y2 = P.linear(x_dev, enc, workspace=ws)
    assert torch.max(torch.abs(y1 - y2)).item() <= 1e-6 * torch.max(torch.abs(y1)).item()
    # K = 64 at block 64, OSR 2: 128 ternary codes = 2 chunks, the smallest K segment
    small, _ = _oracle_codes_on_device(torch, 256, 64, 2.0, 3, seed=2, block=64)
    assert small.layout.n_chunks <= 2
    xs, _ = to_device_x(synth.activations_f32(1, 0, 1, 64), "f16", torch)
    assert torch.equal(P.linear(xs, small), P.linear(xs, small))


def test_split_entry_points_share_one_expansion():
    # One expansion serves two linears with the same (k, block, M, levels).
    torch = require_gpu()
    import paper_2510_03275_amd as P
    a, ra = _oracle_codes_on_device(torch, 300, 1024, 2.0, 3, seed=11)
    b, rb = _oracle_codes_on_device(torch, 1100, 1024, 2.0, 3, seed=12)
    for m in (1, 5, 40):
        x_dev, x64 = to_device_x(synth.activations_f32(21, 0, m, 1024), "f16", torch)
        need = max(P.sdq_linear_workspace_bytes(a.layout, m), P.sdq_linear_workspace_bytes(b.layout, m))
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        P.sdq_expand_activations(x_dev, a.layout, ws)
        ya = torch.empty((m, 300), dtype=torch.float32, device="cuda")
        yb = torch.empty((m, 1100), dtype=torch.float32, device="cuda")
        P.sdq_linear_expanded(m, a.codes, a.scales, a.layout, ya, ws)
        P.sdq_linear_expanded(m, b.codes, b.scales, b.layout, yb, ws)
        for y, r in ((ya, ra), (yb, rb)):
            ref = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up)
            assert np.all(OL.rel_err_rows(y.cpu().numpy().astype(np.float64), ref) <= TOL)


@pytest.mark.parametrize("n,k,m", [(256, 256, 1), (4096, 2048, 1), (300, 1024, 5), (300, 1024, 40)])
def test_linear_accumulate(n, k, m):
    # accumulate=1 adds x W_hat^T onto y: decode with one K segment (plain
    # read-modify-write), decode split over K (atomics onto y), prefill.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    enc, r = _oracle_codes_on_device(torch, n, k, 2.0, 3, seed=n + k + m)
    x_dev, x64 = to_device_x(synth.activations_f32(31, 0, m, k), "f16", torch)
    y_plain = P.linear(x_dev, enc)
    y0 = torch.from_numpy(synth.activations_f32(32, 0, m, n)).cuda()
    y = y0.clone()
    P.linear(x_dev, enc, out=y, accumulate=True)
    expect = y0 + y_plain
    torch.cuda.synchronize()
    assert torch.max(torch.abs(y - expect)).item() <= 1e-5 * torch.max(torch.abs(expect)).item()
    # the accumulated product still meets the tolerance against the oracle
    err = OL.rel_err_rows((y - y0).cpu().numpy().astype(np.float64),
                          OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
    assert np.all(err <= TOL), err.max()
    # the split entry point accumulates the same way
    ws = torch.empty(P.sdq_linear_workspace_bytes(enc.layout, m), dtype=torch.uint8, device="cuda")
    P.sdq_expand_activations(x_dev, enc.layout, ws)
    y2 = y0.clone()
    P.sdq_linear_expanded(m, enc.codes, enc.scales, enc.layout, y2, ws, accumulate=True)
    torch.cuda.synchronize()
    assert torch.max(torch.abs(y2 - expect)).item() <= 1e-5 * torch.max(torch.abs(expect)).item()


@pytest.mark.parametrize("n,k,osr,levels", [(4096, 2048, 1.5, 2), (3000, 1024, 2.0, 3), (256, 64, 2.0, 3)])
def test_decode_repeated_inputs_on_one_workspace(n, k, osr, levels):
    # Successive one-row calls on one workspace with different inputs each see
    # their own x_tilde, and agree with the split entry points.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    block = 64 if k == 64 else 256
    enc, r = _oracle_codes_on_device(torch, n, k, osr, levels, seed=n + k, block=block)
    ws = torch.empty(P.sdq_linear_workspace_bytes(enc.layout, 1), dtype=torch.uint8, device="cuda")
    y = torch.empty((1, n), dtype=torch.float32, device="cuda")
    y2 = torch.empty((1, n), dtype=torch.float32, device="cuda")
    for it in range(6):
        x_dev, x64 = to_device_x(synth.activations_f32(40 + it, 0, 1, k), "f16", torch)
        P.linear(x_dev, enc, workspace=ws, out=y)
        ws2 = torch.empty_like(ws)
        P.sdq_expand_activations(x_dev, enc.layout, ws2)
        P.sdq_linear_expanded(1, enc.codes, enc.scales, enc.layout, y2, ws2)
        torch.cuda.synchronize()
        ref = OL.linear_fp64(x64, r.codes, r.scales, block, r.m_up)
        got = y.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(got)), it
        assert np.all(OL.rel_err_rows(got, ref) <= TOL), it
        assert torch.max(torch.abs(y - y2)).item() <= 1e-6 * torch.max(torch.abs(y2)).item(), it


def test_linear_empty_batch():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    enc, _ = _oracle_codes_on_device(torch, 64, 256, 2.0, 3, seed=2)
    x = torch.empty((0, 256), dtype=torch.float16, device="cuda")
    assert P.linear(x, enc).shape == (0, 64)


def _workload_case(torch, wl, lin, osr, ms, n_sample=32):
    """GPU: generate W on the device, encode, run the linear at batch m.
    Oracle: regenerate sampled rows on the host, encode, fp64 linear."""
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    w_dev = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
    enc = gpu_encode(w_dev, osr, wl.levels)
    del w_dev
    rng = np.random.default_rng(lin.linear_id + 99)
    rows = np.unique(np.concatenate([[0, lin.n - 1], rng.choice(lin.n, n_sample, replace=False)]))
    w_rows = synth.weight_rows(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers, rows=rows)
    r = oracle.encode(w_rows, osr, wl.levels)
    for m in ms:
        x32 = SG.activations_gpu(wl.seed, 100 + m, m, lin.k).cpu().numpy()
        x_dev, x64 = to_device_x(x32, wl.x_dtype, torch)
        y = P.linear(x_dev, enc)
        torch.cuda.synchronize()
        y_s = y[:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
        y_ref = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up)
        err = OL.rel_err_rows(y_s, y_ref)
        assert np.all(err <= TOL), (lin.name, m, err.max())
    torch.cuda.empty_cache()


def test_linear_opt125m_q_proj():
    torch = require_gpu()
    wl = synth.workload(1)
    _workload_case(torch, wl, wl.linears[0], wl.osr, wl.batches, n_sample=200)


def test_linear_llama7b_down_proj_decode():
    torch = require_gpu()
    wl = synth.workload(2)
    _workload_case(torch, wl, wl.linears[0], wl.osr, wl.batches)


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_linear_llama70b_decode_and_prefill(idx):
    torch = require_gpu()
    wl = synth.workload(4)
    _workload_case(torch, wl, wl.linears[idx], wl.osr, wl.batches + wl.prefill, n_sample=16)


def test_linear_llama7b_layer_multiosr():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    wl = synth.workload(3)
    var = [lin.sigma ** 2 for lin in wl.linears]
    n = [lin.n * lin.k for lin in wl.linears]
    osr = P.sdq_multiosr(var, n, [lin.layer for lin in wl.linears], *wl.multiosr)
    for lin, o in zip(wl.linears, osr):
        _workload_case(torch, wl, lin, float(o), wl.batches, n_sample=8)


def test_weight_moments_match_oracle():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    for n, k in ((1, 1), (300, 777), (4096, 4096)):
        w = synth.weight_rows(n, 0, n, k, 0.02, True) + np.float32(0.5)
        w_dev = torch.from_numpy(w).cuda()
        out = torch.zeros(2, dtype=torch.float64, device="cuda")
        ws = torch.empty(P.sdq_moments_workspace_bytes(w.size), dtype=torch.uint8, device="cuda")
        P.sdq_weight_moments(w_dev, out, ws)
        got = out.cpu().numpy()
        x = w.astype(np.float64)
        assert abs(got[0] - x.mean()) <= 1e-12 * max(1.0, abs(x.mean()))
        assert abs(got[1] - oracle.variance_fp64(w)) <= 1e-10 * max(oracle.variance_fp64(w), 1e-30)


def _row_factors(kind, m):
    """Power-of-two factors per activation row: one for every row, or a spread."""
    if kind == "mixed":
        return np.array([2.0 ** ((7 * i) % 81 - 40) for i in range(m)], dtype=np.float64)
    return np.full(m, 2.0 ** kind)


@pytest.mark.parametrize("dtype,kind", [("f16", 12), ("f16", -16), ("f16", "mixed12"),
                                        ("bf16", 12), ("bf16", -16), ("bf16", 40), ("bf16", -40),
                                        ("bf16", "mixed"), ("f32", 12), ("f32", -16), ("f32", 40),
                                        ("f32", -40), ("f32", "mixed")])
@pytest.mark.parametrize("m", [1, 8, 64])
def test_linear_activation_magnitudes(dtype, kind, m):
    # Activations far outside N(0, 1): every path keeps 1e-3 whatever a row's
    # magnitude -- the prefill path stores x_tilde in fp16 (normal range
    # 2^-14 .. 65504) and scales each row by a power of two first.  The fp16
    # cases stay inside fp16's own range (at most 2^12 times N(0, 1)).
    torch = require_gpu()
    enc, r = _oracle_codes_on_device(torch, 200, 1024, 2.0, 3, seed=31)
    if kind == "mixed12":
        f = np.array([2.0 ** ((5 * i) % 25 - 12) for i in range(m)])
    else:
        f = _row_factors(kind, m)
    x32 = (synth.activations_f32(41, 0, m, 1024).astype(np.float64) * f[:, None]).astype(np.float32)
    x_dev, x64 = to_device_x(x32, dtype, torch)
    y = _run_linear(torch, enc, x_dev)
    assert np.all(np.isfinite(y))
    err = OL.rel_err_rows(y, OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
    assert np.all(err <= TOL), (dtype, kind, m, err.max())


@pytest.mark.parametrize("had", ["none", "sylvester"])
def test_linear_prefill_magnitudes_fp16_pair(had):
    # Layouts without Had keep x_tilde as an fp16 pair hi + lo: both halves
    # are scaled by the row's power of two.  Codes from the oracle encoder.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    n, k, m = 130, 768, 40
    w = synth.weight_rows(77, 2, n, k, 0.02, True)
    hd_o = OH.HAD_NONE if had == "none" else OH.HAD_SYLVESTER
    r = oracle.encode(w, 2.0, 3, 256, hd_o)
    L = P.sdq_layout_init(n, k, 2.0, 3)
    P.sdq_layout_set_hadamard(L, P.SDQ_HAD_NONE if had == "none" else P.SDQ_HAD_SYLVESTER)
    enc = P.Encoded(L, torch.from_numpy(LY.pack(r.codes, 3)).cuda(), torch.from_numpy(r.scales).cuda())
    f = np.array([2.0 ** ((11 * i) % 61 - 30) for i in range(m)])
    x32 = (synth.activations_f32(5, 0, m, k).astype(np.float64) * f[:, None]).astype(np.float32)
    x_dev, x64 = to_device_x(x32, "bf16", torch)
    y = _run_linear(torch, enc, x_dev)
    err = OL.rel_err_rows(y, OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up, hd_o))
    assert np.all(err <= TOL), err.max()


def test_linear_prefill_whole_and_half_tiles():
    # 2 x 160 GEMM tiles of 256 x 256: on a 256-CU part the first 256 run as
    # whole tiles and the last 64 as 128 half tiles; rows 300..511 of the
    # second row tile are past m.  All weight rows are checked.
    torch = require_gpu()
    n, k, m = 40960, 256, 300
    enc, r = _oracle_codes_on_device(torch, n, k, 2.0, 3, seed=404)
    x_dev, x64 = to_device_x(synth.activations_f32(404, 0, m, k), "bf16", torch)
    y = _run_linear(torch, enc, x_dev)
    err = OL.rel_err_rows(y, OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
    assert np.all(err <= TOL), err.max()
