"""GPU parity of base-3 packed ternary codes (five codes per byte, 1.6 bits per
weight of Eq. 14): the encoder's bytes against the oracle packer, and
sdq_linear on base-3 codes (read directly by the one-row table GEMV, unpacked
to 2-bit fields by every other path) against the fp64 definition."""
import numpy as np
import pytest

import oracle
import synth
from oracle import compensation as OC
from oracle import layout as LY
from oracle import linear as OL
from tests.gpu_common import TOL, host_bytes, require_gpu, to_device_x

pytestmark = pytest.mark.gpu


def _base3_layout(n, k, osr, block=256):
    import paper_2510_03275_amd as P
    return P.sdq_layout_set_packing(P.sdq_layout_init(n, k, osr, 3, block), P.SDQ_PACK_BASE3)


ENC = [
    # (n, k, osr, block): ragged panels, K_up a multiple of 80 or not, every block size
    (1, 256, 2.0, 256),
    (100, 768, 2.0, 256),       # K_up = 1536: 19.2 chunks
    (64, 1024, 2.5, 256),       # K_up = 2560 = 32 chunks of 80
    (70, 512, 1.625, 256),      # M = 416
    (33, 256, 1.0, 256),
    (130, 512, 2.25, 128),
    (50, 256, 1.5, 64),
]


@pytest.mark.parametrize("n,k,osr,block", ENC)
def test_encoder_base3_bytes_bit_exact(n, k, osr, block):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    w = synth.weight_rows(60 + n, 1, n, k, 0.02, True)
    enc = P.quantize(torch.from_numpy(w).cuda(), osr, 3, block, packing=P.SDQ_PACK_BASE3)
    r = oracle.encode(w, osr, 3, block)
    want = LY.pack_base3(r.codes)
    got = host_bytes(enc.codes)
    assert enc.layout.packing == P.SDQ_PACK_BASE3 and got.size == want.size
    assert np.array_equal(host_bytes(enc.scales).view(np.uint32), r.scales.view(np.uint32))
    assert np.array_equal(got, want)


def _oracle_base3_on_device(torch, n, k, osr, seed, block=256):
    """Oracle codes, packed by the oracle's base-3 packer, uploaded."""
    import paper_2510_03275_amd as P
    w = synth.weight_rows(seed, 2, n, k, 0.02, True)
    r = oracle.encode(w, osr, 3, block)
    L = _base3_layout(n, k, osr, block)
    enc = P.Encoded(L, torch.from_numpy(LY.pack_base3(r.codes)).cuda(), torch.from_numpy(r.scales).cuda())
    return enc, r


def _check_linear(torch, enc, r, m, seed, dtype="f16", block=256):
    import paper_2510_03275_amd as P
    x_dev, x64 = to_device_x(synth.activations_f32(seed, 0, m, enc.layout.k), dtype, torch)
    y = P.linear(x_dev, enc)
    torch.cuda.synchronize()
    err = OL.rel_err_rows(y.cpu().numpy().astype(np.float64),
                          OL.linear_fp64(x64, r.codes, r.scales, block, r.m_up))
    assert np.all(err <= TOL), (m, err.max())


@pytest.mark.parametrize("m", [1, 2, 3, 8, 16, 17, 40, 130])
@pytest.mark.parametrize("n,k,osr", [(130, 768, 2.0), (100, 512, 1.625), (200, 1024, 2.5), (33, 256, 1.5)])
def test_linear_base3_matches_oracle(n, k, osr, m):
    torch = require_gpu()
    enc, r = _oracle_base3_on_device(torch, n, k, osr, seed=n + m)
    _check_linear(torch, enc, r, m, seed=m)


@pytest.mark.parametrize("m", [1, 2, 16])
def test_linear_base3_single_output_row(m):
    # One weight row: the per-row error takes its maximum over one output, so
    # this runs the decode sizes only (fp32 tables and exact integer sums,
    # errors near 1e-6 of the output scale; the prefill path's fp16 x_tilde is
    # checked on wider layers above).
    torch = require_gpu()
    enc, r = _oracle_base3_on_device(torch, 1, 256, 1.5, seed=1 + m)
    _check_linear(torch, enc, r, m, seed=m)


@pytest.mark.parametrize("n,k,osr", [(64, 8192, 2.0), (96, 16384, 3.0), (300, 2048, 2.0)])
def test_linear_base3_one_row_every_segment_size(n, k, osr):
    # The table GEMV's K segments of 2, 4 and 8 chunks (several segments per
    # output, added atomically), long rows, and n past one workgroup's panels.
    torch = require_gpu()
    enc, r = _oracle_base3_on_device(torch, n, k, osr, seed=k)
    for dtype in ("f16", "bf16", "f32"):
        _check_linear(torch, enc, r, 1, seed=3, dtype=dtype)


@pytest.mark.parametrize("block,osr", [(128, 2.25), (64, 1.5), (64, 2.5)])
def test_linear_base3_block_sizes(block, osr):
    torch = require_gpu()
    enc, r = _oracle_base3_on_device(torch, 70, 8 * block, osr, seed=block, block=block)
    for m in (1, 4, 24):
        _check_linear(torch, enc, r, m, seed=m, block=block)


@pytest.mark.parametrize("m", [1, 5, 33])
def test_linear_base3_split_entry_points_and_accumulate(m):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    enc, r = _oracle_base3_on_device(torch, 130, 1024, 2.0, seed=m)
    x_dev, x64 = to_device_x(synth.activations_f32(m, 0, m, 1024), "f16", torch)
    ws = torch.empty(P.sdq_linear_workspace_bytes(enc.layout, m), dtype=torch.uint8, device="cuda")
    y0 = torch.from_numpy(synth.activations_f32(9, 0, m, 130)).cuda()
    y = y0.clone()
    P.sdq_expand_activations(x_dev, enc.layout, ws)
    P.sdq_linear_expanded(m, enc.codes, enc.scales, enc.layout, y, ws, accumulate=True)
    torch.cuda.synchronize()
    want = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up)
    got = y.cpu().numpy().astype(np.float64) - y0.cpu().numpy().astype(np.float64)
    assert np.all(OL.rel_err_rows(got, want) <= TOL)


def test_linear_base3_from_the_device_encoder():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    n, k = 192, 1536
    w = synth.weight_rows(17, 3, n, k, 0.02, True)
    enc = P.quantize(torch.from_numpy(w).cuda(), 2.0, 3, packing=P.SDQ_PACK_BASE3)
    r = oracle.encode(w, 2.0, 3, 256)
    for m in (1, 7, 48):
        _check_linear(torch, enc, r, m, seed=m)


def test_compensated_base3_is_the_compensated_fields_repacked():
    # The compensated encoder on a base-3 layout: the same codes as on the
    # 2-bit layout (the same device passes, repacked at the end), and block 0
    # bit-exact against the oracle.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    n, k = 96, 768
    w = synth.weight_rows(5, 6, n, k, 0.02, True)
    rng = np.random.default_rng(8)
    x = (rng.standard_normal((2048, 16)) @ rng.standard_normal((16, k)) + 0.1 * rng.standard_normal((2048, k)))
    h = OC.hessian_fp64(x)
    u = OC.inverse_cholesky_upper(h, 0.01 * np.mean(np.diag(h)))
    u_dev, w_dev = torch.from_numpy(u).cuda(), torch.from_numpy(w).cuda()
    e3 = P.quantize_compensated(w_dev, 2.0, 3, u_dev, packing=P.SDQ_PACK_BASE3)
    e2 = P.quantize_compensated(w_dev, 2.0, 3, u_dev)
    k_up = e2.layout.k_up
    c3 = LY.unpack_base3(host_bytes(e3.codes), n, k_up)
    c2 = LY.unpack(host_bytes(e2.codes), n, k_up, 3)
    assert np.array_equal(c3, c2)
    assert np.array_equal(host_bytes(e3.scales), host_bytes(e2.scales))
    ro = OC.encode_compensated(w, 2.0, 3, 256, u)
    assert np.array_equal(c3[:, :512], ro.codes[:, :512])
