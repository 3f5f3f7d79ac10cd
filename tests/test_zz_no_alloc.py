"""sdq_linear_noalloc (the entry point for callers that cannot allocate)
against sdq_linear, through the C ABI: two calls in a row on the library's
fixed scratch, the second with a smaller input, on every path (one-row table
GEMV, 2..16-row matrix-core decode, prefill) and with base-3 codes; results
within 1e-6 of sdq_linear's (the split-K decode adds partials with atomics,
so the last bits may differ; unsplit decodes and prefill are identical) and
within the 1e-3 parity bar of the fp64 oracle."""
import numpy as np
import pytest

import oracle
import synth
from oracle import layout as LY
from oracle import linear as OL
from tests.gpu_common import TOL, require_gpu, to_device_x

pytestmark = pytest.mark.gpu


def _encoded(torch, n, k, osr, levels, seed, packing=0):
    import paper_2510_03275_amd as P
    w = synth.weight_rows(seed, 4, n, k, 0.02, True)
    r = oracle.encode(w, osr, levels)
    L = P.sdq_layout_init(n, k, osr, levels)
    if packing:
        P.sdq_layout_set_packing(L, packing)
        buf = LY.pack_base3(r.codes)
    else:
        buf = LY.pack(r.codes, levels)
    return P.Encoded(L, torch.from_numpy(buf).cuda(), torch.from_numpy(r.scales).cuda()), r


@pytest.mark.parametrize("n,k,osr,levels,packing,ms", [
    (256, 8192, 2.0, 3, 0, (1, 1)),           # one row, k_up 16384: matrix-core decode on compact planes
    (768, 4096, 2.0, 3, 0, (1, 1)),           # one row, k_up 8192: table GEMV, split over K
    (700, 2048, 1.5, 2, 0, (8, 3)),           # matrix-core decode
    (600, 1024, 2.5, 3, 0, (130, 40)),        # prefill
    (600, 2048, 2.0, 3, 1, (1, 1)),           # base-3, one row
    (600, 2048, 2.0, 3, 1, (16, 5)),          # base-3, unpacked into the scratch first
])
def test_noalloc_matches_linear_on_two_calls(n, k, osr, levels, packing, ms):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    enc, r = _encoded(torch, n, k, osr, levels, seed=n + k + ms[0], packing=packing)
    P.sdq_prepare_layout(enc.layout)
    for call, m in enumerate(ms):
        x_dev, x64 = to_device_x(synth.activations_f32(60 + call, 0, m, k), "f16", torch)
        y_ref = P.linear(x_dev, enc)
        y = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
        P.sdq_linear_noalloc(x_dev, enc.codes, enc.scales, enc.layout, y)
        torch.cuda.synchronize()
        assert torch.all(torch.isfinite(y)), (call, m)
        diff = torch.max(torch.abs(y - y_ref)).item()
        assert diff <= 1e-6 * torch.max(torch.abs(y_ref)).item(), (call, m, diff)
        err = OL.rel_err_rows(y.cpu().numpy().astype(np.float64),
                              OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
        assert np.all(err <= TOL), (call, m, err.max())
        # accumulate onto y
        y2 = y.clone()
        P.sdq_linear_noalloc(x_dev, enc.codes, enc.scales, enc.layout, y2, accumulate=True)
        torch.cuda.synchronize()
        assert torch.max(torch.abs(y2 - 2 * y_ref)).item() <= 1e-5 * torch.max(torch.abs(y_ref)).item()


def test_noalloc_rejects_oversized_calls_and_missing_tables():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    # prefill of 2048 rows over k_up = 57344: 235 MB of expansion, beyond the scratch
    L = P.sdq_layout_init(64, 28672, 2.0, 3)
    assert P.sdq_linear_workspace_bytes(L, 2048) > P.SDQ_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((2048, 28672), dtype=torch.float16, device="cuda")
    codes = torch.zeros(P.sdq_codes_bytes(L), dtype=torch.uint8, device="cuda")
    scales = torch.zeros(64, dtype=torch.float32, device="cuda")
    y = torch.zeros((2048, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(P.SdqError) as ei:
        P.sdq_linear_noalloc(x, codes, scales, L, y)
    assert ei.value.status == -6
    # a layout whose tables were never built on this device (OSR 2.875, signed Had)
    L2 = P.sdq_layout_init(64, 256, 2.875, 3)
    P.sdq_layout_set_hadamard(L2, P.SDQ_HAD_SIGNED, synth.hadamard_signs(99, 256))
    x2 = torch.zeros((1, 256), dtype=torch.float16, device="cuda")
    c2 = torch.zeros(P.sdq_codes_bytes(L2), dtype=torch.uint8, device="cuda")
    y2 = torch.zeros((1, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(P.SdqError) as ei:
        P.sdq_linear_noalloc(x2, c2, scales, L2, y2)
    assert ei.value.status == -9
    # after sdq_prepare_layout the same call runs (all-zero codes: y = 0)
    P.sdq_prepare_layout(L2)
    y2.fill_(1.0)
    P.sdq_linear_noalloc(x2, c2, scales, L2, y2)
    torch.cuda.synchronize()
    assert torch.count_nonzero(y2).item() == 0
