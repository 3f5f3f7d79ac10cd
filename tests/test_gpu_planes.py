"""GPU parity of the two front ends of the 2-16-row plane expansion: the fp32
VALU dot products (every activation dtype) and the matrix-core ones (fp16 and
bf16 x: x_b times E as the fp16 pair hi + lo).  Both must meet the 1e-3
budget against the fp64 oracle on every layout kind, including binary codes
without the Hadamard (the layout most sensitive to noise in x_tilde), base-3
codes and blocks of 64 and 128; the matrix-core one (one block per workgroup,
or two sharing the columns of E) is also held to 1e-4."""
import numpy as np
import pytest

import oracle
import synth
from oracle import layout as LY
from oracle import linear as OL
from tests.gpu_common import TOL, require_gpu, to_device_x

pytestmark = pytest.mark.gpu

CASES = [
    # (n, k, osr, levels, block, had, packing)
    (130, 768, 2.0, 3, 256, 1, "fields"),
    (96, 1024, 1.5, 2, 256, 0, "fields"),      # binary, no Hadamard
    (70, 512, 1.625, 3, 256, 1, "fields"),     # blocks start inside chunks
    (64, 512, 2.5, 2, 128, 1, "fields"),
    (50, 256, 1.5, 3, 64, 0, "fields"),
    (100, 512, 1.625, 3, 256, 1, "base3"),
    (80, 768, 2.0, 3, 256, 0, "base3"),
]


def _encoded(torch, n, k, osr, levels, block, had, packing, seed):
    import paper_2510_03275_amd as P
    w = synth.weight_rows(seed, 6, n, k, 0.02, True)
    r = oracle.encode(w, osr, levels, block, had, None)
    L = P.sdq_layout_init(n, k, osr, levels, block)
    P.sdq_layout_set_hadamard(L, had, None)
    if packing == "base3":
        P.sdq_layout_set_packing(L, P.SDQ_PACK_BASE3)
        codes = LY.pack_base3(r.codes)
    else:
        codes = LY.pack(r.codes, levels)
    return P.Encoded(L, torch.from_numpy(codes).cuda(), torch.from_numpy(r.scales).cuda()), r


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("m", [2, 8, 16])
@pytest.mark.parametrize("n,k,osr,levels,block,had,packing", CASES)
def test_plane_front_ends(n, k, osr, levels, block, had, packing, m, dtype, monkeypatch):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    enc, r = _encoded(torch, n, k, osr, levels, block, had, packing, seed=n + k + m)
    x_dev, x64 = to_device_x(synth.activations_f32(n + m, 2, m, k), dtype, torch)
    ref = OL.linear_fp64(x64, r.codes, r.scales, block, r.m_up, had, None)
    errs = {}
    # VALU front end; matrix-core front end with one block per workgroup, and
    # with two blocks sharing E (taken where M is a multiple of the chunk).
    for front, mfma, nbw in (("valu", "0", "1"), ("mfma", "1", "1"), ("mfma2", "1", "2")):
        monkeypatch.setenv("SDQ_PLANES_MFMA", mfma)
        monkeypatch.setenv("SDQ_PLANES_NBW", nbw)
        y = P.linear(x_dev, enc)
        torch.cuda.synchronize()
        errs[front] = OL.rel_err_rows(y.cpu().numpy().astype(np.float64), ref).max()
    print(" ".join(f"{f} {e:.3e}" for f, e in errs.items()))
    assert all(e <= TOL for e in errs.values()), errs
    assert errs["mfma"] <= 1e-4 and errs["mfma2"] <= 1e-4, errs
