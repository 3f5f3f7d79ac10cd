"""The 80-layer LLaMA-70B stack (560 linears, MultiOSR at a 2.5 mean OSR,
ternary codes): measured weight variances on the device, the allocation
against the oracle's and its invariants, and bit-exact codes plus linear
parity on seeded row samples of linears from different depths."""
import numpy as np
import pytest

import oracle
import synth
from oracle import layout as LY
from oracle import linear as OL
from oracle import multiosr as OM
from tests.gpu_common import TOL, gpu_encode, require_gpu, to_device_x

pytestmark = pytest.mark.gpu


def _stack_variances(torch, wl):
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    var = []
    out = torch.zeros(2, dtype=torch.float64, device="cuda")
    ws = None
    for lin in wl.linears:
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        need = P.sdq_moments_workspace_bytes(w.numel())
        if ws is None or ws.numel() < need:
            ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        P.sdq_weight_moments(w, out, ws)
        var.append(float(out[1].item()))
        del w
    return np.array(var)


def _sampled_rows_codes(torch, enc, rows):
    """Unpacked codes of `rows` only: gather their chunks on the device into a
    small buffer in the same panel format, then unpack it on the host."""
    L = enc.layout
    nc = int(L.n_chunks)
    dev = enc.codes.view(-1, nc, 64, 16)
    r = torch.from_numpy(rows).cuda()
    picked = dev[r // 64, :, r % 64, :]                       # [len, n_chunks, 16]
    n_small = (len(rows) + 63) // 64 * 64
    small = torch.zeros((n_small // 64, nc, 64, 16), dtype=torch.uint8, device="cuda")
    j = torch.arange(len(rows), device="cuda")
    small[j // 64, :, j % 64, :] = picked
    got = LY.unpack(small.cpu().numpy().reshape(-1), n_small, int(L.k_up), int(L.levels))
    return got[: len(rows)]


def test_llama70b_stack_multiosr_and_sampled_parity():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    wl = synth.workload(5)
    var = _stack_variances(torch, wl)
    # measured variances track the generator's (rows are long: relative 1e-2)
    sig2 = np.array([lin.sigma ** 2 for lin in wl.linears])
    assert np.all(np.abs(var / sig2 - 1.0) < 2e-2)
    nparams = [lin.n * lin.k for lin in wl.linears]
    layers = [lin.layer for lin in wl.linears]
    target, lo, hi = wl.multiosr
    osr = P.sdq_multiosr(var, nparams, layers, target, lo, hi)
    ref = OM.multiosr(var, nparams, layers, target, lo, hi)
    assert np.array_equal(np.asarray(osr), np.asarray(ref))
    o = np.asarray(osr)
    w = np.asarray(nparams, dtype=np.float64)
    mean = float((o * w).sum() / w.sum())
    assert lo <= o.min() and o.max() <= hi
    assert np.allclose(o * 8, np.round(o * 8))
    assert target - 0.125 * w.max() / w.sum() < mean <= target + 1e-12
    # variance rises with depth, so a given projection's OSR never rises with depth
    per_kind = o.reshape(80, 7)
    assert np.all(np.diff(per_kind, axis=0) <= 1e-12)
    # sampled parity on linears from different depths
    rng = np.random.default_rng(5)
    for idx in (0, 7 * 26 + 1, 7 * 53 + 6, 7 * 79 + 5):
        lin = wl.linears[idx]
        w_dev = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        enc = gpu_encode(w_dev, float(o[idx]), wl.levels)
        del w_dev
        rows = np.unique(np.concatenate([[0, lin.n - 1], rng.choice(lin.n, 14, replace=False)]))
        w_rows = synth.weight_rows(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers, rows=rows)
        r = oracle.encode(w_rows, float(o[idx]), wl.levels)
        assert np.array_equal(_sampled_rows_codes(torch, enc, rows), r.codes), lin.name
        sc = enc.scales[torch.from_numpy(rows).cuda()].cpu().numpy()
        assert np.array_equal(sc.view(np.uint32), r.scales.view(np.uint32)), lin.name
        for m in wl.batches:
            x32 = SG.activations_gpu(wl.seed, 200 + m, m, lin.k).cpu().numpy()
            x_dev, x64 = to_device_x(x32, wl.x_dtype, torch)
            y = P.linear(x_dev, enc)
            torch.cuda.synchronize()
            y_s = y[:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
            err = OL.rel_err_rows(y_s, OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
            assert np.all(err <= TOL), (lin.name, m, err.max())
        del enc
        torch.cuda.empty_cache()
