"""Parity on every row of workloads 1-4 and on 64 rows of every linear kind
at eight depths of workload 5, against the oracle run over a process pool.

Workloads 1-4: the device generates W, encodes it and runs sdq_linear at the
workload's batch sizes; the oracle re-generates every row on the host,
encodes whole panels, packs them with its own packer and computes the fp64
layer output.  Packed bytes (padding included) and scales must be identical
for every row; the layer output, over all weight rows, within 1e-3 per
activation row.  For the m = 2048 prefill the oracle's output is formed for
256 activation rows spread over every 256-row tile of the GEMM (all weight
rows).  Workload 5: MultiOSR from the measured variances, then 64 seeded rows
of each of the seven linears of eight layers, codes, scales and layer output
at m = 1 and 8."""
import numpy as np
import pytest

import synth
from oracle import layout as LY
from oracle import linear as OL
from tests import oracle_pool as OP
from tests.gpu_common import TOL, require_gpu, to_device_x

pytestmark = pytest.mark.gpu



def _xspec(wl, lin, m, rows=None):
    return OP.XSpec(wl.seed, 100 + m, m, lin.k, wl.x_dtype, rows)


def _check_every_row(torch, wl, lin, osr, batches):
    """Bit-exact codes and scales on all rows and the layer output at every batch in `batches`."""
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    specs = []
    for m in batches:
        rows = None if m <= 64 else list(range(0, m, max(1, m // 256)))[:256]
        specs.append(_xspec(wl, lin, m, rows))
    tasks = OP.panel_tasks(lin.n, 4 * OP.workers(), seed=wl.seed, linear_id=lin.linear_id, k=lin.k,
                           sigma=lin.sigma, outliers=wl.outliers, osr=osr, levels=wl.levels, xs=specs)
    with OP.pool() as pool:
        pending = OP.submit(pool, tasks)
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        enc = P.quantize(w, osr, wl.levels)
        del w
        ys = []
        for s in specs:
            x_dev, _ = to_device_x(synth.activations_f32(s.seed, s.stream, s.m, s.k), s.dtype, torch)
            y = P.linear(x_dev, enc)
            torch.cuda.synchronize()
            y = y.cpu().numpy().astype(np.float64)
            ys.append(y if s.rows is None else y[np.asarray(s.rows)])
            del x_dev
        codes = enc.codes.cpu().numpy()
        scales = enc.scales.cpu().numpy()
        del enc
        torch.cuda.empty_cache()
        results = OP.gather(pending, len(tasks), lin.name)
    L = P.sdq_layout_init(lin.n, lin.k, osr, wl.levels)
    panel_bytes = int(L.n_chunks) * 64 * 16
    assert codes.size == int(L.n_pad) // 64 * panel_bytes
    y_ref = [np.concatenate([res[2][i] for res in results], axis=1) for i in range(len(specs))]
    for t, (packed, sc, _, _) in zip(tasks, results):
        p0, p1 = t.r0 // 64, -(-t.r1 // 64)
        got = codes[p0 * panel_bytes:p1 * panel_bytes]
        if not np.array_equal(got, packed):
            bad = np.flatnonzero(got != packed)
            raise AssertionError(f"{lin.name}: rows {t.r0}..{t.r1}: {bad.size} packed bytes differ "
                                 f"(first at byte {p0 * panel_bytes + bad[0]})")
        assert np.array_equal(scales[t.r0:t.r1].view(np.uint32), sc.view(np.uint32)), (lin.name, t.r0)
    for s, y, yr in zip(specs, ys, y_ref):
        err = OL.rel_err_rows(y, yr)
        assert np.all(err <= TOL), (lin.name, s.m, float(err.max()))


def test_every_row_opt125m_q_proj():
    torch = require_gpu()
    wl = synth.workload(1)
    _check_every_row(torch, wl, wl.linears[0], wl.osr, wl.batches)


def test_every_row_llama7b_down_proj():
    torch = require_gpu()
    wl = synth.workload(2)
    _check_every_row(torch, wl, wl.linears[0], wl.osr, wl.batches)


@pytest.mark.parametrize("idx", range(7))
def test_every_row_llama7b_layer_multiosr(idx):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    wl = synth.workload(3)
    osr = P.sdq_multiosr([lin.sigma ** 2 for lin in wl.linears], [lin.n * lin.k for lin in wl.linears],
                         [lin.layer for lin in wl.linears], *wl.multiosr)
    _check_every_row(torch, wl, wl.linears[idx], float(osr[idx]), wl.batches)


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_every_row_llama70b_decode_and_prefill(idx):
    torch = require_gpu()
    wl = synth.workload(4)
    _check_every_row(torch, wl, wl.linears[idx], wl.osr, wl.batches + wl.prefill)


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
    return var


def _rows_codes(torch, enc, rows):
    """Unpacked codes of `rows` only: their chunks gathered on the device into a
    small buffer in the same panel format, unpacked on the host."""
    L = enc.layout
    nc = int(L.n_chunks)
    dev = enc.codes.view(-1, nc, 64, 16)
    r = torch.from_numpy(rows).cuda()
    picked = dev[r // 64, :, r % 64, :]
    n_small = (len(rows) + 63) // 64 * 64
    small = torch.zeros((n_small // 64, nc, 64, 16), dtype=torch.uint8, device="cuda")
    j = torch.arange(len(rows), device="cuda")
    small[j // 64, :, j % 64, :] = picked
    return LY.unpack(small.cpu().numpy().reshape(-1), n_small, int(L.k_up), int(L.levels))[:len(rows)]


LAYERS = (0, 11, 22, 33, 44, 55, 66, 79)


def test_llama70b_stack_64_rows_of_every_linear_kind_at_eight_depths():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    from synth import gpu as SG
    wl = synth.workload(5)
    var = _stack_variances(torch, wl)
    osr = P.sdq_multiosr(var, [lin.n * lin.k for lin in wl.linears], [lin.layer for lin in wl.linears],
                         *wl.multiosr)
    picks = []
    for layer in LAYERS:
        for j in range(7):
            lin = wl.linears[7 * layer + j]
            rng = np.random.default_rng(lin.linear_id + 7)
            rows = np.unique(np.concatenate([[0, lin.n - 1], rng.choice(lin.n, 62, replace=False)]))
            while rows.size < 64:
                rows = np.unique(np.concatenate([rows, rng.choice(lin.n, 64 - rows.size, replace=False)]))
            picks.append((lin, float(osr[7 * layer + j]), rows))
    tasks = [OP.Task(seed=wl.seed, linear_id=lin.linear_id, n=lin.n, k=lin.k, sigma=lin.sigma,
                     outliers=wl.outliers, r0=0, r1=0, osr=o, levels=wl.levels, rows=rows.tolist(),
                     xs=[OP.XSpec(wl.seed, 200 + m, m, lin.k, wl.x_dtype) for m in wl.batches])
             for lin, o, rows in picks]
    with OP.pool() as pool:
        pending = OP.submit(pool, tasks)
        got = []
        xs = {}
        for lin, o, rows in picks:
            w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
            enc = P.quantize(w, o, wl.levels)
            del w
            ys = []
            for m in wl.batches:
                if (m, lin.k) not in xs:
                    xs[(m, lin.k)] = to_device_x(synth.activations_f32(wl.seed, 200 + m, m, lin.k), wl.x_dtype,
                                                 torch)[0]
                y = P.linear(xs[(m, lin.k)], enc)
                ys.append(y[:, torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64))
            sc = enc.scales[torch.from_numpy(rows).cuda()].cpu().numpy()
            got.append((_rows_codes(torch, enc, rows), sc, ys))
            del enc
            torch.cuda.empty_cache()
        results = OP.gather(pending, len(tasks), "70B stack rows")
    for (lin, o, rows), (codes, sc, ys), (_, ref_sc, ref_ys, ref_codes) in zip(picks, got, results):
        assert np.array_equal(codes, ref_codes), (lin.name, lin.layer)
        assert np.array_equal(sc.view(np.uint32), ref_sc.view(np.uint32)), (lin.name, lin.layer)
        for m, y, yr in zip(wl.batches, ys, ref_ys):
            err = OL.rel_err_rows(y, yr)
            assert np.all(err <= TOL), (lin.name, lin.layer, m, float(err.max()))
