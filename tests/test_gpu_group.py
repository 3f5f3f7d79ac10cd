"""GPU parity of sdq_linear_group (one expansion and one contraction launch for
several linears that read the same input) against the fp64 oracle and against
each linear's own sdq_linear."""
import numpy as np
import pytest

import oracle
import synth
from oracle import layout as LY
from oracle import linear as OL
from tests.gpu_common import TOL, require_gpu, to_device_x

pytestmark = pytest.mark.gpu


def _members(torch, ns, k, osr, levels, seed, packing=0):
    import paper_2510_03275_amd as P
    out = []
    for j, n in enumerate(ns):
        w = synth.weight_rows(seed, 10 + j, n, k, 0.02, True)
        r = oracle.encode(w, osr, levels)
        L = P.sdq_layout_init(n, k, osr, levels)
        if packing:
            P.sdq_layout_set_packing(L, packing)
            buf = LY.pack_base3(r.codes) if n else np.zeros(0, np.uint8)
        else:
            buf = LY.pack(r.codes, levels) if n else np.zeros(0, np.uint8)
        codes = torch.from_numpy(buf).cuda() if buf.size else torch.zeros(16, dtype=torch.uint8, device="cuda")
        scales = torch.from_numpy(r.scales).cuda() if n else torch.zeros(1, dtype=torch.float32, device="cuda")
        out.append((P.Encoded(L, codes, scales), r))
    return out


@pytest.mark.parametrize("ns,k,osr,levels,packing", [
    ((300, 64, 130), 1024, 2.0, 3, 0),          # q/k/v-like: three row counts, one under a panel
    ((600, 600), 2048, 1.5, 2, 0),              # gate/up-like, binary
    ((520, 0, 200, 64), 768, 2.5, 3, 0),        # four slots, one empty linear
    ((300, 190), 1024, 2.0, 3, 1),              # base-3 codes
])
@pytest.mark.parametrize("m", [1, 3, 16, 40])
def test_group_matches_oracle_and_single_calls(ns, k, osr, levels, packing, m):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    mem = _members(torch, ns, k, osr, levels, seed=sum(ns) + k + m, packing=packing)
    encs = [e for e, _ in mem]
    x_dev, x64 = to_device_x(synth.activations_f32(70 + m, 0, m, k), "f16", torch)
    ys = [torch.full((m, e.layout.n), float("nan"), dtype=torch.float32, device="cuda") for e in encs]
    grp = P.LinearGroup(encs, ys)
    ws = torch.empty(max(1, P.sdq_linear_group_workspace_bytes([e.layout for e in encs], m)),
                     dtype=torch.uint8, device="cuda")
    P.sdq_linear_group(x_dev, grp, ws)
    torch.cuda.synchronize()
    for (enc, r), y in zip(mem, ys):
        if enc.layout.n == 0:
            continue
        got = y.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(got))
        err = OL.rel_err_rows(got, OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up))
        assert np.all(err <= TOL), (enc.layout.n, m, err.max())
        single = P.linear(x_dev, enc)
        torch.cuda.synchronize()
        assert torch.max(torch.abs(single - y)).item() <= 1e-6 * torch.max(torch.abs(single)).item()
    # accumulate: y_j += x W_j^T
    y0 = [y.clone() for y in ys]
    P.sdq_linear_group(x_dev, grp, ws, accumulate=True)
    torch.cuda.synchronize()
    for y, base in zip(ys, y0):
        if y.numel():
            assert torch.max(torch.abs(y - 2 * base)).item() <= 1e-5 * torch.max(torch.abs(base)).item()


def test_group_rejects_mismatched_layouts():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    a = P.sdq_layout_init(64, 512, 2.0, 3)
    b = P.sdq_layout_init(64, 512, 2.5, 3)
    assert P.sdq_linear_group_workspace_bytes([a, b], 1) == 0
    encs = [P.Encoded(L, torch.zeros(P.sdq_codes_bytes(L), dtype=torch.uint8, device="cuda"),
                      torch.zeros(64, dtype=torch.float32, device="cuda")) for L in (a, b)]
    ys = [torch.zeros((1, 64), dtype=torch.float32, device="cuda") for _ in encs]
    x = torch.zeros((1, 512), dtype=torch.float16, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    with pytest.raises(P.SdqError) as ei:
        P.sdq_linear_group(x, P.LinearGroup(encs, ys), ws)
    assert ei.value.status == -1


@pytest.mark.parametrize("m", [1, 8, 33])
def test_group_expanded_matches_the_whole_call(m):
    # sdq_expand_activations once, then the group's contraction alone.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    mem = _members(torch, (260, 64, 64), 1024, 2.0, 3, seed=5 + m)
    encs = [e for e, _ in mem]
    x_dev, _ = to_device_x(synth.activations_f32(90 + m, 0, m, 1024), "f16", torch)
    ys = [torch.empty((m, e.layout.n), dtype=torch.float32, device="cuda") for e in encs]
    ys2 = [torch.empty_like(y) for y in ys]
    ws = torch.empty(P.sdq_linear_group_workspace_bytes([e.layout for e in encs], m), dtype=torch.uint8,
                     device="cuda")
    P.sdq_linear_group(x_dev, P.LinearGroup(encs, ys), ws)
    ws2 = torch.empty_like(ws)
    P.sdq_expand_activations(x_dev, encs[0].layout, ws2)
    P.sdq_linear_group_expanded(m, P.LinearGroup(encs, ys2), ws2)
    torch.cuda.synchronize()
    for y, y2 in zip(ys, ys2):
        assert torch.max(torch.abs(y - y2)).item() <= 1e-6 * torch.max(torch.abs(y)).item()
