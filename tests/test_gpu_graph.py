"""sdq_linear and sdq_quantize captured in a HIP graph (through PyTorch) give
the eager result on every replay, with eager work interleaved (sdq_quantize
bitwise; sdq_linear up to the rounding order of split-K atomics)."""
import numpy as np
import pytest

import synth
from tests.gpu_common import require_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("m", [1, 8, 100])
def test_linear_graph_replays_match_eager(m):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    w = torch.from_numpy(synth.weight_rows(1, 0, 300, 1024, 0.02, True)).cuda()
    enc = P.quantize(w, 2.0, 3)
    x = torch.from_numpy(synth.to_f16(synth.activations_f32(2, 0, m, 1024))).cuda()
    ws = torch.empty(P.sdq_linear_workspace_bytes(enc.layout, m), dtype=torch.uint8, device="cuda")
    y_eager = P.linear(x, enc, workspace=ws).clone()
    y = torch.zeros_like(y_eager)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.sdq_linear(x, enc.codes, enc.scales, enc.layout, y, ws)
    scale = torch.max(torch.abs(y_eager)).item()
    for rep in range(4):
        y.fill_(1e30)       # the graph itself must reset whatever it accumulates into
        g.replay()
        torch.cuda.synchronize()
        # split-K decode accumulates with fp32 atomics: equal up to rounding order
        assert torch.max(torch.abs(y - y_eager)).item() <= 1e-6 * scale, rep
        P.linear(x * 0.5, enc, workspace=ws)       # eager work on the same workspace
        torch.cuda.synchronize()


def test_quantize_graph_replays_match_eager():
    torch = require_gpu()
    import paper_2510_03275_amd as P
    w = torch.from_numpy(synth.weight_rows(3, 0, 200, 768, 0.02, True)).cuda()
    ref = P.quantize(w, 1.5, 2)
    L = ref.layout
    codes = torch.zeros_like(ref.codes)
    scales = torch.zeros_like(ref.scales)
    ws = torch.empty(P.sdq_quantize_workspace_bytes(L), dtype=torch.uint8, device="cuda")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.sdq_quantize(w, L, codes, scales, ws)
    for rep in range(3):
        codes.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(codes, ref.codes) and torch.equal(scales, ref.scales), rep
        P.quantize(w * 2.0, 1.5, 2)
        torch.cuda.synchronize()
