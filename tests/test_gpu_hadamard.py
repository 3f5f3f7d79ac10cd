"""GPU parity of the Had choices (Sylvester, sign-randomised diag(s) H / sqrt(B),
none) against the oracle: bit-exact codes and scales from sdq_quantize, and
sdq_linear within the 1e-3 tolerance on the decode (table and integer-MFMA)
and prefill paths."""
import numpy as np
import pytest

import oracle
import synth
from oracle import layout as LY
from oracle import linear as OL
from tests.gpu_common import TOL, host_bytes, require_gpu, to_device_x

pytestmark = pytest.mark.gpu

SHAPES = [
    # (n, k, osr, levels, block)
    (100, 768, 2.0, 3, 256),
    (130, 512, 1.5, 2, 256),
    (70, 512, 1.625, 3, 256),     # blocks start inside chunks
    (33, 256, 1.0, 3, 256),       # M = B
    (64, 512, 2.5, 2, 128),
    (50, 256, 1.5, 3, 64),
]


def _signs(mode, block, seed):
    return synth.hadamard_signs(seed, block) if mode == 2 else None


@pytest.mark.parametrize("mode", [0, 2])
@pytest.mark.parametrize("n,k,osr,levels,block", SHAPES)
def test_encoder_bit_exact_for_each_had(mode, n, k, osr, levels, block):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    s = _signs(mode, block, n + k)
    w = synth.weight_rows(60 + n, 3, n, k, 0.02, True)
    enc = P.quantize(torch.from_numpy(w).cuda(), osr, levels, block, hadamard=mode, signs=s)
    r = oracle.encode(w, osr, levels, block, mode, s)
    assert np.array_equal(host_bytes(enc.scales).view(np.uint32), r.scales.view(np.uint32))
    assert np.array_equal(host_bytes(enc.codes), LY.pack(r.codes, levels))


@pytest.mark.parametrize("mode", [0, 2])
@pytest.mark.parametrize("n,k,osr,levels,block", SHAPES[:3] + SHAPES[4:])
def test_linear_for_each_had(mode, n, k, osr, levels, block):
    # Codes from the oracle (so the linear is checked on its own), m covering
    # the one-row decode (1), the integer-MFMA decode (3, 16) and prefill (40).
    torch = require_gpu()
    import paper_2510_03275_amd as P
    s = _signs(mode, block, 7 * n)
    w = synth.weight_rows(80 + n, 4, n, k, 0.02, True)
    r = oracle.encode(w, osr, levels, block, mode, s)
    L = P.sdq_layout_init(n, k, osr, levels, block)
    P.sdq_layout_set_hadamard(L, mode, s)
    enc = P.Encoded(L, torch.from_numpy(LY.pack(r.codes, levels)).cuda(), torch.from_numpy(r.scales).cuda())
    for m in (1, 3, 16, 40):
        x_dev, x64 = to_device_x(synth.activations_f32(5, m, m, k), "f16", torch)
        y = P.linear(x_dev, enc)
        torch.cuda.synchronize()
        ref = OL.linear_fp64(x64, r.codes, r.scales, block, r.m_up, mode, s)
        err = OL.rel_err_rows(y.cpu().numpy().astype(np.float64), ref)
        assert np.all(err <= TOL), (mode, m, err.max())


def test_two_had_choices_on_one_block_and_m_keep_their_own_tables():
    # Same (B, M) under the three choices, interleaved calls: each layer is
    # evaluated with its own E = Had D^T.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    n, k, osr, levels = 96, 512, 2.0, 3
    w = synth.weight_rows(91, 5, n, k, 0.02, True)
    layers = []
    for mode in (1, 2, 0):
        s = _signs(mode, 256, 91)
        enc = P.quantize(torch.from_numpy(w).cuda(), osr, levels, 256, hadamard=mode, signs=s)
        layers.append((mode, s, enc, oracle.encode(w, osr, levels, 256, mode, s)))
    assert not np.array_equal(host_bytes(layers[0][2].codes), host_bytes(layers[1][2].codes))
    x_dev, x64 = to_device_x(synth.activations_f32(6, 0, 8, k), "f16", torch)
    for _ in range(2):
        for mode, s, enc, r in layers:
            y = P.linear(x_dev, enc)
            torch.cuda.synchronize()
            ref = OL.linear_fp64(x64, r.codes, r.scales, 256, r.m_up, mode, s)
            assert np.all(OL.rel_err_rows(y.cpu().numpy().astype(np.float64), ref) <= TOL), mode
