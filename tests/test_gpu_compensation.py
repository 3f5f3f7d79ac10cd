"""GPU parity of the block compensation (Algorithm 1's block loop) against the
oracle: the Hessian, the Cholesky factor of its damped inverse, and the
compensated codes."""
import numpy as np
import pytest

import oracle
import synth
from oracle import compensation as OC
from oracle import layout as LY
from oracle import linear as OL
from tests.gpu_common import host_bytes, require_gpu

pytestmark = pytest.mark.gpu


def _calib_x(seed, m, k, rank=16):
    """Correlated calibration activations (shared low-rank part plus noise, uneven
    channel scales), drawn from the seeded generator: fp32 [m, k]."""
    g = synth.activations_f32(seed, 1, k, rank).astype(np.float64)
    ch = np.exp(0.5 * synth.activations_f32(seed, 2, 1, k).astype(np.float64))[0]
    z = synth.activations_f32(seed, 3, m, rank).astype(np.float64)
    e = synth.activations_f32(seed, 4, m, k).astype(np.float64)
    return ((z @ g.T * 0.9 + e) * ch).astype(np.float32)


@pytest.mark.parametrize("m,k", [(300, 192), (1000, 1024)])
def test_hessian_accumulates_twice_the_gram_matrix(m, k):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    x = _calib_x(m + k, m, k)
    h = torch.zeros((k, k), dtype=torch.float64, device="cuda")
    xd = torch.from_numpy(x).cuda()
    P.sdq_hessian_accumulate(xd[: m // 2].contiguous(), h)
    P.sdq_hessian_accumulate(xd[m // 2:].contiguous(), h)
    want = OC.hessian_fp64(x)
    got = h.cpu().numpy()
    assert np.max(np.abs(got - want)) <= 1e-12 * np.max(np.abs(want))


@pytest.mark.parametrize("m,k", [(300, 100), (257, 320)])
def test_hessian_adds_to_any_starting_matrix(m, k):
    # Only tiles on or below the diagonal are multiplied, each added at its own
    # and its transposed position: a non-symmetric starting H keeps both triangles.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    x = _calib_x(3 * k, m, k)
    h0 = np.random.default_rng(k).standard_normal((k, k))
    h = torch.from_numpy(h0.copy()).cuda()
    P.sdq_hessian_accumulate(torch.from_numpy(x).cuda(), h)
    want = h0 + OC.hessian_fp64(x)
    assert np.max(np.abs(h.cpu().numpy() - want)) <= 1e-12 * np.max(np.abs(want))


@pytest.mark.parametrize("k", [64, 128, 320, 1024, 4096])
def test_factor_matches_oracle(k):
    # k = 4096: the size of the compensation bench's factor.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    x = _calib_x(k, 4 * k if k <= 1024 else k + 512, k)
    h = OC.hessian_fp64(x)
    lam = 0.01 * np.mean(np.diag(h))
    u = P.hessian_factor(torch.from_numpy(h).cuda(), lam).cpu().numpy()
    want = OC.inverse_cholesky_upper(h, lam)
    assert np.array_equal(u, np.triu(u))
    assert np.max(np.abs(u - want)) <= 1e-9 * np.max(np.abs(want))
    assert np.max(np.abs(u.T @ u @ (h + lam * np.eye(k)) - np.eye(k))) < 1e-8


@pytest.mark.parametrize("bad", [None, 0, 70, 130])
def test_factor_reports_an_indefinite_matrix(bad):
    # The pivot that fails lies in the first diagonal block (factored on its
    # own) or in a later one (factored by the trailing update producing it).
    # The factor works on the index-reversed matrix, so entry bad of the
    # reversed diagonal is entry k - 1 - bad of H.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    k = 192
    if bad is None:
        h = -torch.eye(k, dtype=torch.float64, device="cuda")
    else:
        h = torch.eye(k, dtype=torch.float64, device="cuda")
        h[k - 1 - bad, k - 1 - bad] = -1.0
    with pytest.raises(P.SdqError) as ei:
        P.hessian_factor(h, 0.0)
    assert ei.value.status == -10
    ok = torch.eye(k, dtype=torch.float64, device="cuda")
    u = P.hessian_factor(ok, 0.0).cpu().numpy()   # the flag does not stick
    assert np.array_equal(u, np.eye(k))


CASES = [
    # (n, k, osr, levels, block)
    (96, 512, 2.0, 3, 256),
    (130, 768, 1.5, 2, 256),
    (64, 512, 2.25, 3, 128),
    (70, 256, 1.5, 3, 64),
]


@pytest.mark.parametrize("update", [0, 1])
@pytest.mark.parametrize("n,k,osr,levels,block", CASES)
def test_compensated_codes_match_oracle(n, k, osr, levels, block, update):
    # Same U on both sides (the oracle's).  Every compensation step is fp64 on
    # both sides but summed in different orders, so a block handed to the fp32
    # encoder can differ in the last fp32 bit where an fp64 value sits at a
    # rounding boundary (about 1e-5 per element per block): the scales and
    # block 0 are bit-exact, nearly every row is, and rows that differ do so
    # from a later block on; the fit to the calibration set agrees.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    w = synth.weight_rows(n + k, 6, n, k, 0.02, True)
    x = _calib_x(7 * k, 4 * k, k)
    h = OC.hessian_fp64(x)
    u = OC.inverse_cholesky_upper(h, 0.01 * np.mean(np.diag(h)))
    enc = P.quantize_compensated(torch.from_numpy(w).cuda(), osr, levels, torch.from_numpy(u).cuda(), block,
                                 update=update)
    r = OC.encode_compensated(w, osr, levels, block, u, update=update)
    got = LY.unpack(host_bytes(enc.codes), n, r.codes.shape[1], levels)
    assert np.array_equal(host_bytes(enc.scales).view(np.uint32), r.scales.view(np.uint32))
    assert np.array_equal(got[:, : r.m_up], r.codes[:, : r.m_up])
    same = np.all(got == r.codes, axis=1)
    assert same.mean() >= 0.95, same.mean()
    y = x.astype(np.float64) @ w.astype(np.float64).T
    fit = []
    for c in (got, r.codes):
        yq = x.astype(np.float64) @ OL.reconstruct_fp64(c, r.scales, block, r.m_up).T
        fit.append(np.linalg.norm(yq - y) / np.linalg.norm(y))
    assert abs(fit[0] - fit[1]) <= 0.01 * fit[1], fit
    plain = oracle.encode(w, osr, levels, block)
    yq = x.astype(np.float64) @ OL.reconstruct_fp64(plain.codes, plain.scales, block, plain.m_up).T
    assert fit[1] < np.linalg.norm(yq - y) / np.linalg.norm(y)


def test_device_pipeline_end_to_end():
    # Hessian, factor and compensated encoding all on the device, against the
    # oracle's pipeline on the same seeded calibration rows.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    n, k = 128, 1024
    w = synth.weight_rows(3, 9, n, k, 0.02, True)
    x = _calib_x(11, 4096, k)
    h = torch.zeros((k, k), dtype=torch.float64, device="cuda")
    P.sdq_hessian_accumulate(torch.from_numpy(x).cuda(), h)
    lam = 0.01 * float(torch.mean(torch.diagonal(h)).item())
    u = P.hessian_factor(h, lam)
    enc = P.quantize_compensated(torch.from_numpy(w).cuda(), 2.0, 3, u)
    hh = OC.hessian_fp64(x)
    r = OC.encode_compensated(w, 2.0, 3, 256, OC.inverse_cholesky_upper(hh, 0.01 * np.mean(np.diag(hh))))
    got = LY.unpack(host_bytes(enc.codes), n, r.codes.shape[1], 3)
    assert np.array_equal(got[:, :512], r.codes[:, :512])
    assert np.all(got == r.codes, axis=1).mean() >= 0.95


@pytest.mark.parametrize("levels", [2, 3])
def test_diagonal_hessian_gives_the_plain_codes(levels):
    torch = require_gpu()
    import paper_2510_03275_amd as P
    n, k = 80, 768
    w = synth.weight_rows(5, 10, n, k, 0.02, True)
    d = 0.5 + np.arange(k) / k
    u = torch.from_numpy(np.diag(1.0 / np.sqrt(d))).cuda()
    enc = P.quantize_compensated(torch.from_numpy(w).cuda(), 2.0, levels, u)
    plain = P.quantize(torch.from_numpy(w).cuda(), 2.0, levels)
    assert torch.equal(enc.codes, plain.codes) and torch.equal(enc.scales, plain.scales)


@pytest.mark.parametrize("update", [0, 1])
@pytest.mark.parametrize("levels", [2, 3])
def test_compensated_codes_bit_exact_on_dyadic_inputs(levels, update):
    # Dyadic W and U at OSR 1 (tests/dyadic_inputs.py): no fp64 step of the
    # block loop rounds on either side (certified on the CPU by
    # test_dyadic_inputs_keep_the_block_loop_exact), so every row's codes must
    # be identical, whatever order the device sums in.
    torch = require_gpu()
    import paper_2510_03275_amd as P
    from tests.dyadic_inputs import dyadic_case
    n, k, b = 70, 1024, 256
    w, u = dyadic_case(n, k, b, seed=3 + levels)
    enc = P.quantize_compensated(torch.from_numpy(w).cuda(), 1.0, levels, torch.from_numpy(u).cuda(), b,
                                 update=update)
    r = OC.encode_compensated(w, 1.0, levels, b, u, update=update)
    assert np.array_equal(host_bytes(enc.scales).view(np.uint32), r.scales.view(np.uint32))
    assert np.array_equal(host_bytes(enc.codes), LY.pack(r.codes, levels))
    # the compensation did act: the codes differ from the plain encoding
    plain = oracle.encode(w, 1.0, levels, b)
    assert np.mean(plain.codes != r.codes) > 0.01
