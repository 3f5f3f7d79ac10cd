"""Helpers shared by the GPU parity tests: run the HIP library through its
binding and the oracle on the same seeded inputs."""
import numpy as np

import oracle
from oracle import layout as LY


def require_gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    return torch


def gpu_encode(w_dev, osr, levels, block=256, check=True):
    import paper_2510_03275_amd as P
    enc = P.quantize(w_dev, osr, levels, block, check=check)
    return enc


def host_bytes(t):
    return t.detach().cpu().numpy()


def oracle_packed(w_np, osr, levels, block=256):
    r = oracle.encode(w_np, osr, levels, block)
    return LY.pack(r.codes, levels), r


def to_device_x(x32, dtype, torch):
    """Activation storage cast on the host (numpy / torch CPU), then upload."""
    import synth
    if dtype == "f16":
        xh = synth.to_f16(x32)
        return torch.from_numpy(xh).cuda(), xh.astype(np.float64)
    if dtype == "bf16":
        bits = synth.to_bf16_bits(x32)
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
        return t, synth.bf16_bits_to_f32(bits).astype(np.float64)
    return torch.from_numpy(x32).cuda(), x32.astype(np.float64)


TOL = 1e-3   # max relative error of sdq_linear against the fp64 definition, per activation row
