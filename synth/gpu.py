"""Device-side generation of the synthetic inputs (HIP twin in csrc/synth_gen.hip).

Produces bit-for-bit the arrays of ``synth.weight_rows`` / ``synth.activations_f32``
directly in device memory; used for workloads too large to generate on the host.
"""
from __future__ import annotations

import ctypes
import os

from . import OUTLIER_THRESHOLD, normal_factor, stream_base

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsdqsynth.so")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2510_03275_amd/build.py")
    import torch  # noqa: F401  (bind to PyTorch's HIP runtime, loaded first)
    lib = ctypes.CDLL(LIB_PATH)
    lib.synth_normal_f32.restype = ctypes.c_int
    lib.synth_normal_f32.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                     ctypes.c_uint64, ctypes.c_double, ctypes.c_int, ctypes.c_uint64,
                                     ctypes.c_void_p]
    lib.synth_read_probe.restype = ctypes.c_int
    lib.synth_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                     ctypes.c_void_p]
    return lib


_lib = _load()


def _fill(out, rows, cols, row0, base, sigma, outliers):
    import torch
    st = _lib.synth_normal_f32(out.data_ptr(), rows, cols, row0, base, normal_factor(sigma),
                               int(outliers), OUTLIER_THRESHOLD, torch.cuda.current_stream().cuda_stream)
    if st != 0:
        raise RuntimeError(f"synth_normal_f32 failed ({st})")
    return out


def weight_rows_gpu(seed: int, linear_id: int, n: int, k: int, sigma: float, outliers: bool,
                    row0: int = 0, rows: int = None, out=None, device="cuda"):
    """fp32 weight rows [row0, row0 + rows) of the synthetic W (n x k) on the device."""
    import torch
    rows = n - row0 if rows is None else rows
    if out is None:
        out = torch.empty((rows, k), dtype=torch.float32, device=device)
    return _fill(out, rows, k, row0, stream_base(seed, 2 * linear_id), sigma, outliers)


def activations_gpu(seed: int, stream: int, m: int, k: int, device="cuda"):
    """fp32 activations ~N(0, 1) [m x k] on the device (cast to fp16 / bf16 by the caller)."""
    import torch
    out = torch.empty((m, k), dtype=torch.float32, device=device)
    return _fill(out, m, k, 0, stream_base(seed, 2 * stream + 1), 1.0, False)


def read_probe(buf, blocks: int, unroll: int, sink) -> None:
    """One streaming read of the device buffer `buf` (a multiple of 16 bytes)."""
    import torch
    st = _lib.synth_read_probe(buf.data_ptr(), buf.numel() * buf.element_size() // 16, blocks, unroll,
                               sink.data_ptr(), torch.cuda.current_stream().cuda_stream)
    if st != 0:
        raise RuntimeError(f"synth_read_probe failed ({st})")
