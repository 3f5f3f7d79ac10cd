"""ctypes binding of libsdq (include/sdq.h).

Argument marshalling only: every step of the hot path runs in the HIP
kernels of libsdq.so.  PyTorch provides device memory and the current
stream.  The library must have been built in-tree (``build.py``); importing
this module without it raises, and there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsdq.so")

SDQ_OK = 0
SDQ_F16, SDQ_BF16, SDQ_F32 = 0, 1, 2
SDQ_HAD_NONE, SDQ_HAD_SYLVESTER, SDQ_HAD_SIGNED = 0, 1, 2
SDQ_PACK_FIELDS, SDQ_PACK_BASE3 = 0, 1
SDQ_COMP_GPTQ, SDQ_COMP_JOINT = 0, 1

STATUS_NAMES = {
    0: "SDQ_OK", -1: "SDQ_ERR_ARG", -2: "SDQ_ERR_SHAPE", -3: "SDQ_ERR_OSR", -4: "SDQ_ERR_LEVELS",
    -5: "SDQ_ERR_NONFINITE", -6: "SDQ_ERR_WORKSPACE", -7: "SDQ_ERR_HIP", -8: "SDQ_ERR_NOMEM",
    -9: "SDQ_ERR_UNSUPPORTED", -10: "SDQ_ERR_NOT_SPD",
}


class SdqError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class sdq_layout(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64), ("k", ctypes.c_int64),
        ("block", ctypes.c_int32), ("m_up", ctypes.c_int32),
        ("levels", ctypes.c_int32), ("bits", ctypes.c_int32),
        ("nb", ctypes.c_int64), ("k_up", ctypes.c_int64),
        ("n_pad", ctypes.c_int64), ("n_chunks", ctypes.c_int64),
        ("codes_per_chunk", ctypes.c_int32), ("hadamard", ctypes.c_int32),
        ("had_signs", ctypes.c_uint32 * 8),
        ("packing", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]

    def __repr__(self):
        return (f"sdq_layout(n={self.n}, k={self.k}, block={self.block}, m_up={self.m_up}, "
                f"levels={self.levels}, k_up={self.k_up}, n_pad={self.n_pad}, n_chunks={self.n_chunks}, "
                f"hadamard={self.hadamard}, packing={self.packing})")


def hip_runtimes_loaded() -> list:
    """Paths of the HIP runtime libraries mapped into this process."""
    with open("/proc/self/maps") as f:
        return sorted({ln.split()[-1] for ln in f if "libamdhip64" in ln})


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libsdq.so is not built ({LIB_PATH}); run paper_2510_03275_amd/build.py")
    # PyTorch ships its own HIP runtime.  Import it first so that libsdq binds
    # to that already-loaded runtime (same SONAME) instead of pulling in a
    # second one: device pointers and streams must belong to one runtime.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    runtimes = hip_runtimes_loaded()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes are loaded in this process: {runtimes}")
    P = ctypes.c_void_p
    L = ctypes.POINTER(sdq_layout)
    sig = {
        "sdq_layout_init": (ctypes.c_int, [L, ctypes.c_int64, ctypes.c_int64, ctypes.c_double,
                                           ctypes.c_int32, ctypes.c_int32]),
        "sdq_layout_set_hadamard": (ctypes.c_int, [L, ctypes.c_int32, P]),
        "sdq_layout_set_packing": (ctypes.c_int, [L, ctypes.c_int32]),
        "sdq_codes_bytes": (ctypes.c_size_t, [L]),
        "sdq_compression_ratio": (ctypes.c_double, [L]),
        "sdq_quantize_workspace_bytes": (ctypes.c_size_t, [L]),
        "sdq_quantize": (ctypes.c_int, [P, L, P, P, P, ctypes.c_size_t, P]),
        "sdq_quantize_check": (ctypes.c_int, [P, P]),
        "sdq_linear_workspace_bytes": (ctypes.c_size_t, [L, ctypes.c_int64]),
        "sdq_linear": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int64, P, P, L, P, ctypes.c_int32,
                                      P, ctypes.c_size_t, P]),
        "sdq_linear_noalloc": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int64, P, P, L, P, ctypes.c_int32, P]),
        "sdq_linear_group_workspace_bytes": (ctypes.c_size_t, [L, ctypes.c_int32, ctypes.c_int64]),
        "sdq_linear_group": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int64, ctypes.c_int32, P, P, L, P,
                                            ctypes.c_int32, P, ctypes.c_size_t, P]),
        "sdq_linear_group_expanded": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, P, P, L, P, ctypes.c_int32,
                                                     P, ctypes.c_size_t, P]),
        "sdq_expand_activations": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int64, L, P,
                                                  ctypes.c_size_t, P]),
        "sdq_linear_expanded": (ctypes.c_int, [ctypes.c_int64, P, P, L, P, ctypes.c_int32, P,
                                               ctypes.c_size_t, P]),
        "sdq_hessian_accumulate": (ctypes.c_int, [P, ctypes.c_int64, ctypes.c_int64, P, P]),
        "sdq_hessian_factor_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64]),
        "sdq_hessian_factor": (ctypes.c_int, [P, ctypes.c_int64, ctypes.c_double, P, P, ctypes.c_size_t, P]),
        "sdq_hessian_check": (ctypes.c_int, [P, P]),
        "sdq_quantize_compensated_workspace_bytes": (ctypes.c_size_t, [L]),
        "sdq_quantize_compensated": (ctypes.c_int, [P, L, P, ctypes.c_int32, P, P, P, ctypes.c_size_t, P]),
        "sdq_multiosr": (ctypes.c_int, [P, P, P, ctypes.c_int64, ctypes.c_double, ctypes.c_double,
                                        ctypes.c_double, ctypes.c_double, P]),
        "sdq_moments_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64]),
        "sdq_weight_moments": (ctypes.c_int, [P, ctypes.c_int64, P, P, ctypes.c_size_t, P]),
        "sdq_unpack_codes": (ctypes.c_int, [L, P, P]),
        "sdq_upsample_table": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, P]),
        "sdq_prepare": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32]),
        "sdq_prepare_layout": (ctypes.c_int, [L]),
        "sdq_release_tables": (None, []),
        "sdq_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "sdq_last_error": (ctypes.c_char_p, []),
        "sdq_version": (ctypes.c_int32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def lib() -> ctypes.CDLL:
    return _lib


def _check(status: int) -> None:
    if status != SDQ_OK:
        raise SdqError(status, _lib.sdq_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _dtype_code(t) -> int:
    import torch
    return {torch.float16: SDQ_F16, torch.bfloat16: SDQ_BF16, torch.float32: SDQ_F32}[t.dtype]


# ---------------------------------------------------------------------------
# Entry points with the C names (tensors in, status checked).
# ---------------------------------------------------------------------------

def sdq_layout_init(n: int, k: int, osr: float, levels: int, block: int = 256) -> sdq_layout:
    out = sdq_layout()
    _check(_lib.sdq_layout_init(ctypes.byref(out), n, k, float(osr), levels, block))
    return out


def sdq_layout_set_hadamard(layout: sdq_layout, mode: int, signs=None) -> sdq_layout:
    """Select Had for the layout (in place; also returned).  ``signs``: `block`
    values of +-1 for SDQ_HAD_SIGNED."""
    buf = None
    if signs is not None:
        buf = np.ascontiguousarray(signs, dtype=np.int8)
    _check(_lib.sdq_layout_set_hadamard(ctypes.byref(layout), int(mode),
                                        None if buf is None else buf.ctypes.data))
    return layout


def sdq_layout_set_packing(layout: sdq_layout, packing: int) -> sdq_layout:
    """Select the code storage of a ternary layout (in place; also returned)."""
    _check(_lib.sdq_layout_set_packing(ctypes.byref(layout), int(packing)))
    return layout


def sdq_codes_bytes(layout: sdq_layout) -> int:
    return int(_lib.sdq_codes_bytes(ctypes.byref(layout)))


def sdq_compression_ratio(layout: sdq_layout) -> float:
    return float(_lib.sdq_compression_ratio(ctypes.byref(layout)))


def sdq_quantize_workspace_bytes(layout: sdq_layout) -> int:
    return int(_lib.sdq_quantize_workspace_bytes(ctypes.byref(layout)))


def sdq_quantize(w, layout: sdq_layout, codes, scales, workspace, stream=None) -> None:
    _check(_lib.sdq_quantize(_ptr(w), ctypes.byref(layout), _ptr(codes), _ptr(scales),
                             _ptr(workspace), workspace.numel() * workspace.element_size(),
                             _stream(stream)))


def sdq_quantize_check(workspace, stream=None) -> None:
    _check(_lib.sdq_quantize_check(_ptr(workspace), _stream(stream)))


def sdq_linear_workspace_bytes(layout: sdq_layout, m: int) -> int:
    return int(_lib.sdq_linear_workspace_bytes(ctypes.byref(layout), m))


def sdq_linear(x, codes, scales, layout: sdq_layout, y, workspace, stream=None,
               accumulate: bool = False) -> None:
    m = x.shape[0] if x.dim() == 2 else 0
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.sdq_linear(_ptr(x), _dtype_code(x), m, _ptr(codes), _ptr(scales),
                           ctypes.byref(layout), _ptr(y), int(bool(accumulate)), _ptr(workspace),
                           ws_bytes, _stream(stream)))


def _layout_array(layouts):
    arr = (sdq_layout * len(layouts))()
    for i, L in enumerate(layouts):
        arr[i] = L
    return arr


def sdq_linear_group_workspace_bytes(layouts, m: int) -> int:
    return int(_lib.sdq_linear_group_workspace_bytes(_layout_array(layouts), len(layouts), m))


class LinearGroup:
    """The host-side argument arrays of sdq_linear_group for fixed linears and
    outputs, built once (the call then only passes pointers)."""

    def __init__(self, encs, ys):
        n = len(encs)
        self.count = n
        self.layouts = _layout_array([e.layout for e in encs])
        self.codes = (ctypes.c_void_p * n)(*[e.codes.data_ptr() for e in encs])
        self.scales = (ctypes.c_void_p * n)(*[e.scales.data_ptr() for e in encs])
        self.ys = (ctypes.c_void_p * n)(*[y.data_ptr() for y in ys])
        self._keep = (list(encs), list(ys))


def sdq_linear_group(x, group: "LinearGroup", workspace, stream=None, accumulate: bool = False) -> None:
    m = x.shape[0] if x.dim() == 2 else 0
    _check(_lib.sdq_linear_group(_ptr(x), _dtype_code(x), m, group.count, group.codes, group.scales,
                                 group.layouts, group.ys, int(bool(accumulate)), _ptr(workspace),
                                 _nbytes(workspace), _stream(stream)))


def sdq_linear_group_expanded(m: int, group: "LinearGroup", workspace, stream=None,
                              accumulate: bool = False) -> None:
    _check(_lib.sdq_linear_group_expanded(m, group.count, group.codes, group.scales, group.layouts, group.ys,
                                          int(bool(accumulate)), _ptr(workspace), _nbytes(workspace),
                                          _stream(stream)))


SDQ_NOALLOC_SCRATCH_BYTES = 32 << 20     # the library's fixed workspace of sdq_linear_noalloc


def sdq_linear_noalloc(x, codes, scales, layout: sdq_layout, y, stream=None, accumulate: bool = False) -> None:
    m = x.shape[0] if x.dim() == 2 else 0
    _check(_lib.sdq_linear_noalloc(_ptr(x), _dtype_code(x), m, _ptr(codes), _ptr(scales), ctypes.byref(layout),
                                   _ptr(y), int(bool(accumulate)), _stream(stream)))


def sdq_expand_activations(x, layout: sdq_layout, workspace, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.sdq_expand_activations(_ptr(x), _dtype_code(x), x.shape[0], ctypes.byref(layout),
                                       _ptr(workspace), ws_bytes, _stream(stream)))


def sdq_linear_expanded(m: int, codes, scales, layout: sdq_layout, y, workspace, stream=None,
                        accumulate: bool = False) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.sdq_linear_expanded(m, _ptr(codes), _ptr(scales), ctypes.byref(layout), _ptr(y),
                                    int(bool(accumulate)), _ptr(workspace), ws_bytes,
                                    _stream(stream)))


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def sdq_hessian_accumulate(x, h, stream=None) -> None:
    """h += 2 x^T x (x fp32 [m, k] device, h fp64 [k, k] device)."""
    _check(_lib.sdq_hessian_accumulate(_ptr(x), x.shape[0], x.shape[1], _ptr(h), _stream(stream)))


def sdq_hessian_factor_workspace_bytes(k: int) -> int:
    return int(_lib.sdq_hessian_factor_workspace_bytes(k))


def sdq_hessian_factor(h, lam: float, u, workspace, stream=None) -> None:
    _check(_lib.sdq_hessian_factor(_ptr(h), h.shape[0], float(lam), _ptr(u), _ptr(workspace),
                                   _nbytes(workspace), _stream(stream)))


def sdq_hessian_check(workspace, stream=None) -> None:
    _check(_lib.sdq_hessian_check(_ptr(workspace), _stream(stream)))


def sdq_quantize_compensated_workspace_bytes(layout: sdq_layout) -> int:
    return int(_lib.sdq_quantize_compensated_workspace_bytes(ctypes.byref(layout)))


def sdq_quantize_compensated(w, layout: sdq_layout, u, codes, scales, workspace, stream=None,
                             update: int = SDQ_COMP_GPTQ) -> None:
    _check(_lib.sdq_quantize_compensated(_ptr(w), ctypes.byref(layout), _ptr(u), int(update), _ptr(codes),
                                         _ptr(scales), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def sdq_multiosr(var: Sequence[float], nparams: Sequence[int], layer_id: Sequence[int],
                 target: float, lo: float, hi: float, grid: float = 0.125) -> np.ndarray:
    var_a = np.ascontiguousarray(var, dtype=np.float64)
    n_a = np.ascontiguousarray(nparams, dtype=np.int64)
    l_a = np.ascontiguousarray(layer_id, dtype=np.int32)
    out = np.zeros(var_a.size, dtype=np.float64)
    _check(_lib.sdq_multiosr(var_a.ctypes.data, n_a.ctypes.data, l_a.ctypes.data, var_a.size,
                             target, lo, hi, grid, out.ctypes.data))
    return out


def sdq_moments_workspace_bytes(count: int) -> int:
    return int(_lib.sdq_moments_workspace_bytes(count))


def sdq_weight_moments(w, out, workspace, stream=None) -> None:
    _check(_lib.sdq_weight_moments(_ptr(w), w.numel(), _ptr(out), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)))


def sdq_unpack_codes(layout: sdq_layout, codes_host: np.ndarray) -> np.ndarray:
    buf = np.ascontiguousarray(codes_host, dtype=np.uint8)
    if buf.size < sdq_codes_bytes(layout):
        raise ValueError("packed buffer too small")
    out = np.empty((layout.n, layout.k_up), dtype=np.int8)
    _check(_lib.sdq_unpack_codes(ctypes.byref(layout), buf.ctypes.data, out.ctypes.data))
    return out


def sdq_upsample_table(block: int, m_up: int) -> np.ndarray:
    out = np.empty(block * m_up, dtype=np.float32)
    _check(_lib.sdq_upsample_table(block, m_up, out.ctypes.data))
    return out


def sdq_prepare(block: int, m_up: int) -> None:
    _check(_lib.sdq_prepare(block, m_up))


def sdq_prepare_layout(layout: sdq_layout) -> None:
    _check(_lib.sdq_prepare_layout(ctypes.byref(layout)))


def sdq_release_tables() -> None:
    _lib.sdq_release_tables()


def sdq_version() -> int:
    return int(_lib.sdq_version())


# ---------------------------------------------------------------------------
# Convenience: allocate outputs and workspaces with torch (device plumbing).
# ---------------------------------------------------------------------------

@dataclass
class Encoded:
    layout: sdq_layout
    codes: "object"     # torch.uint8 tensor of sdq_codes_bytes bytes
    scales: "object"    # torch.float32 tensor [n]


def quantize(w, osr: float, levels: int, block: int = 256, workspace=None, check: bool = True,
             stream=None, hadamard: int = SDQ_HAD_SYLVESTER, signs=None,
             packing: int = SDQ_PACK_FIELDS) -> Encoded:
    """Encode a device fp32 weight [n, k]; returns codes, scales and layout.

    ``hadamard`` / ``signs`` choose Had (see sdq_layout_set_hadamard);
    ``packing`` the code storage of a ternary layout (SDQ_PACK_BASE3: five
    codes per byte)."""
    import torch
    if w.dtype != torch.float32 or not w.is_cuda or not w.is_contiguous():
        raise ValueError("w must be a contiguous fp32 device tensor")
    layout = sdq_layout_init(w.shape[0], w.shape[1], osr, levels, block)
    if hadamard != SDQ_HAD_SYLVESTER:
        sdq_layout_set_hadamard(layout, hadamard, signs)
    if packing != SDQ_PACK_FIELDS:
        sdq_layout_set_packing(layout, packing)
    codes = torch.empty(sdq_codes_bytes(layout), dtype=torch.uint8, device=w.device)
    scales = torch.empty(layout.n, dtype=torch.float32, device=w.device)
    need = sdq_quantize_workspace_bytes(layout)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=w.device)
    sdq_quantize(w, layout, codes, scales, workspace, stream)
    if check:
        sdq_quantize_check(workspace, stream)
    return Encoded(layout, codes, scales)


def hessian_factor(h, lam: float, check: bool = True, stream=None):
    """U = Cholesky((H + lam I)^-1)^T for a device fp64 [k, k] H; returns U (fp64, device)."""
    import torch
    u = torch.empty_like(h)
    ws = torch.empty(sdq_hessian_factor_workspace_bytes(h.shape[0]), dtype=torch.uint8, device=h.device)
    sdq_hessian_factor(h, lam, u, ws, stream)
    if check:
        sdq_hessian_check(ws, stream)
    return u


def quantize_compensated(w, osr: float, levels: int, u, block: int = 256, check: bool = True,
                         stream=None, hadamard: int = SDQ_HAD_SYLVESTER, signs=None,
                         packing: int = SDQ_PACK_FIELDS, update: int = SDQ_COMP_GPTQ) -> Encoded:
    """Encode a device fp32 weight [n, k] with Algorithm 1's block compensation (u: fp64 [k, k];
    ``update``: SDQ_COMP_GPTQ or SDQ_COMP_JOINT)."""
    import torch
    if w.dtype != torch.float32 or not w.is_cuda or not w.is_contiguous():
        raise ValueError("w must be a contiguous fp32 device tensor")
    if u.dtype != torch.float64 or tuple(u.shape) != (w.shape[1], w.shape[1]) or not u.is_contiguous():
        raise ValueError("u must be a contiguous fp64 device tensor [k, k]")
    layout = sdq_layout_init(w.shape[0], w.shape[1], osr, levels, block)
    if hadamard != SDQ_HAD_SYLVESTER:
        sdq_layout_set_hadamard(layout, hadamard, signs)
    if packing != SDQ_PACK_FIELDS:
        sdq_layout_set_packing(layout, packing)
    codes = torch.empty(sdq_codes_bytes(layout), dtype=torch.uint8, device=w.device)
    scales = torch.empty(layout.n, dtype=torch.float32, device=w.device)
    ws = torch.empty(sdq_quantize_compensated_workspace_bytes(layout), dtype=torch.uint8, device=w.device)
    sdq_quantize_compensated(w, layout, u, codes, scales, ws, stream, update)
    if check:
        sdq_quantize_check(ws, stream)
    return Encoded(layout, codes, scales)


def linear(x, enc: Encoded, workspace=None, out=None, stream=None, accumulate: bool = False):
    """y = x W_hat^T for a device activation [m, k] (fp16, bf16 or fp32).

    With accumulate=True the product is added into `out` (which must be given).
    """
    import torch
    if not x.is_cuda or not x.is_contiguous() or x.dim() != 2 or x.shape[1] != enc.layout.k:
        raise ValueError("x must be a contiguous device tensor [m, k]")
    m = x.shape[0]
    if accumulate and out is None:
        raise ValueError("accumulate=True needs out")
    y = out if out is not None else torch.empty((m, enc.layout.n), dtype=torch.float32, device=x.device)
    need = sdq_linear_workspace_bytes(enc.layout, m)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    sdq_linear(x, enc.codes, enc.scales, enc.layout, y, workspace, stream, accumulate)
    return y
