"""The oracle over a process pool, beside the GPU parity tests (test
infrastructure only).

The pool's processes come from a fork server started before anything in the
test process initialises the GPU (``start`` from the test configuration), so
no worker is a fork of a process holding GPU state.  At most 16 processes:
the host share of one GPU.

A task encodes whole 64-row panels of a synthetic weight (regenerated on the
host from its seed) with the oracle, packs them with the oracle's packer (the
bytes of exactly those panels of the device's buffer), and computes the fp64
layer output of those rows for the requested activation matrices (also
regenerated on the host and cast to their storage type).
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

POOL_MAX = 16
_CTX = None


def start() -> None:
    """Start the fork server (call before the GPU is initialised)."""
    global _CTX
    if _CTX is not None:
        return
    import multiprocessing as mp
    from multiprocessing import forkserver
    ctx = mp.get_context("forkserver")
    ctx.set_forkserver_preload(["numpy", "scipy.linalg", "oracle", "synth", "tests.oracle_pool"])
    forkserver.ensure_running()
    _CTX = ctx


def workers() -> int:
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return max(1, min(POOL_MAX, avail))


def pool(n: Optional[int] = None):
    if _CTX is None:
        start()
    return _CTX.Pool(n or workers())


@dataclass
class XSpec:
    """Activations x = cast(synth.activations_f32(seed, stream, m, k)), rows `rows` of it (all when None)."""
    seed: int
    stream: int
    m: int
    k: int
    dtype: str                       # "f16", "bf16" or "f32"
    rows: Optional[List[int]] = None


@dataclass
class Task:
    seed: int
    linear_id: int
    n: int
    k: int
    sigma: float
    outliers: bool
    r0: int                          # first row, a multiple of 64
    r1: int                          # one past the last row
    osr: float
    levels: int
    block: int = 256
    packing: int = 0                 # 0: 2-bit / 1-bit fields, 1: base-3
    xs: List[XSpec] = field(default_factory=list)
    rows: Optional[List[int]] = None  # explicit rows instead of r0..r1 (no packing then)


def host_x(spec: XSpec):
    import numpy as np
    import synth
    x32 = synth.activations_f32(spec.seed, spec.stream, spec.m, spec.k)
    if spec.dtype == "f16":
        x = synth.to_f16(x32).astype(np.float64)
    elif spec.dtype == "bf16":
        x = synth.bf16_bits_to_f32(synth.to_bf16_bits(x32)).astype(np.float64)
    else:
        x = x32.astype(np.float64)
    return x if spec.rows is None else x[np.asarray(spec.rows)]


def run_task(t: Task) -> Tuple:
    """(packed bytes of the task's panels or None, fp32 scales, [y_ref per XSpec], int8 codes or None)."""
    import numpy as np
    from threadpoolctl import threadpool_limits
    import oracle
    import synth
    from oracle import layout as LY
    from oracle import linear as OL
    with threadpool_limits(1):
        rows = np.arange(t.r0, t.r1) if t.rows is None else np.asarray(t.rows)
        w = synth.weight_rows(t.seed, t.linear_id, t.n, t.k, t.sigma, t.outliers, rows=rows)
        r = oracle.encode(w, t.osr, t.levels, t.block)
        packed = None
        if t.rows is None:
            packed = LY.pack_base3(r.codes) if t.packing else LY.pack(r.codes, t.levels)
        ys = [OL.linear_fp64(host_x(s), r.codes, r.scales, t.block, r.m_up) for s in t.xs]
        keep = r.codes if t.rows is not None else None
    return packed, r.scales, ys, keep


def submit(pool, tasks: List[Task]):
    """Start `tasks` on `pool`; results come back in task order through `gather`."""
    return pool.imap(run_task, tasks, chunksize=1)


def gather(pending, count: int, label: str, task_timeout_s: float = 300.0) -> List[Tuple]:
    """The results of `count` submitted tasks, in order; one line on stdout per
    quarter of them done (a long oracle leg stays visibly alive)."""
    out = []
    step = max(1, count // 4)
    for i in range(count):
        out.append(pending.next(timeout=task_timeout_s))
        if (i + 1) % step == 0 or i + 1 == count:
            print(f"[oracle] {label}: {i + 1}/{count} tasks done", flush=True)
    return out


def panel_tasks(n: int, parts: int, **kw) -> List[Task]:
    """Split rows 0..n into at most `parts` tasks of whole 64-row panels."""
    panels = (n + 63) // 64
    per = max(1, -(-panels // parts))
    out = []
    for p0 in range(0, panels, per):
        out.append(Task(n=n, r0=64 * p0, r1=min(n, 64 * (p0 + per)), **kw))
    return out
