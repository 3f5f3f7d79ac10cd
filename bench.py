#!/usr/bin/env python3
"""Benchmark of the SDQ-LLM hot path on one MI355X.

Headline (one JSON line on stdout): decode throughput of the full LLaMA-70B
stack -- 80 layers x 7 linears (hidden 8192, 64 query / 8 key-value heads of
128, FFN 28672), MultiOSR at a mean OSR of 2.5 over the measured weight
variances, ternary codes as 2-bit fields -- at one fp16 activation row, in
GB/s of packed code bytes.

One step = one token through all 560 linears: per layer the q/k/v group, o,
the gate/up group and down (sdq_linear_group: one expansion and one
contraction launch per group of linears that read the same input).  The
stack's codes (42.8 GB) are resident in HBM and far exceed the 256 MB
last-level cache, so every step streams them.  Steps replay one HIP graph
(captured through PyTorch) so that host launch overhead is not timed; exactly
--steps replays are timed between HIP events on the replay stream.  The line
also carries:

* roofline     -- the step's decode contractions (every contraction launch:
                  the one-row matrix-core kernel gemv_mfma_kernel<3,1,*,true>
                  on rows of k_up >= 16384 samples, the table GEMV
                  gemv_lut_kernel<1,3,*> on shorter ones): the step's code
                  bytes / the time of a graph holding only those launches
                  (expansions done beforehand), against 8 TB/s and against
                  the measured streaming-read rate;
* config.m8    -- the same stack at eight activation rows (matrix-core decode);
* phases       -- the LLaMA-7B down_proj decode (workload 2), the LLaMA-7B layer
                  at m = 1, 4, 16 (workload 3), the three LLaMA-70B linears at
                  m = 1 and at m = 2048 prefill (workload 4), the stack on base-3
                  codes, the encoder (rows/s; the stack's quantization), MultiOSR,
                  the continuous-precision sweep and Algorithm 1's block
                  compensation;
* cpu_baseline -- the CPU oracle on 64 rows of each of the stack's seven linear
                  kinds (one mid-depth layer), over a process pool.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sdq_linear decode GB/s (% of HBM peak) and prefill TFLOP/s; rows/s quantized"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
# Separately rounded fp32 mul and add: the published 157.3 TFLOP/s fp32 vector
# peak is 256 CUs x 2.4 GHz x 128 lanes x 2 flops (fused multiply-add); a
# lane-op that is a plain mul or add is one flop, so the same lanes give
# 78.6 TFLOP/s.
VALU_F32_UNFUSED_PEAK_TFLOPS = 256 * 128 * 2.4e9 / 1e12
F64_PEAK_TFLOPS = 78.6
MALL_BYTES = 256 * 1024 * 1024
MIN_CALLS = 200                  # back-to-back calls per timed phase measurement
POOL_MAX = 16                    # oracle workers: the host share of one GPU

# HBM traffic per launch from two rocprofv3 --pmc passes over `bench.py
# --traffic-probe` (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch, averaged over
# the probe's launches of the kernel), scaled by what the same counters read
# for a 268,435,456-byte device copy.  Valid only for the kernel source they
# were taken with: a source whose hash differs reports traffic null.
TRAFFIC_FETCH_SCALE = 1.999749
TRAFFIC_WRITE_SCALE = 1.000000
TRAFFIC_SOURCES = {"linear_decode.hip": "8724ec4b804cf456d816d6cdb6b93a23ca13b410045cd3246f527c3dc50dca07"}
# launch family -> (source, FETCH_SIZE KiB, WRITE_SIZE KiB) per launch: the mean
# over the 325 contraction launches of one m = 1 token step through the stack.
TRAFFIC_KIB = {"m1_step_contractions": ("linear_decode.hip", 65092.0, 1636.6)}


def traffic_bytes(kernel: str):
    """Scaled HBM bytes per launch of `kernel`, or None if unmeasured or its source changed."""
    import hashlib
    entry = TRAFFIC_KIB.get(kernel)
    if entry is None:
        return None
    src, fetch_kib, write_kib = entry
    path = os.path.join(ROOT, "paper_2510_03275_amd", "csrc", src)
    try:
        digest = hashlib.sha256(open(path, "rb").read()).hexdigest()
    except OSError:
        return None
    if digest != TRAFFIC_SOURCES.get(src):
        return None
    return 1024.0 * (fetch_kib * TRAFFIC_FETCH_SCALE + write_kib * TRAFFIC_WRITE_SCALE)


# ---------------------------------------------------------------------------
# Oracle process pool (cpu_baseline).  Started through a fork server before
# the GPU is initialised, so that no worker is a fork of a GPU process.
# ---------------------------------------------------------------------------

def pool_workers() -> int:
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return max(1, min(POOL_MAX, avail))


def start_forkserver():
    import multiprocessing as mp
    ctx = mp.get_context("forkserver")
    ctx.set_forkserver_preload(["numpy", "scipy.linalg", "oracle", "synth"])
    from multiprocessing import forkserver
    forkserver.ensure_running()
    return ctx


def _oracle_encode_task(args):
    from threadpoolctl import threadpool_limits
    import numpy as np
    import oracle
    import synth
    seed, linear_id, n, k, sigma, outliers, rows, osr, levels = args
    with threadpool_limits(1):
        w = synth.weight_rows(seed, linear_id, n, k, sigma, outliers, rows=np.asarray(rows))
        r = oracle.encode(w, osr, levels)
    return r.codes, r.scales, r.m_up


def _oracle_linear_task(args):
    from threadpoolctl import threadpool_limits
    from oracle import linear as OL
    x, codes, scales, m_up = args
    with threadpool_limits(1):
        return OL.linear_fp64(x, codes, scales, 256, m_up)


# ---------------------------------------------------------------------------
# Timing helpers.
# ---------------------------------------------------------------------------

def _capture(torch, fns):
    """One HIP graph holding every call of fns (eager warm-up first)."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for fn in fns:
            fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for fn in fns:
            fn()
    torch.cuda.synchronize()
    return g


def _replay_ms(torch, g, replays: int, warm: int = 1) -> float:
    """Average ms per replay of g over `replays` back-to-back replays, HIP
    events on the replay (current) stream around them."""
    for _ in range(warm):
        g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(replays):
        g.replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / replays


def _graph_ms(torch, fns, min_calls: int = MIN_CALLS, warm: int = 1):
    """ms per call of a graph of fns replayed until >= min_calls calls ran."""
    g = _capture(torch, fns)
    replays = max(1, math.ceil(min_calls / len(fns)))
    ms = _replay_ms(torch, g, replays, warm) / len(fns)
    del g
    return ms, replays * len(fns)


def _rotations(nbytes: int) -> int:
    return max(2, math.ceil(2 * MALL_BYTES / max(nbytes, 1)))


def stream_read_peak(torch, SG, gib: int = 4):
    """Best streaming-read rate (GB/s) of a plain 16-byte-load kernel over a
    `gib` GiB buffer, over a few launch shapes."""
    buf = torch.empty(gib << 30, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.empty(16384, dtype=torch.int32, device="cuda")
    best = (0.0, None)
    for blocks in (1024, 2048, 4096, 8192, 16384):
        for unroll in (2, 4, 8):
            SG.read_probe(buf, blocks, unroll, sink)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(3):
                SG.read_probe(buf, blocks, unroll, sink)
            b.record()
            torch.cuda.synchronize()
            gbs = 3 * buf.numel() / (a.elapsed_time(b) * 1e-3) / 1e9
            if gbs > best[0]:
                best = (gbs, {"blocks": blocks, "loads_in_flight": unroll})
    del buf, sink
    torch.cuda.empty_cache()
    return {"gbs": best[0], "bytes": gib << 30, "launch": best[1], "frac_of_8tbs": best[0] / HBM_PEAK_GBS}


# ---------------------------------------------------------------------------
# Grouping: linears of one layer that read the same input and share
# (k, block, M, levels, Had, packing) run as one sdq_linear_group.
# ---------------------------------------------------------------------------

def layer_groups(encs, idxs, candidates):
    """Split the candidate index lists into groups of equal layout family."""
    groups = []
    for cand in candidates:
        by_key = {}
        for i in cand:
            L = encs[idxs[i]].layout
            key = (L.k, L.block, L.m_up, L.levels, L.hadamard, L.packing)
            by_key.setdefault(key, []).append(idxs[i])
        groups.extend(by_key.values())
    return groups


class StackRun:
    """Group calls of a list of layers (each a list of linear-index groups) at m rows."""

    def __init__(self, torch, P, SG, encs, layers, m, seed, x_dtype="f16"):
        self.torch, self.P = torch, P
        self.encs, self.m = encs, m
        tdt = torch.float16 if x_dtype == "f16" else torch.bfloat16
        ks = sorted({encs[i].layout.k for grp in sum(layers, []) for i in grp})
        self.x = {k: SG.activations_gpu(seed, 300 + k % 97, m, k).to(tdt) for k in ks}
        ns = sorted({encs[i].layout.n for grp in sum(layers, []) for i in grp})
        self.y = {n: torch.empty((m, n), dtype=torch.float32, device="cuda") for n in ns}
        self.calls = []
        need = 1
        for layer in layers:
            for grp in layer:
                es = [encs[i] for i in grp]
                g = P.LinearGroup(es, [self.y[e.layout.n] for e in es])
                need = max(need, P.sdq_linear_group_workspace_bytes([e.layout for e in es], m))
                self.calls.append((es[0].layout.k, g, es))
        self.ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        self.code_bytes = sum(P.sdq_codes_bytes(encs[i].layout) for grp in sum(layers, []) for i in grp)

    def step_fns(self):
        P, ws = self.P, self.ws
        return [lambda k=k, g=g: P.sdq_linear_group(self.x[k], g, ws) for k, g, _ in self.calls]

    def contraction_fns(self):
        """The contraction launches alone: every distinct expansion is computed
        once into its own workspace beforehand; accumulate mode, so no
        zero-fill launches sit between them."""
        P, torch = self.P, self.torch
        ws_by_key = {}
        fns = []
        for k, g, es in self.calls:
            L = es[0].layout
            key = (L.k, L.block, L.m_up, L.levels, L.hadamard, L.packing)
            if key not in ws_by_key:
                need = max(P.sdq_linear_group_workspace_bytes([e.layout for e in es], self.m), 1)
                ws_k = torch.empty(need, dtype=torch.uint8, device="cuda")
                P.sdq_expand_activations(self.x[k], L, ws_k)
                ws_by_key[key] = ws_k
            else:
                need = P.sdq_linear_group_workspace_bytes([e.layout for e in es], self.m)
                if ws_by_key[key].numel() < need:      # a larger group of the same family
                    ws_k = torch.empty(need, dtype=torch.uint8, device="cuda")
                    P.sdq_expand_activations(self.x[k], L, ws_k)
                    ws_by_key[key] = ws_k
            ws_k = ws_by_key[key]
            fns.append(lambda g=g, ws_k=ws_k: P.sdq_linear_group_expanded(self.m, g, ws_k, accumulate=True))
        torch.cuda.synchronize()
        return fns, ws_by_key


# ---------------------------------------------------------------------------
# Workload 5: the LLaMA-70B stack.
# ---------------------------------------------------------------------------

def build_stack(torch, P, synth, SG, base3: bool = False, variances=None):
    """Measure the 560 weight variances on the device, allocate OSRs with
    MultiOSR, generate and quantize every linear (codes kept resident).  The
    quantization alone is timed with HIP events (generation excluded)."""
    wl = synth.workload(5)
    t0 = time.perf_counter()
    if variances is None:
        out = torch.zeros(2, dtype=torch.float64, device="cuda")
        mws = None
        variances = []
        for lin in wl.linears:
            w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
            need = P.sdq_moments_workspace_bytes(w.numel())
            if mws is None or mws.numel() < need:
                mws = torch.empty(need, dtype=torch.uint8, device="cuda")
            P.sdq_weight_moments(w, out, mws)
            variances.append(float(out[1].item()))
            del w
        del mws
    osr = P.sdq_multiosr(variances, [lin.n * lin.k for lin in wl.linears], [lin.layer for lin in wl.linears],
                         *wl.multiosr)
    t1 = time.perf_counter()
    encs = []
    qws = None
    quant_ms = 0.0
    packing = P.SDQ_PACK_BASE3 if base3 else P.SDQ_PACK_FIELDS
    for lin, o in zip(wl.linears, osr):
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        L = P.sdq_layout_init(lin.n, lin.k, float(o), wl.levels)
        if base3:
            P.sdq_layout_set_packing(L, packing)
        need = P.sdq_quantize_workspace_bytes(L)
        if qws is None or qws.numel() < need:
            qws = torch.empty(need, dtype=torch.uint8, device="cuda")
        codes = torch.empty(P.sdq_codes_bytes(L), dtype=torch.uint8, device="cuda")
        scales = torch.empty(L.n, dtype=torch.float32, device="cuda")
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        P.sdq_quantize(w, L, codes, scales, qws)
        b.record()
        b.synchronize()
        quant_ms += a.elapsed_time(b)
        P.sdq_quantize_check(qws)
        encs.append(P.Encoded(L, codes, scales))
        del w
    del qws
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    torch.cuda.empty_cache()
    rows = sum(lin.n for lin in wl.linears)
    layers = []
    for layer in range(80):
        idxs = list(range(7 * layer, 7 * layer + 7))
        layers.append(layer_groups(encs, idxs, [[0, 1, 2], [3], [4, 5], [6]]))
    info = {"linears": len(encs), "rows": rows, "params": int(sum(lin.n * lin.k for lin in wl.linears)),
            "weighted_mean_osr": float(sum(float(o) * lin.n * lin.k for o, lin in zip(osr, wl.linears))
                                       / sum(lin.n * lin.k for lin in wl.linears)),
            "osr_first_layer": [float(o) for o in osr[:7]], "osr_last_layer": [float(o) for o in osr[-7:]],
            "code_bytes": int(sum(P.sdq_codes_bytes(e.layout) for e in encs)),
            "groups_per_step": sum(len(lg) for lg in layers),
            "variances_and_allocation_s": t1 - t0, "generate_and_quantize_s": t2 - t1,
            "quantize_ms": quant_ms, "quantize_rows_per_s": rows / (quant_ms * 1e-3)}
    return wl, encs, layers, variances, osr, info


def stack_decode(torch, P, SG, wl, encs, layers, m, steps, warmup):
    run = StackRun(torch, P, SG, encs, layers, m, wl.seed)
    g = _capture(torch, run.step_fns())
    ms = _replay_ms(torch, g, steps, warmup)
    del g
    gbs = run.code_bytes / (ms * 1e-3) / 1e9
    return run, {"m": m, "ms_per_step": ms, "tokens_per_s": m * 1e3 / ms, "gbs": gbs,
                 "frac_of_hbm_peak": gbs / HBM_PEAK_GBS, "code_bytes": int(run.code_bytes),
                 "launches_per_step": 2 * len(run.calls), "steps": steps, "warmup": warmup}


def stack_gemv_roofline(torch, run, replays: int = 3):
    """The contraction launches of one step alone, in one graph."""
    fns, ws = run.contraction_fns()
    g = _capture(torch, fns)
    ms = _replay_ms(torch, g, replays, 1)
    del g, ws
    torch.cuda.empty_cache()
    return ms, len(fns)


# ---------------------------------------------------------------------------
# Phases: workloads 2, 3 and 4; encoder; MultiOSR; sweep; compensation.
# ---------------------------------------------------------------------------

def decode_single(torch, P, synth, SG, wl_index, lin_index, m, x_dtype, base3=False, seed_stream=1):
    """sdq_linear at m rows on one linear of a workload, over rotating copies
    of its codes (working set >= 2x the last-level cache), >= MIN_CALLS calls:
    the whole call and the contraction alone."""
    wl = synth.workload(wl_index)
    lin = wl.linears[lin_index]
    w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
    enc = P.quantize(w, wl.osr, wl.levels, packing=P.SDQ_PACK_BASE3 if base3 else P.SDQ_PACK_FIELDS)
    del w
    L = enc.layout
    nbytes = P.sdq_codes_bytes(L)
    rot = _rotations(nbytes)
    codes = [enc.codes.clone() for _ in range(rot)]
    tdt = torch.float16 if x_dtype == "f16" else torch.bfloat16
    x = SG.activations_gpu(wl.seed, seed_stream, m, lin.k).to(tdt)
    y = torch.empty((m, lin.n), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.sdq_linear_workspace_bytes(L, m), dtype=torch.uint8, device="cuda")
    ms_step, calls = _graph_ms(torch, [lambda i=i: P.sdq_linear(x, codes[i], enc.scales, L, y, ws)
                                       for i in range(rot)])
    P.sdq_expand_activations(x, L, ws)
    ms_gemv, _ = _graph_ms(torch, [lambda i=i: P.sdq_linear_expanded(m, codes[i], enc.scales, L, y, ws,
                                                                     accumulate=True)
                                   for i in range(rot)])
    del codes, ws, enc
    torch.cuda.empty_cache()
    gbs = nbytes / (ms_step * 1e-3) / 1e9
    gemv_gbs = nbytes / (ms_gemv * 1e-3) / 1e9
    return {"n": lin.n, "k": lin.k, "osr": L.m_up / L.block, "levels": L.levels, "m": m,
            "code_bytes": int(nbytes), "rotating_code_buffers": rot, "calls_timed": calls,
            "ms": ms_step, "gbs": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS,
            "ms_contraction": ms_gemv, "contraction_gbs": gemv_gbs,
            "contraction_frac_of_hbm_peak": gemv_gbs / HBM_PEAK_GBS}


def prefill_single(torch, P, synth, SG, lin_index, reps: int = 8):
    """Workload 4 at m = 2048 (bf16 activations): the whole sdq_linear (fp16
    expansion + MFMA GEMM) and the GEMM alone, 2 m N K_up flops."""
    wl = synth.workload(4)
    lin = wl.linears[lin_index]
    m = wl.prefill[0]
    w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
    enc = P.quantize(w, wl.osr, wl.levels)
    del w
    L = enc.layout
    x = SG.activations_gpu(wl.seed, 2, m, lin.k).to(torch.bfloat16)
    y = torch.empty((m, lin.n), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.sdq_linear_workspace_bytes(L, m), dtype=torch.uint8, device="cuda")
    ms_total, _ = _graph_ms(torch, [lambda: P.sdq_linear(x, enc.codes, enc.scales, L, y, ws)] * reps, reps)
    P.sdq_expand_activations(x, L, ws)
    ms_gemm, _ = _graph_ms(torch, [lambda: P.sdq_linear_expanded(m, enc.codes, enc.scales, L, y, ws)] * reps,
                           reps)
    flops = 2.0 * m * L.n * L.k_up
    del ws, y, x, enc
    torch.cuda.empty_cache()
    return {"n": lin.n, "k": lin.k, "m": m, "flops": flops, "ms": ms_total, "tflops": flops / (ms_total * 1e-3) / 1e12,
            "frac_of_mfma_peak": flops / (ms_total * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS,
            "ms_gemm": ms_gemm, "gemm_tflops": flops / (ms_gemm * 1e-3) / 1e12,
            "gemm_frac_of_mfma_peak": flops / (ms_gemm * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS}


def bench_workload3(torch, P, synth, SG):
    """The LLaMA-7B layer (7 linears, MultiOSR from the measured variances,
    ternary): one layer step (q/k/v, o, gate/up and down groups) at
    m = 1, 4, 16 over rotating copies of the layer's codes."""
    wl = synth.workload(3)
    out = torch.zeros(2, dtype=torch.float64, device="cuda")
    var = []
    for lin in wl.linears:
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        ws = torch.empty(P.sdq_moments_workspace_bytes(w.numel()), dtype=torch.uint8, device="cuda")
        P.sdq_weight_moments(w, out, ws)
        var.append(float(out[1].item()))
        del w, ws
    osr = P.sdq_multiosr(var, [lin.n * lin.k for lin in wl.linears], [lin.layer for lin in wl.linears],
                         *wl.multiosr)
    base = []
    for lin, o in zip(wl.linears, osr):
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        base.append(P.quantize(w, float(o), wl.levels))
        del w
    layer_bytes = sum(P.sdq_codes_bytes(e.layout) for e in base)
    rot = _rotations(layer_bytes)
    encs = list(base)
    for _ in range(rot - 1):
        encs += [P.Encoded(e.layout, e.codes.clone(), e.scales) for e in base]
    layers = [layer_groups(encs, list(range(7 * r, 7 * r + 7)), [[0, 1, 2], [3], [4, 5], [6]])
              for r in range(rot)]
    res = {"osr": [float(o) for o in osr], "layer_code_bytes": int(layer_bytes), "rotating_copies": rot}
    for m in wl.batches:
        run = StackRun(torch, P, SG, encs, layers, m, wl.seed)
        fns = run.step_fns()
        ms, calls = _graph_ms(torch, fns)
        ms_layer = ms * len(fns) / rot
        gbs = layer_bytes / (ms_layer * 1e-3) / 1e9
        res[f"m{m}"] = {"ms_per_layer_step": ms_layer, "gbs": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS,
                        "group_calls_timed": calls}
        del run
    del encs, base
    torch.cuda.empty_cache()
    return res


def bench_encoder(torch, P, synth, SG, reps: int = 5):
    wl = synth.workload(2)
    lin = wl.linears[0]
    w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
    L = P.sdq_layout_init(w.shape[0], w.shape[1], wl.osr, wl.levels)
    codes = torch.empty(P.sdq_codes_bytes(L), dtype=torch.uint8, device="cuda")
    scales = torch.empty(L.n, dtype=torch.float32, device="cuda")
    ws = torch.empty(P.sdq_quantize_workspace_bytes(L), dtype=torch.uint8, device="cuda")
    P.sdq_quantize(w, L, codes, scales, ws)
    P.sdq_quantize_check(ws)
    ms, _ = _graph_ms(torch, [lambda: P.sdq_quantize(w, L, codes, scales, ws)] * reps, 3 * reps)
    g0 = math.gcd(L.block, L.m_up)
    m_nz = L.m_up - g0
    flops = 2.0 * L.n * L.nb * m_nz * L.block       # separately rounded mul + add per term
    tflops = flops / (ms * 1e-3) / 1e12
    del ws, w
    torch.cuda.empty_cache()
    return {
        "workload": "llama7b_down_proj_4096x11008_osr1.5_binary",
        "rows_per_s": L.n / (ms * 1e-3), "ms": ms,
        "roofline": {"bound": "alu", "achieved": tflops, "peak": VALU_F32_UNFUSED_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": tflops / VALU_F32_UNFUSED_PEAK_TFLOPS,
                     "traffic": None, "note": "whole sdq_quantize call (4 kernels); flops = "
                     "2 * rows * blocks * dense samples per block * B"},
    }


def bench_multiosr(torch, P, synth, SG):
    wl = synth.workload(3)
    var, nparams = [], []
    t0 = time.perf_counter()
    out = torch.zeros(2, dtype=torch.float64, device="cuda")
    for lin in wl.linears:
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        ws = torch.empty(P.sdq_moments_workspace_bytes(w.numel()), dtype=torch.uint8, device="cuda")
        P.sdq_weight_moments(w, out, ws)
        var.append(float(out[1].item()))
        nparams.append(lin.n * lin.k)
    t1 = time.perf_counter()
    osr = P.sdq_multiosr(var, nparams, [lin.layer for lin in wl.linears], *wl.multiosr)
    t2 = time.perf_counter()
    return {"workload": "llama7b_layer_7_linears", "osr": [float(o) for o in osr],
            "weighted_mean_osr": float(sum(o * n for o, n in zip(osr, nparams)) / sum(nparams)),
            "moments_s_incl_generation": t1 - t0, "allocate_ms": (t2 - t1) * 1e3}


SWEEP_OSRS = tuple(1.0 + 0.25 * i for i in range(13))      # 1.0 .. 4.0


def precision_sweep(torch, P, synth, SG, n: int = 4096, k: int = 4096, m: int = 64,
                    osrs=SWEEP_OSRS, hads=(1, 2, 0), levels_list=(3, 2), seed: int = 2516):
    """Continuous precision and the Hadamard ablation on one synthetic layer
    (LLaMA-7B q_proj shape, N(0, 0.02^2) weights with x10 outliers): for every
    (levels, Had, OSR) the codes' bits per weight, the layer-output error
    ||y - x W^T|| / ||x W^T|| on m fp16 activation rows (y from sdq_linear,
    x W^T in fp64 on the host), and the weight reconstruction SNR
    10 log10(||W||^2 / ||W - W_hat||^2) with W_hat^T = sdq_linear of the
    identity.  Hads: 1 Sylvester, 2 sign-randomised, 0 none."""
    import numpy as np
    w = SG.weight_rows_gpu(seed, 0, n, k, 0.02, True)
    x = SG.activations_gpu(seed, 7, m, k).to(torch.float16)
    y_ref = x.double().cpu().numpy() @ w.double().cpu().numpy().T
    ref_norm = float(np.linalg.norm(y_ref))
    w_sq = float(torch.sum(w.double() ** 2).item())
    eye = torch.eye(k, dtype=torch.float16, device="cuda")
    signs = synth.hadamard_signs(seed, 256)
    rows = []
    for levels in levels_list:
        for had in hads:
            for osr in osrs:
                enc = P.quantize(w, osr, levels, hadamard=had, signs=signs if had == 2 else None)
                y = P.linear(x, enc).double().cpu().numpy()
                w_hat_t = P.linear(eye, enc)                     # (k, n) = W_hat^T
                err_sq = float(torch.sum((w_hat_t.t().double() - w.double()) ** 2).item())
                rows.append({"levels": levels, "had": had, "osr": osr,
                             "bits_per_weight": (1 if levels == 2 else 2) * enc.layout.m_up / enc.layout.block,
                             "out_rel_err": float(np.linalg.norm(y - y_ref)) / ref_norm,
                             "weight_snr_db": 10.0 * math.log10(w_sq / err_sq)})
                del enc, w_hat_t
    del w, x, eye
    torch.cuda.empty_cache()
    return rows


def multiosr_ablation(torch, P, synth, SG, targets=(1.5, 2.0, 2.5, 3.0), lo: float = 1.0,
                      hi: float = 4.0, m: int = 16):
    """MultiOSR against one uniform OSR at the same parameter-weighted mean, on
    the seven LLaMA-7B linears of one layer (per-linear variances log-uniform in
    [1e-4, 1e-3], ternary): the parameter-weighted mean and the largest
    per-linear output error ||y - x W^T|| / ||x W^T||."""
    import numpy as np
    wl = synth.workload(3)
    out = torch.zeros(2, dtype=torch.float64, device="cuda")
    var, refs = [], []
    for lin in wl.linears:
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        ws = torch.empty(P.sdq_moments_workspace_bytes(w.numel()), dtype=torch.uint8, device="cuda")
        P.sdq_weight_moments(w, out, ws)
        var.append(float(out[1].item()))
        x = SG.activations_gpu(wl.seed, 40 + lin.linear_id, m, lin.k).to(torch.float16)
        refs.append((x, x.double().cpu().numpy() @ w.double().cpu().numpy().T))
        del w, ws
    nparams = np.array([lin.n * lin.k for lin in wl.linears], dtype=np.float64)
    res = []
    for target in targets:
        alloc = {"uniform": [target] * len(wl.linears),
                 "multiosr": [float(o) for o in P.sdq_multiosr(var, nparams.astype(np.int64),
                                                               [lin.layer for lin in wl.linears],
                                                               target, lo, hi)]}
        entry = {"target_mean_osr": target}
        for name, osrs in alloc.items():
            errs = []
            for lin, o, (x, y_ref) in zip(wl.linears, osrs, refs):
                w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
                enc = P.quantize(w, o, wl.levels)
                y = P.linear(x, enc).double().cpu().numpy()
                errs.append(float(np.linalg.norm(y - y_ref) / np.linalg.norm(y_ref)))
                del w, enc
            entry[name] = {"osr": osrs, "mean_osr": float(np.dot(osrs, nparams) / nparams.sum()),
                           "weighted_mean_out_rel_err": float(np.dot(errs, nparams) / nparams.sum()),
                           "max_out_rel_err": max(errs)}
        res.append(entry)
    del refs
    torch.cuda.empty_cache()
    return {"workload": "llama7b_layer_7_linears_ternary", "lo": lo, "hi": hi, "m": m, "rows": res}


def bench_compensation(torch, P, synth, SG, n: int = 4096, k: int = 4096, m_cal: int = 16384,
                       m_test: int = 256, rank: int = 32, osr: float = 2.0, levels: int = 3,
                       seed: int = 2517):
    """Algorithm 1's block compensation on a LLaMA-7B q_proj-sized layer: the
    Hessian of m_cal calibration rows, its damped inverse's Cholesky factor and
    the compensated encoding (both updates), each timed (fp64 throughput
    against the fp64 peak), and the layer-output error on m_test held-out rows
    of the same input distribution with and without compensation.  Inputs: a
    shared low-rank part plus noise with uneven channel scales (the seeded
    generator's normals combined on the device)."""
    import numpy as np
    w = SG.weight_rows_gpu(seed, 0, n, k, 0.02, True)
    mix = SG.activations_gpu(seed, 11, k, rank)
    ch = torch.exp(0.5 * SG.activations_gpu(seed, 12, 1, k))

    def draw(stream, m):
        z = SG.activations_gpu(seed, stream, m, rank)
        e = SG.activations_gpu(seed, stream + 1, m, k)
        return ((z @ mix.t()) * 0.9 + e) * ch

    x_cal = draw(13, m_cal).contiguous()
    x_test = draw(15, m_test).contiguous()

    def timed(fn):
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        out = fn()
        b.record()
        torch.cuda.synchronize()
        return out, a.elapsed_time(b)

    h = torch.zeros((k, k), dtype=torch.float64, device="cuda")
    P.sdq_hessian_accumulate(x_cal[:64].contiguous(), h)          # warm-up (and discarded)
    h.zero_()
    _, ms_h = timed(lambda: P.sdq_hessian_accumulate(x_cal, h))
    lam = 0.01 * float(torch.mean(torch.diagonal(h)).item())
    u = P.hessian_factor(h, lam)                                   # warm-up
    u, ms_f = timed(lambda: P.hessian_factor(h, lam, check=False))
    ws = torch.empty(P.sdq_hessian_factor_workspace_bytes(k), dtype=torch.uint8, device="cuda")
    P.sdq_hessian_factor(h, lam, u, ws)
    P.sdq_hessian_check(ws)
    y_ref = x_test.double().cpu().numpy() @ w.double().cpu().numpy().T
    res = {}
    errs = {}
    for name, upd in (("gptq", P.SDQ_COMP_GPTQ), ("joint", P.SDQ_COMP_JOINT)):
        P.quantize_compensated(w, osr, levels, u, update=upd)          # warm-up
        enc_c, ms_c = timed(lambda: P.quantize_compensated(w, osr, levels, u, check=False, update=upd))
        res[f"compensated_{name}_quantize_ms"] = ms_c
        y = P.linear(x_test, enc_c).double().cpu().numpy()
        errs[name] = float(np.linalg.norm(y - y_ref) / np.linalg.norm(y_ref))
        del enc_c
    enc_p, ms_p = timed(lambda: P.quantize(w, osr, levels, check=False))
    y = P.linear(x_test, enc_p).double().cpu().numpy()
    errs["plain"] = float(np.linalg.norm(y - y_ref) / np.linalg.norm(y_ref))
    flops_h = 1.0 * m_cal * k * (k + 1)   # symmetric rank-m update: one triangle plus the diagonal
    flops_f = 2.0 * k ** 3 / 3.0          # Cholesky k^3/3 plus triangular inverse k^3/3
    tf = lambda f, ms: f / (ms * 1e-3) / 1e12
    del h, u, x_cal, enc_p, w, ws
    torch.cuda.empty_cache()
    res.update({"workload": f"llama7b_q_proj_{n}x{k}_osr{osr:g}_ternary_compensated_{m_cal}_calibration_rows",
                "hessian_ms": ms_h, "hessian_tflops": tf(flops_h, ms_h),
                "factor_ms": ms_f, "factor_tflops": tf(flops_f, ms_f), "plain_quantize_ms": ms_p,
                "out_rel_err_plain": errs["plain"], "out_rel_err_gptq": errs["gptq"],
                "out_rel_err_joint": errs["joint"],
                "roofline": {"bound": "mfma", "achieved": tf(flops_h, ms_h), "peak": F64_PEAK_TFLOPS,
                             "unit": "TFLOP/s", "frac": tf(flops_h, ms_h) / F64_PEAK_TFLOPS, "traffic": None,
                             "kernel": "gemm64_kernel<float,float> (Hessian)",
                             "note": "fp64 matrix-core GEMM over the tiles on or below the diagonal "
                                     "(each added at its transposed position too); flops = m * k * (k + 1), "
                                     "the count of a symmetric rank-m update"}})
    return res


def bench_sweep(torch, P, synth, SG):
    t0 = time.perf_counter()
    rows = precision_sweep(torch, P, synth, SG)
    t1 = time.perf_counter()
    abl = multiosr_ablation(torch, P, synth, SG)
    t2 = time.perf_counter()
    return {"workload": "llama7b_q_proj_4096x4096_outliers_sweep_osr1to4", "rows": rows,
            "configs_per_s": len(rows) / (t1 - t0), "sweep_s": t1 - t0,
            "multiosr_ablation": abl, "ablation_s": t2 - t1}


# ---------------------------------------------------------------------------
# The oracle beside it.
# ---------------------------------------------------------------------------

def cpu_baseline(ctx, synth, wl, osr, layer: int = 40, rows_per_kind: int = 512, chunk: int = 32):
    """The oracle on 512 rows of each of the seven linear kinds of one stack
    layer (at their MultiOSR OSRs): the encoder over a process pool, then the
    fp64 linear (Algorithm 1's reconstruction, one activation row) over the
    same pool.  value = code bytes of the sampled rows / linear wall time."""
    import numpy as np
    workers = pool_workers()
    enc_tasks, meta = [], []
    code_bytes = 0
    for j in range(7):
        lin = wl.linears[7 * layer + j]
        o = float(osr[7 * layer + j])
        rows = np.random.default_rng(lin.linear_id).choice(lin.n, rows_per_kind, replace=False)
        m_up = int(round(o * 256))
        code_bytes += rows_per_kind * math.ceil(lin.k // 256 * m_up / 64) * 16
        for c0 in range(0, rows_per_kind, chunk):
            enc_tasks.append((wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers,
                              rows[c0:c0 + chunk].tolist(), o, wl.levels))
            meta.append(lin.k)
    with ctx.Pool(workers) as pool:
        t0 = time.perf_counter()
        encoded = pool.map(_oracle_encode_task, enc_tasks, chunksize=1)
        t_enc = time.perf_counter() - t0
        xs = {k: synth.to_f16(synth.activations_f32(wl.seed, 300 + k % 97, 1, k)).astype(np.float64)
              for k in set(meta)}
        lin_tasks = [(xs[k], c, s, mu) for k, (c, s, mu) in zip(meta, encoded)]
        t1 = time.perf_counter()
        pool.map(_oracle_linear_task, lin_tasks, chunksize=1)
        t_lin = time.perf_counter() - t1
    n_rows = 7 * rows_per_kind
    return {"value": code_bytes / t_lin / 1e9, "unit": "GB/s", "cores": workers, "kind": "oracle",
            "sample": f"{rows_per_kind} seeded rows of each of the 7 linears of layer {layer} of the LLaMA-70B "
                      f"stack ({n_rows} rows, {code_bytes} code bytes): oracle encode, then its fp64 linear "
                      f"at one activation row (reconstruct W_hat by FFT Resample and Had^T, then x W_hat^T), "
                      f"tasks of {chunk} rows over a pool of {workers} processes with one BLAS thread each",
            "oracle_encoder_rows_per_s": n_rows / t_enc, "oracle_encoder_s": t_enc, "oracle_linear_s": t_lin,
            "pool_processes": workers, "blas_threads_per_process": 1, "host_cpu_count": os.cpu_count()}


# ---------------------------------------------------------------------------
# Counter and trace probes (short eager runs for rocprofv3).
# ---------------------------------------------------------------------------

def traffic_probe(torch, P, synth, SG) -> None:
    """A short eager run for hardware-counter passes: one 256 MiB device copy
    of known size (to scale FETCH_SIZE / WRITE_SIZE), then the contraction
    launches of one token step through the LLaMA-70B stack (m = 1, expansions
    once before), the same at m = 8, the LLaMA-7B down_proj GEMV and the
    LLaMA-70B prefill GEMMs, and the 28672x8192 layer with base-3 codes at m = 8.
    Prints what it ran and the code bytes of the stack's launches."""
    nbytes = 256 << 20
    a = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    del a, b
    print(f"copy: {nbytes} bytes", flush=True)
    wl, encs, layers, _, _, info = build_stack(torch, P, synth, SG)
    run = StackRun(torch, P, SG, encs, layers, 1, wl.seed)
    fns, ws = run.contraction_fns()
    for fn in fns:
        fn()
    torch.cuda.synchronize()
    print(f"stack m=1 contraction: {len(fns)} launches, code bytes {run.code_bytes}", flush=True)
    del run, fns, ws
    run = StackRun(torch, P, SG, encs, layers, 8, wl.seed)
    fns, ws = run.contraction_fns()
    for fn in fns:
        fn()
    torch.cuda.synchronize()
    print(f"stack m=8 contraction: {len(fns)} launches, code bytes {run.code_bytes}", flush=True)
    del run, fns, ws, encs
    torch.cuda.empty_cache()
    for wl_i, lin_i, m, xdt, pack, label in (
            (2, 0, 1, torch.float16, P.SDQ_PACK_FIELDS, "down_proj 4096x11008 m=1"),
            (4, 0, 2048, torch.bfloat16, P.SDQ_PACK_FIELDS, "70B 8192x8192 m=2048"),
            (4, 1, 2048, torch.bfloat16, P.SDQ_PACK_FIELDS, "70B 28672x8192 m=2048"),
            (4, 2, 2048, torch.bfloat16, P.SDQ_PACK_FIELDS, "70B 8192x28672 m=2048"),
            (4, 1, 8, torch.float16, P.SDQ_PACK_BASE3, "70B 28672x8192 m=8 base-3")):
        wl = synth.workload(wl_i)
        lin = wl.linears[lin_i]
        w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
        enc = P.quantize(w, wl.osr, wl.levels, packing=pack)
        del w
        L = enc.layout
        x = SG.activations_gpu(wl.seed, 5, m, lin.k).to(xdt)
        y = torch.zeros((m, lin.n), dtype=torch.float32, device="cuda")
        ws = torch.empty(P.sdq_linear_workspace_bytes(L, m), dtype=torch.uint8, device="cuda")
        P.sdq_expand_activations(x, L, ws)
        for _ in range(4):
            P.sdq_linear_expanded(m, enc.codes, enc.scales, L, y, ws, accumulate=True)
        torch.cuda.synchronize()
        print(f"{label}: code bytes {P.sdq_codes_bytes(L)}, x_tilde bytes {2 * m * L.n_chunks * 64 if m > 16 else 0}, "
              f"4 launches", flush=True)
        del enc, x, y, ws
        torch.cuda.empty_cache()


def encoder_probe(torch, P, synth, SG) -> None:
    """Three sdq_quantize calls on the LLaMA-7B down_proj layer (4096 x 11008,
    OSR 1.5, binary), after the weight generation.  Prints what it ran."""
    wl = synth.workload(2)
    lin = wl.linears[0]
    w = SG.weight_rows_gpu(wl.seed, lin.linear_id, lin.n, lin.k, lin.sigma, wl.outliers)
    L = P.sdq_layout_init(w.shape[0], w.shape[1], wl.osr, wl.levels)
    codes = torch.empty(P.sdq_codes_bytes(L), dtype=torch.uint8, device="cuda")
    scales = torch.empty(L.n, dtype=torch.float32, device="cuda")
    ws = torch.empty(P.sdq_quantize_workspace_bytes(L), dtype=torch.uint8, device="cuda")
    for _ in range(3):
        P.sdq_quantize(w, L, codes, scales, ws)
    torch.cuda.synchronize()
    print(f"encoder probe: 3 x sdq_quantize {lin.n}x{lin.k} osr {wl.osr} levels {wl.levels}", flush=True)


def _phase(line, name, fn):
    t = time.perf_counter()
    try:
        line["phases"][name] = fn()
    except Exception as exc:  # noqa: BLE001 -- report, keep the headline line
        line["phases"][name] = {"error": repr(exc)}
    print(f"[bench] phase {name}: {time.perf_counter() - t:.1f} s", file=sys.stderr, flush=True)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50, help="timed token steps through the stack")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-phases", action="store_true", help="headline, roofline and m = 8 only")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="short eager run for rocprofv3 --pmc passes (prints no JSON line)")
    ap.add_argument("--encoder-probe", action="store_true",
                    help="three encoder calls on the LLaMA-7B down_proj layer, for rocprofv3 --pmc passes")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: the SDQ hot path has no multi-GPU step "
              f"(requested --gpus {args.gpus}, WORLD_SIZE {world})", file=sys.stderr)
        return 2
    if args.steps < 1 or args.warmup < 0:
        print("need --steps >= 1 and --warmup >= 0", file=sys.stderr)
        return 2
    ctx = None
    if not (args.no_cpu_baseline or args.traffic_probe or args.encoder_probe):
        ctx = start_forkserver()          # before anything initialises the GPU

    import torch
    import paper_2510_03275_amd as P
    import synth
    from synth import gpu as SG

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    torch.cuda.synchronize()
    if args.traffic_probe:
        traffic_probe(torch, P, synth, SG)
        return 0
    if args.encoder_probe:
        encoder_probe(torch, P, synth, SG)
        return 0
    t_start = time.perf_counter()
    peak = stream_read_peak(torch, SG)
    wl, encs, layers, variances, osr, info = build_stack(torch, P, synth, SG)
    print(f"[bench] stack built: {info['code_bytes']} code bytes, {time.perf_counter() - t_start:.1f} s",
          file=sys.stderr, flush=True)
    run1, dec1 = stack_decode(torch, P, SG, wl, encs, layers, 1, args.steps, args.warmup)
    ms_gemv, n_gemv = stack_gemv_roofline(torch, run1)
    del run1
    torch.cuda.empty_cache()
    run8, dec8 = stack_decode(torch, P, SG, wl, encs, layers, 8, max(5, args.steps // 5), 2)
    del run8
    torch.cuda.empty_cache()
    gbs = dec1["gbs"]
    gemv_gbs = info["code_bytes"] / (ms_gemv * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": gbs,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dec1["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "llama70b_stack_80x7_multiosr2.5_ternary_decode_m1",
            "layers": 80, "linears": 560, "hidden": 8192, "ffn": 28672, "m": 1, "x_dtype": "f16",
            "levels": 3, "code_packing": "2-bit fields", "code_bytes": info["code_bytes"],
            "weighted_mean_osr": info["weighted_mean_osr"], "hip_graph": True,
            "launches_per_step": dec1["launches_per_step"],
            "percent_of_hbm_peak": 100.0 * gbs / HBM_PEAK_GBS,
            "percent_of_stream_read_peak": 100.0 * gbs / peak["gbs"],
            "tokens_per_s": dec1["tokens_per_s"],
            "m8": dict(dec8, percent_of_stream_read_peak=100.0 * dec8["gbs"] / peak["gbs"]),
            "stream_read_peak": peak,
            "quantize": {k: info[k] for k in ("rows", "params", "quantize_ms", "quantize_rows_per_s",
                                              "generate_and_quantize_s", "variances_and_allocation_s",
                                              "groups_per_step", "osr_first_layer", "osr_last_layer")},
        },
        "roofline": {"bound": "hbm", "achieved": gemv_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gemv_gbs / HBM_PEAK_GBS, "traffic": traffic_bytes("m1_step_contractions"),
                     "kernel": "every decode contraction launch of one token step: gemv_mfma_kernel<3,1,*,true> "
                               "(rows of k_up >= 16384 samples) and gemv_lut_kernel<1,3,*> (shorter rows)",
                     "launches": n_gemv, "ms_per_step_of_launches": ms_gemv,
                     "bytes_per_launch": info["code_bytes"] / n_gemv,
                     "frac_of_stream_read_peak": gemv_gbs / peak["gbs"],
                     "note": "algorithmic bytes = the step's packed codes (N * K_up / 4 per linear) over its "
                             "contraction launches; achieved = those bytes / the launches' time from HIP "
                             "events around a graph of them alone; traffic = counted HBM bytes per launch "
                             "(fetch + write)"},
    }
    print(f"[bench] headline done: {gbs:.0f} GB/s, {time.perf_counter() - t_start:.1f} s", file=sys.stderr,
          flush=True)
    if not args.no_phases:
        line["phases"] = {}
        del encs
        torch.cuda.empty_cache()

        def stack_base3():
            _, e3, l3, _, _, i3 = build_stack(torch, P, synth, SG, base3=True, variances=variances)
            r1, d1 = stack_decode(torch, P, SG, wl, e3, l3, 1, max(5, args.steps // 2), 2)
            del r1
            r8, d8 = stack_decode(torch, P, SG, wl, e3, l3, 8, max(5, args.steps // 5), 2)
            del r8, e3
            torch.cuda.empty_cache()
            return {"code_bytes": i3["code_bytes"], "bits_per_code": 1.6, "m1": d1, "m8": d8}

        _phase(line, "stack_70b_base3", stack_base3)
        _phase(line, "llama7b_down_proj_decode_m1", lambda: decode_single(torch, P, synth, SG, 2, 0, 1, "f16"))
        _phase(line, "llama7b_layer_multiosr", lambda: bench_workload3(torch, P, synth, SG))
        for i, nm in enumerate(("8192x8192", "28672x8192", "8192x28672")):
            _phase(line, f"llama70b_{nm}_decode_m1",
                   lambda i=i: decode_single(torch, P, synth, SG, 4, i, 1, "bf16", seed_stream=3))
            _phase(line, f"llama70b_{nm}_prefill_m2048", lambda i=i: prefill_single(torch, P, synth, SG, i))
        _phase(line, "encoder", lambda: bench_encoder(torch, P, synth, SG))
        _phase(line, "multiosr", lambda: bench_multiosr(torch, P, synth, SG))
        _phase(line, "precision_sweep", lambda: bench_sweep(torch, P, synth, SG))
        _phase(line, "compensation", lambda: bench_compensation(torch, P, synth, SG))
    if ctx is not None:
        line["cpu_baseline"] = cpu_baseline(ctx, synth, wl, osr)
    line["wall_s"] = time.perf_counter() - t_start
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
