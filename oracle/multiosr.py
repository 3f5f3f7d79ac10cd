"""MultiOSR: layer- and linear-wise OSR allocation (Section 3.4, Fig. 4).

The paper states the rule in words only: given a target average OSR, layers
are ranked by their weight variance and receive OSR accordingly; inside a
layer the layer's OSR is spread over its linear modules inversely to each
module's weight variance and in proportion to its size.  No formula is given,
so the exact allocation below is a reading (parity of its values is unpinned
by the paper; the tests pin its invariants):

1. layer level: pooled variance V_l = sum_j n_j var_j / N_l over the layer's
   linears (N_l = sum_j n_j parameters); score a_l = 1 / V_l; the layer OSR is
   clip(lambda * a_l, lo, hi) with lambda chosen so that the parameter-weighted
   mean over layers equals the target T;
2. linear level: score b_j = n_j / var_j; OSR_j = clip(mu_l * b_j, lo, hi) with
   mu_l chosen so that the parameter-weighted mean inside layer l equals the
   layer OSR;
3. both scale factors are found by fp64 bisection on the monotone weighted
   mean (a variance <= 0 gives an infinite score, i.e. the upper bound hi);
4. snap to the grid g: every OSR is floored to a multiple of g (with a 1e-9
   guard), then, taking linears in order of decreasing fractional remainder
   (ties to the lower index), one step g is added to a linear when it stays
   <= hi and the parameter-weighted mean of the whole model stays <= T.  The
   memory budget T is therefore never exceeded.
"""
from __future__ import annotations

import math

import numpy as np

BISECT_STEPS = 200


def variance_fp64(w: np.ndarray) -> float:
    """Population variance of all entries, two-pass, fp64."""
    x = np.asarray(w, dtype=np.float64).reshape(-1)
    mu = x.sum() / x.size
    return float(((x - mu) ** 2).sum() / x.size)


def _weighted_clip(scale: float, scores, weights, lo: float, hi: float) -> float:
    tot = 0.0
    for sc, wt in zip(scores, weights):
        val = hi if math.isinf(sc) else min(max(scale * sc, lo), hi)
        tot += wt * val
    return tot


def _allocate(scores, weights, target: float, lo: float, hi: float):
    """Values clip(c * score, lo, hi) whose weights-weighted mean is target."""
    wsum = float(sum(weights))
    if target <= lo:
        return [lo] * len(scores)
    if target >= hi:
        return [hi] * len(scores)
    finite = [sc for sc in scores if not math.isinf(sc)]
    if not finite:
        return [hi] * len(scores)
    c_lo, c_hi = 0.0, hi / min(finite)
    goal = target * wsum
    for _ in range(BISECT_STEPS):
        mid = 0.5 * (c_lo + c_hi)
        if _weighted_clip(mid, scores, weights, lo, hi) < goal:
            c_lo = mid
        else:
            c_hi = mid
    return [hi if math.isinf(sc) else min(max(c_hi * sc, lo), hi) for sc in scores]


def multiosr_continuous(var, nparams, layer_id, target: float, lo: float, hi: float):
    """Steps 1-3: continuous per-linear OSR (fp64 list)."""
    var = [float(v) for v in var]
    nparams = [int(n) for n in nparams]
    layer_id = [int(l) for l in layer_id]
    layers = sorted(set(layer_id))
    members = {l: [j for j in range(len(var)) if layer_id[j] == l] for l in layers}
    lay_n = []
    lay_score = []
    for l in layers:
        js = members[l]
        n_l = sum(nparams[j] for j in js)
        pooled = sum(nparams[j] * var[j] for j in js) / n_l
        lay_n.append(n_l)
        lay_score.append(math.inf if pooled <= 0 else 1.0 / pooled)
    lay_osr = _allocate(lay_score, lay_n, target, lo, hi)
    out = [0.0] * len(var)
    for l, osr_l in zip(layers, lay_osr):
        js = members[l]
        scores = [math.inf if var[j] <= 0 else nparams[j] / var[j] for j in js]
        vals = _allocate(scores, [nparams[j] for j in js], osr_l, lo, hi)
        for j, v in zip(js, vals):
            out[j] = v
    return out


def snap_to_grid(cont, nparams, target: float, lo: float, hi: float, grid: float):
    """Step 4: floor to the grid, then add steps by largest remainder within budget."""
    k_lo = math.ceil(lo / grid - 1e-9)
    k_hi = math.floor(hi / grid + 1e-9)
    ks = []
    rem = []
    for c in cont:
        q = c / grid
        k = min(max(math.floor(q + 1e-9), k_lo), k_hi)
        ks.append(k)
        rem.append(q - k)
    budget = target / grid * float(sum(nparams))
    used = sum(n * k for n, k in zip(nparams, ks))
    order = sorted(range(len(cont)), key=lambda j: (-rem[j], j))
    for j in order:
        if ks[j] + 1 <= k_hi and used + nparams[j] <= budget:
            ks[j] += 1
            used += nparams[j]
    return [k * grid for k in ks]


def multiosr(var, nparams, layer_id, target: float, lo: float, hi: float,
             grid: float = 0.125):
    """Per-linear OSR on the grid (list of floats)."""
    if not (lo <= target <= hi) or lo <= 0 or grid <= 0:
        raise ValueError("need 0 < lo <= target <= hi and grid > 0")
    if len(var) == 0:
        return []
    cont = multiosr_continuous(var, nparams, layer_id, target, lo, hi)
    return snap_to_grid(cont, [int(n) for n in nparams], target, lo, hi, grid)
