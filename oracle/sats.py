"""SATS: sensitivity-aware threshold calibration (Section 3.1, Eq. 6-10).

TEST INFRASTRUCTURE ONLY (see the package docstring).

For layer l, a candidate threshold t and a calibration input x (the layer's
input on the base path), let y(x) be the dense MLP output and y_t(x) the
output with every neuron whose post-gate magnitude |SiLU(x W_gate)_j| is
below t removed (the CATS mask of Eq. 4-5).  The local thresholding error is

    Err_l(t) = mean over x of ||y(x) - y_t(x)||_2 / (||y(x)||_2 + eps)     Eq. 6

Candidates T_l come from the calibration post-gate magnitudes, as in CATS
(Eq. 3 percentiles at a grid of levels).  For a layer-wise budget b,

    t_l*(b) = max{ t in T_l : Err_l(t) <= b }                               Eq. 7
    T*(b)   = [t_1*(b), ..., t_L*(b)]                                       Eq. 8
    S(b)    = (1/L) sum_l sp_l(t_l*(b))                                     Eq. 9
    b*      = argmin_b | S(b) - s_tar |                                     Eq. 10

with sp_l(t) the expected sparsity at layer l under t (the fraction of
calibration post-gate magnitudes below t).  The search is coarse to fine:
a coarse candidate grid first, then, per layer, denser candidates around
the threshold the coarse search chose.  The final layer keeps its CATS
threshold (Section 4, the guardrail used in the paper's experiments).

Readings where the paper is silent (listed in the design notes):
  * eps = 1e-6 (a "small constant").
  * T_l = {0} and the Eq. 3 percentile thresholds at the levels of a grid;
    t = 0 (nothing removed, Err = 0) keeps the max of Eq. 7 defined for
    every b >= 0.
  * S(b) changes only where b crosses some Err_l(t), so the budgets tried are
    exactly those values; ties of |S(b) - s_tar| go to the smallest b.
  * Refinement: the Eq. 3 percentiles at levels spaced `fine_step` apart
    strictly between the two coarse levels adjacent to the coarse level of
    the choice (so on both sides of it; the smallest coarse level whose
    percentile is the chosen threshold, 0 for t = 0), added to T_l; the
    selection is then repeated on the union.
  * The guardrail layer's sparsity counts in S(b) at its fixed threshold.

Arithmetic: float64 on the exact stored inputs, with the masked output
computed explicitly for every candidate (the definition, not a shortcut).
Parity pinned by tests: brute force on tiny shapes (Python loops over
neurons), Err(0) = 0, Err above every magnitude equal to the all-removed
value, sp against the empirical CDF, monotonicity of t*(b) and S(b), and
b* against a dense sweep of budgets.
"""
from __future__ import annotations

import numpy as np

from .calibrate import percentile_threshold
from .mlp import glue, silu
from .numerics import decode

ERR_EPS = 1e-6


def layer_terms(H, wg, wu_t, wd):
    """Dense layer on the rows of H (float64): g = SiLU(H W_gate) and the
    per-neuron products p = g * (H W_up) (Eq. 1-2), and y = p W_down."""
    H = np.asarray(H, dtype=np.float64)
    g = silu(H @ wg)
    p = g * (H @ wu_t.T)
    return g, p, p @ wd


def err_curve(H, wg, wu_t, wd, ts, eps=ERR_EPS, per_token=False):
    """Err_l(t) for every t in ts (Eq. 6), with y_t computed by masking.

    Returns err[k] (and, with per_token, e[n][k] = ||y - y_t|| / (||y|| + eps)).
    """
    g, p, y = layer_terms(H, wg, wu_t, wd)
    ny = np.linalg.norm(y, axis=1)
    e = np.zeros((len(H), len(ts)))
    for k, t in enumerate(ts):
        keep = np.abs(g) >= t              # CATS mask: removed iff |g| < t
        y_t = np.where(keep, p, 0.0) @ wd
        e[:, k] = np.linalg.norm(y - y_t, axis=1) / (ny + eps)
    err = e.mean(axis=0)
    return (err, e) if per_token else err


def sparsity_curve(g, ts):
    """sp_l(t): fraction of calibration post-gate magnitudes below t."""
    a = np.abs(np.asarray(g, dtype=np.float64)).ravel()
    return np.array([np.mean(a < t) for t in ts])


def candidates(absg, levels):
    """T_l: 0 and the Eq. 3 percentile thresholds at `levels`, ascending, distinct."""
    ts = [0.0] + [percentile_threshold(absg, q) for q in levels]
    return np.unique(np.asarray(ts, dtype=np.float64))


def select_threshold(ts, err, b):
    """t*(b) = max{t in T : Err(t) <= b} (Eq. 7); the index into ts."""
    ok = np.nonzero(np.asarray(err) <= b)[0]
    return int(ok.max()) if ok.size else 0


def select_budget(curves, s_tar, fixed=None):
    """b* over the breakpoints of S(b) (Eq. 8-10).

    curves: per layer (ts, err, sp) arrays; fixed: {layer: sparsity} for
    layers whose threshold is not chosen by the budget (the guardrail).
    Returns (b*, [index of t_l*(b*) or None for fixed layers], S(b*)).
    """
    fixed = fixed or {}
    L = len(curves)
    budgets = np.unique(np.concatenate([[0.0]] + [c[1] for i, c in enumerate(curves) if i not in fixed]))
    best = None
    for b in budgets:                      # ascending: ties keep the smallest b
        idx, s = [], 0.0
        for i, (ts, err, sp) in enumerate(curves):
            if i in fixed:
                idx.append(None)
                s += fixed[i]
            else:
                k = select_threshold(ts, err, b)
                idx.append(k)
                s += sp[k]
        s /= L
        if best is None or abs(s - s_tar) < abs(best[2] - s_tar):
            best = (float(b), idx, s)
    return best


def coarse_levels(step=0.05):
    """The coarse grid of Eq. 3 levels: step, 2 step, ..., 1 - step."""
    n = int(round(1.0 / step))
    return [round(i * step, 10) for i in range(1, n)]


def coarse_level_of(t, absg, coarse):
    """The coarse level a chosen candidate comes from: 0 for t = 0, else the
    smallest coarse level whose Eq. 3 percentile is t."""
    if t == 0.0:
        return 0.0
    return min(q for q in coarse if percentile_threshold(absg, q) == t)


def fine_levels(q, coarse, fine_step):
    """Levels fine_step apart strictly between the coarse neighbours of q
    (q itself a coarse level: the range spans both sides of it)."""
    lo = max([c for c in coarse if c < q - 1e-12], default=0.0)
    hi = min([c for c in coarse if c > q + 1e-12], default=1.0)
    out, i = [], 1
    while lo + i * fine_step < hi - 1e-9:
        out.append(round(lo + i * fine_step, 10))
        i += 1
    return out


def calibrate(x_cal, W_gate, W_up_T, W_down, s_tar, dtype, coarse_step=0.05, fine_step=0.005,
              guardrail=True, eps=ERR_EPS, layer_inputs=None):
    """SATS thresholds for a stack (coarse-to-fine search of Eq. 7-10).

    Calibration tokens run through the base stack with the inter-layer glue;
    at every layer the candidate curves are measured on that layer's inputs
    (or on layer_inputs[l], stored values, when given: lets a comparison use
    another implementation's own layer inputs).
    Returns a dict: thresholds (float32 [L]), budget b*, realized S(b*), and
    the per-layer candidate sets, error and sparsity curves of both stages.
    """
    H = decode(x_cal, dtype)
    L = len(W_gate)
    coarse = coarse_levels(coarse_step)
    layers = []
    for l in range(L):
        if layer_inputs is not None:
            H = decode(layer_inputs[l], dtype)
        wg, wu, wd = (decode(w[l], dtype) for w in (W_gate, W_up_T, W_down))
        g, p, y = layer_terms(H, wg, wu, wd)
        absg = np.abs(g)
        layers.append(dict(H=H, w=(wg, wu, wd), absg=absg))
        if l < L - 1:
            H = np.stack([glue(y[i], dtype) for i in range(len(y))])
    fixed = {}
    if guardrail and L > 1:
        t_last = percentile_threshold(layers[-1]["absg"], s_tar)
        fixed[L - 1] = float(np.mean(layers[-1]["absg"] < t_last))

    def curves_for(level_sets):
        out = []
        for l, lv in enumerate(level_sets):
            d = layers[l]
            ts = candidates(d["absg"], lv)
            err = err_curve(d["H"], *d["w"], ts, eps=eps)
            out.append((ts, err, sparsity_curve(d["absg"], ts)))
        return out

    c1 = curves_for([coarse] * L)
    b1, idx1, s1 = select_budget(c1, s_tar, fixed)
    # refinement on both sides of each layer's coarse choice (its Eq. 3 level)
    levels2 = []
    for l in range(L):
        if l in fixed:
            levels2.append(coarse)
            continue
        q = coarse_level_of(c1[l][0][idx1[l]], layers[l]["absg"], coarse)
        levels2.append(sorted(set(coarse) | set(fine_levels(q, coarse, fine_step))))
    c2 = curves_for(levels2)
    b2, idx2, s2 = select_budget(c2, s_tar, fixed)
    ts_out = np.zeros(L, dtype=np.float32)
    for l in range(L):
        ts_out[l] = np.float32(t_last if l in fixed else c2[l][0][idx2[l]])
    return dict(thresholds=ts_out, budget=b2, realized=s2, coarse=(b1, idx1, s1, c1), fine=(b2, idx2, s2, c2),
                guardrail=fixed)
