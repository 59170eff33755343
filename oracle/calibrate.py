"""CATS percentile thresholds (Section 2, Eq. 3).  TEST INFRASTRUCTURE ONLY.

For a sparsity level k, CATS takes the activations of a calibration subset and
sets the threshold to their k-th percentile: with F the empirical distribution
function of the pooled values |SiLU(x W_gate)|,

    t = min{ t' : F(t') >= k }.

F(t') = #{v <= t'} / N jumps only at sample values, so the minimum is the
order statistic v_(m), m = ceil(k N) (1-based), for 0 < k <= 1, with k read
as the decimal fraction it is written as.  For k <= 0
every t' qualifies; the threshold is then 0, which keeps every activation.

Parity pinned: equals numpy.quantile(v, k, method="inverted_cdf"); on the
calibration set itself (no ties) exactly m - 1 of the N values fall below t.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

from .mlp import silu, glue
from .numerics import decode


def percentile_threshold(values: np.ndarray, k: float) -> float:
    """t = min{t' : F(t') >= k} over the pooled values (Eq. 3)."""
    v = np.sort(np.asarray(values, dtype=np.float64).ravel())
    if k <= 0:
        return 0.0
    n = v.size
    # k is read as the decimal it prints as (0.01 means 1/100, not the nearest
    # binary double just above it); ceil(k N) is then exact
    m = math.ceil(Fraction(repr(float(k))) * n)
    m = min(max(m, 1), n)
    return float(v[m - 1])


def calibrate_stack(x_cal, W_gate, W_up_T, W_down, ks, dtype, return_values=False):
    """Per-layer CATS thresholds for a stack.

    Calibration tokens run through the base (unmasked) stack with the same
    inter-layer glue as the forward pass; at layer l the threshold is the
    k_l-percentile of |SiLU(h_l W_gate_l)| pooled over tokens and neurons.
    The thresholds are returned as float32 values (the type the library
    takes them in).
    """
    H = decode(x_cal, dtype)                 # [n_cal][d]
    L = len(W_gate)
    ts = np.zeros(L, dtype=np.float32)
    vals = []
    for l in range(L):
        wg = decode(W_gate[l], dtype)
        g = silu(H @ wg)
        t = percentile_threshold(np.abs(g), float(ks[l]))
        ts[l] = np.float32(t)
        if return_values:
            vals.append(np.abs(g))
        if l < L - 1:
            wu = decode(W_up_T[l], dtype)
            wd = decode(W_down[l], dtype)
            Y = (g * (H @ wu.T)) @ wd        # base path for all calibration tokens
            H = np.stack([glue(Y[i], dtype) for i in range(len(Y))])
    return (ts, vals) if return_values else ts
