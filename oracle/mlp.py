"""Routed, threshold-sparsified gated MLP: the plain definition.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per token, independently (Section 3.2 routes on the current token alone):

  route    r = table[id]  (1: base path, 0: sparse path)         Eq. 13
  for each layer l:
    a    = h . W_gate                                               Eq. 1
    g    = a / (1 + exp(-a))                                        Eq. 2
    m_j  = 1 if r == 1 else (|g_j| >= t_l)                          Eq. 4-5
    u    = h . W_up      (W_up held transposed: u_j = W_up_T[j] . h) Eq. 1
    p_j  = g_j * u_j if m_j else 0
    y    = p . W_down                                               Eq. 1
    h    = rho(y / sqrt(mean(y^2) + 1e-6))    between layers (glue)
  out = rho(y of the last layer)

The table stores the routing decision of Eq. 13 directly: a token whose
score is below tau takes the sparse path, every other token the base path
("otherwise" in Eq. 13, so a tie goes to the base path).  No table at all
means every token takes the sparse path (the static sparse model).

The base path is the original MLP of Eq. 1; the sparse path is the same
weights with the CATS function of Eq. 5 applied to SiLU(x W_gate) (Section
3.2: both paths share the model weights, only the MLP activation changes).

Arithmetic is float64 on the exact stored values; the only roundings are
``rho`` (to the activation storage type) on each layer input after the first
and on the output.
"""
from __future__ import annotations

import numpy as np

from .numerics import decode, rho

GLUE_EPS = 1e-6


def silu(a: np.ndarray) -> np.ndarray:
    """SiLU(a) = a * sigmoid(a) = a / (1 + e^-a)   (Section 2, Eq. 2).

    Parity pinned: closed form against scipy's expit, SiLU(0) = 0, and the
    minimum -W(1/e) at a = -1 - W(1/e) (W = Lambert W).
    """
    a = np.asarray(a, dtype=np.float64)
    with np.errstate(over="ignore"):
        return a / (1.0 + np.exp(-a))


def cats_keep(g: np.ndarray, t: float) -> np.ndarray:
    """CATS_t keeps g_j when |g_j| >= t and zeroes it when |g_j| < t (Eq. 4-5).

    NaN compares false and is therefore dropped.
    """
    return np.abs(g) >= t


def route(token_ids, route_lut) -> np.ndarray:
    """Per-token path choice (Eq. 13, decisions held in the table): 1 base, 0 sparse."""
    ids = np.asarray(token_ids, dtype=np.int64)
    if route_lut is None:
        return np.zeros(ids.shape, dtype=np.uint8)
    lut = np.asarray(route_lut, dtype=np.uint8)
    return (lut[ids] != 0).astype(np.uint8)


def layer(h, W_gate, W_up_T, W_down, t, base: bool, mask=None):
    """One gated-MLP layer on one token (Eq. 1 with the Eq. 5 mask on the sparse path).

    h: float64[d]; W_gate float64[d][d_ff]; W_up_T, W_down float64[d_ff][d].
    ``mask`` (bool[d_ff]) replaces the computed keep set when given; tests use
    it to replay the GPU's own decision for gate values lying within rounding
    distance of the threshold.

    Returns (y, a, g, keep).
    """
    a = h @ W_gate                           # x W_gate
    g = silu(a)
    if mask is not None:
        keep = np.asarray(mask, dtype=bool)
    elif base:
        keep = np.ones(g.shape, dtype=bool)  # base path: the unmodified MLP
    else:
        keep = cats_keep(g, t)
    u = W_up_T @ h                           # x W_up, one entry per W_up column
    p = np.where(keep, g * u, 0.0)
    y = p @ W_down
    return y, a, g, keep


def glue(y: np.ndarray, dtype: str) -> np.ndarray:
    """Input of the next layer of a stack: rho(y / sqrt(mean(y^2) + 1e-6)).

    Not from the paper, which places each MLP inside a full transformer block;
    a gain-free RMS normalisation keeps a stack of bare MLPs at unit scale.
    Parity unpinned by the paper; pinned by invariants (zero stays zero,
    mean square ms/(ms+eps) before rounding, invariance to a positive scale).
    """
    ms = float(np.mean(y * y))
    return rho(y / np.sqrt(ms + GLUE_EPS), dtype)


def forward(x, token_ids, W_gate, W_up_T, W_down, thresholds, route_lut, dtype,
            masks=None, trace=False):
    """Full call: route, then every layer, token by token.

    x: storage [n][d]; W_*: storage [L][...]; thresholds: float[L];
    route_lut: uint8[vocab] or None; dtype: "f32" | "bf16".
    masks: optional masks[l][i] (bool[d_ff]) overriding the keep sets.

    Returns out (float64[n][d], values of the storage type) and, when
    ``trace`` is set, a dict with route, and per layer/token: layer input h,
    gate pre-activation a, g, keep set and y.
    """
    xs = decode(x, dtype)
    n, d = xs.shape
    L = len(W_gate)
    r = route(token_ids, route_lut) if n else np.zeros(0, np.uint8)
    out = np.zeros((n, d))
    tr = dict(route=r, h=[], a=[], g=[], keep=[], y=[]) if trace else None
    for l in range(L):
        if tr is not None:
            for k in ("h", "a", "g", "keep", "y"):
                tr[k].append([None] * n)
    hs = [xs[i].copy() for i in range(n)]
    for l in range(L):
        wg = decode(W_gate[l], dtype)
        wu = decode(W_up_T[l], dtype)
        wd = decode(W_down[l], dtype)
        t = float(thresholds[l])
        for i in range(n):
            m = None if masks is None else masks[l][i]
            y, a, g, keep = layer(hs[i], wg, wu, wd, t, bool(r[i]), m)
            if tr is not None:
                tr["h"][l][i] = hs[i]
                tr["a"][l][i] = a
                tr["g"][l][i] = g
                tr["keep"][l][i] = keep
                tr["y"][l][i] = y
            if l < L - 1:
                hs[i] = glue(y, dtype)
            else:
                out[i] = rho(y, dtype)
    return (out, tr) if trace else out


def forward_dense(x, W_gate, W_up_T, W_down, dtype):
    """Base path for every token (Eq. 1 unmasked), through the same glue."""
    n = len(x)
    lut = np.ones(1, dtype=np.uint8)
    return forward(x, np.zeros(n, dtype=np.int32), W_gate, W_up_T, W_down,
                   np.zeros(len(W_gate)), lut, dtype)
