"""LoRA-aware routed sparse MLP (Section 5, "Fine-tuning Methods").

TEST INFRASTRUCTURE ONLY (see the package docstring).

The fine-tuned routed models of Section 5 keep one set of base weights for
both paths: a base-path token runs the base MLP of Eq. 1, and a sparse-path
token runs the fine-tuned sparse model, i.e. the base weights plus low-rank
(LoRA) updates, under the CATS mask.  Because both paths share the base
weights, the updates cannot be merged into them; the sparse path computes
"the thresholded base MLP computation and the LoRA update" together.

Readings (the paper names neither the adapted modules nor the rank; listed
in the design notes):
  * every layer's three MLP projections carry a rank-r adapter with scale s:
        W_gate' = W_gate + s A_g B_g      A_g [d][r],    B_g [r][d_ff]
        W_up'   = W_up   + s A_u B_u      A_u [d][r],    B_u [r][d_ff]
        W_down' = W_down + s A_d B_d      A_d [d_ff][r], B_d [r][d]
    (B_u is held transposed, B_u^T [d_ff][r], like W_up);
  * the CATS threshold applies to |SiLU(h W_gate')| (the adapted gate);
  * base-path tokens use the base weights only.

The definition written out here merges the effective weights explicitly and
runs the plain layer of ``mlp.layer`` on them, in float64 on the exact stored
values.  Pinned by tests: zero scale (or zero adapters) equals the plain
routed layer; base-path tokens ignore the adapters; a brute-force loop over
neurons that applies each adapter factor separately and restricts the up and
down adapters to the kept neurons; threshold 0 equals the dense MLP on the
effective weights; a hand-worked case with d = d_ff = 2, r = 1; linearity of
the output change in the down adapter.
"""
from __future__ import annotations

import numpy as np

from .mlp import glue, layer, route
from .numerics import decode, rho


def effective_weights(wg, wu_t, wd, ag, bg, au, bu_t, ad, bd, s):
    """W + s A B for the three projections (float64); W_up held transposed."""
    wg_e = wg + s * (ag @ bg)
    wu_t_e = wu_t + s * (bu_t @ au.T)      # (W_up + s A_u B_u)^T = W_up_T + s B_u^T A_u^T
    wd_e = wd + s * (ad @ bd)
    return wg_e, wu_t_e, wd_e


def layer_lora(h, wg, wu_t, wd, adapters, s, t, base, mask=None):
    """One layer on one token: base weights on the base path, adapted weights
    (``adapters`` = (A_g, B_g, A_u, B_u^T, A_d, B_d), float64) on the sparse path.
    Returns (y, a, g, keep) as ``mlp.layer``."""
    if base:
        return layer(h, wg, wu_t, wd, t, True, mask)
    return layer(h, *effective_weights(wg, wu_t, wd, *adapters, s), t, False, mask)


def forward_lora(x, token_ids, W_gate, W_up_T, W_down, adapters, scale, thresholds, route_lut, dtype,
                 masks=None, trace=False):
    """Full call, as ``mlp.forward`` with the sparse path on the adapted weights.

    adapters: (A_g, B_g, A_u, B_u^T, A_d, B_d), each stacked [L][...] in the
    storage type.  Returns out (and the trace dict when ``trace``).
    """
    xs = decode(x, dtype)
    n, d = xs.shape
    L = len(W_gate)
    r = route(token_ids, route_lut) if n else np.zeros(0, np.uint8)
    out = np.zeros((n, d))
    tr = dict(route=r, h=[], a=[], g=[], keep=[], y=[]) if trace else None
    hs = [xs[i].copy() for i in range(n)]
    for l in range(L):
        if tr is not None:
            for k in ("h", "a", "g", "keep", "y"):
                tr[k].append([None] * n)
        wg, wu, wd = (decode(w[l], dtype) for w in (W_gate, W_up_T, W_down))
        ad_l = tuple(decode(m[l], dtype) for m in adapters)
        t = float(thresholds[l])
        for i in range(n):
            m = None if masks is None else masks[l][i]
            y, a, g, keep = layer_lora(hs[i], wg, wu, wd, ad_l, float(scale), t, bool(r[i]), m)
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
