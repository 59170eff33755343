"""Shared helpers of the GPU parity tests: upload seeded inputs, call the HIP
library through its C ABI, and compare with the CPU oracle.

Comparison rules
  * routing decisions: exact.
  * keep sets: exact for every column whose oracle gate value is not within
    1e-3 (relative) of the threshold; the GPU's list must be ascending and
    without repeats.  No band when t = 0 or t = +inf.
  * outputs: per token, max_k |o_k - r_k| / max_k |r_k| <= tol (2e-2 bf16,
    1e-5 f32), where r is the oracle re-run on the GPU's own layer input with
    the GPU's decisions substituted inside the band (so that a legitimate
    flip of a borderline column is not counted as arithmetic error).  A zero
    reference requires an exact zero.
  * layer l > 0: each layer is recomputed from the GPU's own input of that
    layer, and the GPU's input of layer l+1 is compared with the oracle's glue
    of the recomputed layer l, under the same output tolerance.
"""
from __future__ import annotations

import numpy as np

from oracle import mlp, numerics

BAND = 1e-3
TOL = {"bf16": 2e-2, "f32": 1e-5}


def torch_mod():
    import torch
    return torch


def to_dev(a, dtype: str):
    torch = torch_mod()
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def gate_dev(w_gate, dtype: str):
    """W_gate ([.., d, d_ff], the orientation of x W_gate) on the device in the
    library's layout: one row of d weights per neuron, [.., d_ff, d]."""
    return to_dev(np.ascontiguousarray(np.swapaxes(np.asarray(w_gate), -1, -2)), dtype)


def weights_dev(case, dtype: str):
    """The three weight stacks of `case` on the device, as the library takes them."""
    return gate_dev(case["W_gate"], dtype), to_dev(case["W_up_T"], dtype), to_dev(case["W_down"], dtype)


def from_dev(t):
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def act_torch_dtype(dtype):
    torch = torch_mod()
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def run_gpu(case, thresholds, lut, dtype, inspect=True, dense=False, out_is_x=False):
    """Run the library on `case` (storage arrays); returns a dict of numpy results."""
    import paper_2607_08991_amd as sats
    torch = torch_mod()
    x = case["x"]
    n, d = x.shape
    L, _, d_ff = case["W_gate"].shape
    dx = to_dev(x, dtype)
    wg, wu, wd = weights_dev(case, dtype)
    ids = to_dev(np.asarray(case["token_ids"], np.int32), dtype)
    thr = torch.tensor(np.asarray(thresholds, np.float32)).cuda()
    dl = to_dev(lut, dtype) if lut is not None else None
    out = dx if out_is_x else torch.empty((n, d), dtype=act_torch_dtype(dtype), device="cuda")
    res = {}
    if dense:
        sats.sats_mlp_dense(dx, wg, wu, wd, out, n, d, d_ff, L)
    elif inspect:
        route = torch.full((max(n, 1),), 7, dtype=torch.uint8, device="cuda")
        cnt = torch.full((L, max(n, 1)), -1, dtype=torch.int32, device="cuda")
        idx = torch.full((L, max(n, 1), d_ff), -1, dtype=torch.int32, device="cuda")
        lin = torch.empty((L, max(n, 1), d), dtype=act_torch_dtype(dtype), device="cuda")
        sats.sats_mlp_forward_inspect(dx, ids if lut is not None else None, wg, wu, wd, thr, dl, out,
                                      n, d, d_ff, L, route_out=route, active_count=cnt,
                                      active_idx=idx, layer_in=lin)
        torch.cuda.synchronize()
        res.update(route=route.cpu().numpy()[:n], count=cnt.cpu().numpy()[:, :n],
                   idx=idx.cpu().numpy()[:, :n], layer_in=from_dev(lin)[:, :n])
    else:
        sats.sats_mlp_forward(dx, ids if lut is not None else None, wg, wu, wd, thr, dl, out,
                              n, d, d_ff, L)
    torch.cuda.synchronize()
    sats.sats_device_status()
    res["out"] = from_dev(out)
    return res


def rel_err(o, r):
    o = np.asarray(o, np.float64)
    r = np.asarray(r, np.float64)
    scale = np.max(np.abs(r)) if r.size else 0.0
    if scale == 0.0:
        return 0.0 if np.all(o == 0) else np.inf
    return float(np.max(np.abs(o - r)) / scale)


def band_mask(g, t):
    if t == 0.0 or not np.isfinite(t):
        return np.zeros(g.shape, dtype=bool)
    return np.abs(np.abs(g) - t) <= BAND * t


def check_layer(h_gpu, gpu_keep_idx, gpu_cnt, wg, wu, wd, t, base, dtype):
    """Recompute one layer from the GPU's input; check the keep set; return (y, keep_used, n_band)."""
    y, a, g, keep = mlp.layer(h_gpu, wg, wu, wd, t, base)
    d_ff = g.size
    lst = np.asarray(gpu_keep_idx[:gpu_cnt])
    assert 0 <= gpu_cnt <= d_ff
    assert np.all(np.diff(lst) > 0), "keep list must be ascending without repeats"
    assert lst.size == 0 or (lst[0] >= 0 and lst[-1] < d_ff)
    gk = np.zeros(d_ff, dtype=bool)
    gk[lst] = True
    band = np.zeros(d_ff, dtype=bool) if base else band_mask(g, t)
    bad = (gk != keep) & ~band
    assert not bad.any(), f"keep set differs outside the band at columns {np.nonzero(bad)[0][:10]}"
    if band.any() and (gk != keep).any():
        y, _, _, _ = mlp.layer(h_gpu, wg, wu, wd, t, base, mask=gk)
    return y, gk, int(band.sum())


def check_against_oracle(case, thresholds, lut, dtype, res, layers=None, tokens=None, weights=None):
    """Compare an inspect run with the oracle; returns the worst relative error seen.

    `weights(l)` may supply decoded float64 (W_gate, W_up_T, W_down) of layer l
    (defaults to decoding case arrays).
    """
    x = case["x"]
    n = x.shape[0]
    L = len(thresholds)
    tokens = range(n) if tokens is None else tokens
    layers = range(L) if layers is None else layers
    tol = TOL[dtype]
    r = mlp.route(case["token_ids"], lut)
    np.testing.assert_array_equal(res["route"], r)
    # layer 0 input is the call input, bit for bit
    lin0 = res["layer_in"][0]
    np.testing.assert_array_equal(lin0.view(lin0.dtype), np.asarray(x).view(lin0.dtype))
    worst = 0.0
    for l in layers:
        if weights is not None:
            wg, wu, wd = weights(l)
        else:
            wg, wu, wd = (numerics.decode(case[k][l], dtype) for k in ("W_gate", "W_up_T", "W_down"))
        t = float(np.float32(thresholds[l]))
        for i in tokens:
            h = numerics.decode(res["layer_in"][l][i], dtype)
            y, gk, _ = check_layer(h, res["idx"][l][i], res["count"][l][i], wg, wu, wd, t,
                                   bool(r[i]), dtype)
            if l < L - 1:
                ref = mlp.glue(y, dtype)
                got = numerics.decode(res["layer_in"][l + 1][i], dtype)
            else:
                ref = numerics.rho(y, dtype)
                got = numerics.decode(res["out"][i], dtype)
            e = rel_err(got, ref)
            assert e <= tol, f"layer {l} token {i}: relative error {e:.3g} > {tol}"
            worst = max(worst, e)
    return worst
