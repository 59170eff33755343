"""Seeded generators for every input of the routed sparse gated MLP.

Every array comes from ``numpy.random.default_rng([seed, stream, layer, ...])``
(PCG64 through SeedSequence), so the same seed yields the same bytes on any
machine with this numpy.  Large matrices are drawn in fixed row chunks, each
chunk from its own key, so the values do not depend on how many threads draw
them.

Storage formats: ``"f32"`` arrays are float32; ``"bf16"`` arrays are uint16
bit patterns of bfloat16, converted from float32 by round-to-nearest-even
(torch's conversion).  Nothing here computes any part of the method.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

# stream ids of the seed key
S_WEIGHTS, S_CAL, S_DECODE, S_IDS, S_LUT, S_KLEVEL, S_TEST = 0, 1, 2, 3, 4, 5, 6
# matrix ids inside the weight stream
M_GATE, M_UP_T, M_DOWN = 0, 1, 2
# LoRA adapter stream and its matrix ids
S_LORA = 7
# routing-corpus stream
S_ROUTE = 8
M_A_GATE, M_B_GATE, M_A_UP, M_B_UP_T, M_A_DOWN, M_B_DOWN = 0, 1, 2, 3, 4, 5
LORA_A_STD = 0.02

WEIGHT_STD = 0.02
_ROW_CHUNK = 256


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def gen(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(k) for k in key])


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """float32 array -> storage array ("f32": float32 copy, "bf16": uint16 bits)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    if dtype != "bf16":
        raise ValueError(dtype)
    import torch
    t = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16)
    return t.numpy().view(np.uint16)


def normal_matrix(rows: int, cols: int, std: float, key, dtype: str) -> np.ndarray:
    """rows x cols of N(0, std^2) in storage format; row chunk c uses key + (c,)."""
    out = np.empty((rows, cols), dtype=np.float32 if dtype == "f32" else np.uint16)
    chunks = [(r0, min(rows, r0 + _ROW_CHUNK)) for r0 in range(0, rows, _ROW_CHUNK)]

    def fill(ci):
        r0, r1 = chunks[ci]
        v = gen(*key, ci).standard_normal((r1 - r0, cols), dtype=np.float32)
        v *= np.float32(std)
        out[r0:r1] = to_storage(v, dtype)

    if len(chunks) == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(len(chunks))))
    return out


def layer_weights(seed: int, layer: int, d: int, d_ff: int, dtype: str, copy: int = 0):
    """(W_gate [d][d_ff], W_up_T [d_ff][d], W_down [d_ff][d]) of one layer.

    W_gate is in the x.W orientation of the gated MLP; W_up is stored
    transposed so that each of its d_ff rows is one contiguous column of W_up.
    """
    base = (seed, S_WEIGHTS, layer, copy)
    wg = normal_matrix(d, d_ff, WEIGHT_STD, base + (M_GATE,), dtype)
    wu = normal_matrix(d_ff, d, WEIGHT_STD, base + (M_UP_T,), dtype)
    wd = normal_matrix(d_ff, d, WEIGHT_STD, base + (M_DOWN,), dtype)
    return wg, wu, wd


def stack_weights(seed: int, n_layers: int, d: int, d_ff: int, dtype: str):
    """Stacked [L][...] weights; layer l equals ``layer_weights(seed, l, ...)``."""
    dt = np.float32 if dtype == "f32" else np.uint16
    wg = np.empty((n_layers, d, d_ff), dtype=dt)
    wu = np.empty((n_layers, d_ff, d), dtype=dt)
    wd = np.empty((n_layers, d_ff, d), dtype=dt)
    for l in range(n_layers):
        wg[l], wu[l], wd[l] = layer_weights(seed, l, d, d_ff, dtype)
    return wg, wu, wd


def lora_adapters(seed: int, layer: int, d: int, d_ff: int, rank: int, dtype: str):
    """(A_gate [d][r], B_gate [r][d_ff], A_up [d][r], B_up_T [d_ff][r], A_down [d_ff][r],
    B_down [r][d]) of one layer: A entries N(0, 0.02^2), B entries N(0, (0.1 / sqrt(r))^2),
    so that with scale 2 each adapter product is about a fifth of its weight matrix."""
    base = (seed, S_LORA, layer)
    b_std = 0.1 / float(np.sqrt(rank))
    return (normal_matrix(d, rank, LORA_A_STD, base + (M_A_GATE,), dtype),
            normal_matrix(rank, d_ff, b_std, base + (M_B_GATE,), dtype),
            normal_matrix(d, rank, LORA_A_STD, base + (M_A_UP,), dtype),
            normal_matrix(d_ff, rank, b_std, base + (M_B_UP_T,), dtype),
            normal_matrix(d_ff, rank, LORA_A_STD, base + (M_A_DOWN,), dtype),
            normal_matrix(rank, d, b_std, base + (M_B_DOWN,), dtype))


def stack_lora_adapters(seed: int, n_layers: int, d: int, d_ff: int, rank: int, dtype: str):
    """The six adapter matrices stacked [L][...]; layer l equals ``lora_adapters(seed, l, ...)``."""
    per = [lora_adapters(seed, l, d, d_ff, rank, dtype) for l in range(n_layers)]
    return tuple(np.stack([p[k] for p in per]) for k in range(6))


def activations(seed: int, stream: int, n: int, d: int, dtype: str, idx: int = 0) -> np.ndarray:
    """n x d tokens with entries N(0, 1), in storage format."""
    v = gen(seed, stream, 0, idx).standard_normal((n, d), dtype=np.float32)
    return to_storage(v, dtype)


def decode_x(cfg, n: int, idx: int = 0) -> np.ndarray:
    return activations(cfg.seed, S_DECODE, n, cfg.d, cfg.dtype, idx)


def calibration_x(cfg) -> np.ndarray:
    return activations(cfg.seed, S_CAL, cfg.n_cal, cfg.d, cfg.dtype)


def route_lut(vocab: int, n_dense: int, seed: int) -> np.ndarray:
    """uint8[vocab]: 1 for the ``n_dense`` ids first in a seeded permutation, else 0."""
    perm = gen(seed, S_LUT).permutation(vocab)
    lut = np.zeros(vocab, dtype=np.uint8)
    lut[perm[:n_dense]] = 1
    return lut


def zipf_ids(n: int, vocab: int, s: float, key) -> np.ndarray:
    """Token ids with P(id = r - 1) proportional to r^-s, r in [1, vocab] (inverse CDF)."""
    r = np.arange(1, vocab + 1, dtype=np.float64)
    cdf = np.cumsum(r ** (-s))
    cdf /= cdf[-1]
    u = gen(*key).random(n)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, vocab - 1).astype(np.int32)


def routing_corpus(seed: int, n: int, vocab: int, s: float = 1.1, split: int = 0):
    """A synthetic routing corpus (stand-in for per-occurrence next-token losses of a
    language model on the base and sparse paths): ids Zipf(s) over the vocabulary; each
    id a sensitivity k_x ~ Exp(mean 0.15) (shared by every split of one seed); base
    loss ~ Gamma(2, 1.2) nats; sparse loss = base + k_x + N(0, 0.3^2); float32.
    Returns (ids int32 [n], loss_base float32 [n], loss_sparse float32 [n])."""
    kappa = gen(seed, S_ROUTE, 0).exponential(0.15, vocab)
    ids = zipf_ids(n, vocab, s, (seed, S_ROUTE, 1, split))
    g = gen(seed, S_ROUTE, 2, split)
    lb = g.gamma(2.0, 1.2, n).astype(np.float32)
    ls = (lb + kappa[ids] + g.normal(0.0, 0.3, n)).astype(np.float32)
    return ids, lb, ls


def uniform_ids(n: int, vocab: int, key) -> np.ndarray:
    return gen(*key).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def token_ids(cfg, n: int, idx: int = 0) -> np.ndarray:
    if cfg.vocab is None:
        return np.zeros(n, dtype=np.int32)
    key = (cfg.seed, S_IDS, 0, idx)
    if cfg.id_dist == "zipf":
        return zipf_ids(n, cfg.vocab, cfg.zipf_s, key)
    return uniform_ids(n, cfg.vocab, key)


def config_lut(cfg):
    if cfg.vocab is None:
        return None
    return route_lut(cfg.vocab, cfg.n_dense_ids, cfg.seed)


def k_levels(cfg) -> np.ndarray:
    """Per-layer CATS percentile levels (float64[L])."""
    if cfg.k_fixed is not None:
        return np.full(cfg.n_layers, float(cfg.k_fixed))
    lo, hi = cfg.k_range
    return gen(cfg.seed, S_KLEVEL).uniform(lo, hi, size=cfg.n_layers)


# ---------------------------------------------------------------- small cases

def small_case(seed: int, n_layers: int, d: int, d_ff: int, dtype: str, n_tokens: int,
               vocab: int = 64, n_dense_ids: int = 16, w_std: float = 0.1):
    """A complete random input set for parity tests at arbitrary small shapes.

    Returns a dict of storage arrays: x, token_ids, W_gate, W_up_T, W_down,
    route_lut (thresholds are chosen by the caller).
    """
    wg = np.empty((n_layers, d, d_ff), dtype=np.float32 if dtype == "f32" else np.uint16)
    wu = np.empty((n_layers, d_ff, d), dtype=wg.dtype)
    wd = np.empty((n_layers, d_ff, d), dtype=wg.dtype)
    for l in range(n_layers):
        base = (seed, S_TEST, l, 0)
        wg[l] = normal_matrix(d, d_ff, w_std, base + (M_GATE,), dtype)
        wu[l] = normal_matrix(d_ff, d, w_std, base + (M_UP_T,), dtype)
        wd[l] = normal_matrix(d_ff, d, w_std, base + (M_DOWN,), dtype)
    x = activations(seed, S_TEST, n_tokens, d, dtype, idx=1)
    ids = uniform_ids(n_tokens, vocab, (seed, S_TEST, 0, 2))
    lut = route_lut(vocab, n_dense_ids, seed + 7)
    return dict(x=x, token_ids=ids, W_gate=wg, W_up_T=wu, W_down=wd, route_lut=lut)
