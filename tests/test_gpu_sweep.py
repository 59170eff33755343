"""Seeded random parity cases of the single-token path (decode batch 1) and of the batch paths.

Each case draws a shape, a precision, a number of layers, a threshold level
(CATS percentiles of Eq. 3, or t = 0), a route (with or without a routing
table, a random id) and a number of gate columns per workgroup, then checks
the library against the oracle under the rules of tests/harness.py and a
second call bit for bit.  The draws reach the cases the kernels treat apart:
workgroups that keep no row, one row or a few, groups with one to several
row batches, an odd number of gate pieces per wavefront, tilings from one
column per workgroup to a full ballot, and layers of both precisions.
"""
import numpy as np
import pytest

from harness import check_against_oracle, run_gpu
from test_gpu_parity import case_thresholds
from workloads import synth
from paper_2607_08991_amd import SATS_PATH_SINGLE_TOKEN, sats_query_path
from paper_2607_08991_amd import options as sats_options

pytestmark = pytest.mark.gpu


def draw(i):
    rng = np.random.default_rng(1000 + i)
    dtype = "bf16" if rng.random() < 0.6 else "f32"
    vec = 8 if dtype == "bf16" else 4
    big = i % 4 == 3  # every fourth case at the Llama / Qwen widths
    d = int(rng.choice([1024, 2048, 4096] if big else [64, 128, 192, 256, 320, 512, 768, 1024]))
    dff = int(rng.choice([4096, 12288, 14336] if big else [64, 128, 256, 448, 512, 1000, 1536, 3000]))
    dff -= dff % vec
    # column blocks the single-token plan accepts (at most 4096 workgroups)
    cols = [c for c in (0, 0, 1, 3, 7, 16, 33, 56, 64) if c == 0 or -(-dff // c) <= 4096]
    return dict(dtype=dtype, d=d, dff=dff, L=int(rng.integers(1, 3 if big else 4)),
                k=float(rng.choice([0.0, 0.3, 0.5, 0.7, 0.9, 0.97])),
                cols=int(rng.choice(cols)), seed=int(rng.integers(0, 10000)),
                lut=bool(rng.random() < 0.5), n_dense_ids=int(rng.integers(0, 20)), tok=int(rng.integers(0, 40)))


@pytest.mark.parametrize("i", range(48))
def test_single_token_random_case(i):
    p = draw(i)
    dtype, d, dff = p["dtype"], p["d"], p["dff"]
    c = synth.small_case(p["seed"], p["L"], d, dff, dtype, 1, vocab=40, n_dense_ids=p["n_dense_ids"],
                         w_std=1.0 / np.sqrt(d))
    ts = case_thresholds(c, dtype, k=p["k"] if p["k"] > 0 else 0.5, seed=p["seed"])
    if p["k"] == 0.0:
        ts = np.zeros_like(ts)
    lut = c["route_lut"] if p["lut"] else None
    c["token_ids"] = np.asarray([p["tok"]], np.int32)
    print(f"case {i}: {p}", flush=True)
    with sats_options(**({"dec_block_cols": p["cols"]} if p["cols"] else {})):
        assert sats_query_path(1, d, dff, 2 if dtype == "bf16" else 4) == SATS_PATH_SINGLE_TOKEN
        r1 = run_gpu(c, ts, lut, dtype)
        r2 = run_gpu(c, ts, lut, dtype)
    check_against_oracle(c, ts, lut, dtype, r1)
    for key in ("out", "layer_in", "count", "idx", "route"):
        np.testing.assert_array_equal(r1[key], r2[key])


def draw_batch(i):
    rng = np.random.default_rng(2000 + i)
    dtype = "bf16" if rng.random() < 0.75 else "f32"
    dff = int(rng.choice([64, 128, 192, 448, 512, 1024, 1536, 3072, 4096]))
    return dict(dtype=dtype, d=int(rng.choice([128, 256, 384, 512, 1024, 2048, 4096])),
                dff=dff - dff % 4 if dtype == "f32" else dff,
                n=int(rng.choice([2, 3, 5, 8, 15, 16, 17, 31, 33, 48, 63, 64, 65, 100])),
                L=int(rng.integers(1, 4)), k=float(rng.choice([0.0, 0.3, 0.5, 0.7, 0.9])),
                seed=int(rng.integers(0, 10000)), n_dense_ids=int(rng.integers(0, 40)),
                path=str(rng.choice(["auto", "split", "compact"])), lut=bool(rng.random() < 0.7))


@pytest.mark.parametrize("i", range(24))
def test_batch_random_case(i):
    """Seeded random batches of 2-100 tokens on the batch paths (the matrix-core kernels where the
    shape is on their tiles, the base-group-only split and the compacted kernels), against the
    oracle and repeated bit for bit."""
    from paper_2607_08991_amd import SATS_BATCH_COMPACT, SATS_BATCH_SPLIT
    p = draw_batch(i)
    dtype, d, dff, n = p["dtype"], p["d"], p["dff"], p["n"]
    c = synth.small_case(p["seed"], p["L"], d, dff, dtype, n, vocab=40, n_dense_ids=p["n_dense_ids"],
                         w_std=1.0 / np.sqrt(d))
    ts = case_thresholds(c, dtype, k=p["k"] if p["k"] > 0 else 0.5, seed=p["seed"])
    if p["k"] == 0.0:
        ts = np.zeros_like(ts)
    lut = c["route_lut"] if p["lut"] else None
    print(f"case {i}: {p}", flush=True)
    opt = {} if p["path"] == "auto" else {"batch_path": SATS_BATCH_SPLIT if p["path"] == "split" else SATS_BATCH_COMPACT}
    with sats_options(**opt):
        r1 = run_gpu(c, ts, lut, dtype)
        r2 = run_gpu(c, ts, lut, dtype)
    check_against_oracle(c, ts, lut, dtype, r1)
    for key in ("out", "layer_in", "count", "idx", "route"):
        np.testing.assert_array_equal(r1[key], r2[key])
