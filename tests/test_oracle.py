"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a closed
form worked by hand, a library routine, an invariant of the definition, or
brute force on tiny shapes.  The last group plants mistakes in the oracle and
checks that the pins catch them.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

from oracle import calibrate, mlp, numerics
from workloads import synth

LN3 = math.log(3.0)


# --------------------------------------------------------------- bf16 storage

def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x0001, 0x7F7F, 0x3EAB], np.uint16)
    v = numerics.bf16_decode(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == 0.0
    assert v[3] == 0.0 and math.copysign(1, v[3]) == -1.0
    assert v[4] == 2.0 ** -133                      # smallest subnormal
    assert v[5] == (2 - 2 ** -7) * 2.0 ** 127       # largest finite
    assert v[6] == 0.333984375


def test_bf16_rounding_matches_torch_rne():
    rng = np.random.default_rng(5)
    f = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-39).astype(np.float32),   # subnormal range
        (rng.standard_normal(2000) * 1e30).astype(np.float32),
    ])
    # exact ties: low 16 bits 0x8000, with even and odd kept parts
    hi = rng.integers(0x0080, 0x7F00, 4000).astype(np.uint32) << 16
    ties = (hi | 0x8000).view(np.float32)
    f = np.concatenate([f, ties, -ties])
    ours = numerics.bf16_encode(f.astype(np.float64))
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


# ---------------------------------------------------------------- SiLU, Eq. 2

def test_silu_matches_expit():
    a = np.linspace(-60, 60, 10001)
    np.testing.assert_allclose(mlp.silu(a), a * scipy.special.expit(a), rtol=1e-14, atol=1e-300)


def test_silu_closed_forms():
    assert mlp.silu(np.array([0.0]))[0] == 0.0
    # sigmoid(ln 3) = 3/4, sigmoid(-ln 3) = 1/4, sigmoid(2 ln 3) = 9/10
    got = mlp.silu(np.array([LN3, -LN3, 2 * LN3]))
    np.testing.assert_allclose(got, [0.75 * LN3, -0.25 * LN3, 1.8 * LN3], rtol=1e-15)
    # minimum: d/da [a sigmoid(a)] = 0  <=>  a = -1 - W(1/e), value a + 1 = -W(1/e)
    w = scipy.special.lambertw(1 / math.e).real
    a_star = -1 - w
    assert abs(mlp.silu(np.array([a_star]))[0] - (-w)) < 1e-15
    grid = np.linspace(-5, 5, 200001)
    assert mlp.silu(grid).min() >= -w - 1e-15
    # large negative inputs give -0 without overflow trouble
    assert mlp.silu(np.array([-1e4]))[0] == 0.0


# ------------------------------------------------------- worked example, Eq. 1-5, 13

def _hand_example():
    """d = 2, d_ff = 4, x = [1, 2], weights chosen so every step has a closed form.

    a = x W_gate = [ln3, -ln3, 2 ln3, 0]
    g = SiLU(a)  = [0.75 ln3, -0.25 ln3, 1.8 ln3, 0]   (sigmoid(ln3) = 3/4 etc.)
    u = W_up_T x = [3, -1, 1, 1]
    dense: p = g u = [2.25, 0.25, 1.8, 0] ln3,  y = p W_down = [4.05, -1.55] ln3
    t = 0 keeps all four (|0| >= 0: the rule is "at least t", Eq. 4)
    t = 0.5 keeps {0, 2}: y = [4.05, -1.8] ln3
    t = 1.0 keeps {2}:    y = [1.8, -1.8] ln3
    t = 2.0 keeps none:   y = [0, 0]
    """
    wg = np.array([[LN3, LN3, 0.0, 2.0], [0.0, -LN3, LN3, -1.0]])
    wu = np.array([[1.0, 1.0], [1.0, -1.0], [-1.0, 1.0], [0.5, 0.25]])
    wd = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, -1.0], [7.0, 3.0]])
    x = np.array([1.0, 2.0])
    return x, wg, wu, wd


@pytest.mark.parametrize("t,keep,y", [
    (0.0, [1, 1, 1, 1], [4.05, -1.55]),
    (0.5, [1, 0, 1, 0], [4.05, -1.8]),
    (1.0, [0, 0, 1, 0], [1.8, -1.8]),
    (2.0, [0, 0, 0, 0], [0.0, 0.0]),
])
def test_worked_example_layer(t, keep, y):
    x, wg, wu, wd = _hand_example()
    yy, a, g, kk = mlp.layer(x, wg, wu, wd, t, base=False)
    np.testing.assert_allclose(a, [LN3, -LN3, 2 * LN3, 0.0], rtol=1e-15, atol=0)
    np.testing.assert_array_equal(kk, np.array(keep, bool))
    np.testing.assert_allclose(yy, np.array(y) * LN3, rtol=1e-14, atol=1e-15)
    # the base path ignores the threshold (Eq. 13 "base path" = unmodified MLP)
    yb, _, _, kb = mlp.layer(x, wg, wu, wd, t, base=True)
    assert kb.all()
    np.testing.assert_allclose(yb, np.array([4.05, -1.55]) * LN3, rtol=1e-14)


def test_worked_example_through_forward_and_routing():
    x, wg, wu, wd = _hand_example()
    f32 = lambda v: np.asarray(v, np.float32)
    X = f32([x, x])
    ids = np.array([3, 5], np.int32)
    lut = np.zeros(8, np.uint8)
    lut[5] = 1                                   # id 5 takes the base path
    out, tr = mlp.forward(X, ids, f32([wg]), f32([wu]), f32([wd]), np.array([1.0]), lut,
                          "f32", trace=True)
    np.testing.assert_array_equal(tr["route"], [0, 1])
    np.testing.assert_allclose(out[0], np.array([1.8, -1.8]) * LN3, rtol=2e-7)
    np.testing.assert_allclose(out[1], np.array([4.05, -1.55]) * LN3, rtol=2e-7)
    # values are float32 numbers (rho = storage rounding)
    assert np.all(out == out.astype(np.float32))


# ------------------------------------------------------------------ brute force

def _brute_forward(x, ids, wg, wu, wd, ts, lut, dtype):
    """Index-by-index loops over plain Python floats."""
    dec = lambda a: numerics.decode(a, dtype).tolist()
    X = dec(x)
    L = len(wg)
    outs = []
    for i, xi in enumerate(X):
        base = lut is not None and int(lut[int(ids[i])]) != 0
        h = list(xi)
        for l in range(L):
            G, U, D = dec(wg[l]), dec(wu[l]), dec(wd[l])
            d, dff = len(G), len(G[0])
            p = []
            for j in range(dff):
                a = 0.0
                for k in range(d):
                    a += h[k] * G[k][j]
                g = a * (1.0 / (1.0 + math.exp(-a))) if a > -700 else 0.0
                u = 0.0
                for k in range(d):
                    u += h[k] * U[j][k]
                p.append(g * u if (base or abs(g) >= ts[l]) else 0.0)
            y = []
            for c in range(d):
                s = 0.0
                for j in range(dff):
                    s += p[j] * D[j][c]
                y.append(s)
            if l < L - 1:
                ms = sum(v * v for v in y) / d
                h = numerics.rho(np.array(y) / math.sqrt(ms + 1e-6), dtype).tolist()
        outs.append(numerics.rho(np.array(y), dtype))
    return np.array(outs)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed,L,d,dff,n", [(1, 1, 3, 5, 3), (2, 2, 6, 4, 4), (3, 3, 5, 9, 2)])
def test_brute_force_tiny(dtype, seed, L, d, dff, n):
    c = synth.small_case(seed, L, d, dff, dtype, n, vocab=8, n_dense_ids=3, w_std=0.7)
    ts = np.array([0.15, 0.3, 0.05][:L])
    got = mlp.forward(c["x"], c["token_ids"], c["W_gate"], c["W_up_T"], c["W_down"], ts,
                      c["route_lut"], dtype)
    ref = _brute_forward(c["x"], c["token_ids"], c["W_gate"], c["W_up_T"], c["W_down"], ts,
                         c["route_lut"], dtype)
    # identical roundings, different summation order: at most one storage ulp apart
    tol = 1e-12 if dtype == "f32" else 0
    for i in range(n):
        scale = max(np.max(np.abs(ref[i])), 1e-30)
        assert np.max(np.abs(got[i] - ref[i])) <= max(tol, 2 ** -7) * scale


# ------------------------------------------------------------------ invariants

@pytest.fixture(scope="module")
def case():
    return synth.small_case(11, 3, 40, 96, "bf16", 6, vocab=32, n_dense_ids=8, w_std=0.15)


def _fwd(c, ts, lut, **kw):
    return mlp.forward(c["x"], c["token_ids"], c["W_gate"], c["W_up_T"], c["W_down"],
                       np.asarray(ts, float), lut, "bf16", **kw)


def test_threshold_zero_is_dense(case):
    sparse = _fwd(case, [0, 0, 0], None)
    dense = mlp.forward_dense(case["x"], case["W_gate"], case["W_up_T"], case["W_down"], "bf16")
    np.testing.assert_array_equal(sparse, dense)


def test_threshold_inf_gives_zero(case):
    out = _fwd(case, [np.inf] * 3, None)
    assert np.all(out == 0)
    out = _fwd(case, [0.0, np.inf, 0.1], None)   # a zero layer stays zero through the glue
    assert np.all(out == 0)


def test_sparse_equals_dense_on_masked_activation(case):
    """Gathered form sum_{j in A} g_j u_j W_down[j] equals the masked dense form."""
    x = numerics.decode(case["x"][0], "bf16")
    wg, wu, wd = (numerics.decode(case[k][0], "bf16") for k in ("W_gate", "W_up_T", "W_down"))
    y, a, g, keep = mlp.layer(x, wg, wu, wd, 0.05, base=False)
    A = np.nonzero(keep)[0]
    assert 0 < len(A) < len(keep)
    y_gather = np.zeros_like(y)
    for j in A:
        y_gather += (g[j] * float(wu[j] @ x)) * wd[j]
    np.testing.assert_allclose(y, y_gather, rtol=1e-12, atol=1e-15)
    # and the masked activation pushed through the unmasked formula
    gm = np.where(keep, g, 0.0)
    np.testing.assert_allclose(y, (gm * (wu @ x)) @ wd, rtol=1e-12, atol=1e-15)


def test_keep_sets_nest_and_count(case):
    x = numerics.decode(case["x"][1], "bf16")
    wg = numerics.decode(case["W_gate"][0], "bf16")
    g = mlp.silu(x @ wg)
    prev = None
    for t in [0.0, 0.01, 0.05, 0.1, 0.2, 0.5]:
        k = mlp.cats_keep(g, t)
        assert k.sum() == sum(1 for v in g if abs(v) >= t)
        if prev is not None:
            assert np.all(k <= prev)
        prev = k
    # above max |SiLU| of a negative input only positive pre-activations survive
    w = scipy.special.lambertw(1 / math.e).real
    k = mlp.cats_keep(g, w + 1e-9)
    assert np.all((x @ wg)[k] > 0)


def test_scaling_up_and_down_weights_scales_output():
    c = synth.small_case(4, 1, 16, 48, "f32", 3, w_std=0.3)
    ts = np.array([0.05])
    y1, tr1 = mlp.forward(c["x"], c["token_ids"], c["W_gate"], c["W_up_T"], c["W_down"], ts, None,
                          "f32", trace=True)
    y2, tr2 = mlp.forward(c["x"], c["token_ids"], c["W_gate"], c["W_up_T"] * 2, c["W_down"] * 4,
                          ts, None, "f32", trace=True)
    for i in range(3):
        np.testing.assert_array_equal(tr1["keep"][0][i], tr2["keep"][0][i])  # mask from gate only
        np.testing.assert_array_equal(tr2["y"][0][i], 8 * tr1["y"][0][i])


def test_routing_lut_semantics(case):
    ts = [0.05, 0.08, 0.03]
    ids = case["token_ids"]
    lut = case["route_lut"]
    out, tr = _fwd(case, ts, lut, trace=True)
    r = tr["route"]
    np.testing.assert_array_equal(r, lut[ids])
    assert 0 < r.sum() < len(r)
    dense = mlp.forward_dense(case["x"], case["W_gate"], case["W_up_T"], case["W_down"], "bf16")
    sparse = _fwd(case, ts, None)
    for i in range(len(r)):
        np.testing.assert_array_equal(out[i], dense[i] if r[i] else sparse[i])
    np.testing.assert_array_equal(_fwd(case, ts, np.ones_like(lut)), dense)
    np.testing.assert_array_equal(_fwd(case, ts, np.zeros_like(lut)), sparse)


def test_rows_are_independent_and_permutation_equivariant(case):
    ts = [0.05, 0.08, 0.03]
    lut = case["route_lut"]
    full = _fwd(case, ts, lut)
    for i in range(len(full)):
        one = mlp.forward(case["x"][i:i + 1], case["token_ids"][i:i + 1], case["W_gate"],
                          case["W_up_T"], case["W_down"], np.array(ts), lut, "bf16")
        np.testing.assert_array_equal(one[0], full[i])
    perm = np.array([3, 0, 5, 1, 4, 2])
    sub = dict(case, x=case["x"][perm], token_ids=case["token_ids"][perm])
    np.testing.assert_array_equal(_fwd(sub, ts, lut), full[perm])


def test_glue_invariants():
    rng = np.random.default_rng(3)
    y = rng.standard_normal(512) * 37.0
    ms = np.mean(y * y)
    # before rounding the mean square is ms / (ms + eps)
    h_exact = y / np.sqrt(ms + mlp.GLUE_EPS)
    assert abs(np.mean(h_exact ** 2) - ms / (ms + mlp.GLUE_EPS)) < 1e-12
    h = mlp.glue(y, "f32")
    np.testing.assert_allclose(h, h_exact, rtol=1e-7)
    np.testing.assert_array_equal(mlp.glue(np.zeros(8), "bf16"), np.zeros(8))
    np.testing.assert_array_equal(mlp.glue(y * 1024.0, "bf16"), mlp.glue(y, "bf16"))


# ------------------------------------------------------------------ calibration, Eq. 3

def test_percentile_matches_inverted_cdf_quantile():
    rng = np.random.default_rng(9)
    for n in [1, 2, 7, 10, 1000, 4099]:
        v = np.abs(rng.standard_normal(n))
        for k in [0.01, 0.3, 0.5, 0.7, 0.95, 1.0]:
            assert calibrate.percentile_threshold(v, k) == np.quantile(v, k, method="inverted_cdf")
    assert calibrate.percentile_threshold(np.array([3.0, 1.0]), 0.0) == 0.0


def test_percentile_realized_fraction_on_calibration_set():
    rng = np.random.default_rng(10)
    v = np.abs(rng.standard_normal(393216))
    for k in [0.4, 0.5, 0.6371, 0.7]:
        t = calibrate.percentile_threshold(v, k)
        m = math.ceil(k * v.size)
        assert np.count_nonzero(v < t) == m - 1        # masked share (m - 1) / N
        assert np.count_nonzero(v <= t) / v.size >= k  # F(t) >= k
        assert np.count_nonzero(v < t) / v.size < k    # no smaller sample value qualifies


def test_calibrate_stack_first_layer_and_propagation():
    c = synth.small_case(6, 2, 24, 64, "bf16", 1, w_std=0.2)
    xcal = synth.activations(6, synth.S_CAL, 50, 24, "bf16")
    ts, vals = calibrate.calibrate_stack(xcal, c["W_gate"], c["W_up_T"], c["W_down"], [0.5, 0.6],
                                         "bf16", return_values=True)
    H = numerics.decode(xcal, "bf16")
    g0 = np.abs(mlp.silu(H @ numerics.decode(c["W_gate"][0], "bf16")))
    assert ts[0] == np.float32(np.quantile(g0, 0.5, method="inverted_cdf"))
    # layer 1 sees the dense stack's glue output of layer 0
    _, tr = mlp.forward(xcal, np.zeros(50, np.int32), c["W_gate"], c["W_up_T"], c["W_down"],
                        np.zeros(2), np.ones(1, np.uint8), "bf16", trace=True)
    g1 = np.abs(np.stack(tr["g"][1]))
    assert ts[1] == np.float32(np.quantile(g1, 0.6, method="inverted_cdf"))


# ------------------------------------------------------------------ planted mistakes

def _pins_pass():
    """The closed-form example and a brute-force case, as a yes/no."""
    try:
        for t, keep, y in [(0.0, [1, 1, 1, 1], [4.05, -1.55]), (0.5, [1, 0, 1, 0], [4.05, -1.8])]:
            test_worked_example_layer(t, keep, y)
        test_brute_force_tiny("f32", 2, 2, 6, 4, 4)
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("mistake", ["silu_sign", "strict_threshold", "transposed_up",
                                     "dropped_up", "glue_no_eps_sqrt"])
def test_pins_catch_planted_mistakes(monkeypatch, mistake):
    assert _pins_pass()
    orig_layer = mlp.layer
    if mistake == "silu_sign":
        monkeypatch.setattr(mlp, "silu", lambda a: np.asarray(a) / (1 + np.exp(np.asarray(a))))
    elif mistake == "strict_threshold":
        monkeypatch.setattr(mlp, "cats_keep", lambda g, t: np.abs(g) > t)
    elif mistake == "transposed_up":
        def bad(h, wg, wu, wd, t, base, mask=None):
            wu2 = np.resize(wu.T, wu.shape)
            return orig_layer(h, wg, wu2, wd, t, base, mask)
        monkeypatch.setattr(mlp, "layer", bad)
    elif mistake == "dropped_up":
        def bad(h, wg, wu, wd, t, base, mask=None):
            return orig_layer(h, wg, np.ones_like(wu) / h.size, wd, t, base, mask)
        monkeypatch.setattr(mlp, "layer", bad)
    elif mistake == "glue_no_eps_sqrt":
        monkeypatch.setattr(mlp, "glue", lambda y, dt: numerics.rho(y / np.mean(y * y), dt))
    assert not _pins_pass()
