"""Pins of the LoRA-aware sparse MLP oracle (Section 5, fine-tuned routed models).

Each test checks oracle/lora.py against something other than its merged-weight
definition: a case worked by hand, the plain routed layer when the adapters
vanish, brute force over neurons with every adapter factor applied separately
and the up and down adapters restricted to the kept neurons, invariants, and
planted mistakes that the pins must catch.
"""
import math

import numpy as np
import pytest

from oracle import lora, mlp, numerics

LN3 = math.log(3.0)


def _case(seed, d=5, dff=9, r=3, scale=0.7):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal(d)
    wg = rng.standard_normal((d, dff))
    wu = rng.standard_normal((dff, d))
    wd = rng.standard_normal((dff, d))
    ad = (rng.standard_normal((d, r)), rng.standard_normal((r, dff)), rng.standard_normal((d, r)),
          rng.standard_normal((dff, r)), rng.standard_normal((dff, r)), rng.standard_normal((r, d)))
    return h, wg, wu, wd, ad, scale


def _brute(h, wg, wu, wd, ad, s, t):
    """The sparse path neuron by neuron: adapter factors applied one after the
    other, the up adapter only for kept neurons, the down adapter's first
    factor only over kept neurons."""
    A_g, B_g, A_u, B_uT, A_d, B_d = ad
    d, dff = wg.shape
    r = A_g.shape[1]
    vg = [sum(h[k] * A_g[k][i] for k in range(d)) for i in range(r)]
    vu = [sum(h[k] * A_u[k][i] for k in range(d)) for i in range(r)]
    y = [0.0] * d
    z = [0.0] * r
    for j in range(dff):
        a = sum(h[k] * wg[k][j] for k in range(d)) + s * sum(vg[i] * B_g[i][j] for i in range(r))
        g = a / (1.0 + math.exp(-a))
        if not abs(g) >= t:
            continue
        u = sum(h[k] * wu[j][k] for k in range(d)) + s * sum(vu[i] * B_uT[j][i] for i in range(r))
        p = g * u
        for c in range(d):
            y[c] += p * wd[j][c]
        for i in range(r):
            z[i] += p * A_d[j][i]
    for c in range(d):
        y[c] += s * sum(z[i] * B_d[i][c] for i in range(r))
    return np.array(y)


def test_hand_worked_two_neurons_rank_one():
    # h = (1, 0); W_gate = 0 and the gate adapter gives a = (ln 3, 0), so
    # g = (0.75 ln 3, 0); u = W_up_T h + (h A_u) B_u = (1, 0) + 2 (1, 1) = (3, 2);
    # t = 0.5 keeps neuron 0 only: p = (2.25 ln 3, 0); y = p W_down + (p A_d) B_d
    # = (2.25 ln 3, 0) + 2.25 ln 3 (0, 1).
    h = np.array([1.0, 0.0])
    wg = np.zeros((2, 2))
    wu = np.eye(2)
    wd = np.eye(2)
    ad = (np.array([[1.0], [0.0]]), np.array([[LN3, 0.0]]), np.array([[2.0], [0.0]]),
          np.array([[1.0], [1.0]]), np.array([[1.0], [1.0]]), np.array([[0.0, 1.0]]))
    y, a, g, keep = lora.layer_lora(h, wg, wu, wd, ad, 1.0, 0.5, False)
    assert a == pytest.approx([LN3, 0.0])
    assert list(keep) == [True, False]
    assert y == pytest.approx([2.25 * LN3, 2.25 * LN3], rel=1e-14)
    # the base path sees only the base weights: a = 0, so y = 0
    yb, *_ = lora.layer_lora(h, wg, wu, wd, ad, 1.0, 0.5, True)
    assert np.all(yb == 0.0)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_matches_brute_force_over_neurons(seed):
    h, wg, wu, wd, ad, s = _case(seed)
    for t in (0.0, 0.3, 1.0, 1e9):
        y, *_ = lora.layer_lora(h, wg, wu, wd, ad, s, t, False)
        np.testing.assert_allclose(y, _brute(h, wg, wu, wd, ad, s, t), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("seed", [4, 5])
def test_vanishing_adapters_give_the_plain_layer(seed):
    h, wg, wu, wd, ad, s = _case(seed)
    for t in (0.0, 0.5):
        plain = mlp.layer(h, wg, wu, wd, t, False)[0]
        np.testing.assert_array_equal(lora.layer_lora(h, wg, wu, wd, ad, 0.0, t, False)[0], plain)
        zero = tuple(np.zeros_like(m) for m in ad)
        np.testing.assert_array_equal(lora.layer_lora(h, wg, wu, wd, zero, s, t, False)[0], plain)


def test_base_path_ignores_the_adapters():
    h, wg, wu, wd, ad, s = _case(6)
    big = tuple(1e3 * m for m in ad)
    np.testing.assert_array_equal(lora.layer_lora(h, wg, wu, wd, big, s, 0.5, True)[0],
                                  mlp.layer(h, wg, wu, wd, 0.5, True)[0])


def test_threshold_zero_is_the_dense_adapted_mlp():
    # every neuron kept: y = (SiLU(h Wg') * (h Wu')) Wd' with no mask
    h, wg, wu, wd, ad, s = _case(7)
    A_g, B_g, A_u, B_uT, A_d, B_d = ad
    a = h @ wg + s * (h @ A_g) @ B_g
    u = h @ wu.T + s * (h @ A_u) @ B_uT.T
    p = mlp.silu(a) * u
    y = p @ wd + s * (p @ A_d) @ B_d
    np.testing.assert_allclose(lora.layer_lora(h, wg, wu, wd, ad, s, 0.0, False)[0], y, rtol=1e-12, atol=1e-12)


def test_output_is_affine_in_the_down_adapter():
    # the keep set does not depend on B_d, and y is linear in it
    h, wg, wu, wd, ad, s = _case(8)
    ys = []
    for c in (0.0, 1.0, 2.0):
        a2 = ad[:5] + (c * ad[5],)
        ys.append(lora.layer_lora(h, wg, wu, wd, a2, s, 0.4, False)[0])
    np.testing.assert_allclose(ys[2] - ys[1], ys[1] - ys[0], rtol=1e-11, atol=1e-11)
    assert np.abs(ys[1] - ys[0]).max() > 1e-3


def test_stack_with_zero_adapters_equals_the_plain_forward():
    rng = np.random.default_rng(9)
    L, n, d, dff, r = 2, 3, 8, 16, 8
    x = numerics.bf16_encode(rng.standard_normal((n, d)))
    W = [numerics.bf16_encode(0.3 * rng.standard_normal(s)) for s in ((L, d, dff), (L, dff, d), (L, dff, d))]
    zero = tuple(numerics.bf16_encode(np.zeros(s)) for s in ((L, d, r), (L, r, dff), (L, d, r), (L, dff, r),
                                                                (L, dff, r), (L, r, d)))
    ids = np.array([0, 1, 2], np.int32)
    lut = np.array([0, 1, 0], np.uint8)
    thr = np.array([0.1, 0.2])
    np.testing.assert_array_equal(lora.forward_lora(x, ids, *W, zero, 0.5, thr, lut, "bf16"),
                                  mlp.forward(x, ids, *W, thr, lut, "bf16"))


# ------------------------------------------------------------------ planted mistakes

def _pins_pass():
    """True when every pin above passes on the (possibly patched) oracle."""
    try:
        test_hand_worked_two_neurons_rank_one()
        for sd in (1, 2, 3):
            test_matches_brute_force_over_neurons(sd)
        test_base_path_ignores_the_adapters()
        test_threshold_zero_is_the_dense_adapted_mlp()
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("mistake", ["no_scale", "up_uses_gate_factor", "down_transposed_order",
                                     "adapters_on_base", "threshold_on_base_gate"])
def test_pins_catch_planted_mistakes(monkeypatch, mistake):
    assert _pins_pass()
    orig_eff, orig_layer = lora.effective_weights, lora.layer_lora
    if mistake == "no_scale":
        monkeypatch.setattr(lora, "effective_weights",
                            lambda wg, wu, wd, ag, bg, au, bu, a_d, b_d, s: orig_eff(wg, wu, wd, ag, bg, au, bu,
                                                                                    a_d, b_d, 1.0))
    elif mistake == "up_uses_gate_factor":
        def eff(wg, wu, wd, ag, bg, au, bu, a_d, b_d, s):
            e = orig_eff(wg, wu, wd, ag, bg, au, bu, a_d, b_d, s)
            return e[0], wu + s * (bu @ ag.T), e[2]
        monkeypatch.setattr(lora, "effective_weights", eff)
    elif mistake == "down_transposed_order":
        def eff(wg, wu, wd, ag, bg, au, bu, a_d, b_d, s):
            e = orig_eff(wg, wu, wd, ag, bg, au, bu, a_d, b_d, s)
            return e[0], e[1], wd + s * (a_d @ b_d)[::-1]
        monkeypatch.setattr(lora, "effective_weights", eff)
    elif mistake == "adapters_on_base":
        def lay(h, wg, wu, wd, adapters, s, t, base, mask=None):
            return mlp.layer(h, *lora.effective_weights(wg, wu, wd, *adapters, s), t, base, mask)
        monkeypatch.setattr(lora, "layer_lora", lay)
    elif mistake == "threshold_on_base_gate":
        def lay(h, wg, wu, wd, adapters, s, t, base, mask=None):
            if base:
                return mlp.layer(h, wg, wu, wd, t, True, mask)
            keep = mlp.cats_keep(mlp.silu(h @ wg), t) if mask is None else mask
            return mlp.layer(h, *lora.effective_weights(wg, wu, wd, *adapters, s), t, False, keep)
        monkeypatch.setattr(lora, "layer_lora", lay)
    assert not _pins_pass(), mistake
    lora.effective_weights, lora.layer_lora = orig_eff, orig_layer
