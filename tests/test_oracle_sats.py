"""Pins of the SATS calibration oracle (Section 3.1, Eq. 6-10).

Each test checks oracle/sats.py against something other than its own code: a
closed form worked by hand, brute force over neurons in Python loops written
from the removed-neuron side of Eq. 6, the Gram-matrix form of the same
norm, invariants of the selection rules, and a dense sweep of budgets.  The
last group plants mistakes in the oracle and checks that the pins catch them.
"""
import math

import numpy as np
import pytest

from oracle import calibrate, sats
from workloads import synth

LN3 = math.log(3.0)


def _tiny(seed, n=5, d=3, dff=7):
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((n, d))
    wg = rng.standard_normal((d, dff))
    wu = rng.standard_normal((dff, d))
    wd = rng.standard_normal((dff, d))
    return H, wg, wu, wd


def _brute_err(H, wg, wu, wd, t, eps=sats.ERR_EPS):
    """Eq. 6 by loops: y - y_t is the sum of the removed neurons' terms."""
    n, d = H.shape
    dff = wg.shape[1]
    tot = 0.0
    for i in range(n):
        y = [0.0] * d
        removed = [0.0] * d
        for j in range(dff):
            a = sum(H[i][k] * wg[k][j] for k in range(d))
            g = a / (1.0 + math.exp(-a))
            u = sum(H[i][k] * wu[j][k] for k in range(d))
            for c in range(d):
                y[c] += g * u * wd[j][c]
                if abs(g) < t:
                    removed[c] += g * u * wd[j][c]
        tot += math.sqrt(sum(v * v for v in removed)) / (math.sqrt(sum(v * v for v in y)) + eps)
    return tot / n


# ------------------------------------------------------------------ Eq. 6

def test_err_closed_form_one_input_two_neurons():
    # a = (ln 3, 2 ln 3): g = (0.75 ln 3, 1.8 ln 3); u = (1, 1); W_down = (2, -1)
    # y = 1.5 ln 3 - 1.8 ln 3 = -0.3 ln 3.  A threshold between the two
    # magnitudes removes neuron 1: ||y - y_t|| = 1.5 ln 3.
    H = np.array([[1.0]])
    wg = np.array([[LN3, 2 * LN3]])
    wu = np.array([[1.0], [1.0]])
    wd = np.array([[2.0], [-1.0]])
    ts = [0.0, 1.0, 1.8 * LN3 * (1 - 1e-12), 10.0]
    err = sats.err_curve(H, wg, wu, wd, ts)
    assert err[0] == 0.0
    assert err[1] == pytest.approx(1.5 * LN3 / (0.3 * LN3 + 1e-6), rel=1e-12)
    # just below |g_2| neuron 2 is still kept (removed only below t)
    assert err[2] == pytest.approx(1.5 * LN3 / (0.3 * LN3 + 1e-6), rel=1e-12)
    assert err[3] == pytest.approx(0.3 * LN3 / (0.3 * LN3 + 1e-6), rel=1e-12)
    # candidates are sample magnitudes (Eq. 3 order statistics): a threshold
    # equal to |g_2| bit for bit keeps neuron 2 (Eq. 4-5 keep on >=)
    t2 = float(np.abs(sats.layer_terms(H, wg, wu, wd)[0][0, 1]))
    assert sats.err_curve(H, wg, wu, wd, [t2])[0] == pytest.approx(1.5 * LN3 / (0.3 * LN3 + 1e-6), rel=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_err_matches_brute_force_over_neurons(seed):
    H, wg, wu, wd = _tiny(seed)
    g = np.sort(np.abs(sats.layer_terms(H, wg, wu, wd)[0]).ravel())
    ts = [0.0] + list((g[:-1:3] + g[1::3]) / 2) + [g.max() * 2]   # between magnitudes: no ties
    err = sats.err_curve(H, wg, wu, wd, ts)
    for k, t in enumerate(ts):
        assert err[k] == pytest.approx(_brute_err(H, wg, wu, wd, t), rel=1e-10, abs=1e-14)


def test_err_matches_gram_quadratic_form():
    # ||sum_{j removed} p_j w_j||^2 = p_M^T (W W^T) p_M
    H, wg, wu, wd = _tiny(7, n=4, d=5, dff=9)
    g, p, y = sats.layer_terms(H, wg, wu, wd)
    gram = wd @ wd.T
    ts = [0.0, 0.3, 0.8, 1.5, 100.0]
    _, e = sats.err_curve(H, wg, wu, wd, ts, per_token=True)
    for i in range(len(H)):
        ny = math.sqrt(p[i] @ gram @ p[i])
        for k, t in enumerate(ts):
            pm = np.where(np.abs(g[i]) < t, p[i], 0.0)
            assert e[i, k] == pytest.approx(math.sqrt(max(pm @ gram @ pm, 0.0)) / (ny + 1e-6), rel=1e-9, abs=1e-12)


def test_err_limits():
    H, wg, wu, wd = _tiny(3)
    g, p, y = sats.layer_terms(H, wg, wu, wd)
    ny = np.linalg.norm(y, axis=1)
    err = sats.err_curve(H, wg, wu, wd, [0.0, np.abs(g).max() * 1.0001])
    assert err[0] == 0.0                                   # t = 0 removes nothing
    assert err[1] == pytest.approx(np.mean(ny / (ny + 1e-6)), rel=1e-12)   # everything removed


# ------------------------------------------------------------------ candidates and sparsity

def test_sparsity_is_empirical_cdf_strictly_below():
    v = np.array([0.1, 0.2, 0.2, 0.5, 0.9])
    assert list(sats.sparsity_curve(v, [0.0, 0.2, 0.21, 1.0])) == [0.0, 0.2, 0.6, 1.0]


def test_candidates_are_zero_and_eq3_percentiles():
    rng = np.random.default_rng(4)
    v = np.abs(rng.standard_normal(1000))
    ts = sats.candidates(v, [0.25, 0.5, 0.75])
    assert ts[0] == 0.0 and len(ts) == 4
    assert list(ts[1:]) == [float(np.quantile(v, q, method="inverted_cdf")) for q in (0.25, 0.5, 0.75)]
    # each percentile candidate masks ceil(qN) - 1 values (no ties)
    assert list(sats.sparsity_curve(v, ts[1:])) == [0.249, 0.499, 0.749]


def test_grids():
    assert sats.coarse_levels(0.25) == [0.25, 0.5, 0.75]
    assert sats.fine_levels(0.5, [0.25, 0.5, 0.75], 0.05) == [0.3, 0.35, 0.4, 0.45, 0.5, 0.55, 0.6, 0.65, 0.7]
    assert sats.fine_levels(0.2, [0.25, 0.5], 0.1) == [0.1, 0.2]


# ------------------------------------------------------------------ Eq. 7-10

def test_select_threshold_rule():
    ts = np.array([0.0, 0.1, 0.2, 0.3])
    err = np.array([0.0, 0.05, 0.2, 0.1])                 # not monotone: the max admissible t wins
    assert sats.select_threshold(ts, err, 0.0) == 0
    assert sats.select_threshold(ts, err, 0.05) == 1
    assert sats.select_threshold(ts, err, 0.1) == 3
    assert sats.select_threshold(ts, err, 0.15) == 3
    assert sats.select_threshold(ts, err, 1.0) == 3


def _random_curves(rng, L=4, K=9):
    out = []
    for _ in range(L):
        ts = np.concatenate([[0.0], np.sort(rng.uniform(0.01, 1.0, K - 1))])
        err = np.concatenate([[0.0], np.sort(rng.uniform(0.0, 0.5, K - 1)) + rng.uniform(-0.05, 0.05, K - 1)])
        err = np.maximum(err, 0.0)
        sp = np.concatenate([[0.0], np.sort(rng.uniform(0.0, 1.0, K - 1))])
        out.append((ts, err, sp))
    return out


@pytest.mark.parametrize("seed", range(5))
def test_budget_selection_matches_dense_sweep(seed):
    rng = np.random.default_rng(seed)
    curves = _random_curves(rng)
    fixed = {3: 0.4}
    s_tar = float(rng.uniform(0.2, 0.8))
    b, idx, s = sats.select_budget(curves, s_tar, fixed)
    # S(b) on a dense sweep of budgets, computed directly from Eq. 7 and 9
    best = None
    for bb in np.linspace(0.0, 0.6, 20001):
        tot = fixed[3]
        for i in range(3):
            ts, err, sp = curves[i]
            ok = [k for k in range(len(ts)) if err[k] <= bb]
            tot += sp[max(ok)]
        S = tot / 4
        if best is None or abs(S - s_tar) < best - 1e-15:
            best = abs(S - s_tar)
    assert abs(s - s_tar) == pytest.approx(best, abs=1e-12)
    assert idx[3] is None


@pytest.mark.parametrize("seed", range(3))
def test_thresholds_and_sparsity_grow_with_the_budget(seed):
    rng = np.random.default_rng(seed + 10)
    curves = _random_curves(rng)
    prev_t, prev_s = None, -1.0
    for b in np.linspace(0, 0.6, 200):
        tt = [c[0][sats.select_threshold(c[0], c[1], b)] for c in curves]
        S = np.mean([c[2][sats.select_threshold(c[0], c[1], b)] for c in curves])
        if prev_t is not None:
            assert all(x >= y for x, y in zip(tt, prev_t))
        assert S >= prev_s
        prev_t, prev_s = tt, S


def test_calibrate_stack_end_to_end_small():
    c = synth.small_case(5, 3, 16, 40, "f32", 1, w_std=0.25)
    xcal = synth.activations(905, synth.S_CAL, 48, 16, "f32")
    r = sats.calibrate(xcal, c["W_gate"], c["W_up_T"], c["W_down"], 0.5, "f32", coarse_step=0.1, fine_step=0.02)
    ts = r["thresholds"]
    # the guardrail layer keeps its CATS threshold
    cats = calibrate.calibrate_stack(xcal, c["W_gate"], c["W_up_T"], c["W_down"], [0.5] * 3, "f32")
    assert ts[2] == cats[2]
    # the other layers' thresholds are candidates whose error fits the budget
    b2, idx2, s2, c2 = r["fine"]
    for l in range(2):
        tsl, err, sp = c2[l]
        assert ts[l] == np.float32(tsl[idx2[l]]) and err[idx2[l]] <= b2
        assert not np.any(err[idx2[l] + 1:] <= b2)
    # the refined search is no further from the target than the coarse one
    assert abs(s2 - 0.5) <= abs(r["coarse"][2] - 0.5) + 1e-12
    # layer 0's curve is measured on the calibration inputs themselves
    err0 = sats.err_curve(xcal.astype(np.float64), c["W_gate"][0].astype(np.float64),
                          c["W_up_T"][0].astype(np.float64), c["W_down"][0].astype(np.float64), c2[0][0])
    np.testing.assert_allclose(err0, c2[0][1], rtol=1e-12)


# ------------------------------------------------------------------ planted mistakes

@pytest.mark.parametrize("mistake", ["no_eps", "keep_strict", "kept_not_removed", "sparsity_le"])
def test_pins_catch_planted_mistakes(monkeypatch, mistake):
    if mistake == "no_eps":
        monkeypatch.setattr(sats, "ERR_EPS", 0.0)
        orig = sats.err_curve
        monkeypatch.setattr(sats, "err_curve", lambda *a, eps=0.0, **k: orig(*a, eps=0.0, **k))
    elif mistake == "keep_strict":
        def bad(H, wg, wu, wd, ts, eps=sats.ERR_EPS, per_token=False):
            g, p, y = sats.layer_terms(H, wg, wu, wd)
            ny = np.linalg.norm(y, axis=1)
            e = np.stack([np.linalg.norm(y - np.where(np.abs(g) > t, p, 0) @ wd, axis=1) / (ny + eps)
                          for t in ts], 1)
            return (e.mean(0), e) if per_token else e.mean(0)
        monkeypatch.setattr(sats, "err_curve", bad)
    elif mistake == "kept_not_removed":
        def bad(H, wg, wu, wd, ts, eps=sats.ERR_EPS, per_token=False):
            g, p, y = sats.layer_terms(H, wg, wu, wd)
            ny = np.linalg.norm(y, axis=1)
            e = np.stack([np.linalg.norm(np.where(np.abs(g) >= t, p, 0) @ wd, axis=1) / (ny + eps)
                          for t in ts], 1)
            return (e.mean(0), e) if per_token else e.mean(0)
        monkeypatch.setattr(sats, "err_curve", bad)
    elif mistake == "sparsity_le":
        monkeypatch.setattr(sats, "sparsity_curve",
                            lambda g, ts: np.array([np.mean(np.abs(np.ravel(g)) <= t) for t in ts]))
    caught = 0
    for pin in (test_err_closed_form_one_input_two_neurons, test_err_limits,
                test_sparsity_is_empirical_cdf_strictly_below, test_candidates_are_zero_and_eq3_percentiles,
                lambda: test_err_matches_brute_force_over_neurons(0)):
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught >= 1, f"no pin caught the planted mistake {mistake}"


# ------------------------------------------------------------------ refinement

def _one_layer_refined(s_tar, seed=7, one_sided=False, monkeypatch=None):
    c = synth.small_case(seed, 1, 16, 64, "f32", 1, w_std=0.25)
    xcal = synth.activations(907, synth.S_CAL, 96, 16, "f32")
    if one_sided:  # the mistake: refine only below the coarse choice
        orig = sats.fine_levels
        monkeypatch.setattr(sats, "fine_levels",
                            lambda q, coarse, f: [v for v in orig(q, coarse, f) if v < q - 1e-12])
    return sats.calibrate(xcal, c["W_gate"], c["W_up_T"], c["W_down"], s_tar, "f32", coarse_step=0.1,
                          fine_step=0.01, guardrail=False)


def test_refinement_spans_both_sides_of_the_coarse_choice(monkeypatch):
    """Section 3.1 refines the search around the coarse choice.  One layer
    whose error curve grows with t: S(b) can reach every candidate's
    sparsity, so b* picks the candidate nearest s_tar.  At s_tar = 0.52 the
    coarse grid (step 0.1) chooses level 0.5, and the nearest refined level
    (0.52) lies ABOVE it: a refinement that looks only below the coarse
    choice cannot get closer than the coarse 0.5."""
    r = _one_layer_refined(0.52)
    b1, idx1, s1, c1 = r["coarse"]
    b2, idx2, s2, c2 = r["fine"]
    ts, err, sp = c2[0]
    assert np.all(np.diff(err) >= 0), "precondition: the error grows with the threshold"
    N = 96 * 64
    assert abs(s1 - 0.5) <= 2.0 / N                       # the coarse choice: level 0.5
    assert abs(s2 - 0.52) <= 2.0 / N                      # the refined choice: level 0.52, above it
    assert ts[idx2[0]] > c1[0][0][idx1[0]]
    # the candidate nearest the target among all refined ones
    assert abs(s2 - 0.52) == pytest.approx(np.min(np.abs(sp - 0.52)), abs=1e-15)
    # and a refinement below the coarse choice only stays at 0.5: the pin catches it
    bad = _one_layer_refined(0.52, one_sided=True, monkeypatch=monkeypatch)
    assert abs(bad["fine"][2] - 0.52) > abs(s2 - 0.52) + 0.01


def test_coarse_level_of_a_candidate():
    v = np.abs(np.random.default_rng(3).standard_normal(1000))
    coarse = [0.25, 0.5, 0.75]
    assert sats.coarse_level_of(0.0, v, coarse) == 0.0
    for q in coarse:
        assert sats.coarse_level_of(float(np.quantile(v, q, method="inverted_cdf")), v, coarse) == q
