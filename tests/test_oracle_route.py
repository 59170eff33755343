"""Pins of the routing-table oracle (Section 3.2, Eq. 11-14).

Each test checks oracle/route.py against something other than its own code:
a corpus worked by hand, brute force with Python loops and exact rationals,
invariants of R(tau) and of the table, and a dense sweep of thresholds; the
last group plants mistakes in the oracle and checks that the pins catch them.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import route


def test_hand_worked_corpus():
    # id 0: (1.0, 1.5), (2.0, 1.0) -> d = 0.5, 0 -> s = 0.25; id 1: (1, 3) -> 2;
    # id 2: (0.5, 0.5) twice -> 0; id 3: never seen -> +inf (base path)
    ids = [0, 0, 1, 2, 2]
    lb = [1.0, 2.0, 1.0, 0.5, 0.5]
    ls = [1.5, 1.0, 3.0, 0.5, 0.5]
    s, sums, counts = route.scores(ids, lb, ls, 4)
    assert list(s[:3]) == [0.25, 2.0, 0.0] and s[3] == np.inf
    assert list(counts) == [2, 1, 2, 0]
    held = [0, 1, 2, 2, 3, 0]
    # candidates 0, 0.25, 2, inf -> R = 0, 2/6, 4/6, 5/6
    assert [route.routed_fraction(s, held, t) for t in (0.0, 0.25, 2.0, np.inf)] == [0.0, 2 / 6, 4 / 6, 5 / 6]
    for r_tar, tau, table in ((0.6, 2.0, [0, 1, 0, 1]), (0.9, np.inf, [0, 0, 0, 1]), (0.0, 0.0, [1, 1, 1, 1]),
                              (0.3, 0.25, [1, 1, 0, 1])):
        t, r = route.select_tau(s, held, r_tar)
        assert t == tau, r_tar
        assert list(route.route_table(s, t)) == table


def test_exact_tie_goes_to_the_smallest_threshold():
    # scores 0, 1, 2, 3 and one held-out occurrence each: R moves in exact quarters,
    # so r_tar = 0.375 is exactly as far from R(1) = 0.25 as from R(2) = 0.5
    s, _, _ = route.scores([0, 1, 2, 3], [1.0] * 4, [1.0, 2.0, 3.0, 4.0], 4)
    assert list(s) == [0.0, 1.0, 2.0, 3.0]
    tau, r = route.select_tau(s, [0, 1, 2, 3], 0.375)
    assert (tau, r) == (1.0, 0.25)
    assert list(route.route_table(s, tau)) == [0, 1, 1, 1]


def _case(seed, n=400, nh=300, vocab=37):
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, vocab - 3, n)           # the last ids never occur in the routing split
    lb = rng.gamma(2.0, 1.0, n).astype(np.float32)
    ls = (lb + rng.normal(0.2, 0.5, n)).astype(np.float32)
    held = rng.integers(0, vocab, nh)
    return ids, lb, ls, held, vocab


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_scores_match_exact_rational_loops(seed):
    ids, lb, ls, held, V = _case(seed)
    s, _, counts = route.scores(ids, lb, ls, V)
    for x in range(V):
        occ = [i for i in range(len(ids)) if ids[i] == x]
        if not occ:
            assert s[x] == np.inf
            continue
        tot = Fraction(0)
        for i in occ:
            d = max(np.float32(0.0), np.float32(ls[i]) - np.float32(lb[i]))   # float32 difference
            tot += Fraction(round(Fraction(float(d)) * 2 ** 32))              # half-even on the exact value
        assert counts[x] == len(occ)
        assert s[x] == float(tot / len(occ)) / 2 ** 32   # the correctly rounded mean (sums below 2^53)
        assert abs(s[x] - np.mean([max(0.0, float(np.float32(ls[i]) - np.float32(lb[i]))) for i in occ])) < 1e-9


@pytest.mark.parametrize("seed", [4, 5])
def test_tau_against_a_dense_sweep(seed):
    ids, lb, ls, held, V = _case(seed)
    s, _, _ = route.scores(ids, lb, ls, V)
    for r_tar in (0.0, 0.1, 0.37, 0.5, 0.8, 1.0):
        tau, r = route.select_tau(s, held, r_tar)
        assert r == route.routed_fraction(s, held, tau)
        # no threshold does better: every score, midpoints and extremes
        fin = np.unique(s[np.isfinite(s)])
        sweep = list(fin) + list((fin[1:] + fin[:-1]) / 2) + [-1.0, 1e9, np.inf]
        best = min(abs(route.routed_fraction(s, held, t) - r_tar) for t in sweep)
        assert abs(r - r_tar) <= best


def test_invariants():
    ids, lb, ls, held, V = _case(6)
    d = route.excess_damage(lb, ls)
    assert np.all(d >= 0) and np.all(d[ls <= lb] == 0)
    s, _, counts = route.scores(ids, lb, ls, V)
    cands = sorted(set(s[held][np.isfinite(s[held])])) + [np.inf]
    rs = [route.routed_fraction(s, held, t) for t in cands]
    assert rs[0] == 0.0 and all(a <= b for a, b in zip(rs, rs[1:]))
    seen = counts[held] > 0
    assert rs[-1] == np.count_nonzero(seen) / len(held)
    for r_tar in (0.0, 0.5, 1.0):
        table, tau, r, _ = route.build(ids, lb, ls, held, V, r_tar)
        assert np.all(table[counts == 0] == 1)          # no estimate: base path
        assert np.all(table[np.asarray(s) < tau] == 0) and np.all(table[np.asarray(s) >= tau] == 1)
    assert route.build(ids, lb, ls, held, V, 0.0)[2] == 0.0
    # a token whose sparse loss never exceeds its base loss scores 0 and goes sparse for any tau > 0
    lb2 = np.array([1.0, 2.0, 3.0], np.float32)
    s2, _, _ = route.scores([5, 5, 5], lb2, lb2 - 1, 8)
    assert s2[5] == 0.0


# ------------------------------------------------------------------ planted mistakes

def _pins_pass():
    try:
        test_hand_worked_corpus()
        test_exact_tie_goes_to_the_smallest_threshold()
        for sd in (1, 2, 3):
            test_scores_match_exact_rational_loops(sd)
        for sd in (4, 5):
            test_tau_against_a_dense_sweep(sd)
        test_invariants()
    except AssertionError:
        return False
    return True


@pytest.mark.parametrize("mistake", ["no_clamp", "rule_le", "unseen_sparse", "ties_largest", "sum_not_mean"])
def test_pins_catch_planted_mistakes(monkeypatch, mistake):
    assert _pins_pass()
    if mistake == "no_clamp":
        monkeypatch.setattr(route, "excess_damage",
                            lambda lb, ls: (np.asarray(ls, np.float32) - np.asarray(lb, np.float32)).astype(np.float32))
        monkeypatch.setattr(route, "quantize",
                            lambda d: [round(float(v) * (1 << route.Q_BITS)) for v in np.asarray(d, np.float32)])
    elif mistake == "rule_le":
        monkeypatch.setattr(route, "route_table",
                            lambda score, tau: np.where(np.asarray(score) <= tau, 0, 1).astype(np.uint8))
        monkeypatch.setattr(route, "routed_fraction",
                            lambda score, ids, tau: float(np.count_nonzero(score[np.asarray(ids)] <= tau)) / len(ids))
    elif mistake == "unseen_sparse":
        orig = route.scores

        def sc(ids, lb, ls, vocab):
            s, sums, counts = orig(ids, lb, ls, vocab)
            s = np.where(counts == 0, 0.0, s)
            return s, sums, counts
        monkeypatch.setattr(route, "scores", sc)
    elif mistake == "ties_largest":
        def sel(score, ids_heldout, r_tar):
            ids = np.asarray(ids_heldout)
            fin = score[ids][np.isfinite(score[ids])]
            best = None
            for tau in list(np.unique(fin)) + [np.inf]:
                r = route.routed_fraction(score, ids, tau)
                if best is None or abs(r - r_tar) <= abs(best[1] - r_tar):
                    best = (float(tau), r)
            return best
        monkeypatch.setattr(route, "select_tau", sel)
    elif mistake == "sum_not_mean":
        orig = route.scores

        def sc(ids, lb, ls, vocab):
            s, sums, counts = orig(ids, lb, ls, vocab)
            return np.where(counts > 0, s * np.maximum(counts, 1), s), sums, counts
        monkeypatch.setattr(route, "scores", sc)
    assert not _pins_pass(), mistake
