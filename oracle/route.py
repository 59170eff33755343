"""Routing-table construction (Section 3.2, Eq. 11-14).

TEST INFRASTRUCTURE ONLY (see the package docstring).

From a routing corpus with per-occurrence next-token losses of the base and
sparse paths, each vocabulary id gets a score, the mean excess damage of the
sparse path over its occurrences; a threshold tau on the score picks the
path of each id, and tau is calibrated on a held-out split so that the
fraction of tokens routed to the sparse path is as close as possible to a
target:

    d_i    = max(0, l_sparse,i - l_base,i)                               Eq. 11
    s(x)  ~= E[d_i | x_i = x], estimated over I_x = {i : x_i = x}        Eq. 12
    route(x; tau) = sparse if s(x) < tau, else base                      Eq. 13
    tau*   = argmin_tau |R(tau) - r_tar|                                 Eq. 14
    R(tau) = fraction of held-out occurrences routed to the sparse path

Readings (listed in the design notes):
  * the estimator's own equation is missing from the text (it introduces
    "the token score is estimated as" and then shows Eq. 13): the empirical
    mean over I_x; an id without occurrences has no estimate and takes the
    base path (score +inf);
  * d_i is formed in float32 from float32 losses, then rounded to a multiple
    of 2^-32 (round half to even) so that the per-id sums S_x (in units of
    2^-32) are exact integers whatever the order of addition;
    s(x) = 2^-32 (double(S_x) / double(|I_x|)) in IEEE double arithmetic (the
    decision s(x) < tau is taken on that value);
  * the candidate thresholds are the distinct finite scores of the held-out
    ids and +inf (R only changes there); ties of |R - r_tar| go to the
    smallest tau, and R(tau) = double(count) / double(n_heldout);
  * the table stores the decision: 1 = base path, 0 = sparse path.

Parity pinned by tests: a hand-worked corpus, brute force with Python loops
and exact rationals, invariants of R(tau) and of the table.
"""
from __future__ import annotations

import math

import numpy as np

Q_BITS = 32  # d_i in units of 2^-32


def excess_damage(loss_base, loss_sparse):
    """d_i = max(0, l_sparse - l_base) in float32 (Eq. 11)."""
    lb = np.asarray(loss_base, dtype=np.float32)
    ls = np.asarray(loss_sparse, dtype=np.float32)
    d = (ls - lb).astype(np.float32)
    return np.maximum(d, np.float32(0.0))


def quantize(d):
    """d_i as integers in units of 2^-Q_BITS, rounded half to even (exact Python ints)."""
    return [round(float(v) * (1 << Q_BITS)) for v in np.asarray(d, dtype=np.float32)]


def scores(ids, loss_base, loss_sparse, vocab):
    """s(x) for every id (Eq. 12 by the empirical mean); +inf for ids without occurrences.

    Returns (scores float64[vocab], sums [vocab] Python ints, counts int64[vocab]).
    """
    q = quantize(excess_damage(loss_base, loss_sparse))
    sums = [0] * vocab
    counts = np.zeros(vocab, dtype=np.int64)
    for x, v in zip(np.asarray(ids, dtype=np.int64), q):
        sums[x] += v
        counts[x] += 1
    s = np.full(vocab, np.inf)
    for x in range(vocab):
        if counts[x]:
            s[x] = math.ldexp(float(sums[x]) / float(counts[x]), -Q_BITS)  # power-of-two scaling: exact
    return s, sums, counts


def routed_fraction(score, ids_heldout, tau):
    """R(tau): fraction of held-out occurrences whose id takes the sparse path (Eq. 13)."""
    ids = np.asarray(ids_heldout, dtype=np.int64)
    if ids.size == 0:
        return 0.0
    return float(np.count_nonzero(score[ids] < tau)) / float(ids.size)


def select_tau(score, ids_heldout, r_tar):
    """tau* = argmin |R(tau) - r_tar| over the candidate thresholds (Eq. 14).

    Returns (tau*, R(tau*)).
    """
    ids = np.asarray(ids_heldout, dtype=np.int64)
    fin = score[ids][np.isfinite(score[ids])]
    cands = list(np.unique(fin)) + [np.inf]
    best = None
    for tau in cands:                      # ascending: ties keep the smallest tau
        r = routed_fraction(score, ids, tau)
        if best is None or abs(r - r_tar) < abs(best[1] - r_tar):
            best = (float(tau), r)
    return best


def route_table(score, tau):
    """uint8[vocab]: 1 = base path, 0 = sparse path (Eq. 13)."""
    return np.where(np.asarray(score) < tau, 0, 1).astype(np.uint8)


def build(ids, loss_base, loss_sparse, ids_heldout, vocab, r_tar):
    """The whole construction: (table, tau*, R(tau*), scores)."""
    s, _, _ = scores(ids, loss_base, loss_sparse, vocab)
    tau, r = select_tau(s, ids_heldout, r_tar)
    return route_table(s, tau), tau, r, s
