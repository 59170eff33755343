"""GPU parity of the routing-table construction (Eq. 11-14) through the C ABI,
against oracle/route.py.

The scores are compared bit for bit (both sides sum d in exact integer units
of 2^-32 and divide in IEEE double), so tau*, R(tau*) and the table must be
identical.  At the full vocabulary and corpus size the scores are still
compared in full; tau* is checked by its defining property over every
candidate threshold (the oracle's candidate loop is quadratic).
"""
import sys

import numpy as np
import pytest

from oracle import route
from workloads import synth

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2607_08991_amd as sats
    sats.load()


def run(ids, lb, ls, held, vocab, r_tar):
    import torch
    import paper_2607_08991_amd as sats
    dev = lambda a, dt: None if a is None or len(a) == 0 else torch.from_numpy(np.ascontiguousarray(a, dt)).cuda()
    table = torch.full((vocab,), 7, dtype=torch.uint8, device="cuda")
    scores = torch.empty(vocab, dtype=torch.float64, device="cuda")
    tau, r = sats.sats_route_table(dev(lb, np.float32), dev(ls, np.float32), dev(ids, np.int32),
                                   dev(held, np.int32), vocab, r_tar, table, scores)
    return table.cpu().numpy(), tau, r, scores.cpu().numpy()


CASES = [
    # seed, n_route, n_heldout, vocab
    (1, 1000, 500, 50),
    (2, 5000, 3000, 1000),      # two chunks and a ragged third; many ids unseen
    (3, 4096, 4096, 7),         # whole chunks of few ids: long runs
    (4, 0, 300, 40),            # empty routing split: every score +inf
    (5, 2000, 0, 40),           # empty held-out split
]


@pytest.mark.parametrize("seed,n,nh,vocab", CASES)
def test_route_table_matches_oracle(seed, n, nh, vocab):
    say(f"route case seed={seed} n={n} nh={nh} vocab={vocab}")
    ids, lb, ls = synth.routing_corpus(seed, n, vocab)
    held = synth.routing_corpus(seed, nh, vocab, split=1)[0]
    s_ref, _, _ = route.scores(ids, lb, ls, vocab)
    for r_tar in (0.0, 0.25, 0.5, 0.75, 1.0):
        table, tau, r, s = run(ids, lb, ls, held, vocab, r_tar)
        np.testing.assert_array_equal(s, s_ref)
        t_ref, r_ref = route.select_tau(s_ref, held, r_tar)
        assert (tau, r) == (t_ref, r_ref), (r_tar, tau, t_ref)
        np.testing.assert_array_equal(table, route.route_table(s_ref, t_ref))


def test_out_of_range_id_is_an_error():
    import paper_2607_08991_amd as sats
    ids, lb, ls = synth.routing_corpus(6, 100, 20)
    ids = ids.copy()
    ids[17] = 20
    with pytest.raises(sats.SatsError) as e:
        run(ids, lb, ls, ids[:10] % 20, 20, 0.5)
    assert "outside" in str(e.value)


def test_route_table_full_vocabulary():
    """Vocabulary 128256, 2^22 routing occurrences and 2^20 held-out ones, Zipf(1.1) ids."""
    V, n, nh = 128256, 1 << 22, 1 << 20
    ids, lb, ls = synth.routing_corpus(7, n, V)
    held = synth.routing_corpus(7, nh, V, split=1)[0]
    say("full-size oracle scores")
    s_ref, _, _ = route.scores(ids, lb, ls, V)
    for r_tar in (0.25, 0.5, 0.75):
        table, tau, r, s = run(ids, lb, ls, held, V, r_tar)
        np.testing.assert_array_equal(s, s_ref)
        # tau* by its definition: every candidate (distinct finite held-out scores, +inf) is no closer
        hs = s_ref[held]
        fin = np.sort(hs[np.isfinite(hs)])
        cands = np.unique(fin)
        below = np.searchsorted(fin, cands, side="left")            # occurrences scoring below each candidate
        rs = np.concatenate([below / nh, [fin.size / nh]])
        err = np.abs(rs - r_tar)
        k = int(np.argmin(err))                                      # first minimum: the smallest tau on ties
        t_ref = float(np.append(cands, np.inf)[k])
        assert tau == t_ref and r == rs[k]
        assert r == route.routed_fraction(s_ref, held, tau)
        np.testing.assert_array_equal(table, route.route_table(s_ref, tau))
        say(f"  r_tar {r_tar}: tau {tau:.6g}, R {r:.4f}, sparse ids {int((table == 0).sum())}")


@pytest.mark.parametrize("vocab", [1_500_000, 1 << 22, (1 << 22) + 4099])
def test_route_table_wide_vocabularies(vocab):
    """Id ranges of 2048 and 4096 ids (the widest the partitioned sums take),
    and a vocabulary past 2^22 ids, whose chunk tables are added with global
    atomics instead.  A third of the ids are drawn uniformly over the whole
    vocabulary so that every range is hit; these calls also reuse the kept
    device buffers at other sizes."""
    n, nh = 20000, 3000
    ids, lb, ls = synth.routing_corpus(8, n, vocab)
    held = synth.routing_corpus(8, nh, vocab, split=1)[0]
    ids, held = ids.copy(), held.copy()
    ids[::3] = synth.uniform_ids(n, vocab, (8, synth.S_ROUTE, 7))[::3]
    held[::3] = synth.uniform_ids(nh, vocab, (8, synth.S_ROUTE, 8))[::3]
    say(f"route wide vocabulary {vocab}")
    s_ref, _, _ = route.scores(ids, lb, ls, vocab)
    for r_tar in (0.3, 0.6):
        table, tau, r, s = run(ids, lb, ls, held, vocab, r_tar)
        np.testing.assert_array_equal(s, s_ref)
        t_ref, r_ref = route.select_tau(s_ref, held, r_tar)
        assert (tau, r) == (t_ref, r_ref), (r_tar, tau, t_ref)
        np.testing.assert_array_equal(table, route.route_table(s_ref, t_ref))
