"""Pins for the inference tail of the oracle: t_m, the m most probable tags (Section 4.4), and
the counts behind p@m (Eq. 4) and q@m (Eq. 5).

Independent checks: numpy's lexsort and argmax, brute force with Python sets, the
hand-worked fixture tests/golden/topm_tiny.json, and the m = V identities."""
import json
import os

import numpy as np
import pytest

from paper_1704_06363_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_topm_golden(orc):
    g = json.load(open(os.path.join(GOLD, "topm_tiny.json")))
    top = orc.topm(np.array(g["logits"]), g["m"])
    assert top.tolist() == g["top"]
    p, q = orc.topm_hits(top, g["row_ptr"], g["tag"], g["q_sample"], g["q_tag"])
    assert p.tolist() == g["p_hits"] and q.tolist() == g["q_hits"]


@pytest.mark.parametrize("m", [1, 5, 10, 16])
def test_topm_matches_lexsort_with_ties(orc, m):
    rs = np.random.default_rng(m)
    L = rs.integers(-6, 7, size=(50, 40)).astype(np.float64)  # many exact ties
    top = orc.topm(L, m)
    ref = np.lexsort((np.broadcast_to(np.arange(40), L.shape), -L), axis=-1)[:, :m]
    assert np.array_equal(top, ref)


def test_top1_is_first_argmax_and_constant_rows(orc):
    rs = np.random.default_rng(3)
    L = rs.normal(size=(30, 25))
    L[5] = 2.0
    assert np.array_equal(orc.topm(L, 1)[:, 0], np.argmax(L, axis=1))
    assert orc.topm(L, 7)[5].tolist() == list(range(7))


def test_hits_brute_force_and_full_ranking(orc):
    rs = np.random.default_rng(4)
    n, V, m = 40, 30, 6
    L = rs.normal(size=(n, V))
    rp, tg = W.zipf_labels(n, V, 5, seed=5)
    qs, qt = W.q_draws(rp, tg, 500, seed=6)
    top = orc.topm(L, m)
    p, q = orc.topm_hits(top, rp, tg, qs, qt)
    for k in range(1, m + 1):
        assert p[k - 1] == sum(len(set(top[i, :k]) & set(tg[rp[i]:rp[i + 1]])) for i in range(n))
        assert q[k - 1] == sum(int(qt[s] in set(top[qs[s], :k])) for s in range(len(qs)))
    assert np.all(np.diff(p) >= 0) and np.all(np.diff(q) >= 0)
    # with every tag ranked (m = V) each positive and each draw is a hit
    full = orc.topm(L, V)
    pf, qf = orc.topm_hits(full, rp, tg, qs, qt)
    assert pf[-1] == rp[-1] and qf[-1] == len(qs)


def test_q_draws_are_labelled_and_cover_tags():
    rp, tg = W.zipf_labels(200, 50, 4, seed=7)
    qs, qt = W.q_draws(rp, tg, 5000, seed=8)
    for s, t in zip(qs[:500], qt[:500]):
        assert t in tg[rp[s]:rp[s + 1]]
    # tags are drawn uniformly over the present ones, not by frequency
    present = np.unique(tg)
    counts = np.bincount(np.searchsorted(present, qt), minlength=len(present))
    assert counts.min() > 0.5 * 5000 / len(present)
