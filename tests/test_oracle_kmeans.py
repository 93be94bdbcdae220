"""Pins for the gater half of the oracle: nearest-centroid assignment (Eq. 2), k-means++
seeding, the Lloyd update with reseeding, and the fixed-iteration fit (Section 2).

Every expected value here comes from a library routine independent of the oracle (scipy's
cdist, numpy's mean / var / argsort), a closed form, or a hand-worked fixture under
tests/golden/.  Nothing comes from the HIP library."""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ------------------------------------------------------------------ assignment (Eq. 2)

def test_assign_golden(orc):
    g = _gold("assign_2d.json")
    a, d1, d2 = orc.assign(np.array(g["X"], float), np.array(g["C"], float))
    assert a.tolist() == g["a"]
    np.testing.assert_array_equal(d1, g["d1"])
    np.testing.assert_array_equal(d2, g["d2"])


@pytest.mark.parametrize("n,d,K", [(257, 3, 1), (300, 7, 5), (1000, 33, 17), (64, 128, 64)])
def test_assign_matches_scipy_cdist(orc, n, d, K):
    rs = np.random.default_rng(n + d + K)
    X = rs.normal(size=(n, d))
    C = rs.normal(size=(K, d))
    a, d1, d2 = orc.assign(X, C)
    ref = cdist(X, C, "sqeuclidean")
    assert np.array_equal(a, np.argmin(ref, axis=1))  # argmin returns the first minimum
    np.testing.assert_allclose(d1, ref.min(axis=1), rtol=1e-12, atol=1e-12)
    if K > 1:
        np.testing.assert_allclose(d2, np.sort(ref, axis=1)[:, 1], rtol=1e-12, atol=1e-12)
    else:
        assert np.all(np.isinf(d2))
        assert np.all(a == 0)


def test_assign_special_cases(orc):
    rs = np.random.default_rng(3)
    C = rs.normal(size=(6, 9))
    C[4] = C[1]  # duplicate centroid: the lower index must win
    X = np.concatenate([C, rs.normal(size=(50, 9))])
    a, d1, _ = orc.assign(X, C)
    assert a[:6].tolist() == [0, 1, 2, 3, 1, 5]
    assert np.all(d1[:6] == 0.0)
    assert not np.any(a == 4)


def test_near_tie_rule(orc):
    d1 = np.array([1.0, 1.0, 0.0, 0.0, 10.0])
    d2 = np.array([1.0 + 0.5e-5, 1.0 + 2e-5, 0.0, 1e-30, 10.0 + 0.5e-4])
    assert orc.near_tie(d1, d2).tolist() == [True, False, True, False, True]


# ------------------------------------------------------------------ k-means++ seeding

def test_kmeanspp_golden(orc):
    g = _gold("kmeanspp_1d.json")
    X = np.array(g["X"], float)
    for case in g["cases"]:
        assert orc.kmeanspp(X, 2, np.array(case["u"])).tolist() == case["idx"]


def test_kmeanspp_first_pick_and_n_equals_k(orc):
    rs = np.random.default_rng(5)
    X = rs.normal(size=(37, 4))
    u = rs.random(37)
    idx = orc.kmeanspp(X, 37, u)
    assert idx[0] == int(np.floor(u[0] * 37))
    assert sorted(idx.tolist()) == list(range(37))  # every point chosen exactly once


def test_kmeanspp_all_identical_points(orc):
    X = np.ones((5, 3))
    idx = orc.kmeanspp(X, 3, np.array([0.5, 0.3, 0.9]))
    # D^2 is zero everywhere after the first pick: the lowest unchosen rows follow.
    assert idx.tolist() == [2, 0, 1]


def test_kmeanspp_second_pick_is_d2_weighted(orc):
    """Second centre frequencies follow D^2 / sum D^2 (chi-square test over many draws)."""
    X = np.array([[0.0], [1.0], [2.0], [4.0], [7.0]])
    rs = np.random.default_rng(11)
    n_draw = 4000
    counts = np.zeros(5)
    for _ in range(n_draw):
        u = np.array([0.0, rs.random()])  # first pick is always row 0
        counts[orc.kmeanspp(X, 2, u)[1]] += 1
    D2 = (X[:, 0] - 0.0) ** 2
    expect = n_draw * D2 / D2.sum()
    mask = expect > 0
    assert counts[~mask].sum() == 0
    chi2 = ((counts[mask] - expect[mask]) ** 2 / expect[mask]).sum()
    assert chi2 < 16.27  # 3 degrees of freedom, p = 0.001


# ------------------------------------------------------------------ Lloyd update + reseed

def test_update_k1_is_mean_and_total_sum_of_squares(orc):
    rs = np.random.default_rng(7)
    X = rs.normal(size=(500, 6)) * 3 + 1
    r = orc.fit(X, 1, 3, C0=X[:1])
    np.testing.assert_allclose(r["C"][0], X.mean(axis=0), rtol=1e-6, atol=1e-6)  # fp32 store
    tss = X.var(axis=0).sum() * X.shape[0]
    np.testing.assert_allclose(r["J"][1:], tss, rtol=1e-6)
    assert np.all(r["a"] == 0)


def test_update_two_blobs_converge_in_one_step(orc):
    rs = np.random.default_rng(8)
    A = rs.normal(size=(100, 2)) + np.array([-50.0, 0.0])
    B = rs.normal(size=(80, 2)) + np.array([50.0, 0.0])
    X = np.concatenate([A, B])
    C0 = np.array([[-60.0, 0.0], [10.0, 0.0]])
    a, d1, _ = orc.assign(X, C0)
    C1, counts, _ = orc.update(X, a, d1, C0)
    np.testing.assert_allclose(C1[0], A.mean(axis=0), rtol=1e-12)
    np.testing.assert_allclose(C1[1], B.mean(axis=0), rtol=1e-12)
    assert counts.tolist() == [100, 80]


def test_reseed_golden(orc):
    g = _gold("reseed_1d.json")
    for case in g["cases"]:
        X = np.array(case["X"], float)
        C0 = np.array(case["C0"], float)
        a, d1, _ = orc.assign(X, C0)
        assert a.tolist() == case["a_in"]
        C, counts, a2 = orc.update(X, a, d1, C0, reseed=True)
        np.testing.assert_allclose(C, np.array(case["C"], float), rtol=0, atol=1e-12)
        assert a2.tolist() == case["a"]
        assert counts.tolist() == case["counts"]


def test_update_without_reseed_keeps_empty_centre(orc):
    X = np.array([[0.0], [1.0]])
    C0 = np.array([[0.0], [100.0]])
    a, d1, _ = orc.assign(X, C0)
    C, counts, a2 = orc.update(X, a, d1, C0, reseed=False)
    assert counts.tolist() == [2, 0]
    assert C.tolist() == [[0.5], [100.0]]
    assert a2.tolist() == [0, 0]


def test_fit_objective_non_increasing_and_fixed_point(orc):
    rs = np.random.default_rng(9)
    means = rs.normal(size=(12, 16)) * 2
    X = (means[rs.integers(0, 12, 3000)] + rs.normal(size=(3000, 16))).astype(np.float32)
    r = orc.fit(X, 8, 100, u=rs.random(8))
    J = r["J"]
    assert np.all(J[1:] <= J[:-1] * (1 + 1e-6))
    # the k-means++ picks are rows of X
    np.testing.assert_array_equal(r["C"].shape, (8, 16))
    # at convergence assign(update(a)) == a
    a, d1, _ = orc.assign(X, r["C"])
    C1, _, _ = orc.update(X, a, d1, r["C"])
    a1, _, _ = orc.assign(X, orc.round_store(C1, "f32"))
    assert np.array_equal(a1, a)
    # objective is the sum of squared distances to the assigned centres
    ref = cdist(X.astype(float), r["C"], "sqeuclidean")
    np.testing.assert_allclose(J[-1], ref[np.arange(3000), r["a"]].sum(), rtol=1e-9)


def test_fit_init_is_kmeanspp(orc):
    rs = np.random.default_rng(10)
    X = rs.normal(size=(200, 5)).astype(np.float32).astype(float)
    u = rs.random(6)
    r = orc.fit(X, 6, 0, u=u)
    idx = orc.kmeanspp(X, 6, u)
    assert r["init_idx"].tolist() == idx.tolist()
    np.testing.assert_array_equal(r["C"], X[idx])


def test_bf16_rounding(orc):
    # 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7: ties go to even (1.0);
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: ties go to even (1 + 2^-6).
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -3.0, 0.0, 1e-30])
    y = orc.round_store(x, "bf16")
    assert y[0] == 1.0
    assert y[1] == 1 + 2 ** -6
    assert y[2] == 1 + 2 ** -7
    assert y[3] == -3.0 and y[4] == 0.0
    # agrees with torch's own fp32 -> bf16 conversion on values exact in fp32
    import torch
    z = np.random.default_rng(0).normal(size=1000).astype(np.float32)
    tb = torch.from_numpy(z).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(orc.round_store(z.astype(float), "bf16"), tb)
