"""Parity at the full workload sizes, in the launch configuration the bench times.

The oracle cannot redo a whole full-size step, so each test checks what it can compute one
sample (or one expert) at a time -- sampled rows of the assignment, the expert outputs, the
loss and dX; the complete gradients of the experts that receive only a few samples; k-means++
picks and one Lloyd update -- plus properties that hold at any size.  Oracle inputs come from
the generators only."""
import numpy as np
import pytest
import torch
from scipy.spatial.distance import cdist

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import RTOL, assert_assign, assert_close, assert_grad_close, np64, npi

pytestmark = pytest.mark.gpu
RT = RTOL["bf16"]


def _rows(t, idx):
    return np64(t[torch.as_tensor(idx, dtype=torch.long, device=t.device)])


def _sub_labels(rp, tg, idx):
    cnt = rp[1:] - rp[:-1]
    sub_rp = np.concatenate([[0], np.cumsum(cnt[idx])]).astype(np.int32)
    sub_tg = np.concatenate([tg[rp[i]:rp[i + 1]] for i in idx]).astype(np.int32)
    return sub_rp, sub_tg


def _routed_step(inp, ids=None):
    s = inp["shape"]
    X = inp["X"]
    if ids is None:
        a, md = hmoe.kmeans_assign(X, inp["C"])
    else:
        a, md = torch.as_tensor(ids, dtype=torch.int32).cuda(), None
    d = hmoe.moe_dispatch(a, s["K"], rows=X)
    rp = torch.as_tensor(inp["row_ptr"]).cuda()
    tg = torch.as_tensor(inp["tag"]).cuda()
    f = hmoe.moe_forward(inp["params"], d["rows_sorted"], d["offsets"], d["perm"], rp, tg,
                         save_logits=True)
    g = hmoe.moe_backward(inp["params"], d["rows_sorted"], d["offsets"], d["perm"], d["inv"], rp,
                          tg, f["H1_sorted"], f["H"], f["lse"], logits=f["logits"],
                          logit_anchor=f["logit_anchor"])
    torch.cuda.synchronize()
    return a, md, d, f, g


def _check_sampled_rows(inp, a_np, d, f, g, rows):
    """Oracle forward + per-sample backward on `rows` (scale 1/n of the full batch)."""
    s = inp["shape"]
    p = inp["params"]
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    Xs = _rows(inp["X"], rows)
    srp, stg = _sub_labels(inp["row_ptr"], inp["tag"], rows)
    ids = a_np[rows]
    ref = O.moe_forward(Xs, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], srp, stg,
                        store="bf16")
    inv = npi(d["inv"])
    assert_close(_rows(f["H1_sorted"], inv[rows]), ref["H1"], RT, "H1 (sampled rows)")
    assert_close(_rows(f["H"], rows), ref["H"], RT, "H (sampled rows)")
    assert_close(np64(f["lse"])[rows], ref["lse"], RT, "lse (sampled rows)")
    assert_close(np64(f["loss"])[rows], ref["loss"], RT, "loss (sampled rows)")
    args = (Xs, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], srp, stg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, scale=1.0 / s["n"], store="bf16")
    gm = O.moe_backward(*args, scale=1.0 / s["n"], magnitude=True)
    assert_grad_close(_rows(g["dX"], rows), gr["dX"], gm["dX"], "bf16", "dX (sampled rows)")
    return ph


def _check_invariants(inp, f, g, ph):
    # softmax rows sum to one and the targets carry unit mass: sum_j dbD_j = 0, sum_v dD_v = 0
    dbD = np64(g["dbD"])
    assert abs(dbD.sum()) <= 1e-3 * np.abs(dbD).sum()
    dD = np64(g["dD"])
    assert np.all(np.abs(dD.sum(axis=0)) <= 1e-2 * np.abs(dD).sum(axis=0) + 1e-12)
    # the expert-side bias gradients add up to D^T dbD (both equal sum_i D^T g_i)
    lhs = np64(g["db2"]).sum(axis=0)
    rhs = ph["D"].T @ dbD
    assert_close(lhs, rhs, RT, "sum_e db2_e vs D^T dbD")
    assert abs(float(f["loss_mean"].item()) - float(np64(f["loss"]).mean())) <= 1e-4 * abs(
        float(np64(f["loss"]).mean()))


def test_balanced_step_full_size():
    inp = W.balanced_inputs(device="cuda", seed=0)
    s = inp["shape"]
    a, md, d, f, g = _routed_step(inp)
    rs = np.random.default_rng(0)
    # gater assignment on 8192 sampled rows
    rows = np.sort(rs.choice(s["n"], 8192, replace=False))
    a_ref, d1, d2 = O.assign(_rows(inp["X"], rows), np64(inp["C"]))
    assert_assign(npi(a)[rows], a_ref, d1, d2)
    assert_close(np64(md)[rows], d1, 1e-4, "min_dist (sampled rows)")
    # buckets are roughly balanced (the centres are spread for that)
    counts = npi(d["counts"])
    assert counts.sum() == s["n"] and counts.min() > 0.5 * s["n"] / s["K"]
    # experts, decoder, loss and dX on 24 sampled rows (routed by the oracle's own ids)
    a_np = npi(a).copy()
    rows = np.sort(rs.choice(s["n"], 24, replace=False))
    a_or, d1, d2 = O.assign(_rows(inp["X"], rows), np64(inp["C"]))
    keep = ~O.near_tie(d1, d2)
    assert np.array_equal(a_np[rows][keep], a_or[keep])
    ph = _check_sampled_rows(inp, a_np, d, f, g, rows[keep])
    _check_invariants(inp, f, g, ph)


def test_skewed_step_full_size():
    inp = W.skewed_inputs(device="cuda", seed=0)
    s = inp["shape"]
    ids = inp["ids"]
    a, _, d, f, g = _routed_step(inp, ids=ids)
    counts, offsets, perm, inv = O.dispatch(ids, s["K"])
    assert npi(d["counts"]).tolist() == counts.tolist()
    assert np.array_equal(npi(d["perm"]), perm) and np.array_equal(npi(d["inv"]), inv)
    rs = np.random.default_rng(1)
    rows = np.sort(rs.choice(s["n"], 16, replace=False))
    ph = _check_sampled_rows(inp, ids, d, f, g, rows)
    _check_invariants(inp, f, g, ph)
    # the experts with 1..3 samples: their whole gradients from the oracle, run on those experts
    # alone (ids remapped to 0..m-1).  Each entry is a sum of one to three per-sample terms that
    # can cancel, so the bar takes the oracle's magnitude of each entry (assert_grad_close).
    small = np.flatnonzero((counts >= 1) & (counts <= 3))
    assert len(small) >= 4
    rows = np.flatnonzero(np.isin(ids, small))
    sub = np.searchsorted(small, ids[rows]).astype(np.int32)
    pw = {k: ph[k][small] for k in ("W1", "W2")}
    pb = {k: (ph[k][small] if ph[k] is not None else None) for k in ("b1", "b2")}
    Xs = _rows(inp["X"], rows)
    keys = ("dW1", "db1", "dW2", "db2")
    srp, stg = _sub_labels(inp["row_ptr"], inp["tag"], rows)
    ref = O.moe_forward(Xs, sub, pw["W1"], pb["b1"], pw["W2"], pb["b2"], ph["D"], ph["bD"], srp,
                        stg, store="bf16")
    args = (Xs, sub, pw["W1"], pw["W2"], ph["D"], ph["bD"], srp, stg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, scale=1.0 / s["n"], store="bf16", want_dX=False)
    gm = O.moe_backward(*args, scale=1.0 / s["n"], want_dX=False, magnitude=True)
    sel = torch.as_tensor(small, dtype=torch.long, device="cuda")
    for k in keys:
        assert_grad_close(np64(g[k][sel]), gr[k], gm[k], "bf16", k + " (experts with 1-3 samples)")
    empty = np.flatnonzero(counts == 0)
    assert len(empty) >= 2
    sel = torch.as_tensor(empty, dtype=torch.long, device="cuda")
    for k in ("dW1", "db1", "dW2", "db2"):
        assert torch.count_nonzero(g[k][sel]) == 0


def test_gater_fit_full_size():
    c = W.CONFIGS["gater_fit"]
    X = W.gmm_features(c.n, c.d, c.extra["n_comp"], seed=0, dtype="f32", device="cuda",
                       dirichlet_alpha=c.extra["alpha"])
    u = W.uniforms(c.K, 1)
    out = hmoe.kmeans_fit(X, c.K, c.n_iter, init_uniforms=u)
    torch.cuda.synchronize()
    Xh = np64(X)
    # k-means++ picks over all 2^20 rows
    idx = O.kmeanspp(Xh, c.K, u)
    assert npi(out["init_idx"]).tolist() == idx.tolist()
    # one Lloyd step from the seeding, at full size: assignment, then the update fed with the
    # oracle's assignment
    C0 = Xh[idx]
    a0, d10, d20 = O.assign(Xh, C0)
    ga, gmd = hmoe.kmeans_assign(X, torch.tensor(C0, dtype=torch.float32, device="cuda"))
    assert_assign(ga, a0, d10, d20)
    assert_close(gmd, d10, 1e-4, "min_dist")
    C1, cnt1, a1 = O.update(Xh, a0, d10, C0, reseed=True)
    at = torch.tensor(a0, dtype=torch.int32, device="cuda")
    Ct = torch.tensor(C0, dtype=torch.float32, device="cuda")
    sums = torch.zeros(c.K, c.d, dtype=torch.float64, device="cuda")
    cnt = torch.zeros(c.K, dtype=torch.int64, device="cuda")
    hmoe.kmeans_update(X, c.K, at, torch.tensor(d10, dtype=torch.float32, device="cuda"), sums, cnt,
                       Ct, mode=hmoe.UPDATE_FULL, reseed=True)
    assert npi(cnt).tolist() == cnt1.tolist()
    assert np.array_equal(npi(at), a1)
    assert_close(Ct, O.round_store(C1, "f32"), 1e-5, "centres after one update")
    # properties of the finished fit: J non-increasing, the final assignment is the nearest
    # centre (library distance on sampled rows), J_T = sum of the final min distances
    J = npi(out["objective"])
    assert np.all(J[1:] <= J[:-1] * (1 + 1e-6))
    rows = np.random.default_rng(2).choice(c.n, 4096, replace=False)
    D = cdist(Xh[rows], np64(out["C"]), "sqeuclidean")
    best = D.min(axis=1)
    fa = npi(out["assign"])[rows]
    near = np.sort(D, axis=1)[:, 1] - best <= 1e-5 * best
    assert np.all((fa == D.argmin(axis=1)) | near)
    assert abs(J[-1] - np64(out["min_dist"]).sum()) <= 1e-6 * J[-1]


def test_large_assign_full_size():
    c = W.CONFIGS["large_assign"]
    chunk = c.extra["chunk"]
    n_chunks = c.n // chunk
    means = W.gmm_means(c.extra["n_comp"], c.d, seed=2, device="cuda")
    rs = np.random.default_rng(3)
    g = torch.Generator(device="cpu").manual_seed(3)
    sums = torch.zeros(c.K, c.d, dtype=torch.float64, device="cuda")
    cnt = torch.zeros(c.K, dtype=torch.int64, device="cuda")
    Cn = torch.zeros(c.K, c.d, dtype=torch.float32, device="cuda")
    ref_sum = torch.zeros(3, c.d, dtype=torch.float64, device="cuda")
    ref_cnt = torch.zeros(3, dtype=torch.int64, device="cuda")
    probe = None
    samples_X, samples_a = [], []
    C = None
    for ci in range(n_chunks):
        x = W.gmm_features(chunk, c.d, c.extra["n_comp"], seed=100 + ci, dtype="bf16",
                           device="cuda", means=means)
        if C is None:
            C = x[torch.randperm(chunk, generator=g)[:c.K].cuda()].contiguous()
            probe = torch.tensor(rs.choice(c.K, 3, replace=False), dtype=torch.long, device="cuda")
        a, md = hmoe.kmeans_assign(x, C)
        hmoe.kmeans_update(x, c.K, a, md, sums, cnt, Cn, mode=hmoe.UPDATE_ACCUMULATE, reseed=False)
        if ci % 4 == 0:
            rows = rs.choice(chunk, 256, replace=False)
            samples_X.append(_rows(x, rows))
            samples_a.append(npi(a)[rows])
        # library reference for the update of three clusters: fp64 sums of their rows
        for q in range(3):
            m = a.long() == probe[q]
            ref_sum[q] += x[m].double().sum(dim=0)
            ref_cnt[q] += m.sum()
        del x
    hmoe.kmeans_update(None, c.K, None, None, sums, cnt, Cn, mode=hmoe.UPDATE_FINALIZE)
    torch.cuda.synchronize()
    assert int(npi(cnt).sum()) == c.n
    a_ref, d1, d2 = O.assign(np.concatenate(samples_X), np64(C))
    assert_assign(np.concatenate(samples_a), a_ref, d1, d2)
    for q in range(3):
        k = int(probe[q])
        assert int(cnt[k]) == int(ref_cnt[q])
        if int(ref_cnt[q]) > 0:
            assert_close(Cn[k], (ref_sum[q] / ref_cnt[q]).float(), 1e-5, f"centre {k}")


def test_gater_pca_full_size():
    # the bench's PCA: 2^20 fp32 rows of width 512 (a 256-component Dirichlet(0.5) mixture) to
    # 256 components with 20 subspace iterations, against the oracle's fp64 covariance of the
    # same rows and LAPACK's eigenpairs.  Its spectrum has near-equal neighbours (relative gaps
    # down to 0.2% among the leading 128) and reaches the noise floor well before 256, so
    # single directions are compared only where both neighbouring gaps exceed 2%; every one of
    # the leading 128 computed pairs must be an eigenpair of the fp64 covariance (residual),
    # and the span of the leading k is compared at the largest gap.
    c = W.CONFIGS["gater_fit"]
    r, lead = 256, 128
    X = W.gmm_features(c.n, c.d, c.extra["n_comp"], seed=0, dtype="f32", device="cuda",
                       dirichlet_alpha=c.extra["alpha"])
    mean, comps, ev = hmoe.pca_fit(X, r, 20, seed=0)
    Z = hmoe.pca_project(X, mean, comps)
    Xh = np64(X)
    m_ref, c_ref, e_ref = O.pca(Xh, r)
    assert_close(mean, m_ref, 1e-5, "mean")
    assert_close(ev[:lead], e_ref[:lead], 1e-3, "leading eigenvalues")
    U = np64(comps)[:lead]
    Cov = np.cov(Xh, rowvar=False)
    res = np.linalg.norm(Cov @ U.T - U.T * np64(ev)[:lead], axis=0)
    assert res.max() < 1e-3 * e_ref[0], res.max() / e_ref[0]
    gap = (e_ref[:-1] - e_ref[1:]) / e_ref[:-1]
    single = [j for j in range(1, lead) if gap[j - 1] > 0.02 and gap[j] > 0.02]
    assert len(single) >= 8
    cos = np.abs(np.sum(U[single] * c_ref[single], axis=1))
    assert cos.min() > 0.999, cos.min()
    k = 16 + int(np.argmax(gap[16:lead]))  # span of the leading k + 1 at the largest gap
    sv = np.linalg.svd(U[:k + 1] @ c_ref[:k + 1].T, compute_uv=False)
    assert sv.min() > 0.999, (k, sv.min())
    idx = np.random.default_rng(7).choice(c.n, 4096, replace=False)
    Zr = O.pca_project(Xh[idx], np64(mean), np64(comps))
    assert_close(_rows(Z, idx), Zr, 1e-4, "projection (sampled rows)")
