"""bf16 parity of the routed step and the gater against the fp64 oracle at sizes the oracle
finishes in seconds, spanning several 128-wide tiles with ragged tails, plus the degenerate
cases (empty experts, K = 1, n = 0)."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import (RTOL, anchored, assert_assign, assert_close, assert_grad_close, assert_scalar_close,
                          assert_stored_logits, np64, npi)

pytestmark = pytest.mark.gpu
RT = RTOL["bf16"]


def _step(X, ids, K, p, rp, tg, saved=False):
    a = torch.as_tensor(ids, dtype=torch.int32).cuda()
    d = hmoe.moe_dispatch(a, K, rows=X)
    row_ptr = torch.tensor(rp, device="cuda")
    tag = torch.tensor(tg, device="cuda")
    f = hmoe.moe_forward(p, d["rows_sorted"], d["offsets"], d["perm"], row_ptr, tag,
                         save_logits=saved)
    return d, f, row_ptr, tag


def _check_step(X, ids, K, p, rp, tg, rt=RT, saved=False):
    """Forward on the HIP path vs the oracle; backward from the oracle's saved activations
    (with the saved-logits path, from the oracle's logits in the stored form) against the
    oracle's gradient of Eq. 3."""
    d, f, row_ptr, tag = _step(X, ids, K, p, rp, tg, saved)
    Xh = np64(X)
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    ref = O.moe_forward(Xh, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                        store="bf16", want_logits=saved)
    if saved:
        assert_stored_logits(f["logits"], f["logit_anchor"], ref["logits"], "bf16")
    perm = npi(d["perm"])
    counts, offsets, perm_ref, inv_ref = O.dispatch(ids, K)
    assert np.array_equal(perm, perm_ref)
    assert_close(f["H1_sorted"], ref["H1"][perm], rt, "H1_sorted")
    assert_close(f["H"], ref["H"], rt, "H")
    assert_close(f["lse"], ref["lse"], rt, "lse")
    assert_close(f["loss"], ref["loss"], rt, "loss")
    assert_scalar_close(f["loss_mean"].item(), ref["loss_mean"], rt, "loss_mean")
    H1s = torch.tensor(ref["H1"][perm], dtype=torch.float32).to(torch.bfloat16).cuda()
    H = torch.tensor(ref["H"], dtype=torch.float32).to(torch.bfloat16).cuda()
    lse = torch.tensor(ref["lse"], dtype=torch.float32, device="cuda")
    Lg, An = anchored(ref["logits"], torch.bfloat16) if saved else (None, None)
    g = hmoe.moe_backward(p, d["rows_sorted"], d["offsets"], d["perm"], d["inv"], row_ptr, tag,
                          H1s, H, lse, logits=Lg, logit_anchor=An)
    args = (Xh, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store="bf16")
    gm = O.moe_backward(*args, magnitude=True)
    for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD", "dX"):
        assert_grad_close(g[k], gr[k], gm[k], "bf16", k)
    return g, counts


@pytest.mark.parametrize("saved", [False, True])
def test_routed_step_ragged_tiles(saved):
    # n, h, o, V all leave ragged tails in the 256-wide tiles; biases exercised
    inp = W.balanced_inputs(device="cuda", seed=3, n=600, d=256, h=384, o=136, V=1000, K=5,
                            bias=True)
    C = inp["C"]
    a, _ = hmoe.kmeans_assign(inp["X"], C)
    a_ref, d1, d2 = O.assign(np64(inp["X"]), np64(C))
    assert_assign(a, a_ref, d1, d2)
    _check_step(inp["X"], a_ref, 5, inp["params"], inp["row_ptr"], inp["tag"], saved=saved)


def test_skewed_routing_with_empty_experts():
    n, K = 900, 24
    inp = W.skewed_inputs(device="cuda", seed=5, n=n, d=128, h=256, o=64, V=520, K=K)
    ids = inp["ids"]
    g, counts = _check_step(inp["X"], ids, K, inp["params"], inp["row_ptr"], inp["tag"], saved=True)
    empty = np.flatnonzero(counts == 0)
    assert len(empty) >= 2
    for k in ("dW1", "db1", "dW2", "db2"):
        assert torch.count_nonzero(g[k][torch.as_tensor(empty).cuda()]) == 0, k


def test_bucket_sizes_around_the_half_height_tile():
    # a group's last row tile runs at half height (128 rows) when it holds at most 128 rows:
    # buckets on both sides of that boundary and of the 256-row tile, next to empty and
    # one-sample experts, through every row-grouped GEMM (layers 1 and 2, dH1 and dX)
    sizes = [128, 1, 129, 0, 256, 127, 257, 64, 384, 255, 385]
    n, K = sum(sizes), len(sizes)
    ids = np.repeat(np.arange(K, dtype=np.int32), sizes)
    ids = ids[np.random.default_rng(11).permutation(n)]
    inp = W.skewed_inputs(device="cuda", seed=12, n=n, d=256, h=384, o=136, V=600, K=K, bias=True)
    g, counts = _check_step(inp["X"], ids, K, inp["params"], inp["row_ptr"], inp["tag"], saved=True)
    assert counts.tolist() == sizes
    for k in ("dW1", "db1", "dW2", "db2"):
        assert torch.count_nonzero(g[k][3]) == 0, k


def test_single_expert():
    inp = W.skewed_inputs(device="cuda", seed=6, n=300, d=64, h=128, o=64, V=256, K=1)
    ids = np.zeros(300, np.int32)
    _check_step(inp["X"], ids, 1, inp["params"], inp["row_ptr"], inp["tag"])


@pytest.mark.parametrize("n,d,K", [(3000, 2048, 300), (1000, 512, 64), (777, 64, 129)])
def test_assign_bf16_multi_tile(n, d, K):
    X = W.gmm_features(n, d, 40, seed=n, dtype="bf16", device="cuda")
    C = X[torch.randperm(n, generator=torch.Generator().manual_seed(1))[:K].cuda()].contiguous()
    a, md = hmoe.kmeans_assign(X, C)
    a_ref, d1, d2 = O.assign(np64(X), np64(C))
    assert_assign(a, a_ref, d1, d2)
    assert_close(md, d1, 1e-4, "min_dist")  # fp32 accumulation of exact bf16 products


def test_kmeans_fit_bf16():
    n, d, K = 5000, 256, 20
    X = W.gmm_features(n, d, 32, seed=11, dtype="bf16", device="cuda", dirichlet_alpha=0.5)
    u = W.uniforms(K, 12)
    out = hmoe.kmeans_fit(X, K, 6, init_uniforms=u)
    ref = O.fit(np64(X), K, 6, u=u, data_store="bf16")
    assert npi(out["init_idx"]).tolist() == ref["init_idx"].tolist()
    _, d1, d2 = O.assign(np64(X), O.round_store(ref["C"], "bf16"))
    assert_assign(out["assign"], ref["a"], d1, d2)
    assert_close(out["C"], ref["C"], 1e-4, "centres")
    J = npi(out["objective"])
    for t in range(7):
        assert_scalar_close(J[t], ref["J"][t], 1e-4, f"J[{t}]")


def test_update_chunks_and_reseed():
    n, d, K = 4000, 64, 12
    X = W.gmm_features(n, d, 6, seed=21, dtype="f32", device="cuda")
    Xh = np64(X)
    C0 = Xh[:K].copy()
    C0[K - 3:] = 1e3  # three far-away centres: their clusters start empty
    a_ref, d1, _ = O.assign(Xh, C0)
    # full update with reseeding, from the oracle's assignment
    a = torch.tensor(a_ref, dtype=torch.int32, device="cuda")
    md = torch.tensor(d1, dtype=torch.float32, device="cuda")
    C = torch.tensor(C0, dtype=torch.float32, device="cuda")
    sums = torch.zeros(K, d, dtype=torch.float64, device="cuda")
    cnt = torch.zeros(K, dtype=torch.int64, device="cuda")
    hmoe.kmeans_update(X, K, a, md, sums, cnt, C, mode=hmoe.UPDATE_FULL, reseed=True)
    C_ref, counts_ref, a2_ref = O.update(Xh, a_ref, np64(md), C0, reseed=True)
    assert npi(cnt).tolist() == counts_ref.tolist()
    assert np.array_equal(npi(a), a2_ref)
    assert_close(C, O.round_store(C_ref, "f32"), 1e-6, "centres")
    # the same update streamed in three chunks (no reseeding)
    C2 = torch.tensor(C0, dtype=torch.float32, device="cuda")
    sums.zero_()
    cnt.zero_()
    a = torch.tensor(a_ref, dtype=torch.int32, device="cuda")
    for lo, hi in ((0, 1500), (1500, 1501), (1501, n)):
        hmoe.kmeans_update(X[lo:hi].contiguous(), K, a[lo:hi].contiguous(), None, sums, cnt, C2,
                           mode=hmoe.UPDATE_ACCUMULATE, reseed=False)
    hmoe.kmeans_update(None, K, None, None, sums, cnt, C2, mode=hmoe.UPDATE_FINALIZE)
    C_ref2, counts2, _ = O.update(Xh, a_ref, None, C0, reseed=False)
    assert npi(cnt).tolist() == counts2.tolist()
    assert_close(C2, O.round_store(C_ref2, "f32"), 1e-6, "chunked centres")


def test_empty_batch():
    X = torch.empty(0, 64, dtype=torch.bfloat16, device="cuda")
    C = torch.randn(4, 64, device="cuda").to(torch.bfloat16)
    a, md = hmoe.kmeans_assign(X, C)
    assert a.numel() == 0
    d = hmoe.moe_dispatch(torch.empty(0, dtype=torch.int32, device="cuda"), 3)
    assert npi(d["counts"]).tolist() == [0, 0, 0] and npi(d["offsets"]).tolist() == [0, 0, 0, 0]
    p = W.moe_params(3, 64, 128, 64, 80, seed=0, dtype="bf16", device="cuda")
    z = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = hmoe.moe_backward(p, X, d["offsets"], d["perm"], d["inv"], z, z,
                          torch.empty(0, 128, dtype=torch.bfloat16, device="cuda"),
                          torch.empty(0, 64, dtype=torch.bfloat16, device="cuda"),
                          torch.empty(0, device="cuda"), want_dX=False)
    for k in ("dW1", "dW2", "dD", "dbD"):
        assert torch.count_nonzero(g[k]) == 0


@pytest.mark.parametrize("K,n,bad", [(63, 1024 * 1024, 0), (63, 1024 * 1024 + 1, 0), (15, 4096 * 1024, 7),
                                     (15, 4096 * 1024 + 1, 7)])
def test_dispatch_around_the_fused_scan_size(K, n, bad):
    # the column scans and offsets run as one workgroup while (K + 1) ceil(n / 1024) <= 2^16 and
    # as two launches above: both sides of that size, bit-exact against the oracle (with a few
    # out-of-range ids in the last two cases)
    rs = np.random.default_rng(K + n)
    ids = rs.integers(0, K, n).astype(np.int32)
    if bad:
        ids[rs.choice(n, bad, replace=False)] = K + 3
    d = hmoe.moe_dispatch(torch.as_tensor(ids).cuda(), K)
    good = ids[ids < K]
    counts, offsets, perm, inv = O.dispatch(good, K)
    assert npi(d["counts"]).tolist() == counts.tolist()
    assert npi(d["offsets"]).tolist() == offsets.tolist()
    # the in-range rows in expert order match the oracle's order over the same rows
    rows = np.flatnonzero(ids < K)
    assert np.array_equal(npi(d["perm"])[:len(good)], rows[perm])
    assert np.array_equal(np.sort(npi(d["perm"])[len(good):]), np.flatnonzero(ids >= K))
    pv = npi(d["perm"])
    assert np.array_equal(npi(d["inv"])[pv], np.arange(n))


def test_dispatch_out_of_range_ids():
    # ids outside [0, K) are the caller's error: their rows go after every expert's, in sample
    # order, the counts exclude them, and perm / inv stay permutations of all rows
    K, n = 5, 3000
    rs = np.random.default_rng(31)
    ids = rs.integers(0, K, n).astype(np.int32)
    bad = rs.choice(n, 40, replace=False)
    ids[bad[:20]] = -1
    ids[bad[20:]] = K + rs.integers(0, 3, 20)
    X = torch.randn(n, 64, device="cuda").to(torch.bfloat16)
    d = hmoe.moe_dispatch(torch.as_tensor(ids).cuda(), K, rows=X)
    key = np.where((ids >= 0) & (ids < K), ids, K)
    order = np.argsort(key, kind="stable")
    assert npi(d["counts"]).tolist() == np.bincount(ids[key < K], minlength=K).tolist()
    assert npi(d["offsets"]).tolist() == [0] + np.cumsum(np.bincount(ids[key < K], minlength=K)).tolist()
    assert np.array_equal(npi(d["perm"]), order)
    inv = np.empty(n, np.int64)
    inv[order] = np.arange(n)
    assert np.array_equal(npi(d["inv"]), inv)
    assert torch.equal(d["rows_sorted"], X[torch.as_tensor(order).cuda()])
    # the row gather with indices outside [0, n): zero rows, the others gathered
    idx = torch.as_tensor(order.astype(np.int32)).cuda()
    idx[7], idx[100], idx[2999] = -5, n, 1 << 30
    out = hmoe.permute_rows(X, idx)
    ref = X[torch.as_tensor(order).cuda()].clone()
    ref[[7, 100, 2999]] = 0
    assert torch.equal(out, ref)


def _scaled(p, s):
    q = dict(p)
    q["D"] = (p["D"].float() * s).to(torch.bfloat16)
    return q


@pytest.mark.parametrize("scale", [1.0, 8.0])
def test_saved_logits_step_against_eq3(scale):
    """The benchmarked path (bf16, logits saved by the forward) end to end: the HIP forward
    stores the logits, the HIP backward forms g from them, and every gradient is compared with
    the oracle's plain gradient of Eq. 3 (nothing rounded but H1, H and dX).  At the workload's
    N(0, 1/fan_in) decoder and with the decoder scaled by 8, so that the largest logits pass 20
    in magnitude as a trained tagger's do: a bf16 logit of that size is off by up to 0.06, which
    moves its probability by 6%, so the stored form must keep the large logits near fp32."""
    n, d, h, o, V, K = 700, 256, 384, 136, 4104, 5
    inp = W.balanced_inputs(device="cuda", seed=21, n=n, d=d, h=h, o=o, V=V, K=K, bias=True)
    p = _scaled(inp["params"], scale)
    ids = np.random.default_rng(22).integers(0, K, n).astype(np.int32)
    rp, tg = inp["row_ptr"], inp["tag"]
    d_, f, row_ptr, tag = _step(inp["X"], ids, K, p, rp, tg, saved=True)
    g = hmoe.moe_backward(p, d_["rows_sorted"], d_["offsets"], d_["perm"], d_["inv"], row_ptr, tag,
                          f["H1_sorted"], f["H"], f["lse"], logits=f["logits"], logit_anchor=f["logit_anchor"])
    Xh = np64(inp["X"])
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    ref = O.moe_forward(Xh, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                        store="bf16", want_logits=True)
    big = np.abs(ref["logits"]).max()
    assert big > (20.0 if scale > 1 else 2.0), big
    assert_stored_logits(f["logits"], f["logit_anchor"], ref["logits"], "bf16")
    assert_close(f["lse"], ref["lse"], RT, "lse")
    args = (Xh, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store="bf16")
    gm = O.moe_backward(*args, magnitude=True)
    for k in ("dD", "dbD", "dW2", "db2", "dW1", "db1", "dX"):
        assert_grad_close(g[k], gr[k], gm[k], "bf16", k + " (HIP forward and backward)")
    # the backward alone, from the oracle's activations and logits in the stored form
    Lg, An = anchored(ref["logits"], torch.bfloat16)
    perm = npi(d_["perm"])
    tb = lambda a: torch.tensor(a, dtype=torch.float32).to(torch.bfloat16).cuda()  # noqa: E731
    g2 = hmoe.moe_backward(p, d_["rows_sorted"], d_["offsets"], d_["perm"], d_["inv"], row_ptr, tag,
                           tb(ref["H1"][perm]), tb(ref["H"]),
                           torch.tensor(ref["lse"], dtype=torch.float32, device="cuda"), logits=Lg, logit_anchor=An)
    for k in ("dD", "dbD", "dW2", "db2", "dW1", "db1", "dX"):
        assert_grad_close(g2[k], gr[k], gm[k], "bf16", k + " (HIP backward)")


def test_decoder_gradient_whole_and_split_tiles():
    """dD = g^T H with more output tiles than the chip runs at once: V = 16640 and o = 1024
    give 65 x 4 = 260 tiles of 256 x 256, so 256 run whole over all n rows and the last 4 are
    split over the rows.  With saved bf16 logits g is slab-major (2048-column slabs, the last
    one ragged), the layout the balanced step's dD reads; dD and dbD element-wise against the
    oracle's gradient of Eq. 3."""
    n, d, h, o, V, K = 300, 64, 128, 1024, 16640, 3
    inp = W.balanced_inputs(device="cuda", seed=23, n=n, d=d, h=h, o=o, V=V, K=K, bias=True)
    p = inp["params"]
    ids = np.random.default_rng(24).integers(0, K, n).astype(np.int32)
    rp, tg = inp["row_ptr"], inp["tag"]
    d_, f, row_ptr, tag = _step(inp["X"], ids, K, p, rp, tg, saved=True)
    g = hmoe.moe_backward(p, d_["rows_sorted"], d_["offsets"], d_["perm"], d_["inv"], row_ptr, tag,
                          f["H1_sorted"], f["H"], f["lse"], logits=f["logits"], logit_anchor=f["logit_anchor"])
    Xh = np64(inp["X"])
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    ref = O.moe_forward(Xh, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                        store="bf16")
    assert_close(f["H"], ref["H"], RT, "H")
    assert_close(f["lse"], ref["lse"], RT, "lse")
    args = (Xh, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store="bf16", want_dX=False)
    gm = O.moe_backward(*args, want_dX=False, magnitude=True)
    assert_grad_close(g["dD"], gr["dD"], gm["dD"], "bf16", "dD")
    assert_grad_close(g["dbD"], gr["dbD"], gm["dbD"], "bf16", "dbD")
    # the whole tiles are the first 256 in the launch's tile order (bands of 16 row tiles with all
    # four column tiles): vocabulary rows 0 .. 16383
    w = 64 * 256
    assert_grad_close(g["dD"][:w], gr["dD"][:w], gm["dD"][:w], "bf16", "dD (whole tiles)")
    assert_grad_close(g["dD"][w:], gr["dD"][w:], gm["dD"][w:], "bf16", "dD (split tiles)")
