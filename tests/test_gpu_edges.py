"""Edge cases of the HIP path against the fp64 oracle: rows with more tags than the gradient
and loss kernels stage in LDS, the narrowest widths the ABI allows, a single sample, a decoder with more
tiles than the chip holds workgroups at once, the largest K, and exactly duplicated centres
(ties must go to the lower index)."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import (RTOL, anchored, assert_assign, assert_close, assert_grad_close, assert_scalar_close,
                          assert_stored_logits, np64, npi, unanchored)

pytestmark = pytest.mark.gpu


def _step_vs_oracle(X, ids, K, p, rp, tg, store, saved):
    """Forward on the HIP path vs the oracle, then the backward from the oracle's saved
    activations (and, with `saved`, its stored logits)."""
    rt = RTOL[store]
    a = torch.as_tensor(ids, dtype=torch.int32).cuda()
    d = hmoe.moe_dispatch(a, K, rows=X)
    row_ptr = torch.tensor(rp, device="cuda")
    tag = torch.tensor(tg, device="cuda")
    f = hmoe.moe_forward(p, d["rows_sorted"], d["offsets"], d["perm"], row_ptr, tag, save_logits=saved)
    Xh = np64(X)
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    ref = O.moe_forward(Xh, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                        store=store, want_logits=saved)
    perm = npi(d["perm"])
    assert_close(f["H1_sorted"], ref["H1"][perm], rt, "H1_sorted")
    assert_close(f["H"], ref["H"], rt, "H")
    assert_close(f["lse"], ref["lse"], rt, "lse")
    assert_close(f["loss"], ref["loss"], rt, "loss")
    assert_scalar_close(f["loss_mean"].item(), ref["loss_mean"], rt, "loss_mean")
    if saved:
        assert_stored_logits(f["logits"], f["logit_anchor"], ref["logits"], store)
    tdt = torch.bfloat16 if store == "bf16" else torch.float32
    H1s = torch.tensor(ref["H1"][perm], dtype=torch.float32).to(tdt).cuda()
    H = torch.tensor(ref["H"], dtype=torch.float32).to(tdt).cuda()
    lse = torch.tensor(ref["lse"], dtype=torch.float32, device="cuda")
    Lg, An = anchored(ref["logits"], tdt) if saved else (None, None)
    g = hmoe.moe_backward(p, d["rows_sorted"], d["offsets"], d["perm"], d["inv"], row_ptr, tag, H1s, H,
                          lse, logits=Lg, logit_anchor=An)
    args = (Xh, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store=store)
    gm = O.moe_backward(*args, magnitude=True)
    for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD", "dX"):
        assert_grad_close(g[k], gr[k], gm[k], store, k)


@pytest.mark.parametrize("saved", [False, True])
def test_rows_with_many_tags(saved):
    # 17..24 tags on every other row: past the 16 tags per row the gradient kernels stage in LDS,
    # and past the 512 (row, tag) pairs per 64 rows the loss kernel stages at a time
    n, d, h, o, V, K = 300, 64, 128, 64, 264, 3
    rp_few, tg_few = W.zipf_labels(n, V, 3, seed=40)
    rp_many, tg_many = W.zipf_labels(n, V, 24, seed=41, min_tags=17)
    rows = []
    for i in range(n):
        src = (rp_many, tg_many) if i % 2 == 0 else (rp_few, tg_few)
        rows.append(src[1][src[0][i]:src[0][i + 1]])
    rp = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
    tg = np.concatenate(rows).astype(np.int32)
    assert (rp[1:] - rp[:-1]).max() > 16
    assert min(rp[min(i + 64, n)] - rp[i] for i in range(0, n, 64) if i + 64 <= n) > 512
    X = W.rectified_gaussian(n, d, seed=42, dtype="bf16", device="cuda")
    ids = np.random.default_rng(43).integers(0, K, n).astype(np.int32)
    p = W.moe_params(K, d, h, o, V, seed=44, dtype="bf16", device="cuda", bias=True)
    _step_vs_oracle(X, ids, K, p, rp, tg, "bf16", saved)


@pytest.mark.parametrize("store", ["f32", "bf16"])
def test_narrowest_widths(store):
    # every width at the ABI's minimum of 8; n leaves a ragged tail in every tile size
    n, K = 37, 3
    X = W.rectified_gaussian(n, 8, seed=50, dtype=store, device="cuda")
    ids = np.random.default_rng(51).integers(0, K, n).astype(np.int32)
    rp, tg = W.zipf_labels(n, 8, 3, seed=52)
    p = W.moe_params(K, 8, 8, 8, 8, seed=53, dtype=store, device="cuda", bias=True)
    _step_vs_oracle(X, ids, K, p, rp, tg, store, saved=(store == "bf16"))
    C = X[:K].contiguous()
    a, md = hmoe.kmeans_assign(X, C)
    a_ref, d1, d2 = O.assign(np64(X), np64(C))
    assert_assign(a, a_ref, d1, d2)
    assert_close(md, d1, 1e-4, "min_dist")


def test_single_sample():
    X = W.rectified_gaussian(1, 64, seed=60, dtype="bf16", device="cuda")
    rp, tg = W.zipf_labels(1, 96, 5, seed=61)
    p = W.moe_params(4, 64, 64, 32, 96, seed=62, dtype="bf16", device="cuda")
    _step_vs_oracle(X, np.array([2], np.int32), 4, p, rp, tg, "bf16", saved=True)


@pytest.mark.parametrize("saved", [False, True])
def test_decoder_tiles_outnumber_workgroups(saved):
    # 17 x 32 = 544 decoder tiles of 256 x 256 (ragged in rows, columns and K = 136 = 4 x 32 + 8):
    # the persistent decoder forward walks two or three tiles per workgroup
    n, d, h, o, V, K = 4200, 64, 128, 136, 8000, 4
    X = W.rectified_gaussian(n, d, seed=90, dtype="bf16", device="cuda")
    ids = np.random.default_rng(91).integers(0, K, n).astype(np.int32)
    rp, tg = W.zipf_labels(n, V, 8, seed=92)
    p = W.moe_params(K, d, h, o, V, seed=93, dtype="bf16", device="cuda", bias=True)
    _step_vs_oracle(X, ids, K, p, rp, tg, "bf16", saved)


def test_decoder_gradient_tail_in_a_later_slab():
    # bf16 with saved logits keeps g in column slabs of 2048: V = 4104 gives two full slabs and
    # an 8-column third, so dH's last K stage (4104 = 128 x 32 + 8) is a ragged tail read from
    # the third slab and dD's last row tile (8 rows of g^T) starts that slab; n = 700 leaves
    # ragged row tiles
    n, d, h, o, V, K = 700, 64, 128, 64, 4104, 3
    X = W.rectified_gaussian(n, d, seed=95, dtype="bf16", device="cuda")
    ids = np.random.default_rng(96).integers(0, K, n).astype(np.int32)
    rp, tg = W.zipf_labels(n, V, 8, seed=97)
    p = W.moe_params(K, d, h, o, V, seed=98, dtype="bf16", device="cuda", bias=True)
    _step_vs_oracle(X, ids, K, p, rp, tg, "bf16", True)


def test_largest_K_assign_and_dispatch():
    n, d, K = 5000, 64, 4096
    X = W.gmm_features(n, d, 64, seed=70, dtype="bf16", device="cuda")
    C = W.gmm_features(K, d, 64, seed=71, dtype="bf16", device="cuda")
    a, md = hmoe.kmeans_assign(X, C)
    a_ref, d1, d2 = O.assign(np64(X), np64(C))
    assert_assign(a, a_ref, d1, d2)
    assert_close(md, d1, 1e-4, "min_dist")
    ids = np.random.default_rng(72).integers(0, K, n).astype(np.int32)
    dd = hmoe.moe_dispatch(torch.as_tensor(ids).cuda(), K)
    counts, offsets, perm, inv = O.dispatch(ids, K)
    assert npi(dd["counts"]).tolist() == counts.tolist()
    assert npi(dd["offsets"]).tolist() == offsets.tolist()
    assert np.array_equal(npi(dd["perm"]), perm) and np.array_equal(npi(dd["inv"]), inv)


@pytest.mark.parametrize("dtype,K", [("f32", 40), ("f32", 300), ("bf16", 40), ("bf16", 100), ("bf16", 600)])
def test_duplicated_centres_break_ties_low(dtype, K):
    # centre 2j+1 is an exact copy of centre 2j: identical distances, so the lower index wins
    # on every row (the oracle's near-tie exemption would skip these rows, so check directly)
    n, d = 3000, 128
    X = W.gmm_features(n, d, 32, seed=80, dtype=dtype, device="cuda")
    base = X[torch.randperm(n, generator=torch.Generator().manual_seed(81))[:K // 2].cuda()]
    C = base.repeat_interleave(2, dim=0).contiguous()
    a, md = hmoe.kmeans_assign(X, C)
    a = npi(a)
    assert np.all(a % 2 == 0)
    # and the chosen pair is the nearest one (exact duplicates removed: plain parity)
    a_ref, d1, d2 = O.assign(np64(X), np64(base))
    assert_assign(a // 2, a_ref, d1, d2)
    assert_close(md, d1, 1e-4, "min_dist")


def test_reseed_search_across_blocks():
    # 300,000 rows: the first reseed's farthest-row search runs over 74 blocks of the grid and
    # the later ones inside the reseeding block.  Rows 10 and 250,000 (different blocks) are the
    # same far outlier, so their min distances tie: the first empty cluster must take row 10
    # (lowest index), the second then takes row 250,000.
    n, d, K = 300_000, 32, 8
    X = W.gmm_features(n, d, 4, seed=51, dtype="f32", device="cuda")
    X[10] = 40.0
    X[250_000] = 40.0
    Xh = np64(X)
    C0 = Xh[[0, 1, 2, 3, 4, 5, 6, 7]].copy()
    C0[K - 2:] = 1e3  # two far-away centres: their clusters start empty
    a_ref, d1, _ = O.assign(Xh, C0)
    a = torch.tensor(a_ref, dtype=torch.int32, device="cuda")
    md = torch.tensor(d1, dtype=torch.float32, device="cuda")
    C = torch.tensor(C0, dtype=torch.float32, device="cuda")
    sums = torch.zeros(K, d, dtype=torch.float64, device="cuda")
    cnt = torch.zeros(K, dtype=torch.int64, device="cuda")
    hmoe.kmeans_update(X, K, a, md, sums, cnt, C, mode=hmoe.UPDATE_FULL, reseed=True)
    C_ref, counts_ref, a2_ref = O.update(Xh, a_ref, np64(md), C0, reseed=True)
    assert a2_ref[10] == K - 2 and a2_ref[250_000] == K - 1
    assert npi(cnt).tolist() == counts_ref.tolist()
    assert np.array_equal(npi(a), a2_ref)
    assert_close(C, O.round_store(C_ref, "f32"), 1e-6, "centres")


@pytest.mark.parametrize("dtype,K", [("f32", 64), ("f32", 300), ("bf16", 64), ("bf16", 300)])
def test_assign_4096_wide_features(dtype, K):
    # the paper's wider gater features (4096, an AlexNet layer) on the narrow and wide tiles
    n, d = 3000, 4096
    X = W.gmm_features(n, d, 32, seed=80, dtype=dtype, device="cuda")
    C = W.gmm_features(K, d, 32, seed=81, dtype=dtype, device="cuda")
    a, md = hmoe.kmeans_assign(X, C)
    a_ref, d1, d2 = O.assign(np64(X), np64(C))
    assert_assign(a, a_ref, d1, d2)
    assert_close(md, d1, 1e-4, "min_dist")


@pytest.mark.parametrize("store,saved", [("bf16", True), ("bf16", False), ("f32", True)])
def test_vocabulary_padded_to_a_multiple_of_8(store, saved):
    """A vocabulary of 1001 tags runs as 1008: seven zero rows of D with bias -inf.  Every result
    for the 1001 real tags is the unpadded problem's (the oracle runs V = 1001), and the padded
    tags get exact zero gradients."""
    n, d, h, o, V, Vp, K = 500, 64, 128, 72, 1001, 1008, 3
    tdt = torch.bfloat16 if store == "bf16" else torch.float32
    X = W.rectified_gaussian(n, d, seed=70, dtype=store, device="cuda")
    ids = np.random.default_rng(71).integers(0, K, n).astype(np.int32)
    rp, tg = W.zipf_labels(n, V, 8, seed=72)
    p = W.moe_params(K, d, h, o, V, seed=73, dtype=store, device="cuda", bias=True)
    pp = dict(p)
    pp["D"] = torch.cat([p["D"], torch.zeros(Vp - V, o, dtype=tdt, device="cuda")])
    pp["bD"] = torch.cat([p["bD"], torch.full((Vp - V,), float("-inf"), dtype=tdt, device="cuda")])
    rt = RTOL[store]
    a = torch.as_tensor(ids).cuda()
    dd = hmoe.moe_dispatch(a, K, rows=X)
    row_ptr, tag = torch.tensor(rp, device="cuda"), torch.tensor(tg, device="cuda")
    f = hmoe.moe_forward(pp, dd["rows_sorted"], dd["offsets"], dd["perm"], row_ptr, tag, save_logits=saved)
    g = hmoe.moe_backward(pp, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], row_ptr, tag, f["H1_sorted"],
                          f["H"], f["lse"], logits=f["logits"], logit_anchor=f["logit_anchor"])
    Xh = np64(X)
    ph = {k: np64(v) for k, v in p.items()}
    ref = O.moe_forward(Xh, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg, store=store,
                        want_logits=True)
    assert_close(f["lse"], ref["lse"], rt, "lse")
    assert_close(f["loss"], ref["loss"], rt, "loss")
    if saved:
        Lr = unanchored(f["logits"], f["logit_anchor"])
        assert_stored_logits(f["logits"][:, :V], f["logit_anchor"], ref["logits"], store)
        assert np.all(Lr[:, V:] == -np.inf)
    args = (Xh, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store=store)
    gm = O.moe_backward(*args, magnitude=True)
    for k in ("dW1", "db1", "dW2", "db2", "dX"):
        assert_grad_close(g[k], gr[k], gm[k], store, k)
    assert_grad_close(g["dD"][:V], gr["dD"], gm["dD"], store, "dD")
    assert_grad_close(g["dbD"][:V], gr["dbD"], gm["dbD"], store, "dbD")
    assert torch.count_nonzero(g["dD"][V:]).item() == 0 and torch.count_nonzero(g["dbD"][V:]).item() == 0
