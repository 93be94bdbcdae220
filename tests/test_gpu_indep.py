"""The independent-decoder variant (Section 2: every expert has its own decoder D_e, bD_e and a
sample is decoded by its expert's) on the HIP path against the fp64 oracle, in fp32 and bf16,
at ragged multi-tile sizes with an empty expert; and its reduction to the shared decoder when
all the D_e are equal."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import (RTOL, anchored, assert_close, assert_grad_close, assert_scalar_close, assert_stored_logits,
                          np64, npi, unanchored)

pytestmark = pytest.mark.gpu


def _run(n, d, h, o, V, K, store, seed, empty=None, bias=True):
    X = W.rectified_gaussian(n, d, seed=seed, dtype=store, device="cuda")
    ids = np.random.default_rng(seed + 1).integers(0, K, n).astype(np.int32)
    if empty is not None:
        ids[ids == empty] = (empty + 1) % K
    rp, tg = W.zipf_labels(n, V, 8, seed=seed + 2)
    p = W.moe_params(K, d, h, o, V, seed=seed + 3, dtype=store, device="cuda", bias=bias,
                     per_expert_decoders=True)
    return X, ids, rp, tg, p


def _check(X, ids, rp, tg, p, K, store):
    rt = RTOL[store]
    a = torch.as_tensor(ids, dtype=torch.int32).cuda()
    dd = hmoe.moe_dispatch(a, K, rows=X)
    row_ptr = torch.tensor(rp, device="cuda")
    tag = torch.tensor(tg, device="cuda")
    f = hmoe.moe_forward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], row_ptr, tag, save_logits=True)
    Xh = np64(X)
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    ref = O.moe_forward(Xh, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                        store=store, want_logits=True)
    perm = npi(dd["perm"])
    assert_close(f["H1_sorted"], ref["H1"][perm], rt, "H1_sorted")
    assert_close(f["H"], ref["H"], rt, "H")
    assert_close(f["lse"], ref["lse"], rt, "lse")
    assert_close(f["loss"], ref["loss"], rt, "loss")
    assert_scalar_close(f["loss_mean"].item(), ref["loss_mean"], rt, "loss_mean")
    assert_stored_logits(f["logits"], f["logit_anchor"], ref["logits"][perm], store, "stored logits (slot order)")
    # backward from the oracle's saved activations and logits (slot order)
    tdt = torch.bfloat16 if store == "bf16" else torch.float32
    H1s = torch.tensor(ref["H1"][perm], dtype=torch.float32).to(tdt).cuda()
    H = torch.tensor(ref["H"], dtype=torch.float32).to(tdt).cuda()
    lse = torch.tensor(ref["lse"], dtype=torch.float32, device="cuda")
    Lg, An = anchored(ref["logits"][perm], tdt)
    g = hmoe.moe_backward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], row_ptr, tag, H1s, H,
                          lse, logits=Lg, logit_anchor=An)
    args = (Xh, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store=store)
    gm = O.moe_backward(*args, magnitude=True)
    for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD", "dX"):
        assert_grad_close(g[k], gr[k], gm[k], store, k)
    return g


@pytest.mark.parametrize("store", ["f32", "bf16"])
def test_independent_decoders_ragged_with_empty_expert(store):
    # 1100 rows over 5 experts (expert 2 empty), V = 1000 and o = 136: ragged in rows, columns
    # and K; every decoder tile shape and an empty expert's decoder (exact zero gradients)
    n, d, h, o, V, K = 1100, 256, 384, 136, 1000, 5
    X, ids, rp, tg, p = _run(n, d, h, o, V, K, store, seed=100, empty=2)
    g = _check(X, ids, rp, tg, p, K, store)
    assert torch.count_nonzero(g["dD"][2]).item() == 0
    assert torch.count_nonzero(g["dbD"][2]).item() == 0


def test_independent_decoders_one_expert_and_single_sample():
    X, ids, rp, tg, p = _run(300, 64, 64, 64, 264, 1, "bf16", seed=110)
    _check(X, ids, rp, tg, p, 1, "bf16")
    X, ids, rp, tg, p = _run(1, 64, 64, 32, 96, 4, "bf16", seed=111)
    _check(X, ids, rp, tg, p, 4, "bf16")


def test_equal_decoders_reduce_to_the_shared_one():
    """Every expert given the same decoder: the HIP path's per-expert results agree with its
    shared-decoder results (loss exactly per sample up to summation order; dD summed over the
    experts is the shared dD)."""
    n, d, h, o, V, K = 1500, 128, 256, 128, 704, 4
    inp = W.balanced_inputs(device="cuda", seed=120, n=n, d=d, h=h, o=o, V=V, K=K, bias=True)
    ps = inp["params"]
    pe = dict(ps)
    pe["D"] = ps["D"].unsqueeze(0).expand(K, V, o).contiguous()
    pe["bD"] = ps["bD"].unsqueeze(0).expand(K, V).contiguous()
    a, _ = hmoe.kmeans_assign(inp["X"], inp["C"])
    dd = hmoe.moe_dispatch(a, K, rows=inp["X"])
    rp = torch.as_tensor(inp["row_ptr"]).cuda()
    tg = torch.as_tensor(inp["tag"]).cuda()
    args = (dd["rows_sorted"], dd["offsets"], dd["perm"], rp, tg)
    fs = hmoe.moe_forward(ps, *args, save_logits=True)
    fe = hmoe.moe_forward(pe, *args, save_logits=True)
    rt = RTOL["bf16"]
    for k in ("H1_sorted", "H"):
        assert torch.equal(fs[k], fe[k]), k
    assert_close(fe["lse"], fs["lse"], 1e-5, "lse")
    assert_close(fe["loss"], fs["loss"], 1e-5, "loss")
    perm = npi(dd["perm"])
    assert_close(unanchored(fe["logits"], fe["logit_anchor"]),
                 unanchored(fs["logits"], fs["logit_anchor"])[perm], 1e-2, "logits")
    gs = hmoe.moe_backward(ps, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], rp, tg, fs["H1_sorted"],
                           fs["H"], fs["lse"], logits=fs["logits"], logit_anchor=fs["logit_anchor"])
    ge = hmoe.moe_backward(pe, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], rp, tg, fe["H1_sorted"],
                           fe["H"], fe["lse"], logits=fe["logits"], logit_anchor=fe["logit_anchor"])
    for k in ("dW1", "db1", "dW2", "db2", "dX"):
        assert_close(ge[k], gs[k], rt, k)
    assert_close(ge["dD"].sum(0), gs["dD"], rt, "sum_e dD_e")
    assert_close(ge["dbD"].sum(0), gs["dbD"], rt, "sum_e dbD_e")


def test_backward_needs_saved_logits():
    X, ids, rp, tg, p = _run(64, 64, 64, 64, 96, 2, "bf16", seed=130)
    a = torch.as_tensor(ids, dtype=torch.int32).cuda()
    dd = hmoe.moe_dispatch(a, 2, rows=X)
    row_ptr = torch.tensor(rp, device="cuda")
    tag = torch.tensor(tg, device="cuda")
    f = hmoe.moe_forward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], row_ptr, tag, save_logits=True)
    with pytest.raises(hmoe.HmoeError, match="saved logits"):
        hmoe.moe_backward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], row_ptr, tag,
                          f["H1_sorted"], f["H"], f["lse"])


def test_independent_step_full_size():
    """The balanced workload's shapes (n = 65536, d = 2048, MLP 2048-4096-1024, V = 50,000,
    K = 16) with one decoder per expert, in the bench's launch configuration: H, lse, loss and
    dX on sampled rows of two experts against the oracle (the experts remapped to 0 and 1, so
    the oracle widens two decoders instead of sixteen), and per-expert invariants of the
    gradients: sum_v dbD_e = 0, sum_v dD_e = 0, db2_e = D_e^T dbD_e."""
    inp = W.balanced_inputs(device="cuda", seed=0)
    s = inp["shape"]
    n, K, V, o = s["n"], s["K"], s["V"], s["o"]
    p = W.moe_params(K, s["d"], s["h"], o, V, seed=20, dtype="bf16", device="cuda", bias=True,
                     per_expert_decoders=True)
    a, _ = hmoe.kmeans_assign(inp["X"], inp["C"])
    dd = hmoe.moe_dispatch(a, K, rows=inp["X"])
    rp = torch.as_tensor(inp["row_ptr"]).cuda()
    tg = torch.as_tensor(inp["tag"]).cuda()
    f = hmoe.moe_forward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], rp, tg, save_logits=True)
    g = hmoe.moe_backward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], rp, tg, f["H1_sorted"],
                          f["H"], f["lse"], logits=f["logits"], logit_anchor=f["logit_anchor"])
    torch.cuda.synchronize()
    rt = RTOL["bf16"]
    a_np = npi(a)
    rs = np.random.default_rng(1)
    pick = [3, 11]
    rows = np.sort(np.concatenate([rs.choice(np.flatnonzero(a_np == e), 12, replace=False) for e in pick]))
    ids = np.searchsorted(pick, a_np[rows]).astype(np.int32)
    sel = torch.as_tensor(pick, dtype=torch.long, device="cuda")
    ph = {k: np64(v[sel]) for k, v in p.items()}
    Xs = np64(inp["X"][torch.as_tensor(rows, dtype=torch.long, device="cuda")])
    cnt = inp["row_ptr"][1:] - inp["row_ptr"][:-1]
    srp = np.concatenate([[0], np.cumsum(cnt[rows])]).astype(np.int32)
    stg = np.concatenate([inp["tag"][inp["row_ptr"][i]:inp["row_ptr"][i + 1]] for i in rows]).astype(np.int32)
    ref = O.moe_forward(Xs, ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], srp, stg,
                        store="bf16")
    assert_close(np64(f["H"])[rows], ref["H"], rt, "H (sampled rows)")
    assert_close(np64(f["lse"])[rows], ref["lse"], rt, "lse (sampled rows)")
    assert_close(np64(f["loss"])[rows], ref["loss"], rt, "loss (sampled rows)")
    args = (Xs, ids, ph["W1"], ph["W2"], ph["D"], ph["bD"], srp, stg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, scale=1.0 / n, store="bf16")
    gm = O.moe_backward(*args, scale=1.0 / n, magnitude=True)
    assert_grad_close(np64(g["dX"])[rows], gr["dX"], gm["dX"], "bf16", "dX (sampled rows)")
    dbD = np64(g["dbD"])
    assert np.all(np.abs(dbD.sum(axis=1)) <= 1e-3 * np.abs(dbD).sum(axis=1))
    db2 = np64(g["db2"])
    for e in range(K):
        dDe = np64(g["dD"][e])
        assert np.all(np.abs(dDe.sum(axis=0)) <= 1e-2 * np.abs(dDe).sum(axis=0) + 1e-12), e
        assert_close(db2[e], np64(p["D"][e]).T @ dbD[e], rt, f"db2_{e} vs D_{e}^T dbD_{e}")
