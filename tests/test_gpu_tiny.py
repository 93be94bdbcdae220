"""Parity of the whole hot path on the tiny workload (4096 fp32 rows, d=64, K=8, experts
64->128->64, V=1000) against the fp64 oracle.  Every oracle input is generator output;
HIP-path inputs may come from the oracle (never the reverse)."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import (RTOL, anchored, assert_assign, assert_close, assert_grad_close, assert_scalar_close,
                          assert_stored_logits, np64, npi)

pytestmark = pytest.mark.gpu
RT = RTOL["f32"]


@pytest.fixture(scope="module")
def tiny():
    torch.manual_seed(0)
    inp = W.tiny_inputs(device="cuda", seed=0)
    X = inp["X"]
    Xh = np64(X)
    c = inp["cfg"]
    fit = O.fit(Xh, c.K, c.n_iter, u=inp["u"], data_store="f32")
    return {"inp": inp, "X": X, "Xh": Xh, "cfg": c, "fit": fit}


def test_assign_matches_oracle(tiny):
    X, Xh, c = tiny["X"], tiny["Xh"], tiny["cfg"]
    C = torch.tensor(tiny["fit"]["C"], dtype=torch.float32, device="cuda")
    a, md = hmoe.kmeans_assign(X, C)
    a_ref, d1, d2 = O.assign(Xh, np64(C))
    assert_assign(a, a_ref, d1, d2)
    assert_close(md, d1, RT, "min_dist")


def test_kmeans_fit_matches_oracle(tiny):
    X, c, ref = tiny["X"], tiny["cfg"], tiny["fit"]
    out = hmoe.kmeans_fit(X, c.K, c.n_iter, init_uniforms=tiny["inp"]["u"])
    assert npi(out["init_idx"]).tolist() == ref["init_idx"].tolist()
    a_ref, d1, d2 = O.assign(tiny["Xh"], ref["C"])
    assert_assign(out["assign"], ref["a"], d1, d2)
    assert_close(out["C"], ref["C"], RT, "centres")
    J = npi(out["objective"])
    for t in range(c.n_iter + 1):
        assert_scalar_close(J[t], ref["J"][t], RT, f"J[{t}]")
    assert np.all(J[1:] <= J[:-1] * (1 + 1e-6))
    assert npi(out["counts"]).tolist() == np.bincount(ref["a"], minlength=c.K).tolist()
    assert_close(out["min_dist"], d1, RT, "min_dist")


def test_dispatch_bit_exact(tiny):
    X, c = tiny["X"], tiny["cfg"]
    a = torch.tensor(tiny["fit"]["a"], dtype=torch.int32, device="cuda")
    d = hmoe.moe_dispatch(a, c.K, rows=X)
    counts, offsets, perm, inv = O.dispatch(tiny["fit"]["a"], c.K)
    assert npi(d["counts"]).tolist() == counts.tolist()
    assert npi(d["offsets"]).tolist() == offsets.tolist()
    assert np.array_equal(npi(d["perm"]), perm)
    assert np.array_equal(npi(d["inv"]), inv)
    assert torch.equal(d["rows_sorted"], X[torch.from_numpy(perm).long().cuda()])
    back = hmoe.permute_rows(d["rows_sorted"], d["inv"])
    assert torch.equal(back, X)


def _params(tiny, bias):
    inp = W.tiny_inputs(device="cuda", seed=0, bias=bias) if bias else tiny["inp"]
    return inp["params"]


@pytest.mark.parametrize("bias,saved", [(False, False), (True, False), (True, True)])
def test_forward_backward_match_oracle(tiny, bias, saved):
    c = tiny["cfg"]
    X, Xh = tiny["X"], tiny["Xh"]
    p = _params(tiny, bias)
    a_np = tiny["fit"]["a"]
    rp, tg = tiny["inp"]["row_ptr"], tiny["inp"]["tag"]
    a = torch.tensor(a_np, dtype=torch.int32, device="cuda")
    d = hmoe.moe_dispatch(a, c.K, rows=X)
    row_ptr = torch.tensor(rp, device="cuda")
    tag = torch.tensor(tg, device="cuda")
    f = hmoe.moe_forward(p, d["rows_sorted"], d["offsets"], d["perm"], row_ptr, tag,
                         save_logits=saved)
    ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
    ref = O.moe_forward(Xh, a_np, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                        store="f32", want_logits=saved)
    if saved:
        assert_stored_logits(f["logits"], f["logit_anchor"], ref["logits"], "f32")
    perm = npi(d["perm"])
    assert_close(f["H1_sorted"], ref["H1"][perm], RT, "H1_sorted")
    assert_close(f["H"], ref["H"], RT, "H")
    assert_close(f["lse"], ref["lse"], RT, "lse")
    assert_close(f["loss"], ref["loss"], RT, "loss")
    assert_scalar_close(f["loss_mean"].item(), ref["loss_mean"], RT, "loss_mean")
    # backward from the oracle's saved activations
    H1s = torch.tensor(ref["H1"][perm], dtype=torch.float32, device="cuda")
    H = torch.tensor(ref["H"], dtype=torch.float32, device="cuda")
    lse = torch.tensor(ref["lse"], dtype=torch.float32, device="cuda")
    Lg, An = anchored(ref["logits"], torch.float32) if saved else (None, None)
    g = hmoe.moe_backward(p, d["rows_sorted"], d["offsets"], d["perm"], d["inv"], row_ptr, tag,
                          H1s, H, lse, logits=Lg, logit_anchor=An)
    args = (Xh, a_np, ph["W1"], ph["W2"], ph["D"], ph["bD"], rp, tg, ref["H1"], ref["H"], ref["lse"])
    gr = O.moe_backward(*args, store="f32")
    gm = O.moe_backward(*args, magnitude=True)
    for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD", "dX"):
        assert_grad_close(g[k], gr[k], gm[k], "f32", k)
    # invariants: the softmax rows sum to one, so the decoder-bias gradient sums to zero
    assert abs(float(g["dbD"].double().sum())) < 1e-6


def test_determinism(tiny):
    c = tiny["cfg"]
    X = tiny["X"]
    o1 = hmoe.kmeans_fit(X, c.K, 3, init_uniforms=tiny["inp"]["u"])
    o2 = hmoe.kmeans_fit(X, c.K, 3, init_uniforms=tiny["inp"]["u"])
    for k in ("C", "assign", "min_dist", "objective"):
        assert torch.equal(o1[k], o2[k]), k
