"""Pins for the routed half of the oracle: the hard dispatch (Section 2), the shared-decoder
expert forward with the multilabel softmax loss (Section 2; Section 4.1, Eq. 3) and its
gradients.

Independent checks: numpy's stable argsort, scipy's logsumexp, PyTorch CPU fp64 autograd
(per-sample expert selection + cross_entropy with probability targets), central finite
differences, the closed form for a zero decoder, and the hand-worked loss fixture."""
import json
import os

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _case(seed, n=40, d=6, h=9, o=5, V=13, K=3, empty=None, max_tags=4):
    rs = np.random.default_rng(seed)
    X = rs.normal(size=(n, d))
    a = rs.integers(0, K, n).astype(np.int32)
    if empty is not None:
        a[a == empty] = (empty + 1) % K
    W1 = rs.normal(size=(K, h, d)) / np.sqrt(d)
    b1 = rs.normal(size=(K, h)) * 0.3
    W2 = rs.normal(size=(K, o, h)) / np.sqrt(h)
    b2 = rs.normal(size=(K, o)) * 0.3
    D = rs.normal(size=(V, o)) / np.sqrt(o)
    bD = rs.normal(size=V) * 0.3
    cnt = rs.integers(1, max_tags + 1, n)
    tags = [rs.choice(V, c, replace=False) for c in cnt]
    row_ptr = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)
    tag = np.concatenate(tags).astype(np.int32)
    return dict(X=X, a=a, W1=W1, b1=b1, W2=W2, b2=b2, D=D, bD=bD, row_ptr=row_ptr, tag=tag)


def _fwd(orc, c, **kw):
    return orc.moe_forward(c["X"], c["a"], c["W1"], c["b1"], c["W2"], c["b2"], c["D"], c["bD"],
                           c["row_ptr"], c["tag"], **kw)


def _bwd(orc, c, f, **kw):
    return orc.moe_backward(c["X"], c["a"], c["W1"], c["W2"], c["D"], c["bD"], c["row_ptr"],
                            c["tag"], f["H1"], f["H"], f["lse"], **kw)


# ------------------------------------------------------------------ dispatch

@pytest.mark.parametrize("n,K", [(0, 3), (1, 1), (1000, 7), (513, 64)])
def test_dispatch_is_stable_sort(orc, n, K):
    rs = np.random.default_rng(n + K)
    e = rs.integers(0, K, n).astype(np.int32)
    if n > 10:
        e[e == 2] = 3  # force an empty bucket
    counts, offsets, perm, inv = orc.dispatch(e, K)
    assert np.array_equal(perm, np.argsort(e, kind="stable"))
    assert np.array_equal(counts, np.bincount(e, minlength=K))
    assert offsets[0] == 0 and offsets[-1] == n
    assert np.array_equal(np.diff(offsets), counts)
    assert np.array_equal(inv[perm], np.arange(n))
    assert np.array_equal(perm[inv], np.arange(n))
    # combine(dispatch(rows)) is the identity
    rows = rs.normal(size=(n, 3))
    assert np.array_equal(rows[perm][inv], rows)


# ------------------------------------------------------------------ forward

def test_loss_golden(orc):
    g = json.load(open(os.path.join(GOLD, "loss_tiny.json")))
    # One expert whose output is exactly h: d = h = o = 1, W1 = W2 = 1, x = h > 0.
    X = np.array([[g["h"]], [g["h"]]])
    one = np.ones((1, 1, 1))
    D = np.array(g["D"], float)
    row_ptr = np.array(g["row_ptr"], np.int32)
    tag = np.array(g["tag"], np.int32)
    f = orc.moe_forward(X, np.zeros(2, np.int32), one, None, one, None, D, None, row_ptr, tag,
                        want_probs=True)
    np.testing.assert_allclose(f["lse"], g["lse"], rtol=1e-14)
    np.testing.assert_allclose(f["loss"], g["loss"], rtol=1e-14)
    np.testing.assert_allclose(f["probs"][0], g["probs"], rtol=1e-14)
    b = orc.moe_backward(X, np.zeros(2, np.int32), one, one, D, None, row_ptr, tag,
                         f["H1"], f["H"], f["lse"])
    dl = np.array(g["dlogits"])
    # dbD is the batch sum of dloss/dlogits; dD = sum_i dlogits_i * h
    np.testing.assert_allclose(b["dbD"], dl.sum(axis=0), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(b["dD"][:, 0], dl.sum(axis=0) * g["h"], rtol=1e-13, atol=1e-15)


def test_zero_decoder_gives_log_v(orc):
    c = _case(1, V=37)
    c["D"] = np.zeros_like(c["D"])
    c["bD"] = np.zeros_like(c["bD"])
    f = _fwd(orc, c, want_probs=True)
    np.testing.assert_allclose(f["loss"], np.log(37.0), rtol=1e-15)
    np.testing.assert_allclose(f["probs"], 1.0 / 37.0, rtol=1e-14)
    b = _bwd(orc, c, f)
    n = c["X"].shape[0]
    # g = (1/V - y)/n: closed form for dbD
    y = np.zeros((n, 37))
    for i in range(n):
        t = c["tag"][c["row_ptr"][i]:c["row_ptr"][i + 1]]
        y[i, t] = 1.0 / len(t)
    np.testing.assert_allclose(b["dbD"], ((1.0 / 37.0) - y).sum(axis=0) / n, atol=1e-15)


def test_softmax_rows_and_lse(orc):
    c = _case(2, V=50)
    f = _fwd(orc, c, want_probs=True)
    np.testing.assert_allclose(f["probs"].sum(axis=1), 1.0, rtol=1e-13)
    logits = f["H"] @ c["D"].T + c["bD"]
    np.testing.assert_allclose(f["lse"], logsumexp(logits, axis=1), rtol=1e-13)
    assert np.isclose(f["loss_mean"], f["loss"].mean(), rtol=1e-14)


def _torch_loss(c, store_mask=None):
    """The same model written with PyTorch ops (fp64 CPU) for autograd."""
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=k not in ("row_ptr", "tag", "a"))
         for k, v in c.items() if k not in ("row_ptr", "tag", "a")}
    a = torch.tensor(c["a"], dtype=torch.long)
    z = torch.einsum("nhd,nd->nh", t["W1"][a], t["X"]) + t["b1"][a]
    h1 = torch.relu(z)
    y = torch.einsum("noh,nh->no", t["W2"][a], h1) + t["b2"][a]
    logits = y @ t["D"].T + t["bD"]
    n, V = logits.shape
    target = torch.zeros(n, V, dtype=torch.float64)
    for i in range(n):
        tg = c["tag"][c["row_ptr"][i]:c["row_ptr"][i + 1]]
        target[i, torch.tensor(tg, dtype=torch.long)] = 1.0 / len(tg)
    loss = torch.nn.functional.cross_entropy(logits, target)  # mean over the batch
    loss.backward()
    return t, loss, h1, y


@pytest.mark.parametrize("K,empty", [(1, None), (3, None), (4, 2)])
def test_matches_torch_autograd(orc, K, empty):
    c = _case(3 + K, K=K, empty=empty)
    f = _fwd(orc, c)
    b = _bwd(orc, c, f)
    t, loss, h1, y = _torch_loss(c)
    assert np.isclose(f["loss_mean"], loss.item(), rtol=1e-12)
    np.testing.assert_allclose(f["H1"], h1.detach().numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(f["H"], y.detach().numpy(), rtol=1e-12, atol=1e-13)
    for k in ("W1", "b1", "W2", "b2", "D", "bD", "X"):
        np.testing.assert_allclose(b["d" + k], t[k].grad.numpy(), rtol=1e-10, atol=1e-13,
                                   err_msg=k)
    if empty is not None:
        for k in ("dW1", "db1", "dW2", "db2"):
            assert np.all(b[k][empty] == 0.0)


def test_finite_differences(orc):
    """Central differences of loss_mean on the fp64 oracle itself (h = 1e-6)."""
    c = _case(11, n=12, d=4, h=6, o=3, V=7, K=2, max_tags=3)
    # keep pre-activations away from the ReLU kink so the loss is smooth at the probe points
    f = _fwd(orc, c)
    b = _bwd(orc, c, f)
    rs = np.random.default_rng(0)
    eps = 1e-6

    def loss_at(cc):
        return _fwd(orc, cc)["loss_mean"]

    for key, gkey in (("W1", "dW1"), ("b1", "db1"), ("W2", "dW2"), ("b2", "db2"),
                      ("D", "dD"), ("bD", "dbD"), ("X", "dX")):
        for _ in range(4):
            idx = tuple(rs.integers(0, s) for s in c[key].shape)
            cp = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
            cm = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
            cp[key][idx] += eps
            cm[key][idx] -= eps
            fd = (loss_at(cp) - loss_at(cm)) / (2 * eps)
            an = b[gkey][idx]
            assert abs(fd - an) <= 1e-6 * max(abs(an), 1e-3), (key, idx, fd, an)


def test_store_rounding_points(orc):
    """With bf16 storage the hidden activations and outputs are bf16 values and dX too; the
    softmax and the activation gradients g, dh, dz are not rounded."""
    c = _case(12)
    f = _fwd(orc, c, store="bf16")
    for k in ("H1", "H"):
        np.testing.assert_array_equal(orc.round_store(f[k], "bf16"), f[k])
    b = _bwd(orc, c, f, store="bf16")
    np.testing.assert_array_equal(orc.round_store(b["dX"], "bf16"), b["dX"])
    # the gradient of Eq. 3 rounds nothing but the dX it hands back: every other output is the
    # unrounded backward's, bit for bit, and dX is that backward's dX rounded once
    b64 = _bwd(orc, c, f, store="f64")
    for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD"):
        np.testing.assert_array_equal(b[k], b64[k], err_msg=k)
    np.testing.assert_array_equal(b["dX"], orc.round_store(b64["dX"], "bf16"))
    # the diagnostic that rounds g, dh and dz does move the parameter gradients
    bi = _bwd(orc, c, f, store="bf16", internal_store="bf16")
    assert not np.array_equal(bi["dW1"], b64["dW1"])
    np.testing.assert_array_equal(bi["dbD"], b64["dbD"])  # dbD sums the unrounded g
    f64 = _fwd(orc, c, store="f64")
    # the stored H differs from the unrounded one by at most half a bf16 ulp chain
    assert np.max(np.abs(f["H"] - f64["H"])) < 0.05


# ------------------------------------------------------------------ independent decoders

def _case_indep(seed, K=3, empty=None, **kw):
    """_case with one decoder per expert (D [K][V][o], bD [K][V]; Section 2's
    independent-decoder figure)."""
    c = _case(seed, K=K, empty=empty, **kw)
    rs = np.random.default_rng(seed + 1000)
    V, o = c["D"].shape
    c["D"] = rs.normal(size=(K, V, o)) / np.sqrt(o)
    c["bD"] = rs.normal(size=(K, V)) * 0.3
    return c


def _torch_loss_indep(c):
    """Per-sample decoder selection written with PyTorch ops (fp64 CPU) for autograd."""
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True)
         for k, v in c.items() if k not in ("row_ptr", "tag", "a")}
    a = torch.tensor(c["a"], dtype=torch.long)
    h1 = torch.relu(torch.einsum("nhd,nd->nh", t["W1"][a], t["X"]) + t["b1"][a])
    y = torch.einsum("noh,nh->no", t["W2"][a], h1) + t["b2"][a]
    logits = torch.einsum("nvo,no->nv", t["D"][a], y) + t["bD"][a]
    n, V = logits.shape
    target = torch.zeros(n, V, dtype=torch.float64)
    for i in range(n):
        tg = c["tag"][c["row_ptr"][i]:c["row_ptr"][i + 1]]
        target[i, torch.tensor(tg, dtype=torch.long)] = 1.0 / len(tg)
    loss = torch.nn.functional.cross_entropy(logits, target)
    loss.backward()
    return t, loss, logits


@pytest.mark.parametrize("K,empty", [(1, None), (3, None), (4, 1)])
def test_independent_decoders_match_torch_autograd(orc, K, empty):
    c = _case_indep(20 + K, K=K, empty=empty)
    f = _fwd(orc, c, want_logits=True)
    b = _bwd(orc, c, f)
    t, loss, logits = _torch_loss_indep(c)
    assert np.isclose(f["loss_mean"], loss.item(), rtol=1e-12)
    np.testing.assert_allclose(f["logits"], logits.detach().numpy(), rtol=1e-12, atol=1e-13)
    assert b["dD"].shape == c["D"].shape and b["dbD"].shape == c["bD"].shape
    for k in ("W1", "b1", "W2", "b2", "D", "bD", "X"):
        np.testing.assert_allclose(b["d" + k], t[k].grad.numpy(), rtol=1e-10, atol=1e-13,
                                   err_msg=k)
    if empty is not None:
        for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD"):
            assert np.all(b[k][empty] == 0.0), k


def test_independent_decoders_finite_differences(orc):
    c = _case_indep(31, n=12, d=4, h=6, o=3, V=7, K=2, max_tags=3)
    f = _fwd(orc, c)
    b = _bwd(orc, c, f)
    rs = np.random.default_rng(1)
    eps = 1e-6
    for key, gkey in (("D", "dD"), ("bD", "dbD"), ("W2", "dW2"), ("X", "dX")):
        for _ in range(6):
            idx = tuple(rs.integers(0, s) for s in c[key].shape)
            cp = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
            cm = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in c.items()}
            cp[key][idx] += eps
            cm[key][idx] -= eps
            fd = (_fwd(orc, cp)["loss_mean"] - _fwd(orc, cm)["loss_mean"]) / (2 * eps)
            an = b[gkey][idx]
            assert abs(fd - an) <= 1e-6 * max(abs(an), 1e-3), (key, idx, fd, an)


def test_independent_decoders_equal_to_shared_reduce_to_it(orc):
    """K copies of one decoder decode exactly as the shared decoder does; each copy's
    gradient is the shared gradient restricted to its expert's samples, so they sum to it."""
    c = _case(41, K=3)
    ci = dict(c)
    ci["D"] = np.stack([c["D"]] * 3)
    ci["bD"] = np.stack([c["bD"]] * 3)
    f, fi = _fwd(orc, c, want_logits=True), _fwd(orc, ci, want_logits=True)
    for k in ("H1", "H", "lse", "loss", "logits"):
        np.testing.assert_array_equal(fi[k], f[k], err_msg=k)
    b, bi = _bwd(orc, c, f), _bwd(orc, ci, fi)
    for k in ("dW1", "db1", "dW2", "db2", "dX"):
        np.testing.assert_array_equal(bi[k], b[k], err_msg=k)
    np.testing.assert_allclose(bi["dD"].sum(axis=0), b["dD"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(bi["dbD"].sum(axis=0), b["dbD"], rtol=1e-12, atol=1e-15)
    for e in range(3):
        sel = c["a"] == e
        assert np.all(bi["dbD"][e] == 0.0) == (not sel.any())


def test_independent_zero_decoders_give_log_v(orc):
    c = _case_indep(51, K=3)
    c["D"][:] = 0.0
    c["bD"][:] = 0.0
    f = _fwd(orc, c)
    V = c["D"].shape[1]
    np.testing.assert_allclose(f["lse"], np.log(V), rtol=1e-15)
    np.testing.assert_allclose(f["loss"], np.log(V), rtol=1e-15)


def test_backward_magnitude(orc):
    """The magnitude mode is the backward's sums taken over absolute values: it bounds every
    gradient entry (triangle inequality) and equals the chain |G||D| -> |W2| (ReLU mask) -> |W1|
    written out with numpy matrix products per expert (G = (softmax - y)/n from scipy)."""
    from scipy.special import softmax
    c = _case(31, n=60, K=3, empty=1)
    f = _fwd(orc, c)
    b = _bwd(orc, c, f)
    m = _bwd(orc, c, f, magnitude=True)
    for k in ("dW1", "db1", "dW2", "db2", "dD", "dbD", "dX"):
        assert np.all(m[k] >= np.abs(b[k]) * (1 - 1e-12)), k
    n = c["X"].shape[0]
    L = f["H"] @ c["D"].T + c["bD"]
    Y = np.zeros_like(L)
    for i in range(n):
        t = c["tag"][c["row_ptr"][i]:c["row_ptr"][i + 1]]
        Y[i, t] = 1.0 / len(t)
    G = np.abs(softmax(L, axis=1) - Y) / n
    np.testing.assert_allclose(m["dD"], G.T @ np.abs(f["H"]), rtol=1e-12)
    np.testing.assert_allclose(m["dbD"], G.sum(0), rtol=1e-12)
    dH = G @ np.abs(c["D"])
    for e in range(3):
        r = c["a"] == e
        dZ = (dH[r] @ np.abs(c["W2"][e])) * (f["H1"][r] > 0)
        np.testing.assert_allclose(m["dW2"][e], dH[r].T @ np.abs(f["H1"][r]), rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(m["db2"][e], dH[r].sum(0), rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(m["dW1"][e], dZ.T @ np.abs(c["X"][r]), rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(m["db1"][e], dZ.sum(0), rtol=1e-12, atol=1e-300)
        np.testing.assert_allclose(m["dX"][r], dZ @ np.abs(c["W1"][e]), rtol=1e-12, atol=1e-300)
    assert np.all(m["dW1"][1] == 0)  # the empty expert
