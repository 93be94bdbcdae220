"""Full-size gradients of the balanced and skewed steps, element by element, in the bench's
launch configuration (bf16, logits saved by the forward).

The C oracle cannot redo a 65,536-row step in seconds, so the full-size reference here is the
gradient of Eq. 3 (Section 4.1) written out with torch fp64 operations on the GPU, computed from
the step's inputs alone -- features, weights, labels and the routing -- and rounding only H1 and
H to bf16, where the boundary stores them, as the oracle does.  Nothing the HIP library computes
enters it.  Before it is used it is pinned to the C oracle on sampled rows (H1, H, lse, loss to
1e-9).  It then gives:
  * 512 seeded rows of dD and dbD, drawn from both parts of the dD launch: the tiles that run
    whole over all n rows and the last partial round of tiles, which is split over the rows;
  * the whole dW1, db1, dW2 and db2 of the median expert (by bucket size)."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import RTOL, assert_close, np64, npi

pytestmark = pytest.mark.gpu
RT = RTOL["bf16"]
f64 = torch.float64


def _bf16_rne(x):
    """fp64 -> the nearest bf16 value (8 significant bits, ties to even), kept in fp64."""
    m, e = torch.frexp(x)
    return torch.ldexp(torch.round(torch.ldexp(m, torch.full_like(e, 8))), e - 8)


def _dense_targets(row_ptr, tag, rows, cols, V):
    """Y[r, c] = 1/|P_i| if cols[c] is a positive tag of sample rows[r] (else 0), fp64 on the GPU."""
    col_of = np.full(V, -1, np.int64)
    col_of[cols] = np.arange(len(cols))
    Y = np.zeros((len(rows), len(cols)))
    for r, i in enumerate(rows):
        t = tag[row_ptr[i]:row_ptr[i + 1]]
        c = col_of[t]
        Y[r, c[c >= 0]] = 1.0 / len(t)
    return torch.as_tensor(Y, dtype=f64, device="cuda")


class Reference:
    """Forward of the hard mixture in fp64 (Section 2): per expert h1 = relu(W1 x + b1) and
    y = W2 h1 + b2, both rounded to bf16 as stored; lse of the decoder logits D y + bD."""

    def __init__(self, inp, ids):
        s = inp["shape"]
        self.s = s
        self.ids = np.asarray(ids, np.int64)
        self.X = inp["X"].to(f64)
        self.p = {k: (v.to(f64) if v is not None else None) for k, v in inp["params"].items()}
        self.rp, self.tg = inp["row_ptr"], inp["tag"]
        n, h, o = s["n"], s["h"], s["o"]
        self.H1 = torch.empty(n, h, dtype=f64, device="cuda")
        self.H = torch.empty(n, o, dtype=f64, device="cuda")
        ids_t = torch.as_tensor(self.ids, device="cuda")
        p = self.p
        for e in range(s["K"]):
            rows = torch.nonzero(ids_t == e).flatten()
            if rows.numel() == 0:
                continue
            z = self.X[rows] @ p["W1"][e].T + p["b1"][e]
            h1 = _bf16_rne(torch.clamp_min(z, 0.0))
            self.H1[rows] = h1
            self.H[rows] = _bf16_rne(h1 @ p["W2"][e].T + p["b2"][e])
        self.lse = torch.empty(n, dtype=f64, device="cuda")
        for r0 in range(0, n, 4096):
            self.lse[r0:r0 + 4096] = torch.logsumexp(self.logits(slice(r0, r0 + 4096)), dim=1)

    def logits(self, rows, cols=None):
        D, bD = self.p["D"], self.p["bD"]
        if cols is not None:
            ci = torch.as_tensor(np.asarray(cols, np.int64), device="cuda")
            D, bD = D[ci], bD[ci]
        return self.H[rows] @ D.T + bD

    def g(self, rows, cols):
        """(p - y) / n on rows x cols (Section 4.1, Eq. 3, target mass 1/|P_i| per positive)."""
        rows_np = np.asarray(rows)
        ri = torch.as_tensor(rows_np, device="cuda")
        P = torch.exp(self.logits(ri, cols) - self.lse[ri, None])
        return (P - _dense_targets(self.rp, self.tg, rows_np, cols, self.s["V"])) / self.s["n"]

    def decoder_rows(self, cols):
        """dD and dbD on the vocabulary rows `cols`: sum_i g_i,v H_i and sum_i g_i,v."""
        n = self.s["n"]
        dD = torch.zeros(len(cols), self.s["o"], dtype=f64, device="cuda")
        dbD = torch.zeros(len(cols), dtype=f64, device="cuda")
        for r0 in range(0, n, 8192):
            rows = np.arange(r0, min(n, r0 + 8192))
            g = self.g(rows, cols)
            dD += g.T @ self.H[r0:r0 + len(rows)]
            dbD += g.sum(dim=0)
        return dD, dbD

    def expert(self, e):
        """The whole parameter gradient of expert e: dh = D^T g, then back through W2, the ReLU
        and W1 over the expert's own samples (Section 2; ReLU'(0) = 0)."""
        rows = np.flatnonzero(self.ids == e)
        ri = torch.as_tensor(rows, device="cuda")
        p = self.p
        V = self.s["V"]
        dH = torch.zeros(len(rows), self.s["o"], dtype=f64, device="cuda")
        for c0 in range(0, V, 8192):
            cols = np.arange(c0, min(V, c0 + 8192))
            dH += self.g(rows, cols) @ p["D"][c0:c0 + len(cols)]
        H1 = self.H1[ri]
        dZ = (dH @ p["W2"][e]) * (H1 > 0)
        return {"dW2": dH.T @ H1, "db2": dH.sum(0), "dW1": dZ.T @ self.X[ri], "db1": dZ.sum(0)}


def _pin_to_oracle(ref, inp, rows):
    """The fp64 reference's forward equals the C oracle's on `rows` (both fp64, H1 and H rounded
    to bf16 the same way)."""
    # the oracle widens only the experts these rows use (ids remapped to 0 .. m-1)
    uniq = np.unique(ref.ids[rows])
    sel = torch.as_tensor(uniq, device="cuda")
    ph = {k: np64(v[sel] if k in ("W1", "b1", "W2", "b2") else v) for k, v in inp["params"].items()}
    Xs = np64(inp["X"][torch.as_tensor(rows, device="cuda")])
    cnt = inp["row_ptr"][1:] - inp["row_ptr"][:-1]
    srp = np.concatenate([[0], np.cumsum(cnt[rows])]).astype(np.int32)
    stg = np.concatenate([inp["tag"][inp["row_ptr"][i]:inp["row_ptr"][i + 1]] for i in rows]).astype(np.int32)
    orc = O.moe_forward(Xs, np.searchsorted(uniq, ref.ids[rows]).astype(np.int32), ph["W1"], ph["b1"], ph["W2"],
                        ph["b2"], ph["D"], ph["bD"], srp, stg, store="bf16")
    ri = torch.as_tensor(rows, device="cuda")
    assert_close(ref.H1[ri], orc["H1"], 1e-9, "reference H1 vs oracle")
    assert_close(ref.H[ri], orc["H"], 1e-9, "reference H vs oracle")
    assert_close(ref.lse[ri], orc["lse"], 1e-9, "reference lse vs oracle")
    pos = torch.tensor([float(ref.logits(ri[k:k + 1], inp["tag"][inp["row_ptr"][i]:inp["row_ptr"][i + 1]]).mean())
                        for k, i in enumerate(rows)], dtype=f64)
    assert_close((ref.lse[ri].cpu() - pos).numpy(), orc["loss"], 1e-9, "reference loss vs oracle")


def _step(inp, ids):
    s = inp["shape"]
    a = torch.as_tensor(ids, dtype=torch.int32).cuda()
    d = hmoe.moe_dispatch(a, s["K"], rows=inp["X"])
    rp = torch.as_tensor(inp["row_ptr"]).cuda()
    tg = torch.as_tensor(inp["tag"]).cuda()
    f = hmoe.moe_forward(inp["params"], d["rows_sorted"], d["offsets"], d["perm"], rp, tg, save_logits=True)
    g = hmoe.moe_backward(inp["params"], d["rows_sorted"], d["offsets"], d["perm"], d["inv"], rp, tg,
                          f["H1_sorted"], f["H"], f["lse"], logits=f["logits"], logit_anchor=f["logit_anchor"])
    torch.cuda.synchronize()
    return d, f, g


def _decoder_sample(V, o, seed):
    """512 vocabulary rows: the 16 most frequent tags, 432 drawn from the dD tiles that run whole
    and 64 from the last partial round (split over the rows).  The dD launch runs its 256 x 256
    tiles in rounds of 256 (one per CU) in bands of 16 row tiles; the last round's tiles are the
    last 16 * ceil(o / 256)-tile band's remainder."""
    tiles = -(-V // 256) * -(-o // 256)
    whole = tiles - tiles % 256
    v_split = (whole // (16 * -(-o // 256))) * 16 * 256  # first vocabulary row of the split tiles
    rs = np.random.default_rng(seed)
    head = np.arange(16)
    body = rs.choice(np.arange(16, min(v_split, V)), 432, replace=False)
    tail = rs.choice(np.arange(v_split, V), min(64, V - v_split), replace=False) if v_split < V else []
    return np.unique(np.concatenate([head, body, tail]).astype(np.int64)), v_split


def _check(inp, ids, seed):
    s = inp["shape"]
    d, f, g = _step(inp, ids)
    ref = Reference(inp, ids)
    rs = np.random.default_rng(seed)
    _pin_to_oracle(ref, inp, np.sort(rs.choice(s["n"], 6, replace=False)))
    # the forward's per-sample outputs, whole
    assert_close(f["H"], ref.H, RT, "H")
    assert_close(f["lse"], ref.lse, RT, "lse")
    cols, v_split = _decoder_sample(s["V"], s["o"], seed)
    assert (cols >= v_split).sum() >= 32 and (cols < v_split).sum() >= 400
    dD, dbD = ref.decoder_rows(cols)
    ci = torch.as_tensor(cols, device="cuda")
    assert_close(g["dD"][ci], dD, RT, "dD (512 sampled vocabulary rows)")
    assert_close(g["dbD"][ci], dbD, RT, "dbD (512 sampled vocabulary rows)")
    counts = npi(d["counts"])
    e = int(np.argsort(counts, kind="stable")[s["K"] // 2])
    want = ref.expert(e)
    for k in ("dW1", "db1", "dW2", "db2"):
        assert_close(g[k][e], want[k], RT, f"{k} of the median expert {e} ({counts[e]} samples)")
    return counts[e]


def test_balanced_step_gradients_full_size():
    inp = W.balanced_inputs(device="cuda", seed=0)
    # routing by the nearest centre, in fp64 by direct differences (Eq. 2); the HIP step takes
    # these ids, so both sides route every sample the same way
    X = inp["X"].to(f64)
    C = inp["C"].to(f64)
    dist = torch.cdist(X, C, compute_mode="donot_use_mm_for_euclid_dist")
    ids = npi(torch.argmin(dist, dim=1)).astype(np.int32)
    del X, dist
    m = _check(inp, ids, seed=5)
    assert m > 2000


def test_skewed_step_gradients_full_size():
    inp = W.skewed_inputs(device="cuda", seed=0)
    m = _check(inp, inp["ids"], seed=6)
    assert m >= 8
