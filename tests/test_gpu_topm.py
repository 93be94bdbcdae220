"""The inference tail (Section 4.4) on the HIP path against the oracle: t_m per row, bit-exact
indices on the same logits (including forced ties, fp32 and bf16, small and 50,000-wide
vocabularies, m = 1 .. 16 and the full ranking), the counts behind p@m (Eq. 4) and q@m
(Eq. 5), and the whole inference path (forward, then t_m and the counts) against the oracle's
own forward, exempting rows whose m-th and (m+1)-th logits are closer than the two sides'
rounding."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import anchor_of_columns, anchored, np64, npi, unanchored

pytestmark = pytest.mark.gpu


def _logits(n, V, dtype, seed, ties):
    g = torch.Generator(device="cpu").manual_seed(seed)
    if ties:  # small integers: many exact ties per row
        L = torch.randint(-8, 9, (n, V), generator=g).float()
    else:
        L = torch.randn(n, V, generator=g) * 3.0
    return L.to(torch.bfloat16 if dtype == "bf16" else torch.float32).cuda()


@pytest.mark.parametrize("dtype,n,V,m,ties", [
    ("bf16", 1000, 1000, 10, True), ("bf16", 999, 1000, 5, False), ("f32", 777, 520, 16, True),
    ("f32", 300, 64, 1, False), ("bf16", 64, 8, 8, False), ("bf16", 50, 50000, 10, False),
    ("bf16", 37, 50000, 16, True)])
def test_topm_bit_exact(dtype, n, V, m, ties):
    L = _logits(n, V, dtype, seed=n + V + m, ties=ties)
    idx, val = hmoe.topm(L, m, want_values=True)
    ref = O.topm(np64(L), m)
    assert np.array_equal(npi(idx), ref)
    np.testing.assert_array_equal(np64(val), np.take_along_axis(np64(L), ref.astype(np.int64), axis=1))


@pytest.mark.parametrize("dtype,n,V,m", [("bf16", 500, 1000, 10), ("bf16", 33, 50000, 16), ("f32", 200, 520, 5),
                                          ("bf16", 70, 264, 3)])
def test_topm_anchored_bit_exact(dtype, n, V, m):
    """Logits stored as offsets from per-row anchors (the forward's layout): an entry is anchor +
    offset formed in fp32, on both sides.  Anchors differ between the 64-column blocks of a row,
    and the offsets are drawn so that entries of different blocks tie after the addition."""
    g = torch.Generator(device="cpu").manual_seed(n + V)
    nt = (V + 255) // 256
    anc = (torch.randint(-3, 4, (nt, n, 4), generator=g).float() * 0.5)
    off = torch.randint(-12, 1, (n, V), generator=g).float() * 0.25  # exact in bf16; ties across blocks
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    L, A = off.to(tdt).cuda(), anc.cuda()
    idx, val = hmoe.topm(L, m, want_values=True, anchor=A)
    full = (anchor_of_columns(A, V) + np64(L).astype(np.float32)).astype(np.float32)
    ref = O.topm(full, m)
    assert np.array_equal(npi(idx), ref)
    np.testing.assert_array_equal(np64(val), np.take_along_axis(full, ref.astype(np.int64), axis=1))


@pytest.mark.parametrize("dtype,n,V,m,top", [("bf16", 300, 1000, 10, -0.25), ("bf16", 40, 50000, 16, -0.5),
                                              ("f32", 100, 520, 7, -0.25), ("bf16", 90, 64, 16, 0.0),
                                              ("bf16", 50, 136, 16, -0.25), ("f32", 64, 8, 8, 0.0)])
def test_topm_anchored_unattained_anchors(dtype, n, V, m, top):
    """Anchors that only bound their blocks (every offset at most `top` < 0), so a block with a
    high anchor may hold only lower entries, and the blocks whose anchor lies between the row's
    m-th entry and the m-th largest anchor must be read as well; plus rows with fewer 64-column
    blocks than m (V = 64, 136, 8)."""
    g = torch.Generator(device="cpu").manual_seed(7 * n + V)
    nt = (V + 255) // 256
    anc = torch.randint(-4, 5, (nt, n, 4), generator=g).float() * 0.5
    off = torch.randint(-16, 1, (n, V), generator=g).float() * 0.25 + top
    off = torch.minimum(off, torch.tensor(top))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    L, A = off.to(tdt).cuda(), anc.cuda()
    idx, val = hmoe.topm(L, m, want_values=True, anchor=A)
    full = (anchor_of_columns(A, V) + np64(L).astype(np.float32)).astype(np.float32)
    ref = O.topm(full, m)
    assert np.array_equal(npi(idx), ref)
    np.testing.assert_array_equal(np64(val), np.take_along_axis(full, ref.astype(np.int64), axis=1))


@pytest.mark.parametrize("n,V,m", [(64, 50000, 10), (200, 4000, 16), (128, 1000, 1)])
def test_topm_anchored_forward_layout(n, V, m):
    """The forward's own layout (each anchor its block's maximum, offsets rounded to bf16) from
    Gaussian logits of the trained-tagger scale."""
    Lf = np.random.default_rng(n + V).standard_normal((n, V)) * 6.0
    L, A = anchored(Lf, torch.bfloat16)
    idx, val = hmoe.topm(L, m, want_values=True, anchor=A)
    full = unanchored(L, A)
    ref = O.topm(full, m)
    assert np.array_equal(npi(idx), ref)
    np.testing.assert_array_equal(np64(val), np.take_along_axis(full, ref.astype(np.int64), axis=1))


def test_topm_anchored_full_size_sampled_rows():
    """The inference workload's shape and launch (65,536 x 50,000 bf16 logits in the forward's
    anchored layout, m = 10): 512 seeded rows against the oracle on their own entries, plus
    every row's list checked for validity (m distinct in-range indices, values non-increasing
    and equal to the entries they name)."""
    n, V, m = 65536, 50000, 10
    g = torch.Generator(device="cuda").manual_seed(21)
    nt = (V + 255) // 256
    Lp = torch.full((n, nt * 256), -float("inf"), device="cuda")
    Lp[:, :V] = torch.randn(n, V, device="cuda", generator=g) * 6.0
    bm = Lp.view(n, nt, 4, 64).amax(dim=3)  # each 64-column block's maximum: the anchor
    A = bm.permute(1, 0, 2).contiguous()
    L = (Lp.view(n, nt, 4, 64) - bm[..., None]).view(n, nt * 256)[:, :V].to(torch.bfloat16).contiguous()
    del Lp, bm
    idx, val = hmoe.topm(L, m, want_values=True, anchor=A)
    rows = np.sort(np.random.default_rng(22).choice(n, 512, replace=False))
    ri = torch.as_tensor(rows, device="cuda")
    full = (anchor_of_columns(A[:, ri].contiguous(), V) + np64(L[ri]).astype(np.float32)).astype(np.float32)
    ref = O.topm(full, m)
    assert np.array_equal(npi(idx)[rows], ref)
    np.testing.assert_array_equal(np64(val)[rows], np.take_along_axis(full, ref.astype(np.int64), axis=1))
    # every row: distinct in-range indices, non-increasing values equal to anchor + offset there
    it = idx.long()
    assert int(it.min()) >= 0 and int(it.max()) < V
    assert bool((it.sort(dim=1).values.diff(dim=1) > 0).all())
    assert bool((val.diff(dim=1) <= 0).all())
    anc_at = A.permute(1, 0, 2).reshape(n, nt * 4).gather(1, it // 64)
    assert torch.equal(anc_at + L.gather(1, it).float(), val)


def test_hits_exact():
    n, V, m = 3000, 2000, 10
    L = _logits(n, V, "bf16", seed=5, ties=False)
    rp, tg = W.zipf_labels(n, V, 8, seed=6)
    qs, qt = W.q_draws(rp, tg, 100000, seed=7)
    idx = hmoe.topm(L, m)
    dev = lambda a: torch.as_tensor(a).cuda()  # noqa: E731
    hits = hmoe.topm_hits(idx, dev(rp), dev(tg), dev(qs), dev(qt))
    p_ref, q_ref = O.topm_hits(O.topm(np64(L), m), rp, tg, qs, qt)
    assert npi(hits[0]).tolist() == p_ref.tolist()
    assert npi(hits[1]).tolist() == q_ref.tolist()
    # no draws, and draws naming no sample
    h0 = hmoe.topm_hits(idx, dev(rp), dev(tg))
    assert npi(h0[0]).tolist() == p_ref.tolist() and int(npi(h0[1]).sum()) == 0
    bad = hmoe.topm_hits(idx, dev(rp), dev(tg), dev(np.array([-1, n], np.int32)), dev(np.array([0, 0], np.int32)))
    assert int(npi(bad[1]).sum()) == 0


def test_inference_path_against_the_oracle():
    """Forward, then t_10 and the counts.  fp32 (the tiny workload): the lists equal the
    oracle's except on rows with two consecutive ranks closer than 1e-5 (relative).  bf16 (a
    balanced-shape miniature): the stored bf16 logits of a row's top ranks are often equal or
    one rounding apart, so instead every chosen tag must be within two bf16 roundings of the
    oracle's 10th largest logit, and p@m, q@m must agree with the oracle's to 1%."""
    m = 10
    for store, inp in (("f32", W.tiny_inputs(device="cuda", seed=0)),
                       ("bf16", W.balanced_inputs(device="cuda", seed=3, n=2000, d=256, h=512, o=128,
                                                  V=1000, K=4))):
        p = inp["params"]
        n = inp["X"].shape[0]
        K = p["W1"].shape[0]
        ids = np.random.default_rng(1).integers(0, K, n).astype(np.int32)
        dd = hmoe.moe_dispatch(torch.as_tensor(ids).cuda(), K, rows=inp["X"])
        rp, tg = inp["row_ptr"], inp["tag"]
        dev = lambda a: torch.as_tensor(a).cuda()  # noqa: E731
        f = hmoe.moe_forward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dev(rp), dev(tg), save_logits=True)
        idx = npi(hmoe.topm(f["logits"], m, anchor=f["logit_anchor"]))
        ph = {k: (np64(v) if v is not None else None) for k, v in p.items()}
        ref = O.moe_forward(np64(inp["X"]), ids, ph["W1"], ph["b1"], ph["W2"], ph["b2"], ph["D"], ph["bD"], rp, tg,
                            store=store, want_logits=True)
        Lr = ref["logits"]
        top_ref = O.topm(Lr, m + 1)
        srt = np.take_along_axis(Lr, top_ref.astype(np.int64), axis=1)
        qs, qt = W.q_draws(rp, tg, 20000, seed=9)
        hits = npi(hmoe.topm_hits(dev(idx), dev(rp), dev(tg), dev(qs), dev(qt)))
        p_ref, q_ref = O.topm_hits(top_ref[:, :m], rp, tg, qs, qt)
        if store == "f32":
            gap = srt[:, :-1] - srt[:, 1:]
            near = np.any(gap <= 1e-5 * np.maximum(np.abs(srt[:, :-1]), 1.0), axis=1)
            assert near.mean() < 0.05
            assert np.array_equal(idx[~near], top_ref[~near, :m])
            assert np.all(np.abs(hits[0] - p_ref) <= near.sum() * m)
        else:
            chosen = np.take_along_axis(Lr, idx.astype(np.int64), axis=1)
            tenth = srt[:, m - 1:m]
            assert np.all(chosen >= tenth - 2 * 2.0 ** -7 * np.maximum(np.abs(tenth), 1.0))
            assert np.all(np.abs(hits[0] - p_ref) <= 0.01 * rp[-1])
            assert np.all(np.abs(hits[1] - q_ref) <= 0.01 * len(qs))
