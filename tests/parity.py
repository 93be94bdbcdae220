"""Comparison helpers for the HIP-vs-oracle parity tests.

Floats: |gpu - ref| <= rtol * max(|ref|, rms(ref)) elementwise (rtol 1e-4 for fp32 data,
2e-2 for bf16).  Integer / index outputs: bit-exact, except assignment rows whose oracle
runner-up distance is within 1e-5 (relative) of the minimum.

Gradients (assert_grad_close): the same bar, or, for an entry whose sum cancels, the
first-order rounding-error bound of the computation, c u M: M is the oracle's magnitude of the
entry (the backward's sums over absolute values), u the unit roundoff of the data dtype (2^-9
for bf16, 2^-24 for fp32) and c = 4 the number of roundings on the longest chain (g, dH, dZ and
dX, each an MFMA operand or output in the data dtype).  Where the terms do not cancel, M is
|ref| and c u M lies below the 2e-2 bar; the floor only decides entries whose value is a small
remainder of much larger terms, where any evaluation with bf16 operands is off by about u M."""
import numpy as np
import torch

RTOL = {"f32": 1e-4, "bf16": 2e-2}
UNIT_ROUNDOFF = {"f32": 2.0 ** -24, "bf16": 2.0 ** -9}
CHAIN_ROUNDINGS = 4


def np64(t) -> np.ndarray:
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy().astype(np.float64)


def npi(t) -> np.ndarray:
    return t.detach().cpu().numpy() if isinstance(t, torch.Tensor) else np.asarray(t)


def assert_close(gpu, ref, rtol, what="", mass=None):
    g = np64(gpu)
    r = np64(ref)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    if r.size == 0:
        return
    rms = float(np.sqrt(np.mean(r * r)))
    scale = np.maximum(np.abs(r), rms)
    if mass is not None:
        assert mass.shape == r.shape, (what, mass.shape, r.shape)
        scale = np.maximum(scale, mass)
    bound = rtol * scale
    err = np.abs(g - r)
    bad = ~(err <= bound)
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(bad, err / np.maximum(bound, 1e-300), 0)), r.shape)
        raise AssertionError(f"{what}: {int(bad.sum())}/{r.size} outside tolerance; worst at {i}: "
                             f"gpu {g[i]!r} ref {r[i]!r} bound {bound[i]!r} (rms {rms:.3e})")


def assert_grad_close(gpu, ref, mag, store, what=""):
    """rtol * max(|ref|, rms(ref)), or the rounding-error floor c u M (M = mag, the oracle's
    magnitude of each entry)."""
    rt = RTOL[store]
    floor = np64(mag) * (CHAIN_ROUNDINGS * UNIT_ROUNDOFF[store] / rt)
    assert_close(gpu, ref, rt, what, mass=floor)


def assert_scalar_close(gpu, ref, rtol, what=""):
    g, r = float(gpu), float(ref)
    assert abs(g - r) <= rtol * max(abs(r), 1e-30), f"{what}: gpu {g!r} ref {r!r}"


def assert_assign(a_gpu, a_ref, d1_ref, d2_ref, what="assign"):
    from oracle import oracle
    a_gpu = npi(a_gpu)
    exempt = oracle.near_tie(d1_ref, d2_ref)
    bad = (a_gpu != a_ref) & ~exempt
    assert not bad.any(), f"{what}: {int(bad.sum())} rows differ outside the near-tie band " \
                          f"(first {np.flatnonzero(bad)[:5]})"
    return int(exempt.sum())


# ------------------------------------------------------------------ stored-logit layout

ANCHOR_COLS, ANCHOR_TILE = 64, 256  # include/hmoe.h: HMOE_ANCHOR_COLS, HMOE_ANCHOR_TILE
ASLOTS = ANCHOR_TILE // ANCHOR_COLS


def anchor_of_columns(anc, V):
    """[n, V] float32: the anchor of every column, from an anchor array [ceil(V/256), n, 4]."""
    a = np.asarray(npi(anc), dtype=np.float32)
    cols = np.arange(V)
    return a[cols // ANCHOR_TILE, :, (cols % ANCHOR_TILE) // ANCHOR_COLS].T


def anchored(L, dtype):
    """The stored form of logits L [n, V] (float64) in the library's layout: per row and 64
    columns the fp32 maximum as the anchor, and each logit as its fp32 offset from that anchor
    rounded to `dtype` (torch.float32 or torch.bfloat16).  Returns (offsets on the GPU,
    anchors float32 on the GPU, [ceil(V/256), n, 4])."""
    L32 = np.asarray(L, dtype=np.float64).astype(np.float32)
    n, V = L32.shape
    nt = (V + ANCHOR_TILE - 1) // ANCHOR_TILE
    anc = np.full((nt, n, ASLOTS), -np.finfo(np.float32).max, np.float32)
    for b in range((V + ANCHOR_COLS - 1) // ANCHOR_COLS):
        anc[b // ASLOTS, :, b % ASLOTS] = L32[:, b * ANCHOR_COLS:(b + 1) * ANCHOR_COLS].max(axis=1)
    off = (L32 - anchor_of_columns(anc, V)).astype(np.float32)
    return (torch.from_numpy(off).to(dtype).cuda().contiguous(),
            torch.from_numpy(anc).cuda().contiguous())


def unanchored(offsets, anc):
    """float32 logits from the stored form: anchor + offset, the sum formed in fp32."""
    off = np64(offsets).astype(np.float32)
    return (anchor_of_columns(anc, off.shape[1]) + off).astype(np.float32)


def assert_stored_logits(offsets, anc, L, store, what="stored logits"):
    """The stored form against the exact logits L: anchor + offset within rtol * max(|L|, rms),
    or within two roundings of the offset in the data dtype (its own and the fp32 logit it was
    taken from), 2 u |L - anchor|: an entry far below its block's maximum is stored to that
    accuracy."""
    V = L.shape[1]
    a = anchor_of_columns(anc, V).astype(np.float64)
    rep = 2.0 * UNIT_ROUNDOFF[store] * np.abs(L - a) / RTOL[store]
    assert_close(unanchored(offsets, anc), L, RTOL[store], what, mass=rep)
