"""Comparison helpers for the HIP-vs-oracle parity tests.

Floats: |gpu - ref| <= rtol * max(|ref|, rms(ref)) elementwise (rtol 1e-4 for fp32 data,
2e-2 for bf16).  Where a result is a short sum whose terms may cancel, the caller passes the
sum of the terms' magnitudes (`mass`), the usual scale of a summation error bound, and the
bound becomes rtol * max(|ref|, rms(ref), mass).  Integer / index outputs: bit-exact, except
assignment rows whose oracle runner-up distance is within 1e-5 (relative) of the minimum."""
import numpy as np
import torch

RTOL = {"f32": 1e-4, "bf16": 2e-2}


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
