"""The C-ABI library builds, loads and exports every entry point include/hmoe.h declares;
host-side argument checks reject bad calls before anything is launched (no GPU needed)."""
import ctypes
import os
import re

import pytest

from paper_1704_06363_amd import hmoe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "hmoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hmoe_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hmoe.LIB_PATH):
        from paper_1704_06363_amd import build
        build.build()
    return hmoe.lib()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) == 23
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(hmoe.SYMBOLS)


def test_version_and_error_string(lib):
    assert hmoe.version() == 2
    assert isinstance(hmoe.last_error(), str)


def test_workspace_queries(lib):
    assert hmoe.kmeans_assign_workspace(4096, 64, 8, __import__("torch").float32) > 0
    assert lib.hmoe_kmeans_fit_workspace(4096, 64, 8, 0) > 0
    assert lib.hmoe_moe_dispatch_workspace(1000, 7) >= 1000 // 1024 * 7
    p = hmoe.MoeParams(8, 64, 128, 64, 1000, 0, 16, None, 16, None, 16, None)
    assert hmoe.moe_workspace(p, 4096) > 4096 * 1000 * 4  # holds g = (p - y)/n


def test_argument_errors_are_reported_before_launch(lib):
    # d not a multiple of 8
    rc = lib.hmoe_kmeans_assign(16, 0, 10, 12, 16, 3, 16, None, None, 0, None)
    assert rc == -3 and "multiple of 8" in hmoe.last_error()
    # K out of range
    rc = lib.hmoe_kmeans_assign(16, 0, 10, 16, 16, 0, 16, None, None, 0, None)
    assert rc == -1 and "K" in hmoe.last_error()
    # unknown dtype
    rc = lib.hmoe_kmeans_assign(16, 7, 10, 16, 16, 3, 16, None, None, 0, None)
    assert rc == -2
    # workspace too small
    rc = lib.hmoe_kmeans_assign(16, 0, 10, 16, 16, 300, 16, None, None, 0, None)
    assert rc == -4 and "workspace" in hmoe.last_error()
    # misaligned pointer
    rc = lib.hmoe_kmeans_assign(18, 0, 10, 16, 16, 3, 16, None, None, 0, None)
    assert rc == -3 and "aligned" in hmoe.last_error()
    # fit with n < K
    rc = lib.hmoe_kmeans_fit(16, 0, 3, 16, 4, 1, None, 1, 16, 16, None, None, None, None, None, 0,
                             None)
    assert rc == -1 and "n >= K" in hmoe.last_error()
    # dispatch with a NULL perm
    rc = lib.hmoe_moe_dispatch(16, 10, 3, 16, 16, None, 16, None, None, 0, 0, None, 0, None)
    assert rc == -1 and "perm" in hmoe.last_error()
    # the allocation-free dispatch: the same checks, and sizes beyond its scratch array refused
    # before the device is touched (K = 4096 over 2^21 rows needs 32 MiB of bucket counts)
    rc = lib.hmoe_moe_dispatch_noalloc(16, 10, 3, 16, 16, None, 16, None, None, 0, 0, None)
    assert rc == -1 and "perm" in hmoe.last_error()
    rc = lib.hmoe_moe_dispatch_noalloc(16, 1 << 21, 4096, 16, 16, 16, 16, None, None, 0, 0, None)
    assert rc == -4 and "scratch" in hmoe.last_error()
    # moe forward with vocab not a multiple of 8
    p = hmoe.MoeParams(2, 64, 128, 64, 1001, 0, 16, None, 16, None, 16, None)
    lab = hmoe.Labels(16, 16)
    rc = lib.hmoe_moe_forward(ctypes.byref(p), 10, 16, 16, 16, ctypes.byref(lab), 16, 16, None, None,
                              16, 16, 16, None, 0, None)
    assert rc == -3 and "vocab" in hmoe.last_error()
    # stored logits without their anchors
    p = hmoe.MoeParams(2, 64, 128, 64, 1000, 0, 16, None, 16, None, 16, None)
    rc = lib.hmoe_moe_forward(ctypes.byref(p), 10, 16, 16, 16, ctypes.byref(lab), 16, 16, 16, None,
                              16, 16, 16, None, 0, None)
    assert rc == -1 and "logit_anchor" in hmoe.last_error()
    rc = lib.hmoe_moe_backward(ctypes.byref(p), 10, 16, 16, 16, 16, ctypes.byref(lab), 16, 16, 16, None,
                               16, 16, None, 16, None, 16, None, None, None, 0, None)
    assert rc == -1 and "logit_anchor" in hmoe.last_error()
    # update with an unknown mode
    rc = lib.hmoe_kmeans_update(16, 0, 10, 16, 3, 16, 16, 16, 16, 16, 9, 0, None, 0, None)
    assert rc == -1 and "mode" in hmoe.last_error()
    # a decoder count that is neither 1 nor K
    p = hmoe.MoeParams(4, 64, 128, 64, 1000, 0, 16, None, 16, None, 16, None, 3)
    rc = lib.hmoe_moe_forward(ctypes.byref(p), 10, 16, 16, 16, ctypes.byref(lab), 16, 16, None, None,
                              16, 16, 16, None, 0, None)
    assert rc == -1 and "decoders" in hmoe.last_error()
    # top-m: m outside [1, 16], and a vocabulary that is not a multiple of 8
    rc = lib.hmoe_topm(16, None, 1, 10, 64, 17, 16, None, None)
    assert rc == -1 and "m = 17" in hmoe.last_error()
    rc = lib.hmoe_topm(16, None, 1, 10, 60, 5, 16, None, None)
    assert rc == -3 and "vocab" in hmoe.last_error()
    rc = lib.hmoe_topm(16, 20, 1, 10, 64, 5, 16, None, None)  # anchors are read as 16-byte vectors
    assert rc == -3 and "anchor" in hmoe.last_error()
    rc = lib.hmoe_topm_hits(16, 10, 0, ctypes.byref(lab), None, None, 0, 16, None)
    assert rc == -1 and "m = 0" in hmoe.last_error()
    # PCA: more components than dimensions, one sample
    rc = lib.hmoe_pca_fit(16, 0, 100, 64, 72, 5, 0, 16, 16, 16, None, 0, None)
    assert rc == -1 and "exceeds" in hmoe.last_error()
    rc = lib.hmoe_pca_fit(16, 0, 1, 64, 8, 5, 0, 16, 16, 16, None, 0, None)
    assert rc == -1 and "n >= 2" in hmoe.last_error()
    # SGD: momentum without a buffer, a negative learning rate
    rc = lib.hmoe_sgd_step(16, 16, None, None, 1, 100, ctypes.c_float(0.1), ctypes.c_float(0.0),
                           ctypes.c_float(0.9), None)
    assert rc == -1 and "momentum" in hmoe.last_error()
    rc = lib.hmoe_sgd_step(16, 16, None, None, 1, 100, ctypes.c_float(-0.1), ctypes.c_float(0.0),
                           ctypes.c_float(0.0), None)
    assert rc == -1 and "lr" in hmoe.last_error()


def test_binding_refuses_host_tensors(lib):
    import torch
    with pytest.raises(hmoe.HmoeError):
        hmoe.kmeans_assign(torch.zeros(4, 8), torch.zeros(2, 8))


def test_binding_refuses_mismatched_dtypes_and_shapes():
    # checked before any pointer is taken: a tensor of another dtype or size would make the
    # library read or write past its bytes
    import torch
    with pytest.raises(hmoe.HmoeError, match="dtype"):
        hmoe.kmeans_assign(torch.zeros(4, 8), torch.zeros(2, 8, dtype=torch.bfloat16))
    with pytest.raises(hmoe.HmoeError, match="shape"):
        hmoe.kmeans_assign(torch.zeros(4, 8), torch.zeros(2, 16))
    p = {"W1": torch.zeros(2, 16, 8, dtype=torch.bfloat16), "b1": None,
         "W2": torch.zeros(2, 8, 16, dtype=torch.bfloat16), "b2": None,
         "D": torch.zeros(24, 8, dtype=torch.bfloat16), "bD": None}
    with pytest.raises(hmoe.HmoeError, match="X_sorted: dtype"):
        hmoe.moe_forward(p, torch.zeros(4, 8), torch.zeros(3, dtype=torch.int32), torch.zeros(4, dtype=torch.int32),
                         None, None)
    bad = dict(p, W2=torch.zeros(2, 8, 16))
    with pytest.raises(hmoe.HmoeError, match="W2: dtype"):
        hmoe.make_params(bad)
    with pytest.raises(hmoe.HmoeError, match="counts: shape"):
        hmoe.moe_dispatch(torch.zeros(4, dtype=torch.int32), 3, out={"counts": torch.zeros(4, dtype=torch.int32)})
