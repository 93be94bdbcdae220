"""The allocation-free dispatch (hmoe_moe_dispatch_noalloc, for callers that cannot allocate)
against the dispatch with a caller workspace, through the C ABI: bit-identical counts, offsets,
perm, inv and gathered rows on two calls in a row, the second with a smaller input (the scratch
array keeps the first call's contents), then the first size again on another stream."""
import numpy as np
import pytest
import torch

from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W

pytestmark = pytest.mark.gpu


def _same(a, b):
    for k in ("counts", "offsets", "perm", "inv", "rows_sorted"):
        if a[k] is None:
            assert b[k] is None, k
            continue
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("n,K,w,dtype", [(65536, 16, 2048, "bf16"), (1000, 5, 64, "f32")])
def test_noalloc_dispatch_matches_workspace_dispatch(n, K, w, dtype):
    rows = W.rectified_gaussian(n, w, seed=n, dtype=dtype, device="cuda")
    ids = torch.as_tensor(np.random.default_rng(K).integers(0, K, n).astype(np.int32)).cuda()
    ref = hmoe.moe_dispatch(ids, K, rows=rows)
    got = hmoe.moe_dispatch_noalloc(ids, K, rows=rows)
    torch.cuda.synchronize()
    _same(got, ref)
    # second call, smaller (skewed buckets, one empty): the array still holds the first call's counts
    m, K2 = 3001, 128
    ids2 = torch.as_tensor(W.zipf_bucket_ids(m, K2, seed=3)).cuda()
    rows2 = W.rectified_gaussian(m, w, seed=m, dtype=dtype, device="cuda")
    ref2 = hmoe.moe_dispatch(ids2, K2, rows=rows2)
    got2 = hmoe.moe_dispatch_noalloc(ids2, K2, rows=rows2)
    torch.cuda.synchronize()
    _same(got2, ref2)
    assert int((ref2["counts"] == 0).sum()) >= 1
    # the first size again, ids only, on another stream
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        got3 = hmoe.moe_dispatch_noalloc(ids, K)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for k in ("counts", "offsets", "perm", "inv"):
        assert torch.equal(got3[k], ref[k]), k


def test_noalloc_dispatch_refuses_sizes_beyond_its_scratch():
    # K = 4096 over 2^21 rows needs 2048 * 4097 * 4 bytes of bucket counts, more than 16 MiB:
    # refused before any launch, outputs untouched
    n, K = 1 << 21, 4096
    ids = torch.zeros(n, dtype=torch.int32, device="cuda")
    out = {"counts": torch.full((K,), -7, dtype=torch.int32, device="cuda")}
    with pytest.raises(hmoe.HmoeError, match="scratch"):
        hmoe.moe_dispatch_noalloc(ids, K, out=out)
    assert bool((out["counts"] == -7).all())
