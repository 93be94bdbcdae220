"""Seeded input generators: reproducible, with the stated shapes and structure."""
import numpy as np
import torch

from paper_1704_06363_amd import workloads as W


def test_zipf_labels_shape_and_distinct():
    rp, tag = W.zipf_labels(2000, 300, 8, seed=4)
    cnt = np.diff(rp)
    assert cnt.min() >= 1 and cnt.max() <= 8
    assert tag.min() >= 0 and tag.max() < 300
    for i in range(2000):
        t = tag[rp[i]:rp[i + 1]]
        assert len(set(t.tolist())) == len(t)
    # Zipf: rank 1 (tag 0) is the most frequent tag
    assert np.bincount(tag, minlength=300).argmax() == 0
    rp2, tag2 = W.zipf_labels(2000, 300, 8, seed=4)
    assert np.array_equal(rp, rp2) and np.array_equal(tag, tag2)


def test_skewed_bucket_sizes():
    ids = W.zipf_bucket_ids(32768, 128, seed=2)
    sizes = np.sort(np.bincount(ids, minlength=128))
    assert sizes.sum() == 32768
    assert sizes[:8].tolist() == [0, 0, 1, 1, 2, 2, 3, 3]
    assert sizes[-1] > 0.25 * 32768  # the largest bucket holds about 31% of the batch
    assert np.array_equal(ids, W.zipf_bucket_ids(32768, 128, seed=2))


def test_generators_reproducible_and_typed():
    a = W.gmm_features(1000, 16, 4, seed=1, dtype="bf16")
    b = W.gmm_features(1000, 16, 4, seed=1, dtype="bf16")
    assert a.dtype == torch.bfloat16 and torch.equal(a, b)
    x = W.rectified_gaussian(500, 64, seed=3)
    assert x.dtype == torch.bfloat16 and float(x.float().min()) >= 0.0
    c = W.spread_centroids(16, 2048, seed=1)
    norms = (c.float() - 1.0 / np.sqrt(2 * np.pi)).norm(dim=1)
    assert torch.allclose(norms, torch.full_like(norms, 26.42), rtol=0.01)
    p = W.moe_params(3, 8, 16, 4, 10, seed=0, dtype="f32")
    assert p["W1"].shape == (3, 16, 8) and p["W2"].shape == (3, 4, 16) and p["D"].shape == (10, 4)
    assert float(p["b1"].abs().sum()) == 0.0
