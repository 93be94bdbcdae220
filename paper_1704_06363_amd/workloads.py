"""Seeded synthetic inputs for the hard mixture-of-experts hot path.

This module only draws inputs; it holds none of the method's arithmetic (no distances, no
argmin, no routing, no layers).  Both the HIP path (through the tests and the bench) and the
CPU oracle (through the tests) consume what it returns.

The paper's own data (YFCC100M / Instagram images pushed through a trained CNN, Section 4)
is not available, so every workload is synthetic with the shapes of the paper's setting:
gater features from Gaussian mixtures, rectified-Gaussian features for routing, MLP experts
with N(0, 1/fan_in) weights, and multilabel targets whose tags follow a Zipf law.

Generation runs on the device given (``torch.Generator`` seeded per call), so large
workloads never pass through host memory; the CPU and GPU generators give different streams
for the same seed, and each test reads its oracle inputs back from the tensors it made.

Returned tensors live on ``device``.  Real-valued tensors are float32 ("f32") or bfloat16
("bf16"); index tensors are int32.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def torch_dtype(name: str) -> torch.dtype:
    return _DT[name]


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


# ---------------------------------------------------------------- feature matrices

def gmm_means(n_comp: int, d: int, seed: int, device="cpu", std: float = 2.0) -> torch.Tensor:
    """Component means ~ N(0, std^2 I), float32."""
    g = _gen(device, seed)
    return torch.randn(n_comp, d, generator=g, device=device, dtype=torch.float32) * std


def gmm_features(n: int, d: int, n_comp: int, seed: int, dtype: str = "f32", device="cpu",
                 dirichlet_alpha: float | None = None, means: torch.Tensor | None = None,
                 chunk: int = 1 << 20) -> torch.Tensor:
    """n rows from a mixture of `n_comp` isotropic unit-variance Gaussians whose means are
    N(0, 4I); component weights uniform, or Dirichlet(alpha) when given."""
    if means is None:
        means = gmm_means(n_comp, d, seed + 1, device)
    g = _gen(device, seed)
    if dirichlet_alpha is not None:
        rs = np.random.default_rng(seed + 2)
        w = torch.tensor(rs.dirichlet([dirichlet_alpha] * n_comp), dtype=torch.float64)
    else:
        w = torch.full((n_comp,), 1.0 / n_comp, dtype=torch.float64)
    out = torch.empty(n, d, dtype=_DT[dtype], device=device)
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        comp = torch.multinomial(w.to(device), m, replacement=True, generator=g)
        x = means.index_select(0, comp)
        x.add_(torch.randn(m, d, generator=g, device=device, dtype=torch.float32))
        out[s:s + m] = x.to(_DT[dtype])
    return out


def rectified_gaussian(n: int, d: int, seed: int, dtype: str = "bf16", device="cpu") -> torch.Tensor:
    """x = max(0, g), g ~ N(0, I): non-negative features like a ReLU trunk's last layer."""
    g = _gen(device, seed)
    x = torch.randn(n, d, generator=g, device=device, dtype=torch.float32).clamp_min_(0.0)
    return x.to(_DT[dtype])


def spread_centroids(K: int, d: int, seed: int, dtype: str = "bf16", device="cpu") -> torch.Tensor:
    """K centres placed on the sphere where rectified-Gaussian rows concentrate: mu*1 + rho*u/|u|
    with mu = E[max(0,g)] = 1/sqrt(2 pi) and rho = sqrt(d * Var[max(0,g)]).  Random rectified
    rows as centres would give badly unbalanced buckets; these give roughly n/K rows each."""
    g = _gen(device, seed)
    mu = 1.0 / math.sqrt(2.0 * math.pi)
    rho = math.sqrt(d * (0.5 - mu * mu))
    u = torch.randn(K, d, generator=g, device=device, dtype=torch.float32)
    c = mu + rho * u / u.norm(dim=1, keepdim=True)
    return c.to(_DT[dtype])


# ---------------------------------------------------------------- labels

def zipf_labels(n: int, V: int, max_tags: int, seed: int, s: float = 1.1, min_tags: int = 1):
    """Multilabel targets as CSR (row_ptr[n+1], tag[nnz], int32 numpy).  Each row has
    Uniform{min_tags..max_tags} distinct tags; tags are drawn from a Zipf(s) law truncated to
    ranks 1..V (tag id = rank - 1), redrawing duplicates."""
    rs = np.random.default_rng(seed)
    max_tags = min(max_tags, V)
    min_tags = min(min_tags, max_tags)
    cnt = rs.integers(min_tags, max_tags + 1, size=n)
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    tags = [None] * n
    m = 4 * max_tags
    cand = np.minimum(np.searchsorted(cdf, rs.random((n, m)), side="right"), V - 1)
    for i in range(n):
        row = cand[i]
        _, first = np.unique(row, return_index=True)
        first.sort()
        picked = row[first][: cnt[i]]
        while picked.shape[0] < cnt[i]:
            extra = np.minimum(np.searchsorted(cdf, rs.random(m), side="right"), V - 1)
            allv = np.concatenate([picked, extra])
            _, first = np.unique(allv, return_index=True)
            first.sort()
            picked = allv[first][: cnt[i]]
        tags[i] = picked
    row_ptr = np.zeros(n + 1, np.int32)
    row_ptr[1:] = np.cumsum(cnt)
    tag = np.concatenate(tags).astype(np.int32) if n > 0 else np.zeros(0, np.int32)
    return row_ptr, tag


# ---------------------------------------------------------------- experts and decoder

def moe_params(K: int, d: int, h: int, o: int, V: int, seed: int, dtype: str = "bf16",
               device="cpu", bias: bool = False, bias_scale: float = 0.1,
               per_expert_decoders: bool = False) -> dict:
    """Expert MLPs (Linear d->h, ReLU, Linear h->o; [out][in] layout) and the decoder
    (Linear o->V): one shared D [V, o], bD [V], or with per_expert_decoders one per expert,
    D [K, V, o], bD [K, V].  Weights ~ N(0, 1/fan_in).  Biases are zero unless `bias` is set,
    then N(0, bias_scale^2) (used to exercise the bias paths)."""
    g = _gen(device, seed)
    dt = _DT[dtype]

    def w(shape, fan_in):
        return (torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
                / math.sqrt(fan_in)).to(dt)

    def b(shape):
        if bias:
            return (torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
                    * bias_scale).to(dt)
        return torch.zeros(*shape, device=device, dtype=dt)

    dec = (K,) if per_expert_decoders else ()
    return {"W1": w((K, h, d), d), "b1": b((K, h)), "W2": w((K, o, h), h), "b2": b((K, o)),
            "D": w(dec + (V, o), o), "bD": b(dec + (V,))}


def q_draws(row_ptr, tag, S: int, seed: int):
    """The S draws behind q@m (Section 4.4, Eq. 5): each picks a tag uniformly among the tags
    that label at least one sample, then a sample uniformly among the samples it labels.
    Returns (q_sample, q_tag) int32 arrays."""
    row_ptr = np.asarray(row_ptr, dtype=np.int64)
    tag = np.asarray(tag, dtype=np.int64)
    n = row_ptr.shape[0] - 1
    owner = np.repeat(np.arange(n), np.diff(row_ptr))
    order = np.argsort(tag, kind="stable")
    tags_sorted, owners = tag[order], owner[order]
    present, first, count = np.unique(tags_sorted, return_index=True, return_counts=True)
    rs = np.random.default_rng(seed)
    pick = rs.integers(0, present.shape[0], S)
    within = (rs.random(S) * count[pick]).astype(np.int64)
    return (owners[first[pick] + within].astype(np.int32), present[pick].astype(np.int32))


def zipf_bucket_ids(n: int, K: int, seed: int, s: float = 1.3,
                    forced_small=(0, 0, 1, 1, 2, 2, 3, 3)) -> np.ndarray:
    """Expert ids with bucket sizes following Zipf(s) over K ranks: size_r = round(n r^-s / H),
    ranks mapped to experts by a seeded permutation, the len(forced_small) smallest ranks
    forced to the listed sizes (so some experts get 0-3 rows), the surplus or deficit given to
    rank 1, and the ids laid out in a seeded random order.  int32 numpy."""
    rs = np.random.default_rng(seed)
    r = np.arange(1, K + 1, dtype=np.float64)
    w = r ** (-s)
    size = np.rint(n * w / w.sum()).astype(np.int64)
    nf = min(len(forced_small), K - 1)
    if nf > 0:
        size[K - nf:] = np.array(sorted(forced_small[:nf], reverse=True), np.int64)
    size[0] += n - size.sum()
    if size[0] < 0:
        raise ValueError("batch too small for the forced bucket sizes")
    expert_of_rank = rs.permutation(K)
    ids = np.repeat(expert_of_rank, size).astype(np.int32)
    rs.shuffle(ids)
    return ids


def uniforms(k: int, seed: int) -> np.ndarray:
    """k uniform draws in [0, 1) (float64) for the k-means++ seeding."""
    return np.random.default_rng(seed).random(k)


# ---------------------------------------------------------------- the five workloads

@dataclass
class Config:
    name: str
    n: int
    d: int
    dtype: str
    K: int
    h: int = 0
    o: int = 0
    V: int = 0
    max_tags: int = 0
    n_iter: int = 0
    extra: dict = field(default_factory=dict)


CONFIGS = {
    # Tiny: gater fit + routed step, everything fp32.
    "tiny": Config("tiny", n=4096, d=64, dtype="f32", K=8, h=128, o=64, V=1000, max_tags=5,
                   n_iter=10, extra={"n_comp": 16}),
    # Gater fit: 2^20 fp32 rows, d=512, 256-component Dirichlet(0.5) mixture, K=64, 20 Lloyd
    # iterations with farthest-point reseeding.
    "gater_fit": Config("gater_fit", n=1 << 20, d=512, dtype="f32", K=64, n_iter=20,
                        extra={"n_comp": 256, "alpha": 0.5}),
    # Balanced routed training step.
    "balanced": Config("balanced", n=65536, d=2048, dtype="bf16", K=16, h=4096, o=1024,
                       V=50000, max_tags=8),
    # Skewed routing: Zipf(1.3) bucket sizes with some tiny / empty experts.
    "skewed": Config("skewed", n=32768, d=2048, dtype="bf16", K=128, h=2048, o=1024,
                     V=100000, max_tags=8, extra={"zipf_s": 1.3}),
    # Large gater assignment: 2^24 bf16 rows in 2^20-row chunks, K=1024.
    "large_assign": Config("large_assign", n=1 << 24, d=2048, dtype="bf16", K=1024,
                           extra={"n_comp": 4096, "chunk": 1 << 20}),
}


def tiny_inputs(device="cpu", seed: int = 0, n: int | None = None, bias: bool = False) -> dict:
    c = CONFIGS["tiny"]
    n = c.n if n is None else n
    X = gmm_features(n, c.d, c.extra["n_comp"], seed, "f32", device)
    row_ptr, tag = zipf_labels(n, c.V, c.max_tags, seed + 10)
    p = moe_params(c.K, c.d, c.h, c.o, c.V, seed + 20, "f32", device, bias=bias)
    return {"X": X, "u": uniforms(c.K, seed + 30), "row_ptr": row_ptr, "tag": tag, "params": p,
            "cfg": c}


def balanced_inputs(device="cpu", seed: int = 0, n: int | None = None, bias: bool = False,
                    d=None, h=None, o=None, V=None, K=None) -> dict:
    c = CONFIGS["balanced"]
    n = c.n if n is None else n
    d = d or c.d; h = h or c.h; o = o or c.o; V = V or c.V; K = K or c.K
    X = rectified_gaussian(n, d, seed, "bf16", device)
    C = spread_centroids(K, d, seed + 1, "bf16", device)
    row_ptr, tag = zipf_labels(n, V, c.max_tags, seed + 10)
    p = moe_params(K, d, h, o, V, seed + 20, "bf16", device, bias=bias)
    return {"X": X, "C": C, "row_ptr": row_ptr, "tag": tag, "params": p, "cfg": c,
            "shape": dict(n=n, d=d, h=h, o=o, V=V, K=K)}


def skewed_inputs(device="cpu", seed: int = 0, n: int | None = None, bias: bool = False,
                  d=None, h=None, o=None, V=None, K=None) -> dict:
    c = CONFIGS["skewed"]
    n = c.n if n is None else n
    d = d or c.d; h = h or c.h; o = o or c.o; V = V or c.V; K = K or c.K
    X = rectified_gaussian(n, d, seed, "bf16", device)
    ids = zipf_bucket_ids(n, K, seed + 2, c.extra["zipf_s"])
    row_ptr, tag = zipf_labels(n, V, c.max_tags, seed + 10)
    p = moe_params(K, d, h, o, V, seed + 20, "bf16", device, bias=bias)
    return {"X": X, "ids": ids, "row_ptr": row_ptr, "tag": tag, "params": p, "cfg": c,
            "shape": dict(n=n, d=d, h=h, o=o, V=V, K=K)}
