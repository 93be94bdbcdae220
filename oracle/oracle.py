"""numpy front end of the fp64 CPU oracle (``hmoe_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the bench's CPU-baseline leg may
import this module; the product library never does.  It shares no code with the HIP path.

Every function takes and returns numpy arrays.  Real inputs are converted to float64 exactly
(fp32 and bf16 values are representable in fp64), so the oracle sees the same numbers as the
device.  ``store`` names the precision in which the device stores a tensor that a later step
reads back: "f64" (no rounding), "f32" or "bf16" (round to nearest even).

Each function names the part of the paper (Gross, Ranzato & Szlam, arXiv 1704.06363) it
follows; the C file holds the arithmetic, except for the PCA, whose eigensolve is LAPACK's
(numpy.linalg.eigh) applied to the covariance written out in numpy.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hmoe_oracle.c")
_LIB = os.path.join(_HERE, "libhmoe_oracle.so")
_lib = None

_STORE = {"f64": 0, "f32": 1, "bf16": 2}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math) into oracle/libhmoe_oracle.so."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = ctypes.CDLL(_LIB)
    return _lib


def _f64(x):
    return np.ascontiguousarray(x, dtype=np.float64)


def _i32(x):
    return np.ascontiguousarray(x, dtype=np.int32)


def _p(x):
    if x is None:
        return None
    return x.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


def round_store(x, store: str) -> np.ndarray:
    """Round to the storage precision (nearest even)."""
    y = _f64(x).copy()
    _load().hmoe_orc_round(ctypes.c_int64(y.size), _p(y), ctypes.c_int(_STORE[store]))
    return y


def assign(X, C):
    """Eq. 2 (Section 2): nearest centroid by direct squared differences, lowest index on
    ties.  Returns (a int32[n], d1 f64[n], d2 f64[n]) with d2 the runner-up distance."""
    X = _f64(X)
    C = _f64(C)
    n, d = X.shape
    K = C.shape[0]
    a = np.empty(n, np.int32)
    d1 = np.empty(n, np.float64)
    d2 = np.empty(n, np.float64)
    rc = _load().hmoe_orc_assign(ctypes.c_int64(n), ctypes.c_int32(d), ctypes.c_int32(K),
                                 _p(X), _p(C), _p(a), _p(d1), _p(d2))
    _check(rc, "assign")
    return a, d1, d2


def near_tie(d1, d2, rel: float = 1e-5) -> np.ndarray:
    """Rows whose runner-up distance is within `rel` (relative to d1) of the minimum; for
    d1 == 0 only an exact second zero counts."""
    d1 = np.asarray(d1, np.float64)
    d2 = np.asarray(d2, np.float64)
    return (d2 - d1) <= rel * d1


def kmeanspp(X, K: int, u):
    """k-means++ seeding with caller-supplied uniforms u[0..K-1] (the paper leaves the
    initialisation of its K-means step, Section 2, open).  Returns the chosen row ids."""
    X = _f64(X)
    u = _f64(u)
    n, d = X.shape
    idx = np.empty(K, np.int32)
    rc = _load().hmoe_orc_kmeanspp(ctypes.c_int64(n), ctypes.c_int32(d), ctypes.c_int32(K),
                                   _p(X), _p(u), _p(idx))
    _check(rc, "kmeanspp")
    return idx


def update(X, a, d1, C_prev, reseed: bool = True):
    """One Lloyd update (Section 2's K-means) with farthest-point reseeding of empty
    clusters.  Returns (C f64 unrounded, counts int64, a int32 after reseeding)."""
    X = _f64(X)
    a = _i32(a).copy()
    C = _f64(C_prev).copy()
    n, d = X.shape
    K = C.shape[0]
    d1 = _f64(d1) if d1 is not None else np.zeros(n)
    counts = np.empty(K, np.int64)
    rc = _load().hmoe_orc_update(ctypes.c_int64(n), ctypes.c_int32(d), ctypes.c_int32(K),
                                 _p(X), _p(a), _p(d1), ctypes.c_int(1 if reseed else 0),
                                 _p(C), _p(counts))
    _check(rc, "update")
    return C, counts, a


def fit(X, K: int, n_iter: int, u=None, C0=None, data_store: str = "f32", reseed: bool = True):
    """Lloyd's K-means for a fixed number of iterations (Section 2).  Returns a dict with
    C (fp32-rounded, as float64), a (final assignment), J (n_iter+1 objectives), init_idx
    (k-means++ picks, or None) and counts."""
    X = _f64(X)
    n, d = X.shape
    if (u is None) == (C0 is None):
        raise ValueError("give exactly one of u (k-means++) or C0")
    C = np.zeros((K, d)) if C0 is None else _f64(C0).copy()
    a = np.empty(n, np.int32)
    J = np.empty(n_iter + 1, np.float64)
    idx = np.empty(K, np.int32)
    counts = np.empty(K, np.int64)
    uu = _f64(u) if u is not None else None
    rc = _load().hmoe_orc_fit(ctypes.c_int64(n), ctypes.c_int32(d), ctypes.c_int32(K), _p(X),
                              ctypes.c_int32(n_iter), _p(uu), ctypes.c_int(_STORE[data_store]),
                              ctypes.c_int(1 if reseed else 0), _p(C), _p(a), _p(J), _p(idx),
                              _p(counts))
    _check(rc, "fit")
    return {"C": C, "a": a, "J": J, "init_idx": idx if u is not None else None,
            "counts": counts}


def dispatch(e, K: int):
    """Hard partition of the batch by expert (Section 2): stable grouping.  Returns
    (counts, offsets[K+1], perm slot->sample, inv sample->slot), all int32."""
    e = _i32(e)
    n = e.shape[0]
    counts = np.empty(K, np.int32)
    offsets = np.empty(K + 1, np.int32)
    perm = np.empty(n, np.int32)
    inv = np.empty(n, np.int32)
    rc = _load().hmoe_orc_dispatch(ctypes.c_int64(n), ctypes.c_int32(K), _p(e), _p(counts),
                                   _p(offsets), _p(perm), _p(inv))
    _check(rc, "dispatch")
    return counts, offsets, perm, inv


def _ndec(D, K):
    """Decoders in D: [V][o] is one shared decoder, [K][V][o] one per expert."""
    D = np.asarray(D)
    if D.ndim == 2:
        return 1, D.shape[0]
    assert D.ndim == 3 and D.shape[0] == K, D.shape
    return K, D.shape[1]


def moe_forward(X, a, W1, b1, W2, b2, D, bD, row_ptr, tag, store: str = "f64",
                want_probs: bool = False, want_logits: bool = False):
    """Hard MoE forward with the multilabel softmax loss (Section 2; Section 4.1, Eq. 3).
    D [V][o] (bD [V]) is the shared decoder; D [K][V][o] (bD [K][V]) gives every expert its
    own, and each sample is decoded by its expert's.  Per-sample outputs in sample order."""
    X = _f64(X)
    n, d = X.shape
    K, h, _ = W1.shape
    o = W2.shape[1]
    ndec, V = _ndec(D, K)
    W1 = _f64(W1); W2 = _f64(W2); D = _f64(D)
    b1 = _f64(b1) if b1 is not None else None
    b2 = _f64(b2) if b2 is not None else None
    bD = _f64(bD) if bD is not None else None
    a = _i32(a); row_ptr = _i32(row_ptr); tag = _i32(tag)
    H1 = np.empty((n, h)); H = np.empty((n, o)); lse = np.empty(n); loss = np.empty(n)
    lm = np.zeros(1)
    probs = np.empty((n, V)) if want_probs else None
    logits = np.empty((n, V)) if want_logits else None
    rc = _load().hmoe_orc_moe_forward(
        ctypes.c_int64(n), ctypes.c_int32(d), ctypes.c_int32(h), ctypes.c_int32(o),
        ctypes.c_int32(V), ctypes.c_int32(K), ctypes.c_int32(ndec), _p(X), _p(a), _p(W1), _p(b1), _p(W2), _p(b2),
        _p(D), _p(bD), _p(row_ptr), _p(tag), ctypes.c_int(_STORE[store]), _p(H1), _p(H),
        _p(lse), _p(loss), _p(lm), _p(probs), _p(logits))
    _check(rc, "moe_forward")
    out = {"H1": H1, "H": H, "lse": lse, "loss": loss, "loss_mean": float(lm[0])}
    if want_probs:
        out["probs"] = probs
    if want_logits:
        out["logits"] = logits
    return out


def moe_backward(X, a, W1, W2, D, bD, row_ptr, tag, H1, H, lse, scale=None,
                 store: str = "f64", want_dX: bool = True, internal_store: str = "f64",
                 logit_round: bool = False, magnitude: bool = False):
    """Gradients of the mean loss w.r.t. every expert and decoder parameter (and X) given the
    saved activations (Section 2; Section 4.1, Eq. 3; the gater gets none, Section 2.2).
    Decoders as in moe_forward; dD and dbD have D's and bD's shapes.  `store` rounds dX, the
    activation gradient handed to the caller; g, dh and dz stay fp64 (the plain gradient).
    Diagnostics only: internal_store rounds g, dh and dz as a device storing them would, and
    logit_round rounds the logits (in internal_store precision) before the softmax.
    magnitude: the same sums over absolute values (|g| = |p - y| scale, then |a||b| for every
    product, nothing rounded): per output the scale M of the first-order rounding-error bound of
    the computation (an evaluation that rounds its operands with unit roundoff u stays within
    (number of roundings) u M of the exact gradient)."""
    X = _f64(X)
    n, d = X.shape
    K, h, _ = W1.shape
    o = W2.shape[1]
    ndec, V = _ndec(D, K)
    W1 = _f64(W1); W2 = _f64(W2); D = _f64(D)
    bD = _f64(bD) if bD is not None else None
    a = _i32(a); row_ptr = _i32(row_ptr); tag = _i32(tag)
    H1 = _f64(H1); H = _f64(H); lse = _f64(lse)
    if scale is None:
        scale = 1.0 / max(n, 1)
    dW1 = np.empty((K, h, d)); db1 = np.empty((K, h)); dW2 = np.empty((K, o, h))
    db2 = np.empty((K, o))
    per_expert = np.asarray(D).ndim == 3
    dD = np.empty((K, V, o)) if per_expert else np.empty((V, o))
    dbD = np.empty((K, V)) if per_expert else np.empty(V)
    dX = np.empty((n, d)) if want_dX else None
    rc = _load().hmoe_orc_moe_backward(
        ctypes.c_int64(n), ctypes.c_int32(d), ctypes.c_int32(h), ctypes.c_int32(o),
        ctypes.c_int32(V), ctypes.c_int32(K), ctypes.c_int32(ndec), _p(X), _p(a), _p(W1), _p(W2), _p(D), _p(bD),
        _p(row_ptr), _p(tag), _p(H1), _p(H), _p(lse), ctypes.c_double(scale),
        ctypes.c_int(_STORE[store]), ctypes.c_int(_STORE[internal_store]),
        ctypes.c_int(1 if logit_round else 0), ctypes.c_int(1 if magnitude else 0), _p(dW1), _p(db1),
        _p(dW2), _p(db2), _p(dD), _p(dbD), _p(dX))
    _check(rc, "moe_backward")
    return {"dW1": dW1, "db1": db1, "dW2": dW2, "db2": db2, "dD": dD, "dbD": dbD, "dX": dX}


def topm(L, m: int) -> np.ndarray:
    """t_m (Section 4.4): indices of the m largest entries of each row, in decreasing order,
    equal values by increasing index.  L is taken as given (pass the stored logits)."""
    L = _f64(L)
    n, V = L.shape
    idx = np.empty((n, m), dtype=np.int32)
    _check(_load().hmoe_orc_topm(ctypes.c_int64(n), ctypes.c_int32(V), ctypes.c_int32(m), _p(L),
                                 _p(idx)), "topm")
    return idx


def topm_hits(idx, row_ptr, tag, q_sample, q_tag):
    """Counts behind Eq. 4 (p@m) and Eq. 5 (q@m), Section 4.4, for every m' = 1..m of the
    top-m lists idx [n, m]: p_hits[m'-1] = sum_i |t_m'(i) & P_i| and q_hits[m'-1] = number of
    the given (sample, tag) draws whose tag is in the sample's t_m'.  p@m' = p_hits / nnz,
    q@m' = q_hits / S."""
    idx = _i32(idx)
    n, m = idx.shape
    row_ptr = _i32(row_ptr); tag = _i32(tag)
    q_sample = _i32(q_sample); q_tag = _i32(q_tag)
    S = q_sample.shape[0]
    p_hits = np.zeros(m, dtype=np.int64); q_hits = np.zeros(m, dtype=np.int64)
    _check(_load().hmoe_orc_topm_hits(ctypes.c_int64(n), ctypes.c_int32(m), _p(idx), _p(row_ptr),
                                      _p(tag), ctypes.c_int64(S), _p(q_sample), _p(q_tag),
                                      _p(p_hits), _p(q_hits)), "topm_hits")
    return p_hits, q_hits


def sgd_step(w, g, lr: float, weight_decay: float = 0.0, momentum: float = 0.0, v=None):
    """One SGD step (Section 4.2: weight decay; momentum for the trunk, none for the experts).
    Returns the new weights (and the new momentum buffer when momentum > 0); inputs untouched."""
    w = _f64(w).copy()
    shape = w.shape
    w = w.reshape(-1)
    g = _f64(g).reshape(-1)
    vv = None
    if momentum > 0.0:
        vv = (np.zeros_like(w) if v is None else _f64(v).reshape(-1).copy())
    _check(_load().hmoe_orc_sgd_step(ctypes.c_int64(w.shape[0]), _p(w), _p(g), _p(vv),
                                     ctypes.c_double(lr), ctypes.c_double(weight_decay),
                                     ctypes.c_double(momentum)), "sgd_step")
    return (w.reshape(shape), vv.reshape(shape)) if momentum > 0.0 else w.reshape(shape)


def pca(X, r: int):
    """Section 4.2's projection before the K-means: the sample mean and the r leading
    eigenpairs of the sample covariance C = (1/(n-1)) sum_i (x_i - mean)(x_i - mean)^T, by
    LAPACK's symmetric eigensolver.  Components [r, d] in decreasing eigenvalue order, each
    row's sign fixed so that its largest-magnitude entry is positive (lowest index on ties).
    Returns (mean [d], components [r, d], eigenvalues [r])."""
    X = _f64(X)
    n = X.shape[0]
    mean = X.sum(axis=0) / n
    Xc = X - mean
    C = (Xc.T @ Xc) / (n - 1)
    w, U = np.linalg.eigh(C)
    order = np.argsort(-w, kind="stable")[:r]
    comps = U[:, order].T.copy()
    for j in range(r):
        k = int(np.argmax(np.abs(comps[j])))
        if comps[j, k] < 0:
            comps[j] = -comps[j]
    return mean, comps, w[order]


def pca_project(X, mean, comps):
    """The projected features (x_i - mean) U^T that the K-means runs on (Section 4.2)."""
    return (_f64(X) - _f64(mean)) @ _f64(comps).T
