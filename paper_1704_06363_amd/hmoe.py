"""Python binding of libhmoe.so (include/hmoe.h): argument marshalling only.

Tensors are torch tensors on the GPU; every function hands their device pointers, the
current HIP stream and a workspace to the C ABI and returns the output tensors.  No step of
the hot path runs here: if the library is not built, or a call fails, an exception is
raised -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhmoe.so")

F32, BF16 = 0, 1
UPDATE_FULL, UPDATE_ACCUMULATE, UPDATE_FINALIZE = 0, 1, 2
_DT = {torch.float32: F32, torch.bfloat16: BF16}

SYMBOLS = (
    "hmoe_last_error", "hmoe_version",
    "hmoe_kmeans_assign_workspace", "hmoe_kmeans_assign",
    "hmoe_kmeans_fit_workspace", "hmoe_kmeans_fit",
    "hmoe_kmeans_update_workspace", "hmoe_kmeans_update",
    "hmoe_moe_dispatch_workspace", "hmoe_moe_dispatch", "hmoe_moe_dispatch_noalloc", "hmoe_permute_rows",
    "hmoe_moe_workspace", "hmoe_moe_forward", "hmoe_moe_backward",
    "hmoe_pca_workspace", "hmoe_pca_fit", "hmoe_pca_project",
    "hmoe_sgd_step", "hmoe_topm", "hmoe_topm_hits",
    "hmoe_timer_enable", "hmoe_timer_report",
)


class HmoeError(RuntimeError):
    pass


class MoeParams(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int32), ("d_in", ctypes.c_int32), ("d_hid", ctypes.c_int32),
                ("d_out", ctypes.c_int32), ("vocab", ctypes.c_int32), ("dt", ctypes.c_int),
                ("W1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("W2", ctypes.c_void_p),
                ("b2", ctypes.c_void_p), ("D", ctypes.c_void_p), ("bD", ctypes.c_void_p),
                ("decoders", ctypes.c_int32)]


class Labels(ctypes.Structure):
    _fields_ = [("row_ptr", ctypes.c_void_p), ("tag", ctypes.c_void_p)]


_lib = None

_c = ctypes
_I64, _I32, _SZ, _P, _D = _c.c_int64, _c.c_int32, _c.c_size_t, _c.c_void_p, _c.c_double


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise HmoeError("libhmoe.so is not built: run `python -m paper_1704_06363_amd.build` "
                            "(or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        L.hmoe_last_error.restype = _c.c_char_p
        L.hmoe_version.restype = _c.c_int
        for name in ("hmoe_kmeans_assign_workspace", "hmoe_kmeans_fit_workspace",
                     "hmoe_kmeans_update_workspace"):
            getattr(L, name).restype = _SZ
            getattr(L, name).argtypes = [_I64, _I32, _I32, _c.c_int]
        L.hmoe_moe_dispatch_workspace.restype = _SZ
        L.hmoe_moe_dispatch_workspace.argtypes = [_I64, _I32]
        L.hmoe_moe_workspace.restype = _SZ
        L.hmoe_moe_workspace.argtypes = [_c.POINTER(MoeParams), _I64]
        L.hmoe_kmeans_assign.argtypes = [_P, _c.c_int, _I64, _I32, _P, _I32, _P, _P, _P, _SZ, _P]
        L.hmoe_kmeans_fit.argtypes = [_P, _c.c_int, _I64, _I32, _I32, _I32, _P, _I32, _P, _P, _P,
                                      _P, _P, _P, _P, _SZ, _P]
        L.hmoe_kmeans_update.argtypes = [_P, _c.c_int, _I64, _I32, _I32, _P, _P, _P, _P, _P,
                                         _I32, _I32, _P, _SZ, _P]
        L.hmoe_moe_dispatch.argtypes = [_P, _I64, _I32, _P, _P, _P, _P, _P, _P, _c.c_int, _I32,
                                        _P, _SZ, _P]
        L.hmoe_moe_dispatch_noalloc.argtypes = [_P, _I64, _I32, _P, _P, _P, _P, _P, _P, _c.c_int, _I32, _P]
        L.hmoe_permute_rows.argtypes = [_P, _P, _P, _I64, _I32, _c.c_int, _P]
        L.hmoe_moe_forward.argtypes = [_c.POINTER(MoeParams), _I64, _P, _P, _P,
                                       _c.POINTER(Labels), _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]
        L.hmoe_moe_backward.argtypes = [_c.POINTER(MoeParams), _I64, _P, _P, _P, _P,
                                        _c.POINTER(Labels), _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                        _P, _P, _P, _P, _SZ, _P]
        L.hmoe_pca_workspace.restype = _SZ
        L.hmoe_pca_workspace.argtypes = [_I64, _I32, _I32, _c.c_int]
        L.hmoe_pca_fit.argtypes = [_P, _c.c_int, _I64, _I32, _I32, _I32, _c.c_uint64, _P, _P, _P, _P, _SZ, _P]
        L.hmoe_pca_project.argtypes = [_P, _c.c_int, _I64, _I32, _P, _P, _I32, _P, _P, _SZ, _P]
        L.hmoe_sgd_step.argtypes = [_P, _P, _P, _P, _c.c_int, _I64, _c.c_float, _c.c_float, _c.c_float, _P]
        L.hmoe_topm.argtypes = [_P, _P, _c.c_int, _I64, _I32, _I32, _P, _P, _P]
        L.hmoe_topm_hits.argtypes = [_P, _I64, _I32, _c.POINTER(Labels), _P, _P, _I64, _P, _P]
        L.hmoe_timer_enable.argtypes = [_c.c_int]
        L.hmoe_timer_enable.restype = _c.c_int
        L.hmoe_timer_report.argtypes = [_c.c_char_p, _SZ]
        L.hmoe_timer_report.restype = _I64
        for name in ("hmoe_kmeans_assign", "hmoe_kmeans_fit", "hmoe_kmeans_update",
                     "hmoe_moe_dispatch", "hmoe_moe_dispatch_noalloc", "hmoe_permute_rows", "hmoe_moe_forward",
                     "hmoe_moe_backward", "hmoe_pca_fit", "hmoe_pca_project", "hmoe_sgd_step",
                     "hmoe_topm", "hmoe_topm_hits"):
            getattr(L, name).restype = _c.c_int
        _lib = L
    return _lib


def version() -> int:
    return lib().hmoe_version()


def last_error() -> str:
    return lib().hmoe_last_error().decode()


def timer_enable(on: bool = True):
    """Start (or stop) recording HIP events around every kernel the library launches."""
    _chk(lib().hmoe_timer_enable(1 if on else 0), "timer_enable")


def timer_report() -> dict:
    """{kernel label: (launches, total_ms)} for the launches recorded since timer_enable."""
    n = lib().hmoe_timer_report(None, 0)
    if n < 0:
        raise HmoeError(f"timer_report failed ({n}): {last_error()}")
    buf = ctypes.create_string_buffer(int(n) + 1)
    lib().hmoe_timer_report(buf, int(n) + 1)
    out = {}
    for line in buf.value.decode().splitlines():
        label, cnt, ms = line.split("\t")
        out[label] = (int(cnt), float(ms))
    return out


def _out(o, key, make):
    """o[key] when the caller passed it, else a new tensor from make() (only then allocated)."""
    return o[key] if key in o else make()


def _chk(rc: int, what: str):
    if rc != 0:
        raise HmoeError(f"{what} failed ({rc}): {last_error()}")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise HmoeError("tensor is not on the GPU")
    if not t.is_contiguous():
        raise HmoeError("tensor is not contiguous")
    return t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _dt(t):
    try:
        return _DT[t.dtype]
    except KeyError:
        raise HmoeError(f"unsupported dtype {t.dtype}") from None


def _expect(t, shape, dtype, what):
    """t (if given) must have this shape (None entries match any size) and dtype: a tensor of
    another dtype or size would make the library read or write past its bytes."""
    if t is None:
        return
    if dtype is not None and t.dtype != dtype:
        raise HmoeError(f"{what}: dtype {t.dtype}, {dtype} expected")
    if len(t.shape) != len(shape) or any(e is not None and a != e for a, e in zip(t.shape, shape)):
        raise HmoeError(f"{what}: shape {tuple(t.shape)}, {tuple(shape)} expected")


def _workspace(nbytes, ws, device):
    if nbytes == 0:
        return None, 0
    if ws is not None:
        if ws.numel() * ws.element_size() < nbytes:
            raise HmoeError(f"workspace of {ws.numel() * ws.element_size()} bytes, {nbytes} needed")
        return ws, ws.numel() * ws.element_size()
    return torch.empty(nbytes, dtype=torch.uint8, device=device), nbytes


# ------------------------------------------------------------------ gater

def kmeans_assign_workspace(n, d, K, dtype) -> int:
    return lib().hmoe_kmeans_assign_workspace(n, d, K, _DT[dtype])


def kmeans_assign(X, C, assign=None, min_dist=None, want_min_dist=True, ws=None):
    """Eq. 2: nearest centroid per row (ties to the lowest index) and its squared distance."""
    n, d = X.shape
    K = C.shape[0]
    dev = X.device
    _expect(C, (K, d), X.dtype, "C")
    _expect(assign, (n,), torch.int32, "assign")
    _expect(min_dist, (n,), torch.float32, "min_dist")
    if assign is None:
        assign = torch.empty(n, dtype=torch.int32, device=dev)
    if min_dist is None and want_min_dist:
        min_dist = torch.empty(n, dtype=torch.float32, device=dev)
    w, wb = _workspace(kmeans_assign_workspace(n, d, K, X.dtype), ws, dev)
    _chk(lib().hmoe_kmeans_assign(_ptr(X), _dt(X), n, d, _ptr(C), K, _ptr(assign), _ptr(min_dist),
                                  _ptr(w), wb, _stream()), "kmeans_assign")
    return assign, min_dist


def kmeans_fit_workspace(n, d, K, dtype) -> int:
    return lib().hmoe_kmeans_fit_workspace(n, d, K, _DT[dtype])


def kmeans_fit(X, K, n_iter, init_uniforms=None, C=None, reseed=True, ws=None):
    """Lloyd's K-means for n_iter iterations, k-means++ seeded from init_uniforms (K values in
    [0,1)) or started from C.  Returns C (fp32), assign, min_dist, counts, objective,
    init_idx."""
    n, d = X.shape
    dev = X.device
    if (init_uniforms is None) == (C is None):
        raise HmoeError("give exactly one of init_uniforms or C")
    _expect(C, (K, d), torch.float32, "C (fp32 master centres)")
    Cout = torch.empty(K, d, dtype=torch.float32, device=dev) if C is None else C.clone()
    u = None
    if init_uniforms is not None:
        u = torch.as_tensor(init_uniforms, dtype=torch.float64).to(dev).contiguous()
    out = {"C": Cout,
           "assign": torch.empty(n, dtype=torch.int32, device=dev),
           "min_dist": torch.empty(n, dtype=torch.float32, device=dev),
           "counts": torch.empty(K, dtype=torch.int32, device=dev),
           "objective": torch.empty(n_iter + 1, dtype=torch.float64, device=dev),
           "init_idx": torch.empty(K, dtype=torch.int32, device=dev) if u is not None else None}
    w, wb = _workspace(kmeans_fit_workspace(n, d, K, X.dtype), ws, dev)
    _chk(lib().hmoe_kmeans_fit(_ptr(X), _dt(X), n, d, K, n_iter, _ptr(u), 1 if reseed else 0,
                               _ptr(Cout), _ptr(out["assign"]), _ptr(out["min_dist"]),
                               _ptr(out["counts"]), _ptr(out["objective"]), _ptr(out["init_idx"]),
                               _ptr(w), wb, _stream()), "kmeans_fit")
    return out


def kmeans_update_workspace(n, d, K, dtype) -> int:
    return lib().hmoe_kmeans_update_workspace(n, d, K, _DT[dtype])


def kmeans_update(X, K, assign, min_dist, sums, counts, C, mode=UPDATE_FULL, reseed=True,
                  ws=None):
    """One Lloyd centre update (modes: full / accumulate a chunk / finalize).  sums (fp64
    [K,d]), counts (int64 [K]), C (fp32 [K,d]) and assign are updated in place."""
    n, d = (X.shape if X is not None else (0, C.shape[1]))
    dev = C.device
    _expect(C, (K, d), torch.float32, "C")
    _expect(sums, (K, d), torch.float64, "sums")
    _expect(counts, (K,), torch.int64, "counts")
    if X is not None:
        _expect(assign, (n,), torch.int32, "assign")
        _expect(min_dist, (n,), torch.float32, "min_dist")
    dt = _dt(X) if X is not None else F32
    w, wb = _workspace(lib().hmoe_kmeans_update_workspace(n, d, K, dt), ws, dev)
    _chk(lib().hmoe_kmeans_update(_ptr(X), dt, n, d, K, _ptr(assign), _ptr(min_dist), _ptr(sums),
                                  _ptr(counts), _ptr(C), mode, 1 if reseed else 0, _ptr(w), wb,
                                  _stream()), "kmeans_update")


# ------------------------------------------------------------------ routing

def moe_dispatch_workspace(n, K) -> int:
    return lib().hmoe_moe_dispatch_workspace(n, K)


def _check_dispatch(expert, K, rows, o):
    n = expert.shape[0]
    _expect(expert, (n,), torch.int32, "expert")
    for k, shape in (("counts", (K,)), ("offsets", (K + 1,)), ("perm", (n,)), ("inv", (n,))):
        _expect(o.get(k), shape, torch.int32, k)
    if rows is not None:
        _expect(rows, (n, None), None, "rows")
        _expect(o.get("rows_sorted"), tuple(rows.shape), rows.dtype, "rows_sorted")


def moe_dispatch(expert, K, rows=None, out=None, ws=None):
    """Stable bucketing of the batch by expert; optionally gathers rows into expert order."""
    n = expert.shape[0]
    dev = expert.device
    o = out or {}
    _check_dispatch(expert, K, rows, o)
    counts = _out(o, "counts", lambda: torch.empty(K, dtype=torch.int32, device=dev))
    offsets = _out(o, "offsets", lambda: torch.empty(K + 1, dtype=torch.int32, device=dev))
    perm = _out(o, "perm", lambda: torch.empty(n, dtype=torch.int32, device=dev))
    inv = _out(o, "inv", lambda: torch.empty(n, dtype=torch.int32, device=dev))
    rows_sorted = None
    w = 0
    dt = F32
    if rows is not None:
        rows_sorted = _out(o, "rows_sorted", lambda: torch.empty_like(rows))
        w = rows.shape[1]
        dt = _dt(rows)
    wsb, wb = _workspace(moe_dispatch_workspace(n, K), ws, dev)
    _chk(lib().hmoe_moe_dispatch(_ptr(expert), n, K, _ptr(counts), _ptr(offsets), _ptr(perm),
                                 _ptr(inv), _ptr(rows), _ptr(rows_sorted), dt, w, _ptr(wsb), wb,
                                 _stream()), "moe_dispatch")
    return {"counts": counts, "offsets": offsets, "perm": perm, "inv": inv,
            "rows_sorted": rows_sorted}


DISPATCH_SCRATCH_BYTES = 16 << 20  # include/hmoe.h: HMOE_DISPATCH_SCRATCH_BYTES


def moe_dispatch_noalloc(expert, K, rows=None, out=None):
    """moe_dispatch without a workspace: the library's own device scratch array (for callers
    that cannot allocate; calls that overlap on one GPU race on it).  Outputs are allocated here
    unless passed in `out`."""
    n = expert.shape[0]
    dev = expert.device
    o = out or {}
    _check_dispatch(expert, K, rows, o)
    counts = _out(o, "counts", lambda: torch.empty(K, dtype=torch.int32, device=dev))
    offsets = _out(o, "offsets", lambda: torch.empty(K + 1, dtype=torch.int32, device=dev))
    perm = _out(o, "perm", lambda: torch.empty(n, dtype=torch.int32, device=dev))
    inv = _out(o, "inv", lambda: torch.empty(n, dtype=torch.int32, device=dev))
    rows_sorted = None
    w = 0
    dt = F32
    if rows is not None:
        rows_sorted = _out(o, "rows_sorted", lambda: torch.empty_like(rows))
        w = rows.shape[1]
        dt = _dt(rows)
    _chk(lib().hmoe_moe_dispatch_noalloc(_ptr(expert), n, K, _ptr(counts), _ptr(offsets), _ptr(perm), _ptr(inv),
                                         _ptr(rows), _ptr(rows_sorted), dt, w, _stream()), "moe_dispatch_noalloc")
    return {"counts": counts, "offsets": offsets, "perm": perm, "inv": inv, "rows_sorted": rows_sorted}


def permute_rows(inp, index, out=None):
    """out[r] = inp[index[r]]."""
    n = index.shape[0]
    _expect(index, (n,), torch.int32, "index")
    _expect(inp, (n, None), None, "inp")
    _expect(out, tuple(inp.shape), inp.dtype, "out")
    if out is None:
        out = torch.empty((n, inp.shape[1]), dtype=inp.dtype, device=inp.device)
    _chk(lib().hmoe_permute_rows(_ptr(inp), _ptr(out), _ptr(index), n, inp.shape[1], _dt(inp),
                                 _stream()), "permute_rows")
    return out


# ------------------------------------------------------------------ experts + decoder

class _Dims:
    """The sizes of a parameter dict, checked for consistency (shapes and one dtype)."""

    def __init__(self, p: dict):
        K, h, d = p["W1"].shape
        o = p["W2"].shape[1]
        per_expert = p["D"].dim() == 3
        if per_expert and p["D"].shape[0] != K:
            raise HmoeError(f"per-expert decoders need D [K, V, o] with K = {K}, got {tuple(p['D'].shape)}")
        V = p["D"].shape[-2]
        dec = (K,) if per_expert else ()
        for k, shape in (("W1", (K, h, d)), ("b1", (K, h)), ("W2", (K, o, h)), ("b2", (K, o)),
                         ("D", dec + (V, o)), ("bD", dec + (V,))):
            _expect(p.get(k), shape, p["W1"].dtype, k)
        self.K, self.d_in, self.d_hid, self.d_out, self.vocab = K, d, h, o, V


def make_params(p: dict) -> MoeParams:
    """p: W1 [K,h,d], b1 [K,h] or None, W2 [K,o,h], b2 [K,o] or None, and the decoder: shared,
    D [V,o] with bD [V] or None, or one per expert, D [K,V,o] with bD [K,V] or None."""
    _Dims(p)
    K, h, d = p["W1"].shape
    o = p["W2"].shape[1]
    per_expert = p["D"].dim() == 3
    if per_expert and p["D"].shape[0] != K:
        raise HmoeError(f"per-expert decoders need D [K, V, o] with K = {K}, got {tuple(p['D'].shape)}")
    V = p["D"].shape[-2]
    return MoeParams(K, d, h, o, V, _dt(p["W1"]), _ptr(p["W1"]), _ptr(p.get("b1")), _ptr(p["W2"]),
                     _ptr(p.get("b2")), _ptr(p["D"]), _ptr(p.get("bD")), K if per_expert else 1)


def moe_workspace(params: MoeParams, n) -> int:
    return lib().hmoe_moe_workspace(ctypes.byref(params), n)


ANCHOR_COLS, ANCHOR_TILE = 64, 256  # include/hmoe.h: HMOE_ANCHOR_COLS, HMOE_ANCHOR_TILE


def anchor_shape(n: int, V: int):
    """Shape of the anchors of n rows of V stored logits: [ceil(V / 256), n, 4]."""
    return ((V + ANCHOR_TILE - 1) // ANCHOR_TILE, n, ANCHOR_TILE // ANCHOR_COLS)


def _check_moe_io(prm, n, dt, X_sorted, offsets, perm, o):
    """The activations in the parameters' dtype and the shapes the library assumes."""
    _expect(X_sorted, (n, prm.d_in), dt, "X_sorted")
    _expect(offsets, (prm.K + 1,), torch.int32, "offsets")
    _expect(perm, (n,), torch.int32, "perm")
    _expect(o.get("H1_sorted"), (n, prm.d_hid), dt, "H1_sorted")
    _expect(o.get("H"), (n, prm.d_out), dt, "H")


def moe_forward(p: dict, X_sorted, offsets, perm, row_ptr, tag, out=None, ws=None,
                save_logits=False):
    """Expert MLPs + decoder(s) + multilabel softmax loss (Eq. 3).  With save_logits the
    [n, V] logits are returned too (for a backward that does not recompute them; in slot
    order, row p = sample perm[p], when every expert has its own decoder, which needs them),
    stored as offsets from per-row anchors (returned as logit_anchor, anchor_shape(n, V))."""
    dims = _Dims(p)
    n = X_sorted.shape[0]
    dev = X_sorted.device
    dt = p["W1"].dtype
    o = out or {}
    _check_moe_io(dims, n, dt, X_sorted, offsets, perm, o)
    prm = make_params(p)
    _expect(o.get("logits"), (n, prm.vocab), dt, "logits")
    _expect(o.get("logit_anchor"), anchor_shape(n, prm.vocab), torch.float32, "logit_anchor")
    for k in ("lse", "loss"):
        _expect(o.get(k), (n,), torch.float32, k)
    _expect(o.get("loss_mean"), (1,), torch.float32, "loss_mean")
    H1s = _out(o, "H1_sorted", lambda: torch.empty(n, prm.d_hid, dtype=dt, device=dev))
    H = _out(o, "H", lambda: torch.empty(n, prm.d_out, dtype=dt, device=dev))
    lse = _out(o, "lse", lambda: torch.empty(n, dtype=torch.float32, device=dev))
    loss = _out(o, "loss", lambda: torch.empty(n, dtype=torch.float32, device=dev))
    lm = _out(o, "loss_mean", lambda: torch.empty(1, dtype=torch.float32, device=dev))
    lg = o.get("logits")
    if lg is None and save_logits:
        lg = torch.empty(n, prm.vocab, dtype=dt, device=dev)
    anc = o.get("logit_anchor")
    if anc is None and lg is not None:
        anc = torch.empty(anchor_shape(n, prm.vocab), dtype=torch.float32, device=dev)
    lab = Labels(_ptr(row_ptr), _ptr(tag))
    w, wb = _workspace(moe_workspace(prm, n), ws, dev)
    _chk(lib().hmoe_moe_forward(ctypes.byref(prm), n, _ptr(X_sorted), _ptr(offsets), _ptr(perm),
                                ctypes.byref(lab), _ptr(H1s), _ptr(H), _ptr(lg), _ptr(anc), _ptr(lse),
                                _ptr(loss), _ptr(lm), _ptr(w), wb, _stream()), "moe_forward")
    return {"H1_sorted": H1s, "H": H, "lse": lse, "loss": loss, "loss_mean": lm, "logits": lg,
            "logit_anchor": anc}


def moe_backward(p: dict, X_sorted, offsets, perm, inv, row_ptr, tag, H1_sorted, H, lse,
                 want_dX=True, out=None, ws=None, logits=None, logit_anchor=None):
    """Gradients of the mean loss for all expert and decoder parameters (fp32) and dX.  With
    logits and logit_anchor (saved by the forward) the decoder logits are not recomputed."""
    prm = _Dims(p)
    n = X_sorted.shape[0]
    dev = X_sorted.device
    K, d, h, o_, V = prm.K, prm.d_in, prm.d_hid, prm.d_out, prm.vocab
    f32 = torch.float32
    o = out or {}
    dt = p["W1"].dtype
    _check_moe_io(prm, n, dt, X_sorted, offsets, perm, {"H1_sorted": H1_sorted, "H": H})
    _expect(inv, (n,), torch.int32, "inv")
    _expect(lse, (n,), f32, "lse")
    _expect(logits, (n, V), dt, "logits")
    _expect(logit_anchor, anchor_shape(n, V), f32, "logit_anchor")
    if (logits is None) != (logit_anchor is None):
        raise HmoeError("logits and logit_anchor go together (the forward's stored form)")
    for k, shape in (("dW1", (K, h, d)), ("db1", (K, h)), ("dW2", (K, o_, h)), ("db2", (K, o_)),
                     ("dD", tuple(p["D"].shape)), ("dbD", tuple(p["D"].shape[:-1]))):
        _expect(o.get(k), shape, f32, k)
    _expect(o.get("dX"), (n, d), dt, "dX")
    g = {"dW1": _out(o, "dW1", lambda: torch.empty(K, h, d, dtype=f32, device=dev)),
         "db1": _out(o, "db1", lambda: torch.empty(K, h, dtype=f32, device=dev)),
         "dW2": _out(o, "dW2", lambda: torch.empty(K, o_, h, dtype=f32, device=dev)),
         "db2": _out(o, "db2", lambda: torch.empty(K, o_, dtype=f32, device=dev)),
         "dD": _out(o, "dD", lambda: torch.empty(p["D"].shape, dtype=f32, device=dev)),
         "dbD": _out(o, "dbD", lambda: torch.empty(p["D"].shape[:-1], dtype=f32, device=dev)),
         "dX": (_out(o, "dX", lambda: torch.empty(n, d, dtype=dt, device=dev))
                if want_dX else None)}
    prm = make_params(p)
    lab = Labels(_ptr(row_ptr), _ptr(tag))
    w, wb = _workspace(moe_workspace(prm, n), ws, dev)
    _chk(lib().hmoe_moe_backward(ctypes.byref(prm), n, _ptr(X_sorted), _ptr(offsets), _ptr(perm),
                                 _ptr(inv), ctypes.byref(lab), _ptr(H1_sorted), _ptr(H),
                                 _ptr(logits), _ptr(logit_anchor), _ptr(lse),
                                 _ptr(g["dW1"]), _ptr(g["db1"]), _ptr(g["dW2"]), _ptr(g["db2"]),
                                 _ptr(g["dD"]), _ptr(g["dbD"]), _ptr(g["dX"]), _ptr(w), wb,
                                 _stream()), "moe_backward")
    return g


# ------------------------------------------------------------------ inference tail

def topm(logits, m: int, out=None, want_values=False, anchor=None):
    """t_m (Section 4.4): the indices [n, m] of each row's m largest logits, decreasing, equal
    values by increasing index (and their values, fp32, with want_values).  anchor: the
    forward's logit_anchor when logits are its stored offsets (an entry is then anchor +
    offset in fp32; every offset must be <= 0, as the forward writes them)."""
    n, V = logits.shape
    dev = logits.device
    o = out or {}
    _expect(o.get("idx"), (n, m), torch.int32, "idx")
    _expect(o.get("val") if want_values else None, (n, m), torch.float32, "val")
    idx = o["idx"] if "idx" in o else torch.empty(n, m, dtype=torch.int32, device=dev)
    val = None
    if want_values:
        val = o["val"] if "val" in o else torch.empty(n, m, dtype=torch.float32, device=dev)
    _expect(anchor, anchor_shape(n, V), torch.float32, "anchor")
    _chk(lib().hmoe_topm(_ptr(logits), _ptr(anchor), _dt(logits), n, V, m, _ptr(idx), _ptr(val), _stream()),
         "topm")
    return (idx, val) if want_values else idx


def topm_hits(idx, row_ptr, tag, q_sample=None, q_tag=None, out=None):
    """Counts behind p@m' (Eq. 4) and q@m' (Eq. 5) for m' = 1..m: an int64 tensor [2, m] with
    row 0 = sum_i |t_m'(i) & P_i| and row 1 = the draws (q_sample, q_tag) whose tag is in the
    sample's t_m'."""
    n, m = idx.shape
    S = 0 if q_sample is None else q_sample.shape[0]
    hits = out if out is not None else torch.empty(2, m, dtype=torch.int64, device=idx.device)
    lab = Labels(_ptr(row_ptr), _ptr(tag))
    _chk(lib().hmoe_topm_hits(_ptr(idx), n, m, ctypes.byref(lab), _ptr(q_sample), _ptr(q_tag), S, _ptr(hits),
                              _stream()), "topm_hits")
    return hits


# ------------------------------------------------------------------ parameter update

def sgd_step(w, g, lr: float, weight_decay: float = 0.0, momentum: float = 0.0, v=None, w_lo=None):
    """One SGD step in place on the fp32 master weights w (Section 4.2); v is the momentum
    buffer (required when momentum > 0); w_lo, if given, receives the updated weights in its
    dtype (bf16 or fp32)."""
    if w.dtype != torch.float32 or g.dtype != torch.float32 or g.numel() != w.numel():
        raise HmoeError("sgd_step needs fp32 w and g of the same size")
    if w_lo is not None and w_lo.numel() != w.numel():
        raise HmoeError(f"w_lo has {w_lo.numel()} elements, w {w.numel()}")
    if v is not None and (v.dtype != torch.float32 or v.numel() != w.numel()):
        raise HmoeError("v must be fp32 with as many elements as w")
    dt = _dt(w_lo) if w_lo is not None else 1
    _chk(lib().hmoe_sgd_step(_ptr(w), _ptr(g), _ptr(v), _ptr(w_lo), dt, w.numel(), lr, weight_decay, momentum,
                             _stream()), "sgd_step")
    return w


# ------------------------------------------------------------------ PCA before the K-means

def pca_workspace(n, d, r, dtype) -> int:
    return lib().hmoe_pca_workspace(n, d, r, 1 if dtype == torch.bfloat16 else 0)


def pca_fit(X, r: int, n_iter: int = 20, seed: int = 0, ws=None):
    """Section 4.2: mean [d], components [r, d] (the r leading principal directions, decreasing
    eigenvalue, largest-magnitude entry of each positive) and eigenvalues [r], fp32."""
    n, d = X.shape
    dev = X.device
    mean = torch.empty(d, dtype=torch.float32, device=dev)
    comps = torch.empty(r, d, dtype=torch.float32, device=dev)
    ev = torch.empty(r, dtype=torch.float32, device=dev)
    w, wb = _workspace(pca_workspace(n, d, r, X.dtype), ws, dev)
    _chk(lib().hmoe_pca_fit(_ptr(X), _dt(X), n, d, r, n_iter, seed, _ptr(mean), _ptr(comps), _ptr(ev), _ptr(w), wb,
                            _stream()), "pca_fit")
    return mean, comps, ev


def pca_project(X, mean, comps, out=None, ws=None):
    """(X - mean) comps^T in X's dtype: the features the K-means runs on."""
    n, d = X.shape
    r = comps.shape[0]
    _expect(mean, (d,), torch.float32, "mean")
    _expect(comps, (r, d), torch.float32, "comps")
    _expect(out, (n, r), X.dtype, "out")
    Z = out if out is not None else torch.empty(n, r, dtype=X.dtype, device=X.device)
    w, wb = _workspace(pca_workspace(n, d, r, X.dtype), ws, X.device)
    _chk(lib().hmoe_pca_project(_ptr(X), _dt(X), n, d, _ptr(mean), _ptr(comps), r, _ptr(Z), _ptr(w), wb, _stream()),
         "pca_project")
    return Z
