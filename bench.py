"""Benchmark of the hard mixture-of-experts hot path on one MI355X.

One step = one routed training step on the balanced workload: gater assignment of 65,536
bf16 feature rows (d = 2048) to the nearest of K = 16 centres, counting-sort dispatch, the
16 expert MLPs 2048 -> 4096 -> 1024 with the shared 1024 -> 50,000 decoder, multilabel
softmax loss, and the full backward pass (all parameter gradients and dX; the forward saves
the bf16 logits so the backward does not recompute them).  Inputs are seeded synthetic
tensors already resident in HBM.

Printed: one JSON line with the step throughput (samples/s), the roofline of the dominant
kernel (HIP events recorded around every launch in the timed region), the fp64 CPU oracle
timed on a bounded sample of the same workload, and extra legs for the gater fit
(2^20 fp32 rows, K = 64, 20 Lloyd iterations), the skewed routing step (K = 128, V = 100k),
the balanced step with one decoder per expert (the independent-decoder model), inference on
the balanced batch (forward, top-10 tags per row, p@m / q@m counts), the SGD update of the
balanced model's parameters and the large streamed assignment (2^24 bf16 rows, K = 1024).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "k-means assign samples/s; routed MoE fwd+bwd samples/s and % MFMA/HBM peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
LEG_NAMES = ("gater_fit", "gater_pca", "skewed", "independent", "inference", "sgd_update", "large_assign")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ------------------------------------------------------------------ HBM traffic record

TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "decoder_forward_hbm_traffic.md")


def _code_only(text: str) -> str:
    """The source without comments, trailing spaces or blank lines (a comment edit changes no
    kernel)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines())
    return "\n".join(ln for ln in lines if ln)


def kernel_source_digest(read=None, unit="moe.hip"):
    """sha256 over the translation unit that builds the dominant kernel (csrc/moe.hip), the
    headers it includes (recursively) and the C header, without their comments, so a traffic
    figure measured on older kernels is recognised as stale while edits elsewhere (or to
    comments) do not retire it.  `read(relative_path)` supplies the text (default: the tree)."""
    src_rel = "paper_1704_06363_amd/csrc"
    if read is None:
        def read(rel):
            with open(os.path.join(ROOT, rel), encoding="utf-8") as fh:
                return fh.read()
    texts, todo = {}, [f"{src_rel}/{unit}"]
    while todo:
        rel = todo.pop()
        if rel in texts:
            continue
        texts[rel] = read(rel)
        for name in re.findall(r'^\s*#\s*include\s+"([^"]+)"', texts[rel], flags=re.M):
            todo.append(f"include/{name}" if name == "hmoe.h" else f"{src_rel}/{name}")
    h = hashlib.sha256()
    for rel in sorted(texts):
        h.update(rel.encode() + b"\0" + _code_only(texts[rel]).encode())
    return h.hexdigest()[:16]


def recorded_traffic(label):
    """HBM bytes per launch of `label` from the committed counter summary (FETCH_SIZE and
    WRITE_SIZE, scaled by the same counters on a plain copy), or None when there is no record
    for this kernel or the kernel sources changed since it was taken."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    with open(TRAFFIC_PROFILE) as fh:
        m = re.search(r"^traffic-record: (\{.*\})$", fh.read(), re.M)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("kernel") != label or rec.get("source_digest") != kernel_source_digest():
        return None
    return rec


def calib_copy(mib):
    """A plain device-to-device copy of `mib` MiB (twice), the known-size reference for the
    HBM byte counters."""
    import torch
    src = torch.ones(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


# ------------------------------------------------------------------ routed step

def gemm_flops(s):
    """Algorithmic FLOPs per launch of each labelled kernel of one routed step."""
    n, d, h, o, V, K = s["n"], s["d"], s["h"], s["o"], s["V"], s["K"]
    return {
        "assign": 2.0 * n * K * d,
        "expert layer 1": 2.0 * n * d * h,
        "expert layer 2": 2.0 * n * h * o,
        "decoder forward": 2.0 * n * V * o,
        "decoder dH": 2.0 * n * V * o,
        "decoder dD": 2.0 * n * V * o,
        "expert dW2": 2.0 * n * o * h,
        "expert dH1": 2.0 * n * o * h,
        "expert dW1": 2.0 * n * h * d,
        "expert dX": 2.0 * n * h * d,
    }


def step_bytes(s, nnz):
    """Algorithmic HBM bytes per step of each labelled kernel of one routed step (all its
    launches): every operand read once and every output written once, in the stored dtypes
    (bf16 data, fp32 gradients, int32 indices).  Partial sums a kernel keeps for a later one
    (the split-K partials) count for the kernel that writes and the one that reads them."""
    n, d, h, o, V, K = s["n"], s["d"], s["h"], s["o"], s["V"], s["K"]
    b, f, i = 2, 4, 4
    ntv = -(-V // 256)
    nb = -(-n // 1024)
    return {
        "assign": n * d * b + K * d * b + n * (i + f),
        "dispatch hist": n * i + nb * (K + 1) * i,
        "dispatch colscan": 2 * nb * (K + 1) * i + K * i,
        "dispatch offsets": K * i + (K + 1) * i,
        "dispatch scan": 2 * nb * (K + 1) * i + K * i + (K + 1) * i,  # colscan + offsets in one launch
        "dispatch scatter": n * i + nb * (K + 1) * i + 2 * n * i,
        "permute rows": 2 * n * d * b + n * i,
        "expert layer 1": n * d * b + K * h * d * b + n * h * b,
        "expert layer 2": n * h * b + K * o * h * b + n * o * b + n * i,
        # H and D read, logits and their anchors written, the per-tile (max, sum) partials
        "decoder forward": n * o * b + V * o * b + n * V * b + n * ntv * 16 + 2 * n * ntv * f,
        "decoder loss": 2 * n * ntv * f + n * o * b + V * o * b + (n + 1 + nnz) * i + 2 * n * f,
        "decoder grad": n * V * b + n * ntv * 16 + n * f + (n + 1 + nnz) * i + n * V * b + (-(-n // 256)) * V * f,
        "decoder bias grad": (-(-n // 256)) * V * f + V * f,
        "decoder dH": n * V * b + V * o * b + n * o * b + n * i,
        "decoder dD": n * V * b + n * o * b + V * o * f,
        "segsum partial": n * (o + h) * b,
        "expert dW2": n * o * b + n * h * b + K * o * h * f,
        "expert dH1": n * o * b + K * o * h * b + 2 * n * h * b,
        "expert dW1": n * h * b + n * d * b + K * h * d * f,
        "expert dX": n * h * b + K * h * d * b + n * d * b + n * i,
    }


def step_flops(s, assign=True):
    f = gemm_flops(s)
    tot = sum(v for k, v in f.items() if k != "assign")
    return tot + (f["assign"] if assign else 0.0)


class RoutedStep:
    """Preallocated buffers for one routed training step; run() enqueues it on the stream."""

    def __init__(self, inp, routed_by_gater: bool):
        import torch
        from paper_1704_06363_amd import hmoe
        self.h = hmoe
        self.inp = inp
        s = inp["shape"]
        self.s = s
        n, d, h, o, V, K = s["n"], s["d"], s["h"], s["o"], s["V"], s["K"]
        dev = inp["X"].device
        self.routed_by_gater = routed_by_gater
        self.X = inp["X"]
        self.C = inp.get("C")
        self.ids = (torch.empty(n, dtype=torch.int32, device=dev) if routed_by_gater
                    else torch.as_tensor(inp["ids"], dtype=torch.int32).to(dev))
        self.md = torch.empty(n, dtype=torch.float32, device=dev)
        self.row_ptr = torch.as_tensor(inp["row_ptr"]).to(dev)
        self.tag = torch.as_tensor(inp["tag"]).to(dev)
        bf = torch.bfloat16
        self.disp = {"counts": torch.empty(K, dtype=torch.int32, device=dev),
                     "offsets": torch.empty(K + 1, dtype=torch.int32, device=dev),
                     "perm": torch.empty(n, dtype=torch.int32, device=dev),
                     "inv": torch.empty(n, dtype=torch.int32, device=dev),
                     "rows_sorted": torch.empty(n, d, dtype=bf, device=dev)}
        self.fwd = {"H1_sorted": torch.empty(n, h, dtype=bf, device=dev),
                    "H": torch.empty(n, o, dtype=bf, device=dev),
                    "lse": torch.empty(n, dtype=torch.float32, device=dev),
                    "loss": torch.empty(n, dtype=torch.float32, device=dev),
                    "loss_mean": torch.empty(1, dtype=torch.float32, device=dev),
                    "logits": torch.empty(n, V, dtype=bf, device=dev),
                    "logit_anchor": torch.empty(hmoe.anchor_shape(n, V), dtype=torch.float32, device=dev)}
        f32 = torch.float32
        self.grads = {"dW1": torch.empty(K, h, d, dtype=f32, device=dev),
                      "db1": torch.empty(K, h, dtype=f32, device=dev),
                      "dW2": torch.empty(K, o, h, dtype=f32, device=dev),
                      "db2": torch.empty(K, o, dtype=f32, device=dev),
                      "dD": torch.empty(inp["params"]["D"].shape, dtype=f32, device=dev),
                      "dbD": torch.empty(inp["params"]["D"].shape[:-1], dtype=f32, device=dev),
                      "dX": torch.empty(n, d, dtype=bf, device=dev)}
        prm = hmoe.make_params(inp["params"])
        need = max(hmoe.moe_workspace(prm, n), hmoe.moe_dispatch_workspace(n, K),
                   hmoe.kmeans_assign_workspace(n, d, K, bf))
        self.ws = torch.empty(need, dtype=torch.uint8, device=dev)

    def run(self, backward=True):
        h, p = self.h, self.inp["params"]
        if self.routed_by_gater:
            h.kmeans_assign(self.X, self.C, assign=self.ids, min_dist=self.md, ws=self.ws)
        h.moe_dispatch(self.ids, self.s["K"], rows=self.X, out=self.disp, ws=self.ws)
        dd = self.disp
        f = h.moe_forward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], self.row_ptr, self.tag,
                          out=self.fwd, ws=self.ws)
        if not backward:
            return
        h.moe_backward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], self.row_ptr,
                       self.tag, f["H1_sorted"], f["H"], f["lse"], out=self.grads, ws=self.ws,
                       logits=f["logits"], logit_anchor=f["logit_anchor"])


def time_steps(fn, steps, warmup, timer=True):
    import torch
    from paper_1704_06363_amd import hmoe
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    if timer:
        hmoe.timer_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    rep = {}
    if timer:
        rep = hmoe.timer_report()
        hmoe.timer_enable(False)
    return ms, rep


def kernel_table(rep, flops, peak_tflops, steps, nbytes=None):
    """Per kernel label: launches and average time; against the MFMA roof (FLOPs per launch in
    `flops`), against the HBM roof (bytes per step in `nbytes`), and where both are known, the
    roof that bounds it -- the larger of FLOPs / MFMA peak and bytes / HBM peak -- with the
    fraction of that roof reached."""
    out = {}
    for label, (cnt, ms) in rep.items():
        e = {"launches_per_step": cnt / steps, "avg_ms": ms / cnt}
        t_step = ms / steps * 1e-3  # seconds per step in this label
        t_mfma = t_hbm = None
        if label in flops:
            tf = flops[label] / (ms / cnt * 1e-3) / 1e12
            e["tflops"] = round(tf, 2)
            e["frac_mfma_peak"] = round(tf / peak_tflops, 4)
            t_mfma = flops[label] * (cnt / steps) / (peak_tflops * 1e12)
        if nbytes and label in nbytes:
            gbs = nbytes[label] / t_step / 1e9
            e["gb_per_s"] = round(gbs, 1)
            e["frac_hbm_peak"] = round(gbs / PEAK_HBM_GBS, 4)
            t_hbm = nbytes[label] / (PEAK_HBM_GBS * 1e9)
        if t_mfma is not None or t_hbm is not None:
            roof = max(x for x in (t_mfma, t_hbm) if x is not None)
            e["bound"] = "mfma" if (t_mfma or 0.0) >= (t_hbm or 0.0) else "hbm"
            e["frac_roof"] = round(roof / t_step, 4)
        out[label] = e
    return out


def hbm_summary(rep, nbytes, steps, labels):
    """Achieved HBM bandwidth of a group of kernels (bytes per step over their summed time)."""
    ms = sum(rep[k][1] for k in labels if k in rep) / steps
    by = sum(nbytes[k] for k in labels if k in rep)
    if ms <= 0:
        return None
    gbs = by / (ms * 1e-3) / 1e9
    return {"kernels": [k for k in labels if k in rep], "ms": round(ms, 4), "bytes": int(by),
            "gb_per_s": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}


def dominant(rep, flops):
    best = None
    for label, (cnt, ms) in rep.items():
        if label in flops and (best is None or ms > rep[best][1]):
            best = label
    return best


# ------------------------------------------------------------------ CPU oracle baseline

def cpu_baseline(inp, sample: int, routed_by_gater: bool):
    """The fp64 oracle on the first `sample` rows of the same workload: gater assignment
    (if routed by the gater), dispatch, expert + decoder forward and full backward."""
    from oracle import oracle as O
    import torch

    def h64(t):
        return t.detach().to(torch.float64).cpu().numpy()

    s = inp["shape"]
    X = h64(inp["X"][:sample])
    p = {k: (h64(v) if v is not None else None) for k, v in inp["params"].items()}
    rp = inp["row_ptr"][:sample + 1].copy()
    tg = inp["tag"][:rp[-1]].copy()
    C = h64(inp["C"]) if routed_by_gater else None
    ids = None if routed_by_gater else np.asarray(inp["ids"][:sample], np.int32)
    O.build(force=False)
    t0 = time.perf_counter()
    if routed_by_gater:
        ids, _, _ = O.assign(X, C)
    O.dispatch(ids, s["K"])
    f = O.moe_forward(X, ids, p["W1"], p["b1"], p["W2"], p["b2"], p["D"], p["bD"], rp, tg,
                      store="bf16")
    O.moe_backward(X, ids, p["W1"], p["W2"], p["D"], p["bD"], rp, tg, f["H1"], f["H"], f["lse"],
                   store="bf16")
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
    return {"value": round(sample / dt, 3), "unit": "samples/s", "cores": threads,
            "kind": "oracle",
            "sample": f"first {sample} of {s['n']} rows, full widths (d={s['d']}, h={s['h']}, "
                      f"o={s['o']}, V={s['V']}, K={s['K']}): assign+dispatch+fwd+bwd in fp64, "
                      f"{dt:.2f} s"}


# ------------------------------------------------------------------ legs

def leg_gater_fit(steps):
    import torch
    from paper_1704_06363_amd import hmoe
    from paper_1704_06363_amd import workloads as W
    c = W.CONFIGS["gater_fit"]
    X = W.gmm_features(c.n, c.d, c.extra["n_comp"], seed=0, dtype="f32", device="cuda",
                       dirichlet_alpha=c.extra["alpha"])
    u = torch.tensor(W.uniforms(c.K, 1), dtype=torch.float64, device="cuda")
    ws = torch.empty(hmoe.kmeans_fit_workspace(c.n, c.d, c.K, torch.float32), dtype=torch.uint8,
                     device="cuda")

    def fn():
        hmoe.kmeans_fit(X, c.K, c.n_iter, init_uniforms=u, ws=ws)

    ms, rep = time_steps(fn, steps, 1)
    a_cnt, a_ms = rep["assign"]
    a_avg = a_ms / a_cnt
    assign_tf = 2.0 * c.n * c.K * c.d / (a_avg * 1e-3) / 1e12
    upd = sum(v[1] for k, v in rep.items() if k.startswith(("segsum", "dispatch", "reseed",
                                                             "finalize", "permute")))
    upd_iter_ms = upd / (steps * c.n_iter)
    kpp = sum(v[1] for k, v in rep.items() if k.startswith("kmeans++")) / steps
    out = {"workload": f"gater fit: n={c.n} fp32, d={c.d}, K={c.K}, k-means++ + {c.n_iter} "
                       f"Lloyd iterations with reseeding",
           "fit_ms": round(ms, 3),
           "assign_samples_per_s": round(c.n / (a_avg * 1e-3), 1),
           "assign_avg_ms": round(a_avg, 4),
           "assign_tflops": round(assign_tf, 2),
           "assign_frac_fp32_peak": round(assign_tf / PEAK_F32_TFLOPS, 4),
           "update_ms_per_iter": round(upd_iter_ms, 4),
           "update_frac_hbm_peak": round(c.n * c.d * 4 / (upd_iter_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "kmeanspp_ms": round(kpp, 3)}
    del X
    torch.cuda.empty_cache()
    return out


def leg_gater_pca(steps):
    """Section 4.2's gater features: the 512-wide features of the gater-fit workload reduced to
    their 256 leading principal directions (covariance, 20 subspace iterations, Rayleigh-Ritz),
    projected, and clustered on the projection (k-means++ and the same Lloyd iterations)."""
    import torch
    from paper_1704_06363_amd import hmoe
    from paper_1704_06363_amd import workloads as W
    c = W.CONFIGS["gater_fit"]
    r, n_iter = 256, 20
    X = W.gmm_features(c.n, c.d, c.extra["n_comp"], seed=0, dtype="f32", device="cuda",
                       dirichlet_alpha=c.extra["alpha"])
    ws = torch.empty(hmoe.pca_workspace(c.n, c.d, r, torch.float32), dtype=torch.uint8, device="cuda")
    Z = torch.empty(c.n, r, dtype=torch.float32, device="cuda")
    u = torch.tensor(W.uniforms(c.K, 1), dtype=torch.float64, device="cuda")
    kws = torch.empty(hmoe.kmeans_fit_workspace(c.n, r, c.K, torch.float32), dtype=torch.uint8, device="cuda")
    fitted = {}

    def fit():
        fitted["m"], fitted["u"], fitted["ev"] = hmoe.pca_fit(X, r, n_iter, seed=0, ws=ws)

    def proj():
        hmoe.pca_project(X, fitted["m"], fitted["u"], out=Z, ws=ws)

    def km():
        hmoe.kmeans_fit(Z, c.K, c.n_iter, init_uniforms=u, ws=kws)

    fit_ms, frep = time_steps(fit, steps, 1)
    gpu_ms = sum(v[1] for v in frep.values()) / steps
    cov_cnt, cov_ms = frep["pca X^T X"]
    cov_avg = cov_ms / cov_cnt
    cov_tf = 2.0 * c.n * c.d * c.d / (cov_avg * 1e-3) / 1e12
    proj_ms, prep = time_steps(proj, steps, 1)
    p_cnt, p_ms = prep["pca project"]
    p_avg = p_ms / p_cnt
    proj_tf = 2.0 * c.n * c.d * r / (p_avg * 1e-3) / 1e12
    km_ms, krep = time_steps(km, steps, 1)
    a_cnt, a_ms = krep["assign"]
    a_avg = a_ms / a_cnt
    ev = fitted["ev"].double()
    out = {"workload": f"gater features with PCA: n={c.n} fp32, d={c.d} -> r={r} ({n_iter} subspace "
                       f"iterations), projection, K-means K={c.K} with {c.n_iter} Lloyd iterations on the "
                       "projection",
           "pca_fit_ms": round(fit_ms, 3),
           "pca_fit_gpu_kernels_ms": round(gpu_ms, 3),
           "pca_fit_host_ms": round(fit_ms - gpu_ms, 3),
           "covariance_avg_ms": round(cov_avg, 4),
           "covariance_tflops": round(cov_tf, 2),
           "covariance_frac_fp32_peak": round(cov_tf / PEAK_F32_TFLOPS, 4),
           "project_avg_ms": round(p_avg, 4),
           "project_tflops": round(proj_tf, 2),
           "project_frac_fp32_peak": round(proj_tf / PEAK_F32_TFLOPS, 4),
           "kmeans_fit_ms": round(km_ms, 3),
           "kmeans_assign_avg_ms": round(a_avg, 4),
           "kmeans_assign_tflops": round(2.0 * c.n * c.K * r / (a_avg * 1e-3) / 1e12, 2),
           "leading_eigenvalues": [round(float(x), 3) for x in ev[:4].tolist()],
           "kernels_fit": kernel_table(frep, {"pca X^T X": 2.0 * c.n * c.d * c.d}, PEAK_F32_TFLOPS, steps)}
    del X, Z, ws, kws
    torch.cuda.empty_cache()
    return out


def leg_skewed(steps, warmup):
    import torch
    from paper_1704_06363_amd import workloads as W
    inp = W.skewed_inputs(device="cuda", seed=0)
    st = RoutedStep(inp, routed_by_gater=False)
    ms, rep = time_steps(st.run, steps, warmup)
    s = inp["shape"]
    fl = gemm_flops(s)
    nby = step_bytes(s, int(inp["row_ptr"][-1]))
    tot = step_flops(s, assign=False)
    out = {"workload": "skewed routed step: n=32768 bf16, d=2048, K=128 Zipf(1.3) buckets, "
                       "MLP 2048-2048-1024, V=100000, fwd+bwd",
           "samples_per_s": round(s["n"] / (ms * 1e-3), 1), "ms_per_step": round(ms, 3),
           "tflops": round(tot / (ms * 1e-3) / 1e12, 1),
           "frac_bf16_peak": round(tot / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "kernels": kernel_table(rep, fl, PEAK_BF16_TFLOPS, steps, nby),
           "hbm": {"dispatch_row_gather": hbm_summary(rep, nby, steps, ["permute rows"]),
                   "reduction_bias_grads": hbm_summary(rep, nby, steps, ["segsum partial"])}}
    del st, inp
    torch.cuda.empty_cache()
    return out


def leg_independent(steps, warmup):
    """The balanced routed step with one decoder per expert (Section 2's independent-decoder
    model): the same per-sample work, so the same FLOPs per step."""
    import torch
    from paper_1704_06363_amd import workloads as W
    inp = W.balanced_inputs(device="cuda", seed=0)
    s = inp["shape"]
    inp["params"] = W.moe_params(s["K"], s["d"], s["h"], s["o"], s["V"], seed=20, dtype="bf16",
                                 device="cuda", per_expert_decoders=True)
    st = RoutedStep(inp, routed_by_gater=True)
    ms, rep = time_steps(st.run, steps, warmup)
    fl = gemm_flops(s)
    tot = step_flops(s)
    out = {"workload": "independent-decoder routed step: n=65536 bf16, d=2048, K=16 experts each with "
                       "its own decoder (16 x 50000 x 1024), MLP 2048-4096-1024, fwd+bwd",
           "samples_per_s": round(s["n"] / (ms * 1e-3), 1), "ms_per_step": round(ms, 3),
           "tflops": round(tot / (ms * 1e-3) / 1e12, 1),
           "frac_bf16_peak": round(tot / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "kernels": kernel_table(rep, fl, PEAK_BF16_TFLOPS, steps)}
    del st, inp
    torch.cuda.empty_cache()
    return out


def leg_inference(steps, warmup, m=10, draws=100000):
    """Inference on the balanced batch (Section 4.4): gater assignment, dispatch, the forward
    with the logits stored, then t_m of every row and the counts behind p@m and q@m."""
    import torch
    from paper_1704_06363_amd import hmoe
    from paper_1704_06363_amd import workloads as W
    inp = W.balanced_inputs(device="cuda", seed=0)
    s = inp["shape"]
    st = RoutedStep(inp, routed_by_gater=True)
    qs, qt = W.q_draws(inp["row_ptr"], inp["tag"], draws, seed=1)
    qs, qt = torch.as_tensor(qs).cuda(), torch.as_tensor(qt).cuda()
    idx = torch.empty(s["n"], m, dtype=torch.int32, device="cuda")
    hits = torch.empty(2, m, dtype=torch.int64, device="cuda")

    def run():
        st.run(backward=False)
        hmoe.topm(st.fwd["logits"], m, out={"idx": idx}, anchor=st.fwd["logit_anchor"])
        hmoe.topm_hits(idx, st.row_ptr, st.tag, qs, qt, out=hits)

    ms, rp = time_steps(run, steps, warmup)
    k = kernel_table(rp, gemm_flops(s), PEAK_BF16_TFLOPS, steps)
    tk = k.get("top-m", {}).get("avg_ms", float("nan"))
    nnz = int(inp["row_ptr"][-1])
    h = hits.cpu().numpy()
    out = {"workload": f"inference: balanced batch (n=65536, V=50000) forward with stored bf16 logits, "
                       f"then top-{m} per row and p@m / q@m counts ({draws} q draws)",
           "samples_per_s": round(s["n"] / (ms * 1e-3), 1), "ms_per_batch": round(ms, 3),
           "topm_ms": round(tk, 4),
           # the anchored top-m reads the anchors (4 bytes per 64 columns) and about m blocks of
           # 64 bf16 logits per row, not the whole row: the rate of the whole-row scan it replaces
           # is quoted as the logits it did not have to read
           "topm_logits_gb_per_s_equiv": round(s["n"] * s["V"] * 2 / (tk * 1e-3) / 1e9, 1),
           "topm_anchor_bytes": int(s["n"] * -(-s["V"] // 256) * 16),
           "p_at_m": [round(float(x) / nnz, 6) for x in h[0]],
           "q_at_m": [round(float(x) / draws, 6) for x in h[1]],
           "kernels": k}
    del st, inp
    torch.cuda.empty_cache()
    return out


def leg_sgd_update(steps, warmup):
    """One SGD step (Section 4.2: weight decay 1e-4, no momentum for the experts and the
    decoder) over every parameter of the balanced model, fp32 master weights, writing the bf16
    copies the next forward reads."""
    import torch
    from paper_1704_06363_amd import hmoe
    from paper_1704_06363_amd import workloads as W
    c = W.CONFIGS["balanced"]
    p = W.moe_params(c.K, c.d, c.h, c.o, c.V, seed=20, dtype="bf16", device="cuda", bias=True)
    master = {k: v.float() for k, v in p.items()}
    grads = {k: torch.randn_like(v) * 1e-3 for k, v in master.items()}

    def run():
        for k in p:
            hmoe.sgd_step(master[k], grads[k], lr=0.1, weight_decay=1e-4, w_lo=p[k])

    ms, rep = time_steps(run, steps, warmup)
    count = sum(v.numel() for v in master.values())
    out = {"workload": f"SGD step (weight decay, no momentum) over the balanced model's {count} expert and "
                       "decoder parameters, fp32 master weights plus bf16 copies",
           "ms_per_update": round(ms, 3),
           "frac_hbm_peak": round(count * 14 / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "kernels": kernel_table(rep, {}, PEAK_BF16_TFLOPS, steps)}
    del p, master, grads
    torch.cuda.empty_cache()
    return out


def leg_large_assign(n_chunks):
    import torch
    from paper_1704_06363_amd import hmoe
    from paper_1704_06363_amd import workloads as W
    c = W.CONFIGS["large_assign"]
    chunk = c.extra["chunk"]
    means = W.gmm_means(c.extra["n_comp"], c.d, seed=2, device="cuda")
    chunks = [W.gmm_features(chunk, c.d, c.extra["n_comp"], seed=100 + i, dtype="bf16",
                             device="cuda", means=means) for i in range(n_chunks)]
    g = torch.Generator(device="cpu").manual_seed(3)
    C = chunks[0][torch.randperm(chunk, generator=g)[:c.K].cuda()].contiguous()
    a = torch.empty(chunk, dtype=torch.int32, device="cuda")
    md = torch.empty(chunk, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(hmoe.kmeans_assign_workspace(chunk, c.d, c.K, torch.bfloat16),
                         hmoe.kmeans_update_workspace(chunk, c.d, c.K, torch.bfloat16)),
                     dtype=torch.uint8, device="cuda")
    sums = torch.zeros(c.K, c.d, dtype=torch.float64, device="cuda")
    cnt = torch.zeros(c.K, dtype=torch.int64, device="cuda")
    Cn = torch.empty(c.K, c.d, dtype=torch.float32, device="cuda")
    hmoe.kmeans_assign(chunks[0], C, assign=a, min_dist=md, ws=ws)  # warm-up
    torch.cuda.synchronize()
    hmoe.timer_enable(True)
    t0 = time.perf_counter()
    for x in chunks:
        hmoe.kmeans_assign(x, C, assign=a, min_dist=md, ws=ws)
        hmoe.kmeans_update(x, c.K, a, md, sums, cnt, Cn, mode=hmoe.UPDATE_ACCUMULATE,
                           reseed=False, ws=ws)
    hmoe.kmeans_update(None, c.K, None, None, sums, cnt, Cn, mode=hmoe.UPDATE_FINALIZE, ws=ws)
    torch.cuda.synchronize()
    total_ms = (time.perf_counter() - t0) * 1e3
    rep = hmoe.timer_report()
    hmoe.timer_enable(False)
    n = chunk * n_chunks
    a_ms = rep["assign"][1] + rep.get("assign merge", (0, 0.0))[1] + rep["centre norms"][1]
    gemm_ms = rep["assign"][1]
    tf = 2.0 * n * c.K * c.d / (gemm_ms * 1e-3) / 1e12
    upd_ms = total_ms - a_ms
    out = {"workload": f"large assign: {n_chunks} chunks x {chunk} bf16 rows, d={c.d}, K={c.K}, "
                       f"plus one streamed centre-update pass",
           "assign_samples_per_s": round(n / (a_ms * 1e-3), 1),
           "distance_gemm_tflops": round(tf, 1),
           "distance_gemm_frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
           "assign_ms": round(a_ms, 3), "update_pass_ms": round(upd_ms, 3),
           "update_frac_hbm_peak": round(n * c.d * 2 / (upd_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    del chunks
    torch.cuda.empty_cache()
    return out


# ------------------------------------------------------------------ main

def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-legs", action="store_true", help="skip the extra legs (gater fit, gater PCA, skewed, independent decoders, inference, SGD update, large assign)")
    ap.add_argument("--legs", default="", help="comma-separated subset of the legs to run (default: all)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-sample", type=int, default=2048)
    ap.add_argument("--large-chunks", type=int, default=16)
    ap.add_argument("--skip-step", action="store_true",
                    help="run only the legs, not the balanced step (for profiling a leg on its own; the JSON line "
                         "then carries no step figures)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    unknown = set(x for x in args.legs.split(",") if x) - set(LEG_NAMES)
    if unknown:
        raise SystemExit(f"unknown legs: {sorted(unknown)}")
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the multi-GPU layout is "
              f"a design note, not a measured configuration.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1704_06363_amd import hmoe
    from paper_1704_06363_amd import workloads as W
    torch.cuda.set_device(0)
    hmoe.lib()
    if args.calib_copy_mib > 0:
        log(f"calibration copy: {args.calib_copy_mib} MiB")
        calib_copy(args.calib_copy_mib)

    if args.skip_step:
        legs = run_legs(args)
        print(json.dumps({"metric": METRIC, "legs": legs}), flush=True)
        return
    log("balanced step: generating inputs")
    inp = W.balanced_inputs(device="cuda", seed=0)
    s = inp["shape"]
    st = RoutedStep(inp, routed_by_gater=True)
    log("balanced step: timing")
    ms, rep = time_steps(st.run, args.steps, args.warmup)
    fl = gemm_flops(s)
    nnz = int(inp["row_ptr"][-1])
    nby = step_bytes(s, nnz)
    kern = kernel_table(rep, fl, PEAK_BF16_TFLOPS, args.steps, nby)
    dom = dominant(rep, fl)
    cnt, tot_ms = rep[dom]
    avg = tot_ms / cnt
    achieved = fl[dom] / (avg * 1e-3) / 1e12
    tot_flops = step_flops(s)
    tr = recorded_traffic(dom)
    res = {
        "metric": METRIC,
        "value": round(s["n"] / (ms * 1e-3), 1),
        "unit": "samples/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "balanced routed training step: gater assign (K=16 centres) + "
                               "dispatch + 16 expert MLPs 2048-4096-1024 + shared decoder "
                               "1024->50000 + multilabel softmax loss, forward and backward",
                   "batch": s["n"], "d": s["d"], "experts": s["K"], "hidden": s["h"],
                   "expert_out": s["o"], "vocab": s["V"], "max_tags": 8},
        "step_tflops": round(tot_flops / (ms * 1e-3) / 1e12, 1),
        "step_frac_bf16_peak": round(tot_flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": tr["bytes_per_launch"] if tr else None,
                     "avg_ms": round(avg, 4), "flop_per_launch": fl[dom]},
        "kernels": kern,
        # dispatch = the counting sort and the row gather into expert order (the combine is the
        # second expert layer's epilogue, which writes rows back to sample order); reduction =
        # the experts' bias-gradient segmented sums (the centre update's is in legs.gater_fit)
        "hbm": {"dispatch": hbm_summary(rep, nby, args.steps, ["dispatch hist", "dispatch colscan",
                                                               "dispatch offsets", "dispatch scan",
                                                               "dispatch scatter", "permute rows"]),
                "dispatch_row_gather": hbm_summary(rep, nby, args.steps, ["permute rows"]),
                "reduction_bias_grads": hbm_summary(rep, nby, args.steps, ["segsum partial"]),
                "decoder_grad_elementwise": hbm_summary(rep, nby, args.steps, ["decoder grad"])},
    }
    loss = float(st.fwd["loss_mean"].item())
    res["loss_mean"] = round(loss, 5)
    del st
    torch.cuda.empty_cache()
    if not args.no_cpu:
        log("cpu oracle baseline")
        res["cpu_baseline"] = cpu_baseline(inp, args.cpu_sample, routed_by_gater=True)
    del inp
    torch.cuda.empty_cache()
    if not args.no_legs:
        res["legs"] = run_legs(args)
    print(json.dumps(res), flush=True)


def run_legs(args):
    legs = {}
    table = [("gater_fit", "gater fit", lambda: leg_gater_fit(steps=2)),
             ("gater_pca", "gater features with PCA", lambda: leg_gater_pca(steps=2)),
             ("skewed", "skewed routing", lambda: leg_skewed(steps=max(2, args.steps // 2), warmup=1)),
             ("independent", "independent decoders",
              lambda: leg_independent(steps=max(2, args.steps // 2), warmup=1)),
             ("inference", "inference tail", lambda: leg_inference(steps=max(2, args.steps // 2), warmup=1)),
             ("sgd_update", "sgd update", lambda: leg_sgd_update(steps=max(2, args.steps // 2), warmup=1)),
             ("large_assign", "large assign", lambda: leg_large_assign(args.large_chunks))]
    chosen = set(x for x in args.legs.split(",") if x)
    for key, what, run in table:
        if chosen and key not in chosen:
            continue
        log(f"leg: {what}")
        legs[key] = run()
    return legs


if __name__ == "__main__":
    main()
