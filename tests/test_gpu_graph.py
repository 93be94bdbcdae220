"""The routed step is asynchronous and allocation-free inside the library, so it can be captured
in a HIP graph: replays (with other work and synchronisations in between) give bit-identical
results to the eager step, every time.  The kernels are deterministic, so exact equality is the
bar."""
import numpy as np
import pytest
import torch

from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W

pytestmark = pytest.mark.gpu


def _buffers(inp):
    s = inp["shape"]
    n, d, h, o, V, K = s["n"], s["d"], s["h"], s["o"], s["V"], s["K"]
    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    z = lambda *shape, dt: torch.empty(*shape, dtype=dt, device="cuda")  # noqa: E731
    disp = {"counts": z(K, dt=i32), "offsets": z(K + 1, dt=i32), "perm": z(n, dt=i32), "inv": z(n, dt=i32),
            "rows_sorted": z(n, d, dt=bf)}
    fwd = {"H1_sorted": z(n, h, dt=bf), "H": z(n, o, dt=bf), "lse": z(n, dt=f32), "loss": z(n, dt=f32),
           "loss_mean": z(1, dt=f32), "logits": z(n, V, dt=bf),
           "logit_anchor": z(*hmoe.anchor_shape(n, V), dt=f32)}
    grads = {"dW1": z(K, h, d, dt=f32), "db1": z(K, h, dt=f32), "dW2": z(K, o, h, dt=f32), "db2": z(K, o, dt=f32),
             "dD": z(V, o, dt=f32), "dbD": z(V, dt=f32), "dX": z(n, d, dt=bf)}
    prm = hmoe.make_params(inp["params"])
    need = max(hmoe.moe_workspace(prm, n), hmoe.moe_dispatch_workspace(n, K),
               hmoe.kmeans_assign_workspace(n, d, K, bf))
    return {"ids": z(n, dt=i32), "md": z(n, dt=f32), "disp": disp, "fwd": fwd, "grads": grads,
            "ws": torch.empty(need, dtype=torch.uint8, device="cuda")}


def _step(inp, b, rp, tg):
    p = inp["params"]
    hmoe.kmeans_assign(inp["X"], inp["C"], assign=b["ids"], min_dist=b["md"], ws=b["ws"])
    dd = b["disp"]
    hmoe.moe_dispatch(b["ids"], inp["shape"]["K"], rows=inp["X"], out=dd, ws=b["ws"])
    f = hmoe.moe_forward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], rp, tg, out=b["fwd"], ws=b["ws"])
    hmoe.moe_backward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], rp, tg, f["H1_sorted"], f["H"],
                      f["lse"], out=b["grads"], ws=b["ws"], logits=f["logits"], logit_anchor=f["logit_anchor"])


def _snapshot(b):
    out = {"ids": b["ids"].clone(), "md": b["md"].clone()}
    for grp in ("disp", "fwd", "grads"):
        for k, v in b[grp].items():
            out[grp + "." + k] = v.clone()
    return out


def test_captured_step_replays_bit_identical():
    # several 256-wide tiles with ragged tails, K = 5 experts, biases on
    inp = W.balanced_inputs(device="cuda", seed=7, n=1100, d=256, h=384, o=136, V=1000, K=5, bias=True)
    rp = torch.as_tensor(inp["row_ptr"]).cuda()
    tg = torch.as_tensor(inp["tag"]).cuda()
    b = _buffers(inp)
    _step(inp, b, rp, tg)
    torch.cuda.synchronize()
    eager = _snapshot(b)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # warm-up on the capture stream
        _step(inp, b, rp, tg)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(inp, b, rp, tg)
    for rep in range(3):
        for t in b["grads"].values():  # scribble over the outputs between replays
            t.fill_(float("nan")) if t.is_floating_point() else t.fill_(-1)
        junk = torch.randn(1 << 20, device="cuda").sum()  # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(b)
        for k, v in eager.items():
            assert torch.equal(got[k], v), (rep, k)
        del junk


def test_captured_inference_tail_and_update_replay_bit_identical():
    # t_m with values, the p@m / q@m counts and an SGD step with momentum and a bf16 copy, all
    # captured in one graph; SGD works in place, so every replay starts from restored weights
    g = torch.Generator(device="cpu").manual_seed(11)
    n, V, m, S = 700, 3000, 10, 5000
    L = (torch.randn(n, V, generator=g) * 3).to(torch.bfloat16).cuda()
    rp, tg = W.zipf_labels(n, V, 8, seed=12)
    rp_t, tg_t = torch.as_tensor(rp).cuda(), torch.as_tensor(tg).cuda()
    qs, qt = W.q_draws(rp, tg, S, seed=13)
    qs_t, qt_t = torch.as_tensor(qs).cuda(), torch.as_tensor(qt).cuda()
    w0 = torch.randn(100_003, generator=g).cuda()
    gr = torch.randn(100_003, generator=g).cuda()
    v0 = torch.randn(100_003, generator=g).cuda()
    bufs = {"idx": torch.empty(n, m, dtype=torch.int32, device="cuda"),
            "val": torch.empty(n, m, dtype=torch.float32, device="cuda"),
            "hits": torch.empty(2, m, dtype=torch.int64, device="cuda"),
            "w": w0.clone(), "v": v0.clone(), "wlo": torch.empty(100_003, dtype=torch.bfloat16, device="cuda")}

    def run():
        hmoe.topm(L, m, out=bufs, want_values=True)
        hmoe.topm_hits(bufs["idx"], rp_t, tg_t, qs_t, qt_t, out=bufs["hits"])
        hmoe.sgd_step(bufs["w"], gr, lr=0.05, weight_decay=1e-4, momentum=0.9, v=bufs["v"], w_lo=bufs["wlo"])

    run()
    torch.cuda.synchronize()
    eager = {k: t.clone() for k, t in bufs.items()}
    bufs["w"].copy_(w0)
    bufs["v"].copy_(v0)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    for rep in range(3):
        bufs["w"].copy_(w0)
        bufs["v"].copy_(v0)
        for k in ("idx", "hits"):
            bufs[k].fill_(-1)
        bufs["val"].fill_(float("nan"))
        bufs["wlo"].fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in eager.items():
            assert torch.equal(bufs[k], v), (rep, k)
