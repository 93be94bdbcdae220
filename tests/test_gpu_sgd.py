"""The SGD step (Section 4.2) on the HIP path: four steps against the oracle (fp64, same fp32
inputs) with and without momentum, at a ragged size and a large one; the bf16 copy is the
rounding of the fp32 result, bit for bit; and in a whole training step (forward, backward,
update of every expert and decoder parameter) a small step lowers the loss on the batch."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_1704_06363_amd import hmoe
from paper_1704_06363_amd import workloads as W
from tests.parity import assert_close, np64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("count,momentum", [(1003, 0.0), (1003, 0.9), (12_582_917, 0.9)])
def test_sgd_matches_oracle(count, momentum):
    g0 = torch.Generator(device="cuda").manual_seed(count)
    w = torch.randn(count, device="cuda", generator=g0) * 0.02
    v = torch.zeros(count, device="cuda") if momentum > 0 else None
    lo = torch.empty(count, dtype=torch.bfloat16, device="cuda")
    wr, vr = np64(w), None
    for step in range(4):
        g = torch.randn(count, device="cuda", generator=g0) * 1e-3
        hmoe.sgd_step(w, g, lr=0.1, weight_decay=1e-4, momentum=momentum, v=v, w_lo=lo)
        if momentum > 0:
            wr, vr = O.sgd_step(wr, np64(g), 0.1, 1e-4, momentum, vr)
        else:
            wr = O.sgd_step(wr, np64(g), 0.1, 1e-4)
        assert_close(w, wr, 1e-6, f"w after step {step}")
        if momentum > 0:
            assert_close(v, vr, 1e-6, f"v after step {step}")
        assert torch.equal(lo, w.to(torch.bfloat16))


def test_training_step_lowers_the_loss():
    inp = W.balanced_inputs(device="cuda", seed=4, n=4096, d=256, h=512, o=128, V=2000, K=4, bias=True)
    p = inp["params"]
    master = {k: v.float().clone() for k, v in p.items()}
    a, _ = hmoe.kmeans_assign(inp["X"], inp["C"])
    dd = hmoe.moe_dispatch(a, 4, rows=inp["X"])
    rp = torch.as_tensor(inp["row_ptr"]).cuda()
    tg = torch.as_tensor(inp["tag"]).cuda()
    args = (dd["rows_sorted"], dd["offsets"], dd["perm"], rp, tg)
    f0 = hmoe.moe_forward(p, *args, save_logits=True)
    g = hmoe.moe_backward(p, dd["rows_sorted"], dd["offsets"], dd["perm"], dd["inv"], rp, tg, f0["H1_sorted"],
                          f0["H"], f0["lse"], logits=f0["logits"], logit_anchor=f0["logit_anchor"])
    loss0 = f0["loss_mean"].item()
    for k in p:
        hmoe.sgd_step(master[k], g["d" + k], lr=0.5, weight_decay=1e-4, w_lo=p[k])
    f1 = hmoe.moe_forward(p, *args)
    assert f1["loss_mean"].item() < loss0
