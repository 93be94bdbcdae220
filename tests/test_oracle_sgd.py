"""Pins for the oracle's SGD step (Section 4.2: weight decay 1e-4, momentum 0.9 for the trunk,
no momentum for the experts): PyTorch's torch.optim.SGD on fp64 CPU tensors (an independent
implementation of the same update), closed forms, and a hand-worked three-step recursion."""
import numpy as np
import pytest
import torch


@pytest.mark.parametrize("momentum", [0.0, 0.9])
def test_matches_torch_sgd_over_steps(orc, momentum):
    rs = np.random.default_rng(0)
    w0 = rs.normal(size=(7, 13))
    grads = [rs.normal(size=(7, 13)) for _ in range(4)]
    p = torch.nn.Parameter(torch.tensor(w0))
    opt = torch.optim.SGD([p], lr=0.1, momentum=momentum, weight_decay=1e-4)
    w, v = w0, None
    for g in grads:
        p.grad = torch.tensor(g)
        opt.step()
        if momentum > 0:
            w, v = orc.sgd_step(w, g, 0.1, 1e-4, momentum, v)
        else:
            w = orc.sgd_step(w, g, 0.1, 1e-4)
        np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-15, atol=1e-15)


def test_closed_forms(orc):
    w = np.array([1.0, -2.0, 0.5])
    g = np.array([0.5, 0.25, -1.0])
    assert np.array_equal(orc.sgd_step(w, g, 0.0, 1e-4), w)          # lr = 0
    assert np.array_equal(orc.sgd_step(w, g, 0.5), w - 0.5 * g)      # plain SGD
    # weight decay alone shrinks the weights by (1 - lr wd)
    np.testing.assert_allclose(orc.sgd_step(w, np.zeros(3), 0.1, 0.5), w * (1 - 0.05), rtol=1e-15)


def test_momentum_recursion_by_hand(orc):
    # w = 1, g = 1 each step, lr = 0.1, momentum 0.5, no decay:
    # v1 = 1, w1 = 0.9; v2 = 1.5, w2 = 0.75; v3 = 1.75, w3 = 0.575
    w, v = np.array([1.0]), None
    for want_v, want_w in ((1.0, 0.9), (1.5, 0.75), (1.75, 0.575)):
        w, v = orc.sgd_step(w, np.array([1.0]), 0.1, 0.0, 0.5, v)
        assert np.isclose(v[0], want_v, rtol=1e-15) and np.isclose(w[0], want_w, rtol=1e-15)
