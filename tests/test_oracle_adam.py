"""Pins for the oracle's Adam step (the dense update of the embedding and
CTR models): torch.optim.Adam in float64 over several steps, the first step's
closed form lr * g / (|g| + eps'), a zero gradient leaving parameters alone,
and the step-decayed learning rate of section 7.2."""
import numpy as np
import torch

from oracle import oracle


def test_adam_matches_torch_optim_over_steps():
    rng = np.random.default_rng(0)
    p0 = rng.standard_normal(257)
    p = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    mine, m, v = p0.copy(), np.zeros(257), np.zeros(257)
    for t in range(1, 6):
        g = rng.standard_normal(257)
        p.grad = torch.tensor(g)
        opt.step()
        mine, m, v = oracle.adam(mine, g, m, v, lr=1e-3, t=t)
        assert np.abs(mine - p.detach().numpy()).max() < 1e-15


def test_adam_first_step_closed_form_and_zero_gradient():
    rng = np.random.default_rng(1)
    g = rng.standard_normal(64)
    g[5] = 0.0
    p0 = rng.standard_normal(64)
    p, m, v = oracle.adam(p0, g, np.zeros(64), np.zeros(64), lr=0.01, t=1)
    # m_hat = g and v_hat = g^2 after one step: the move is lr * g / (|g| + eps)
    assert np.allclose(p0 - p, 0.01 * g / (np.abs(g) + 1e-8), rtol=1e-12, atol=0)
    assert p[5] == p0[5] and m[5] == 0.0 and v[5] == 0.0


def test_paper_learning_rate_schedule():
    assert oracle.paper_lr(1) == 1e-3 and oracle.paper_lr(24000) == 1e-3
    assert abs(oracle.paper_lr(24001) - 9e-4) < 1e-18
    assert abs(oracle.paper_lr(48001) - 1e-3 * 0.81) < 1e-18
