"""Pins for the oracle's AdamW step."""
import numpy as np
import torch

import oracle


def test_first_step_closed_form():
    rng = np.random.default_rng(0)
    th0 = 0.02 * rng.normal(size=1000)
    g = rng.normal(size=1000) * 1e-3
    lr, wd, eps = 1e-6, 1e-2, 1e-8
    th, m, v = oracle.adamw_step(th0, g, np.zeros(1000), np.zeros(1000), 1, lr=lr,
                                 weight_decay=wd, eps=eps)
    # m_hat = g and v_hat = g^2 after one step
    want = th0 * (1 - lr * wd) - lr * g / (np.abs(g) + eps)
    # up to a few float64 ulps of rounding order
    assert np.all(np.abs(th - want) <= 1e-15 * np.abs(want))
    assert np.all(np.abs(m - 0.1 * g) <= 1e-15 * np.abs(0.1 * g))
    assert np.all(np.abs(v - 0.001 * g * g) <= 4e-15 * 0.001 * g * g)  # 1 - 0.999 != 0.001
    # the update is -lr sign(g) up to eps / |g| and the decay: a dropped term shows here
    step = th - th0 * (1 - lr * wd)
    assert np.all(np.abs(step + lr * np.sign(g)) <= lr * eps / np.abs(g) * 1.01 + 1e-21)


def test_matches_torch_adamw_over_steps():
    rng = np.random.default_rng(1)
    n = 257
    th = torch.tensor(0.02 * rng.normal(size=n), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([th], lr=1e-3, betas=(0.8, 0.95), eps=1e-6, weight_decay=0.1)
    mine = th.detach().numpy().copy()
    m = np.zeros(n)
    v = np.zeros(n)
    for t in range(1, 6):
        g = rng.normal(size=n)
        th.grad = torch.tensor(g)
        opt.step()
        mine, m, v = oracle.adamw_step(mine, g, m, v, t, lr=1e-3, beta1=0.8, beta2=0.95,
                                       eps=1e-6, weight_decay=0.1)
        assert np.abs(mine - th.detach().numpy()).max() < 1e-15
    st = opt.state[th]
    assert np.abs(m - st["exp_avg"].numpy()).max() < 1e-15
    assert np.abs(v - st["exp_avg_sq"].numpy()).max() < 1e-15


def test_zero_gradient_only_decays():
    th0 = np.linspace(-1, 1, 11)
    th, m, v = oracle.adamw_step(th0, np.zeros(11), np.zeros(11), np.zeros(11), 3,
                                 lr=0.5, weight_decay=0.1)
    assert np.allclose(th, th0 * 0.95, rtol=0, atol=1e-16)
    assert not m.any() and not v.any()


def test_grad_scale_is_a_gradient_multiplier():
    rng = np.random.default_rng(2)
    th0, g = rng.normal(size=50), rng.normal(size=50)
    a = oracle.adamw_step(th0, g, np.ones(50), np.ones(50), 4, grad_scale=0.25)
    b = oracle.adamw_step(th0, 0.25 * g, np.ones(50), np.ones(50), 4)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
