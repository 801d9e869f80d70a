"""Pins of the float64 Adam oracle (oracle/adam.py) against torch.optim.AdamW in float64 (independent
code) and closed forms. CPU only."""
import numpy as np
import pytest
import torch

from oracle import adam


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_matches_torch_adamw_over_steps(wd):
    rng = np.random.default_rng(0)
    p0 = rng.standard_normal(257)
    grads = [rng.standard_normal(257) * s for s in (1.0, 1e-3, 5.0, 1e-6, 0.2)]
    t = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.AdamW([t], lr=3e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    p, m, v = p0.copy(), np.zeros(257), np.zeros(257)
    for k, g in enumerate(grads, start=1):
        t.grad = torch.tensor(g)
        opt.step()
        p, m, v = adam.adamw_step(p, g, m, v, k, 3e-3, 0.9, 0.95, 1e-8, wd)
        np.testing.assert_allclose(p, t.detach().numpy(), rtol=1e-13, atol=1e-15)
        st = opt.state[t]
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-13, atol=1e-18)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-24)


def test_first_step_closed_form():
    # At t = 1 the bias correction makes m_hat = g and v_hat = g^2: the step is lr g / (|g| + eps).
    g = np.array([2.0, -3.0, 0.5, 0.0])
    p, m, v = adam.adamw_step(np.zeros(4), g, np.zeros(4), np.zeros(4), 1, lr=0.01, eps=1e-8)
    np.testing.assert_allclose(p, -0.01 * g / (np.abs(g) + 1e-8), rtol=1e-14)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-15)


def test_decoupled_weight_decay_only():
    # A zero gradient leaves the moments at zero, and the parameter only decays: p (1 - lr wd).
    p, m, v = adam.adamw_step(np.full(3, 4.0), np.zeros(3), np.zeros(3), np.zeros(3), 7, lr=0.1,
                              weight_decay=0.5)
    np.testing.assert_allclose(p, 4.0 * (1 - 0.05), rtol=1e-15)
    assert np.all(m == 0) and np.all(v == 0)


def test_step_must_count_from_one():
    with pytest.raises(ValueError):
        adam.adamw_step(np.zeros(1), np.zeros(1), np.zeros(1), np.zeros(1), 0, lr=0.1)
