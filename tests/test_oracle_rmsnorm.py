"""Pins of the float64 RMSNorm + LCE oracle (oracle/rmsnorm_lce.py) against facts that do not come
from it: torch's own rms_norm with autograd in float64 (independent code), central finite
differences, the scale invariance of the normalisation, and the reduction to the plain LCE oracle.
CPU only."""
import numpy as np
import pytest
import torch

import oracle
from oracle import rmsnorm_lce as orn


def _case(N, H, V, seed, h_scale=3.0, ignore=2):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((N, H)) * h_scale + 0.5
    gamma = 1.0 + 0.3 * rng.standard_normal(H)
    W = rng.standard_normal((V, H)) * 0.4
    y = rng.integers(0, V, size=N)
    y[rng.permutation(N)[:ignore]] = -100
    return h, gamma, W, y


@pytest.mark.parametrize("reduction", ["mean", "sum"])
@pytest.mark.parametrize("eps", [1e-5, 0.3])
def test_matches_torch_rms_norm_autograd(reduction, eps):
    h, gamma, W, y = _case(9, 12, 17, seed=1)
    ref = orn.forward_backward(h, gamma, W, y, eps=eps, reduction=reduction)
    ht = torch.tensor(h, requires_grad=True)
    gt = torch.tensor(gamma, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    x = torch.nn.functional.rms_norm(ht, (12,), weight=gt, eps=eps)
    L = torch.nn.functional.cross_entropy(x @ Wt.T, torch.tensor(y), ignore_index=-100, reduction=reduction)
    L.backward()
    assert abs(L.item() - ref["loss"]) <= 1e-12 * max(1.0, abs(ref["loss"]))
    np.testing.assert_allclose(ref["x"], x.detach().numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(ref["dh"], ht.grad.numpy(), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(ref["dgamma"], gt.grad.numpy(), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(ref["dW"], Wt.grad.numpy(), rtol=1e-9, atol=1e-13)


def test_finite_differences():
    h, gamma, W, y = _case(5, 6, 7, seed=2, ignore=1)
    eps, d = 1e-3, 1e-6
    ref = orn.forward_backward(h, gamma, W, y, eps=eps)
    loss = lambda hh, gg: orn.forward(hh, gg, W, y, eps=eps)["loss"]
    for i in range(5):
        for j in range(6):
            hp, hm = h.copy(), h.copy()
            hp[i, j] += d
            hm[i, j] -= d
            fd = (loss(hp, gamma) - loss(hm, gamma)) / (2 * d)
            assert abs(fd - ref["dh"][i, j]) <= 1e-6 * max(1.0, abs(fd)), (i, j)
    for j in range(6):
        gp, gm = gamma.copy(), gamma.copy()
        gp[j] += d
        gm[j] -= d
        fd = (loss(h, gp) - loss(h, gm)) / (2 * d)
        assert abs(fd - ref["dgamma"][j]) <= 1e-6 * max(1.0, abs(fd)), j


def test_scale_invariance_without_eps():
    # With eps = 0 the normalised rows do not depend on the scale of h: the loss is unchanged,
    # d h scales by 1/alpha, and every row's gradient is orthogonal to the row.
    h, gamma, W, y = _case(6, 10, 13, seed=3)
    a = orn.forward_backward(h, gamma, W, y, eps=0.0)
    b = orn.forward_backward(7.5 * h, gamma, W, y, eps=0.0)
    assert abs(a["loss"] - b["loss"]) <= 1e-12 * abs(a["loss"])
    np.testing.assert_allclose(b["dh"] * 7.5, a["dh"], rtol=1e-9, atol=1e-14)
    np.testing.assert_allclose(b["dgamma"], a["dgamma"], rtol=1e-9, atol=1e-14)
    np.testing.assert_allclose(np.sum(a["dh"] * h, axis=1), 0.0, atol=1e-12)


def test_reduces_to_plain_lce_on_unit_rms_rows():
    # Rows of mean square 1, gamma = 1, eps = 0: x = h, so loss, dW and dX are the LCE oracle's.
    rng = np.random.default_rng(4)
    g = rng.standard_normal((8, 16))
    h = g / np.sqrt(np.mean(g * g, axis=1, keepdims=True))
    W = rng.standard_normal((21, 16)) * 0.5
    y = rng.integers(0, 21, size=8)
    a = orn.forward_backward(h, np.ones(16), W, y, eps=0.0)
    b = oracle.forward_backward(h, W, y)
    np.testing.assert_allclose(a["x"], h, rtol=1e-13)
    assert abs(a["loss"] - b["loss"]) <= 1e-13 * abs(b["loss"])
    np.testing.assert_allclose(a["dW"], b["dW"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(a["dX"], b["dH"], rtol=1e-12, atol=1e-15)


def test_constant_rows_closed_form():
    # A row of equal entries c normalises to gamma * c / sqrt(c^2 + eps).
    h = np.full((3, 5), 2.0)
    h[1] = -0.5
    gamma = np.arange(1.0, 6.0)
    x, r = orn.rms_normalise(h, gamma, 0.25)
    for i, c in enumerate([2.0, -0.5, 2.0]):
        np.testing.assert_allclose(x[i], gamma * c / np.sqrt(c * c + 0.25), rtol=1e-14)
        assert abs(r[i] - 1.0 / np.sqrt(c * c + 0.25)) <= 1e-15


def test_zero_gamma():
    # gamma = 0: x = 0, so the loss is ln V and no gradient reaches h; d gamma is still nonzero.
    h, _, W, y = _case(7, 8, 11, seed=5, ignore=0)
    out = orn.forward_backward(h, np.zeros(8), W, y, eps=1e-5)
    assert abs(out["loss"] - np.log(11)) <= 1e-13
    assert np.all(out["dh"] == 0.0)
    assert np.any(out["dgamma"] != 0.0)


def test_sampled_rows_match_full_result():
    h, gamma, W, y = _case(11, 9, 15, seed=6)
    full = orn.forward_backward(h, gamma, W, y, eps=1e-4)
    g, _ = oracle.token_weights(y, -100, "mean", 15)
    rows = [0, 3, 7, 10]
    np.testing.assert_allclose(orn.grad_hidden_rows(h, gamma, W, y, rows, g, eps=1e-4), full["dh"][rows],
                               rtol=1e-11, atol=1e-15)
