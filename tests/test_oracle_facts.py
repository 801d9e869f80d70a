"""Pins for the float64 oracle: facts that do not come from the oracle itself.

Each test names the fact it checks. Together they are chosen so that a dropped
term, a wrong sign, a wrong index or a transposed operand in the oracle fails
at least one of them:

* W = 0 closed form (loss = ln V exactly, dH = 0, dW in closed form);
* softmax rows sum to one, so every dlogits row sums to zero and the columns
  of dW sum to zero;
* ignored tokens give zero dH rows and do not influence loss or dW;
* central finite differences of the loss (float64) against dH and dW;
* an independent library routine: torch's CPU cross_entropy with autograd;
* V = 1 and V = 2 closed forms, equal weight rows;
* invariances: a common shift of W's rows, vocabulary and token permutations;
* sum = n_valid x mean; row-block invariance; the sampled-output helpers;
* hand-derived fixtures under tests/golden/.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _case(N, H, V, seed=0, ignore=(), x_scale=1.0, w_std=0.5):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, H)) * x_scale
    W = rng.standard_normal((V, H)) * w_std
    y = rng.integers(0, V, size=N)
    y[list(ignore)] = -100
    return X, W, y


# P1: W = 0 ----------------------------------------------------------------------------

@pytest.mark.parametrize("V", [1, 2, 7, 4096])
def test_zero_weight_closed_form(V):
    N, H = 9, 5
    X, _, y = _case(N, H, V, seed=1, ignore=(2, 6))
    W = np.zeros((V, H))
    r = oracle.forward_backward(X, W, y, reduction="mean")
    n_valid = N - 2
    assert r["n_valid"] == n_valid
    assert r["loss"] == pytest.approx(math.log(V), rel=1e-15, abs=1e-15)
    assert np.all(r["dH"] == 0.0)
    valid = y != -100
    g = 1.0 / n_valid
    # dW_v = g ((1/V) sum_valid x_i - sum_{valid i: y_i = v} x_i)
    expect = np.tile(g * X[valid].sum(axis=0) / V, (V, 1))
    for i in np.nonzero(valid)[0]:
        expect[y[i]] -= g * X[i]
    np.testing.assert_allclose(r["dW"], expect, rtol=1e-13, atol=1e-15)
    rs = oracle.forward_backward(X, W, y, reduction="sum", want_grads=False)
    assert rs["loss"] == pytest.approx(n_valid * math.log(V), rel=1e-15)


# P2: dlogits rows sum to zero ------------------------------------------------------

def test_dlogits_rows_sum_to_zero():
    X, W, y = _case(12, 6, 40, seed=2, ignore=(0, 5))
    r = oracle.forward_backward(X, W, y)
    colsum = r["dW"].sum(axis=0)
    scale = np.abs(r["dW"]).sum(axis=0)
    assert np.all(np.abs(colsum) <= 1e-13 * scale)
    # The same fact seen through dH: dH = dZ W, so shifting all rows of W by c
    # adds (sum_v dZ_v) c = 0. Checked in the invariance test below.


# P3: ignored tokens ------------------------------------------------------------------

def test_ignored_tokens_have_no_effect():
    X, W, y = _case(10, 4, 13, seed=3, ignore=(1, 4, 9))
    r = oracle.forward_backward(X, W, y)
    assert np.all(r["dH"][[1, 4, 9]] == 0.0)
    assert np.all(r["token_loss"][[1, 4, 9]] == 0.0)
    X2 = X.copy()
    X2[[1, 4, 9]] = np.random.default_rng(7).standard_normal((3, 4)) * 50
    r2 = oracle.forward_backward(X2, W, y)
    assert r2["loss"] == pytest.approx(r["loss"], rel=1e-14)
    np.testing.assert_allclose(r2["dW"], r["dW"], rtol=1e-13, atol=1e-16)


def test_all_ignored_mean_is_zero():
    X, W, y = _case(6, 3, 5, seed=4, ignore=range(6))
    r = oracle.forward_backward(X, W, y, reduction="mean")
    assert r["n_valid"] == 0 and r["loss"] == 0.0
    assert np.all(r["dH"] == 0) and np.all(r["dW"] == 0)


def test_label_out_of_range_raises():
    X, W, y = _case(4, 3, 5, seed=5)
    y[2] = 5
    with pytest.raises(ValueError):
        oracle.forward_backward(X, W, y)
    y[2] = -1  # negative but not the ignore index
    with pytest.raises(ValueError):
        oracle.forward_backward(X, W, y)


# P4: central finite differences ---------------------------------------------------------

def _loss(X, W, y, reduction):
    return oracle.forward(X, W, y, reduction=reduction)["loss"]


@pytest.mark.parametrize("reduction", ["mean", "sum"])
def test_finite_differences_every_entry(reduction):
    X, W, y = _case(5, 7, 11, seed=6, ignore=(3,))
    r = oracle.forward_backward(X, W, y, reduction=reduction)
    eps = 1e-5
    for arr, grad in ((X, r["dH"]), (W, r["dW"])):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + eps
            lp = _loss(X, W, y, reduction)
            arr[idx] = old - eps
            lm = _loss(X, W, y, reduction)
            arr[idx] = old
            num[idx] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(num, grad, rtol=1e-6, atol=1e-9)


def test_finite_differences_random_directions():
    X, W, y = _case(16, 8, 33, seed=7, ignore=(0, 15))
    r = oracle.forward_backward(X, W, y)
    rng = np.random.default_rng(8)
    eps = 1e-5
    for _ in range(4):
        EX = rng.standard_normal(X.shape)
        EW = rng.standard_normal(W.shape)
        num = (_loss(X + eps * EX, W + eps * EW, y, "mean")
               - _loss(X - eps * EX, W - eps * EW, y, "mean")) / (2 * eps)
        ana = np.sum(r["dH"] * EX) + np.sum(r["dW"] * EW)
        assert num == pytest.approx(ana, rel=1e-7)


# P5: independent library routine -------------------------------------------------------

@pytest.mark.parametrize("reduction", ["mean", "sum", "none"])
@pytest.mark.parametrize("shape", [(37, 24, 101), (64, 16, 2), (8, 33, 1000)])
def test_matches_torch_cross_entropy(reduction, shape):
    N, H, V = shape
    X, W, y = _case(N, H, V, seed=N + V, ignore=(0, N // 2), x_scale=2.0)
    Xt = torch.tensor(X, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    yt = torch.tensor(y)
    L = torch.nn.functional.cross_entropy(Xt @ Wt.T, yt, ignore_index=-100, reduction=reduction)
    if reduction == "none":
        r = oracle.forward(X, W, y, reduction="none")
        np.testing.assert_allclose(r["loss"], L.detach().numpy(), rtol=1e-12, atol=1e-13)
        return
    L.backward()
    r = oracle.forward_backward(X, W, y, reduction=reduction)
    assert r["loss"] == pytest.approx(L.item(), rel=1e-12)
    np.testing.assert_allclose(r["dH"], Xt.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(r["dW"], Wt.grad.numpy(), rtol=1e-10, atol=1e-14)
    lse = torch.logsumexp(Xt @ Wt.T, dim=1).detach().numpy()
    np.testing.assert_allclose(r["lse"], lse, rtol=1e-13)


def test_matches_torch_on_tiny_workload():
    d = workloads.make_inputs("tiny_fp32")
    X = d["hidden"].double().requires_grad_(True)
    W = d["weight"].double().requires_grad_(True)
    L = torch.nn.functional.cross_entropy(X @ W.T, d["labels"], ignore_index=-100)
    L.backward()
    r = oracle.forward_backward(d["hidden"], d["weight"], d["labels"])
    assert r["loss"] == pytest.approx(L.item(), rel=1e-12)
    np.testing.assert_allclose(r["dH"], X.grad.numpy(), rtol=1e-9, atol=1e-16)
    np.testing.assert_allclose(r["dW"], W.grad.numpy(), rtol=1e-9, atol=1e-16)


# P6: closed forms ------------------------------------------------------------------------

def test_single_class_vocabulary():
    X, W, y = _case(7, 4, 1, seed=9, ignore=(2,))
    r = oracle.forward_backward(X, W, y)
    assert r["loss"] == 0.0
    assert np.all(np.abs(r["dH"]) == 0) and np.all(np.abs(r["dW"]) == 0)


def test_two_class_softplus():
    X, W, y = _case(9, 3, 2, seed=10)
    r = oracle.forward(X, W, y, reduction="none")
    Z = X @ W.T
    for i in range(9):
        d = Z[i, 1 - y[i]] - Z[i, y[i]]
        assert r["loss"][i] == pytest.approx(math.log1p(math.exp(d)), rel=1e-13)


def test_equal_weight_rows_give_log_v():
    rng = np.random.default_rng(11)
    X = rng.standard_normal((6, 5))
    W = np.tile(rng.standard_normal(5), (17, 1))
    y = rng.integers(0, 17, size=6)
    r = oracle.forward_backward(X, W, y)
    assert r["loss"] == pytest.approx(math.log(17), rel=1e-14)
    np.testing.assert_allclose(r["dH"], 0.0, atol=1e-15)


# P7: invariances ------------------------------------------------------------------------

def test_common_row_shift_of_weight():
    X, W, y = _case(11, 6, 29, seed=12, ignore=(4,))
    c = np.random.default_rng(13).standard_normal(6)
    r = oracle.forward_backward(X, W, y)
    r2 = oracle.forward_backward(X, W + c[None, :], y)
    assert r2["loss"] == pytest.approx(r["loss"], rel=1e-12)
    np.testing.assert_allclose(r2["dH"], r["dH"], rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(r2["dW"], r["dW"], rtol=1e-9, atol=1e-13)


def test_permutations():
    X, W, y = _case(13, 5, 23, seed=14, ignore=(0, 7))
    r = oracle.forward_backward(X, W, y)
    rng = np.random.default_rng(15)
    pv = rng.permutation(23)              # new id j holds old id pv[j]
    inv = np.argsort(pv)
    y2 = np.where(y == -100, -100, inv[np.where(y == -100, 0, y)])
    r2 = oracle.forward_backward(X, W[pv], y2)
    assert r2["loss"] == pytest.approx(r["loss"], rel=1e-13)
    np.testing.assert_allclose(r2["dW"], r["dW"][pv], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(r2["dH"], r["dH"], rtol=1e-12, atol=1e-15)
    pt = rng.permutation(13)
    r3 = oracle.forward_backward(X[pt], W, y[pt])
    assert r3["loss"] == pytest.approx(r["loss"], rel=1e-13)
    np.testing.assert_allclose(r3["dH"], r["dH"][pt], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(r3["dW"], r["dW"], rtol=1e-12, atol=1e-15)


# P8, P9: reductions and row blocks ---------------------------------------------------------

def test_sum_is_n_valid_times_mean():
    X, W, y = _case(20, 6, 31, seed=16, ignore=(1, 2, 3))
    rm = oracle.forward_backward(X, W, y, reduction="mean")
    rs = oracle.forward_backward(X, W, y, reduction="sum")
    assert rs["loss"] == pytest.approx(17 * rm["loss"], rel=1e-14)
    np.testing.assert_allclose(rs["dH"], 17 * rm["dH"], rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(rs["dW"], 17 * rm["dW"], rtol=1e-13, atol=1e-16)
    rn = oracle.forward(X, W, y, reduction="none")
    assert math.fsum(rn["loss"]) == pytest.approx(rs["loss"], rel=1e-14)


@pytest.mark.parametrize("r", [1, 7])
def test_row_block_invariance(r):
    X, W, y = _case(23, 6, 19, seed=17, ignore=(5,))
    full = oracle.forward_backward(X, W, y)
    blk = oracle.forward_backward(X, W, y, rows_per_block=r)
    assert blk["loss"] == pytest.approx(full["loss"], rel=1e-13)
    np.testing.assert_allclose(blk["dH"], full["dH"], rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(blk["dW"], full["dW"], rtol=1e-12, atol=1e-16)


def test_sampled_helpers_match_full_result():
    X, W, y = _case(31, 8, 57, seed=18, ignore=(3, 30))
    full = oracle.forward_backward(X, W, y)
    g, _ = oracle.token_weights(y, -100, "mean", 57)
    rows = [0, 3, 17, 30]
    lse, tl = oracle.row_stats(X, W, y, rows)
    np.testing.assert_allclose(lse, full["lse"][rows], rtol=1e-14)
    np.testing.assert_allclose(tl, full["token_loss"][rows], rtol=1e-13, atol=1e-15)
    dh = oracle.grad_hidden_rows(X, W, y, rows, g)
    np.testing.assert_allclose(dh, full["dH"][rows], rtol=1e-12, atol=1e-16)
    vids = [0, y[5], 56]
    dw = oracle.grad_weight_rows(X, W, y, vids, full["lse"], g)
    np.testing.assert_allclose(dw, full["dW"][vids], rtol=1e-12, atol=1e-16)


# P10: statistical sanity of the generator + oracle -------------------------------------------

def test_tiny_workload_loss_near_expectation():
    # E[loss] ~ ln V + sigma^2/2 with sigma^2 = H * E[x^2] * w_std^2 = 256 * 1 * 4e-4.
    d = workloads.make_inputs("tiny_fp32")
    r = oracle.forward(d["hidden"], d["weight"], d["labels"])
    assert r["n_valid"] == 256 - 13
    assert abs(r["loss"] - (math.log(4096) + 0.5 * 256 * 4e-4)) < 0.1


# Hand-derived fixtures -------------------------------------------------------------------

def test_golden_hand_derived_cases():
    with open(os.path.join(GOLDEN, "hand_derived.json")) as f:
        cases = json.load(f)["cases"]
    assert cases
    for c in cases:
        r = oracle.forward_backward(np.array(c["hidden"], float), np.array(c["weight"], float),
                                    np.array(c["labels"]), c["ignore_index"], c["reduction"])
        assert r["loss"] == pytest.approx(c["loss"], rel=1e-12), c["name"]
        np.testing.assert_allclose(r["dH"], np.array(c["dH"]), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(r["dW"], np.array(c["dW"]), rtol=1e-12, atol=1e-15)


# Generator determinism (the recipe both sides rely on) ----------------------------------------

def test_generator_is_deterministic_and_blocking_free():
    a = workloads.make_inputs("small_bf16", N=64, H=32, V=20000)
    b = workloads.make_inputs("small_bf16", N=64, H=32, V=20000)
    assert workloads.fingerprint(a) == workloads.fingerprint(b)
    # W is drawn in row blocks; one draw of the whole matrix gives the same values.
    from workloads import _streams
    rw = _streams(0)[1]
    whole = torch.from_numpy(rw.standard_normal((20000, 32)) * 0.02).to(torch.bfloat16)
    assert torch.equal(whole, a["weight"])
    assert int((a["labels"] == -100).sum()) == round(0.1 * 64)


def test_prefix_ignore_recipe():
    d = workloads.make_inputs("qwen25_7b", N=4096, H=8, V=1000)
    y = d["labels"].numpy().reshape(4, 1024)
    for row in y:
        k = int(np.argmax(row != -100)) if np.any(row != -100) else 1024
        assert np.all(row[:k] == -100) and np.all(row[k:] != -100)
        assert 0 <= k <= 307
