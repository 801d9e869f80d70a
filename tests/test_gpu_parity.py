"""Parity of the HIP path (through the C ABI) with the float64 oracle, on the same seeded inputs.

Tolerances: loss relative error <= 1e-3 and max|dH - ref|, max|dW - ref| <= 2e-2 * max|ref| for
bf16 operands with fp32 accumulation; 1e-5 for the fp32 path; for fp16 (unit roundoff 2^-11, eight
times finer than bf16's) 1e-3 and 5e-3 * max|ref|, the same margin of about ten unit roundoffs.
The fp32 gradients are sums of K = V (dH) or N (dW) rounded fp32 terms, whose rounding grows like
sqrt(K) 2^-24: their bound is max(1e-5, 2 sqrt(K) 2^-24), which is 1e-5 up to K = 7036 (every fp32
case here but the half-million vocabulary one; 8.4e-5 there, where sequential fp32 sums of that
case's exact dZ in the library's six vocabulary splits already differ from float64 by 3.4e-5).

Small cases run the whole oracle (several tiles, ragged tails, several chunks, split-K). The
full-size workloads compare the loss and every token's log-sum-exp with values the oracle wrote
(tests/golden/make_full_size.py), sampled rows of dH and dW that the oracle recomputes one by one,
and properties that hold at any size (dW columns sum to zero, ignored tokens give zero dH rows,
bitwise determinism).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL = {"bf16": (1e-3, 2e-2), "fp16": (1e-3, 5e-3), "fp32": (1e-5, 1e-5)}


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return m


def _to_dev(d):
    return (d["hidden"].cuda(), d["weight"].cuda(), d["labels"].cuda())


def _rel_max_err(got, ref):
    ref = np.asarray(ref, dtype=np.float64)
    got = np.asarray(got, dtype=np.float64)
    scale = np.max(np.abs(ref))
    err = np.max(np.abs(got - ref))
    return err / scale if scale > 0 else err


def _grad_tol(dtype, N, V):
    tol = TOL[dtype][1]
    if dtype == "fp32":
        tol = max(tol, 2.0 * np.sqrt(max(N, V)) * 2.0 ** -24)
    return tol


def _check_full(lce, d, reduction=None, chunk_tokens=0):
    reduction = reduction or d["reduction"]
    tol_loss = TOL[d["dtype"]][0]
    tol_grad = _grad_tol(d["dtype"], d["N"], d["V"])
    X, W, y = _to_dev(d)
    print(f"case {d['name']} N={d['N']} H={d['H']} V={d['V']} {d['dtype']} {reduction} chunk={chunk_tokens}",
          flush=True)
    loss, dH, dW = lce.forward_backward(X, W, y, d["ignore_index"], reduction, chunk_tokens=chunk_tokens)
    torch.cuda.synchronize()
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], reduction)
    L = loss.item()
    if ref["loss"] == 0.0:
        # Exactly zero in exact arithmetic (V = 1, or no valid token): fp32 rounding only.
        assert abs(L) <= 1e-5, L
    else:
        assert abs(L - ref["loss"]) <= tol_loss * abs(ref["loss"]), (L, ref["loss"])
    eh = _rel_max_err(dH.float().cpu().numpy(), ref["dH"])
    ew = _rel_max_err(dW.float().cpu().numpy(), ref["dW"])
    assert eh <= tol_grad, f"dH rel max err {eh}"
    assert ew <= tol_grad, f"dW rel max err {ew}"
    ignored = (d["labels"] == d["ignore_index"]).numpy()
    if ignored.any():
        assert torch.all(dH[torch.from_numpy(ignored).cuda()] == 0)
    return loss, dH, dW


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16"])
def test_configs_against_full_oracle(lce, name):
    _check_full(lce, workloads.make_inputs(name))


RAGGED = [
    # (N, H, V, dtype, chunk_tokens)
    (37, 72, 1000, "bf16", 0),
    (1, 64, 128, "bf16", 0),
    (300, 136, 4099, "bf16", 64),
    (513, 264, 2050, "bf16", 128),
    (129, 8, 300, "bf16", 0),
    (700, 520, 257, "bf16", 0),
    (64, 1024, 33000, "bf16", 0),
    (37, 72, 1000, "fp32", 0),
    (300, 132, 2049, "fp32", 64),
    (260, 4, 129, "fp32", 0),
    (37, 72, 1000, "fp16", 0),
    (300, 136, 4099, "fp16", 64),
    (513, 264, 2050, "fp16", 128),
    (64, 1024, 33000, "fp16", 0),
    # A vocabulary of a million ids (3907 tile rows, ragged), and eleven chunks (ten dW accumulations).
    (48, 64, 1000003, "bf16", 0),
    (40, 32, 500009, "fp32", 0),
    (700, 72, 1000, "bf16", 64),
]


@pytest.mark.parametrize("N,H,V,dtype,chunk", RAGGED)
def test_ragged_shapes(lce, N, H, V, dtype, chunk):
    d = workloads.random_case(N, H, V, dtype=dtype, seed=N + H + V, x_scale=1.0, w_std=0.5)
    _check_full(lce, d, chunk_tokens=chunk)


def _with_extreme_tokens(d, tokens):
    """Sets, for each (token, alpha), a label and that label's weight row so that the token's
    target logit is alpha (x . w_y = alpha, up to rounding): a large negative alpha gives the token
    a loss far above the others, a large positive one a target far above every other logit."""
    X = d["hidden"].double()
    W = d["weight"].double().clone()
    y = d["labels"].clone()
    for k, (i, alpha) in enumerate(tokens):
        lab = (17 * k + 5) % d["V"]
        y[i] = lab
        W[lab] = alpha * X[i] / float(X[i] @ X[i])
    d = dict(d)
    d["weight"], d["labels"] = W.to(d["weight"].dtype), y
    return d


# Losses of 75 (exp(z - z_target) up to e^75: finite, but above the 60 that the target-referenced
# path accepts) and 120 (exp overflows fp32): the chunk is redone with slice-maximum references.
# A target logit of +100 leaves every other exp(z - z_target) below fp32's range (zero or
# subnormal), where p is that small too. Several chunks, only some of them falling back.
@pytest.mark.parametrize("dtype", ["bf16", "fp32", "fp16"])
@pytest.mark.parametrize("tokens,chunk", [
    ([(5, -75.0)], 0),
    ([(5, -120.0)], 0),
    ([(3, 100.0), (40, 90.0)], 0),
    ([(200, -80.0), (3, 100.0)], 64),
])
def test_extreme_target_logits(lce, dtype, tokens, chunk):
    d = workloads.random_case(300, 64, 300, dtype=dtype, seed=11, w_std=0.3)
    _check_full(lce, _with_extreme_tokens(d, tokens), chunk_tokens=chunk)


@pytest.mark.parametrize("dtype", ["bf16", "fp32", "fp16"])
def test_label_outside_vocabulary(lce, dtype):
    # Reading A4: a non-ignored label outside [0, V) cannot be reported by the call; that token's
    # loss is NaN (so is the reduced loss) and the gradients stay finite. bf16 and fp32 drop the
    # token from the gradients entirely: with the sum, they equal the oracle's with it ignored.
    d = workloads.random_case(150, 64, 700, dtype=dtype, seed=21, w_std=0.3)
    y = d["labels"].clone()
    y[7], y[100] = d["V"] + 3, -5
    X, W = d["hidden"].cuda(), d["weight"].cuda()
    loss, dH, dW = lce.forward_backward(X, W, y.cuda(), d["ignore_index"], "sum", chunk_tokens=64)
    torch.cuda.synchronize()
    assert torch.isnan(loss).item()
    assert torch.isfinite(dH.float()).all() and torch.isfinite(dW.float()).all()
    if dtype != "fp16":
        y_ref = y.clone()
        y_ref[7] = y_ref[100] = d["ignore_index"]
        ref = oracle.forward_backward(d["hidden"], d["weight"], y_ref, d["ignore_index"], "sum")
        tol = TOL[dtype][1]
        assert _rel_max_err(dH.float().cpu().numpy(), ref["dH"]) <= tol
        assert _rel_max_err(dW.float().cpu().numpy(), ref["dW"]) <= tol
        assert torch.all(dH[7] == 0) and torch.all(dH[100] == 0)


@pytest.mark.parametrize("reduction", ["mean", "sum"])
def test_reductions(lce, reduction):
    d = workloads.random_case(200, 96, 3001, seed=3, w_std=0.3)
    _check_full(lce, d, reduction=reduction, chunk_tokens=64)


@pytest.mark.parametrize("reduction", ["mean", "sum"])
def test_fp16_large_vocabulary(lce, reduction):
    # Llama-like inputs at a size the oracle finishes in seconds. With the mean, g p is ~3e-8 here,
    # below fp16's smallest subnormal: this is the case the fp16 storage scales exist for.
    d = workloads.make_inputs("llama3_8b", seed=1, N=1024, H=1024, V=32768, dtype="fp16")
    _check_full(lce, d, reduction=reduction, chunk_tokens=256)


def test_fp16_edge_cases(lce):
    d = workloads.random_case(70, 32, 500, dtype="fp16", seed=5, ignore_frac=1.0)
    loss, dH, dW = _check_full(lce, d)
    assert loss.item() == 0.0 and torch.all(dH == 0) and torch.all(dW == 0)
    d = workloads.random_case(100, 64, 3000, dtype="fp16", seed=8)
    d["weight"] = torch.zeros_like(d["weight"])
    X, W, y = _to_dev(d)
    loss, dH, dW = lce.forward_backward(X, W, y)
    assert abs(loss.item() - np.log(3000)) <= 1e-6 * np.log(3000)
    assert torch.all(dH == 0)
    tl, lse = lce.forward(X, W, y, reduction="none", return_lse=True)
    assert torch.allclose(lse, torch.full_like(lse, float(np.log(3000))), rtol=1e-6)


def test_vocab_of_one_and_two(lce):
    for V in (1, 2):
        d = workloads.random_case(50, 16, V, seed=V, w_std=1.0)
        _check_full(lce, d)


def test_all_tokens_ignored(lce):
    d = workloads.random_case(70, 32, 500, seed=5, ignore_frac=1.0)
    loss, dH, dW = _check_full(lce, d)
    assert loss.item() == 0.0 and torch.all(dH == 0) and torch.all(dW == 0)


def test_no_token_ignored_and_custom_ignore_index(lce):
    d = workloads.random_case(90, 40, 700, seed=6, ignore_frac=0.0)
    _check_full(lce, d)
    d = workloads.random_case(90, 40, 700, seed=7, ignore_frac=0.3, ignore_index=3)
    _check_full(lce, d)


def test_zero_weight_gives_log_v(lce):
    d = workloads.random_case(100, 64, 3000, seed=8)
    d["weight"] = torch.zeros_like(d["weight"])
    X, W, y = _to_dev(d)
    loss, dH, dW = lce.forward_backward(X, W, y)
    assert abs(loss.item() - np.log(3000)) <= 1e-6 * np.log(3000)
    assert torch.all(dH == 0)


def test_chunk_size_invariance(lce):
    d = workloads.random_case(512, 128, 5000, seed=9, w_std=0.3)
    X, W, y = _to_dev(d)
    outs = [lce.forward_backward(X, W, y, chunk_tokens=c) for c in (64, 192, 0, 512)]
    ref = outs[-1]
    for o in outs[:-1]:
        assert abs(o[0].item() - ref[0].item()) <= 1e-5 * abs(ref[0].item())
        assert _rel_max_err(o[1].float().cpu().numpy(), ref[1].float().cpu().numpy()) <= 1e-2
        assert _rel_max_err(o[2].float().cpu().numpy(), ref[2].float().cpu().numpy()) <= 1e-2


def test_forward_only_and_lse(lce):
    d = workloads.random_case(333, 200, 7001, seed=10, w_std=0.3)
    X, W, y = _to_dev(d)
    ref = oracle.forward(d["hidden"], d["weight"], d["labels"], reduction="none")
    tl, lse = lce.forward(X, W, y, reduction="none", return_lse=True)
    np.testing.assert_allclose(lse.cpu().numpy(), ref["lse"], rtol=1e-4)
    np.testing.assert_allclose(tl.cpu().numpy(), ref["token_loss"], rtol=2e-3, atol=2e-3)
    for red in ("mean", "sum"):
        r = oracle.forward(d["hidden"], d["weight"], d["labels"], reduction=red)
        L = lce.forward(X, W, y, reduction=red).item()
        assert abs(L - r["loss"]) <= 1e-3 * abs(r["loss"])


def test_deterministic(lce):
    d = workloads.random_case(600, 256, 9000, seed=11)
    X, W, y = _to_dev(d)
    a = lce.forward_backward(X, W, y, chunk_tokens=128)
    b = lce.forward_backward(X, W, y, chunk_tokens=128)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1]) and torch.equal(a[2], b[2])


def test_autograd_function(lce):
    d = workloads.random_case(64, 32, 900, seed=12, w_std=0.5)
    X, W, y = _to_dev(d)
    X.requires_grad_(True)
    W.requires_grad_(True)
    loss = lce.linear_cross_entropy(X, W, y)
    (3.0 * loss).backward()
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"])
    assert _rel_max_err(X.grad.float().cpu().numpy(), 3.0 * ref["dH"]) <= 2e-2
    assert _rel_max_err(W.grad.float().cpu().numpy(), 3.0 * ref["dW"]) <= 2e-2


# ---- full-size workloads ---------------------------------------------------------------------

FULL = ["llama3_8b", "qwen25_7b", "mistral_large"]


def _golden(name):
    with open(os.path.join(GOLDEN, f"{name}_seed0.json")) as f:
        meta = json.load(f)
    arrs = np.load(os.path.join(GOLDEN, f"{name}_seed0.npz"))
    return meta, arrs["lse"], arrs["token_loss"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_sampled(lce, name):
    meta, lse_ref, tl_ref = _golden(name)
    d = workloads.make_inputs(name, seed=0)
    assert workloads.fingerprint(d) == meta["fingerprint"], "generator output changed"
    X, W, y = _to_dev(d)
    print(f"full-size {name}", flush=True)
    loss, dH, dW = lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"])
    torch.cuda.synchronize()
    L = loss.item()
    assert abs(L - meta["loss"]) <= 1e-3 * abs(meta["loss"]), (L, meta["loss"])

    labels = d["labels"].numpy()
    valid = labels != d["ignore_index"]
    g, n_valid = oracle.token_weights(labels, d["ignore_index"], d["reduction"], d["V"])
    assert n_valid == meta["n_valid"]
    X64 = d["hidden"].double().numpy()
    W64 = d["weight"].double().numpy()

    rng = np.random.default_rng(0)
    rows = sorted(set([0, d["N"] - 1] + list(rng.choice(d["N"], 6, replace=False))
                      + [int(np.nonzero(~valid)[0][0])]))
    dh_ref = oracle.grad_hidden_rows(X64, W64, labels, rows, g, d["ignore_index"])
    dh_got = dH[torch.tensor(rows).cuda()].float().cpu().numpy()
    assert _rel_max_err(dh_got, dh_ref) <= 2e-2

    counts = np.bincount(labels[valid], minlength=d["V"])
    ids = sorted(set([0, int(np.argmax(counts)), d["V"] - 1, int(np.argmin(counts))]
                     + list(rng.choice(d["V"], 4, replace=False))))
    dw_ref = oracle.grad_weight_rows(X64, W64, labels, ids, lse_ref, g, d["ignore_index"])
    dw_got = dW[torch.tensor(ids).cuda()].float().cpu().numpy()
    assert _rel_max_err(dw_got, dw_ref) <= 2e-2
    for k in range(len(ids)):  # every sampled row also against its own scale
        assert _rel_max_err(dw_got[k], dw_ref[k]) <= 2e-2, ids[k]

    # Properties at full size.
    col = dW.float().sum(dim=0)
    scale = dW.float().abs().sum(dim=0)
    assert torch.all(col.abs() <= 2e-2 * scale + 1e-12)
    assert torch.all(dH[torch.from_numpy(~valid).cuda()] == 0)
    assert torch.isfinite(dH.float()).all() and torch.isfinite(dW.float()).all()
    loss2, dH2, dW2 = lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"])
    assert torch.equal(loss, loss2) and torch.equal(dH, dH2) and torch.equal(dW, dW2)


@pytest.mark.parametrize("name", FULL)
def test_full_size_forward_lse(lce, name):
    meta, lse_ref, tl_ref = _golden(name)
    d = workloads.make_inputs(name, seed=0)
    X, W, y = _to_dev(d)
    tl, lse = lce.forward(X, W, y, d["ignore_index"], "none", return_lse=True)
    np.testing.assert_allclose(lse.cpu().numpy(), lse_ref, rtol=1e-4)
    np.testing.assert_allclose(tl.cpu().numpy(), tl_ref, rtol=2e-3, atol=2e-3)
    L = lce.forward(X, W, y, d["ignore_index"], d["reduction"]).item()
    assert abs(L - meta["loss"]) <= 1e-3 * abs(meta["loss"])
