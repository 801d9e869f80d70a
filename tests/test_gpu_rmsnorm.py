"""Parity of the fused RMSNorm + LCE entry points (lce_rmsnorm_forward[_backward], through the C ABI)
with the float64 oracle (oracle/rmsnorm_lce.py), on the same seeded inputs.

Tolerances are those of the plain step (tests/test_gpu_parity.py): loss relative <= 1e-3; gradients
max|got - ref| <= 2e-2 (bf16), 5e-3 (fp16), 1e-5 (fp32) times max|ref|. The normalised rows x and
dX pass through the input dtype once each before the Jacobian, inside that budget.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads
from oracle import rmsnorm_lce as orn

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL = {"bf16": (1e-3, 2e-2), "fp16": (1e-3, 5e-3), "fp32": (1e-5, 1e-5)}


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return m


def _dev(d):
    return tuple(d[k].cuda() for k in ("hidden", "gamma", "weight", "labels"))


def _rel(got, ref):
    ref = np.asarray(ref, dtype=np.float64)
    got = np.asarray(got, dtype=np.float64)
    scale = np.max(np.abs(ref))
    err = np.max(np.abs(got - ref))
    return err / scale if scale > 0 else err


def _check(lce, d, reduction=None, chunk_tokens=0):
    reduction = reduction or d["reduction"]
    tl, tg = TOL[d["dtype"]]
    h, g, W, y = _dev(d)
    print(f"case {d['name']} N={d['N']} H={d['H']} V={d['V']} {d['dtype']} {reduction} chunk={chunk_tokens}",
          flush=True)
    loss, dh, dg, dW = lce.rmsnorm_forward_backward(h, g, W, y, d["eps"], d["ignore_index"], reduction,
                                                    chunk_tokens)
    torch.cuda.synchronize()
    ref = orn.forward_backward(d["hidden"], d["gamma"], d["weight"], d["labels"], d["eps"], d["ignore_index"],
                               reduction)
    assert abs(loss.item() - ref["loss"]) <= tl * abs(ref["loss"]), (loss.item(), ref["loss"])
    for name, got, want in (("dh", dh, ref["dh"]), ("dgamma", dg, ref["dgamma"]), ("dW", dW, ref["dW"])):
        e = _rel(got.float().cpu().numpy(), want)
        assert e <= tg, f"{name} rel max err {e}"
    return loss, dh, dg, dW


@pytest.mark.parametrize("name,dtype", [("tiny_fp32", None), ("small_bf16", None), ("small_bf16", "fp16")])
def test_configs_against_full_oracle(lce, name, dtype):
    _check(lce, workloads.make_rmsnorm_inputs(name, dtype=dtype))


CASES = [
    # (N, H, V, dtype, chunk_tokens)
    (37, 72, 1000, "bf16", 0),
    (300, 136, 4099, "bf16", 64),
    (513, 264, 2050, "fp16", 128),
    (129, 8, 300, "fp32", 0),
    (70, 520, 257, "bf16", 0),
    (1, 64, 128, "bf16", 0),
    # Sixteen chunks: beyond the carry limits of bf16 (4) and fp16 (9), dW is summed over the chunks
    # in the fp32 accumulator while dX comes out of the split dH partials in fp32.
    (1024, 256, 3000, "bf16", 64),
    (1024, 256, 3000, "fp16", 64),
]


@pytest.mark.parametrize("N,H,V,dtype,chunk", CASES)
def test_ragged_shapes(lce, N, H, V, dtype, chunk):
    d = workloads.make_rmsnorm_inputs("llama3_8b", seed=N + H + V, N=N, H=H, V=V, dtype=dtype)
    _check(lce, d, chunk_tokens=chunk)


@pytest.mark.parametrize("reduction", ["mean", "sum"])
def test_reductions_at_medium_size(lce, reduction):
    d = workloads.make_rmsnorm_inputs("llama3_8b", seed=2, N=1024, H=1024, V=32768)
    _check(lce, d, reduction=reduction, chunk_tokens=256)


def test_forward_outputs(lce):
    d = workloads.make_rmsnorm_inputs("llama3_8b", seed=3, N=333, H=200, V=7001)
    h, g, W, y = _dev(d)
    ref = orn.forward(d["hidden"], d["gamma"], d["weight"], d["labels"], d["eps"], reduction="none")
    tl, lse, x = lce.rmsnorm_forward(h, g, W, y, d["eps"], reduction="none", return_lse=True, return_normed=True)
    # x is rounded once to bf16 (relative 2^-9).
    np.testing.assert_allclose(x.float().cpu().numpy(), ref["x"], rtol=2 ** -8, atol=1e-6)
    np.testing.assert_allclose(lse.cpu().numpy(), ref["lse"], rtol=1e-3)
    np.testing.assert_allclose(tl.cpu().numpy(), ref["token_loss"], rtol=2e-2, atol=2e-2)
    L = lce.rmsnorm_forward(h, g, W, y, d["eps"]).item()
    r = orn.forward(d["hidden"], d["gamma"], d["weight"], d["labels"], d["eps"])
    assert abs(L - r["loss"]) <= 1e-3 * abs(r["loss"])


def test_deterministic_and_autograd(lce):
    d = workloads.make_rmsnorm_inputs("llama3_8b", seed=4, N=600, H=256, V=9000)
    h, g, W, y = _dev(d)
    a = lce.rmsnorm_forward_backward(h, g, W, y, d["eps"], chunk_tokens=128)
    b = lce.rmsnorm_forward_backward(h, g, W, y, d["eps"], chunk_tokens=128)
    assert all(torch.equal(p, q) for p, q in zip(a, b))
    h.requires_grad_(True)
    g.requires_grad_(True)
    W.requires_grad_(True)
    loss = lce.rmsnorm_linear_cross_entropy(h, g, W, y, d["eps"])
    (2.5 * loss).backward()
    ref = orn.forward_backward(d["hidden"], d["gamma"], d["weight"], d["labels"], d["eps"])
    assert _rel(h.grad.float().cpu().numpy(), 2.5 * ref["dh"]) <= 2e-2
    assert _rel(g.grad.float().cpu().numpy(), 2.5 * ref["dgamma"]) <= 2e-2
    assert _rel(W.grad.float().cpu().numpy(), 2.5 * ref["dW"]) <= 2e-2


def test_full_size_llama_sampled(lce):
    # Llama-3-8B output layer with the final RMSNorm: loss and every token's lse against the values
    # the oracle wrote (tests/golden/make_full_size.py), sampled rows of d h and dW recomputed by
    # the oracle one by one, and properties at full size.
    with open(os.path.join(GOLDEN, "llama3_8b_rmsnorm_seed0.json")) as f:
        meta = json.load(f)
    arrs = np.load(os.path.join(GOLDEN, "llama3_8b_rmsnorm_seed0.npz"))
    d = workloads.make_rmsnorm_inputs("llama3_8b", seed=0)
    assert workloads.fingerprint(d) == meta["fingerprint"], "generator output changed"
    h, g, W, y = _dev(d)
    print("full-size llama3_8b_rmsnorm", flush=True)
    loss, dh, dg, dW = lce.rmsnorm_forward_backward(h, g, W, y, d["eps"], d["ignore_index"], d["reduction"])
    torch.cuda.synchronize()
    assert abs(loss.item() - meta["loss"]) <= 1e-3 * abs(meta["loss"]), (loss.item(), meta["loss"])
    _, lse = lce.rmsnorm_forward(h, g, W, y, d["eps"], d["ignore_index"], "none", return_lse=True)
    np.testing.assert_allclose(lse.cpu().numpy(), arrs["lse"], rtol=1e-4)

    labels = d["labels"].numpy()
    valid = labels != d["ignore_index"]
    gw, _ = oracle.token_weights(labels, d["ignore_index"], d["reduction"], d["V"])
    rng = np.random.default_rng(0)
    rows = sorted(set([0, d["N"] - 1] + list(rng.choice(d["N"], 6, replace=False))
                      + [int(np.nonzero(~valid)[0][0])]))
    ref_rows = orn.grad_hidden_rows(d["hidden"], d["gamma"], d["weight"], labels, rows, gw, d["eps"])
    got_rows = dh[torch.tensor(rows).cuda()].float().cpu().numpy()
    assert _rel(got_rows, ref_rows) <= 2e-2
    x, _ = orn.rms_normalise(d["hidden"], d["gamma"], d["eps"])
    counts = np.bincount(labels[valid], minlength=d["V"])
    ids = sorted(set([0, int(np.argmax(counts)), d["V"] - 1] + list(rng.choice(d["V"], 3, replace=False))))
    ref_w = oracle.grad_weight_rows(x, d["weight"], labels, ids, arrs["lse"], gw, d["ignore_index"])
    assert _rel(dW[torch.tensor(ids).cuda()].float().cpu().numpy(), ref_w) <= 2e-2
    # Properties: ignored tokens get no gradient; dW columns sum to zero; finite everywhere.
    assert torch.all(dh[torch.from_numpy(~valid).cuda()] == 0)
    col = dW.float().sum(dim=0)
    assert torch.all(col.abs() <= 2e-2 * dW.float().abs().sum(dim=0) + 1e-12)
    assert torch.isfinite(dh.float()).all() and torch.isfinite(dg.float()).all()
