"""The step's launch structure, from the library's own per-kind launch counts (lce_timing_*): the
small bandwidth-bound jobs share launches of aux_kernel, so a two-chunk bf16 step is 15 launches
(the start; per chunk the logits GEMM, combine, the fallback logits GEMM and combine that return at
once, one launch of copies and fallback dlogits, dH, dW), fp16 (no fallback; dlogits with the next
chunk's copy, and the next chunk's unscaled dW operand copy after this chunk's dW) 12, and a
one-chunk forward with a reduced loss 4. Results still match the oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return m


def _counts(lce, fn):
    torch.cuda.synchronize()
    lce.timing_enable(True)
    out = fn()
    torch.cuda.synchronize()
    kern = lce.timing_read()
    lce.timing_enable(False)
    return out, {k: v[1] for k, v in kern.items() if v[1]}


@pytest.mark.parametrize("dtype,expect", [
    ("bf16", {"logits_lse_gemm": 2, "dh_gemm": 2, "dw_gemm": 2, "other": 9}),
    ("fp16", {"logits_lse_gemm": 2, "dh_gemm": 2, "dw_gemm": 2, "dlogits": 2, "other": 4}),
])
def test_step_launches(lce, dtype, expect):
    d = workloads.random_case(512, 256, 3000, dtype=dtype, seed=21, w_std=0.5)
    X, W, y = d["hidden"].cuda(), d["weight"].cuda(), d["labels"].cuda()
    print(f"case 512x256x3000 {dtype} chunk 256", flush=True)
    (loss, dH, dW), counts = _counts(lce, lambda: lce.forward_backward(X, W, y, d["ignore_index"], "mean",
                                                                       chunk_tokens=256))
    assert counts == expect, counts
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], "mean")
    assert abs(loss.item() - ref["loss"]) <= 1e-3 * abs(ref["loss"])
    for got, r in ((dH, ref["dH"]), (dW, ref["dW"])):
        assert np.abs(got.float().cpu().numpy() - r).max() <= 2e-2 * np.abs(r).max()


def test_forward_launches(lce):
    d = workloads.random_case(300, 136, 4099, dtype="bf16", seed=22, w_std=0.5)
    X, W, y = d["hidden"].cuda(), d["weight"].cuda(), d["labels"].cuda()
    loss, counts = _counts(lce, lambda: lce.forward(X, W, y, d["ignore_index"], "mean"))
    assert counts == {"logits_lse_gemm": 1, "other": 3}, counts
    ref = oracle.forward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], "mean")
    assert abs(loss.item() - ref["loss"]) <= 1e-3 * abs(ref["loss"])
