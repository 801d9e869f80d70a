"""lce_forward_no_alloc, called through the C ABI, against lce_forward: identical per-token losses,
log-sum-exps and reduced losses on calls in a row on one device, each smaller than the one before
(the first large enough that the static scratch forces several chunks), with nothing allocated
during the call. Per token, the result does not depend on how the tokens are chunked (each token's
partials over the vocabulary slices are merged in the same fixed order), so the two entry points
agree bit for bit."""
import ctypes

import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

SCRATCH = 64 << 20  # LCE_NO_ALLOC_SCRATCH_BYTES
DT = {torch.float32: 0, torch.bfloat16: 1, torch.float16: 2}
RED = {"none": 0, "mean": 1, "sum": 2}


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return m


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def test_no_alloc_forward_matches_forward(lce):
    lib = lce.load_library()
    cases = [workloads.make_inputs("llama3_8b", seed=0),
             workloads.random_case(300, 136, 4099, dtype="bf16", seed=1, w_std=0.5),
             workloads.random_case(150, 72, 1000, dtype="fp32", seed=2, w_std=0.5),
             workloads.random_case(100, 64, 700, dtype="fp16", seed=3, w_std=0.5)]
    first = cases[0]
    assert lce.workspace_size(first["N"], first["H"], first["V"], torch.bfloat16, False) > SCRATCH
    for d in cases:
        X, W, y = d["hidden"].cuda(), d["weight"].cuda(), d["labels"].cuda()
        N, H = X.shape
        V = W.shape[0]
        for red in ("none", "mean"):
            print(f"case N={N} H={H} V={V} {d['dtype']} {red}", flush=True)
            ref = lce.forward(X, W, y, d["ignore_index"], red, return_lse=True)
            loss = torch.full((N if red == "none" else 1,), float("nan"), dtype=torch.float32, device="cuda")
            lse = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
            stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
            base = torch.cuda.memory_allocated()
            torch.cuda.reset_peak_memory_stats()
            st = lib.lce_forward_no_alloc(_p(X), _p(W), _p(y), N, H, V, DT[X.dtype], d["ignore_index"], RED[red],
                                          _p(loss), _p(lse), stream)
            torch.cuda.synchronize()
            assert st == 0, lce.lce.STATUS.get(st, st)
            assert torch.cuda.max_memory_allocated() == base
            ref_loss = ref[0] if red == "none" else ref[0].reshape(1)
            assert torch.equal(lse, ref[1]), (lse - ref[1]).abs().max().item()
            assert torch.equal(loss, ref_loss), (loss - ref_loss).abs().max().item()
            assert torch.isfinite(lse).all()
