"""Parity of the HIP path (through the C ABI) with the float64 oracle, on the same seeded inputs.

Tolerances: loss relative error <= 1e-3 and max|dH - ref|, max|dW - ref| <= 2e-2 * max|ref| for
bf16 operands with fp32 accumulation; 1e-5 for the fp32 path; for fp16 1e-3 and 5e-3 * max|ref|
(bf16's bar is 5.1 unit roundoffs of bf16, u = 2^-8; fp16's path stores one more rounded value per
logit, and its bar is 10.2 of fp16's u = 2^-11).
fp32 gradients: every dH entry is a sum over K = V rounded fp32 terms and every dW entry a sum over
the K = N tokens; their rounding grows like sqrt(K) 2^-24, so the bounds are max(1e-5,
2 sqrt(K) 2^-24) per tensor: 1e-5 up to K = 7036, i.e. everywhere except dH of the half-million
vocabulary case (8.4e-5). The per-token factor g/S that both carry adds little: S is summed in
short sequential runs (64 terms per lane, then per-slice merges in 16 groups), not in one run of V.

Small cases run the whole oracle (several tiles, ragged tails, several chunks, split-K and the
unsplit dH store, the dW carry in the operand type and in fp32). The full-size workloads compare
every element of the loss, dH and dW with the whole oracle, every token's log-sum-exp with values
the oracle wrote (tests/golden/make_full_size.py), and properties that hold at any size (dW
columns sum to zero, ignored tokens give zero dH rows, bitwise determinism). Each case prints how
it runs (lce_plan_info), and tests/test_abi.py checks on the CPU that the cases cover every path.
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


def _grad_tol(dtype, K):
    """Bar for max|got - ref| / max|ref| of a gradient whose entries sum K terms (dH: K = V, dW:
    K = N; see the module docstring)."""
    tol = TOL[dtype][1]
    if dtype == "fp32":
        tol = max(tol, 2.0 * np.sqrt(K) * 2.0 ** -24)
    return tol


def _nan_workspace(lce, d, chunk_tokens):
    """A workspace whose every byte is 0xFF (NaN as any float type): a kernel that reads a byte of
    it before writing it puts NaN into the results."""
    need = lce.workspace_size(d["N"], d["H"], d["V"], d["hidden"].dtype, True, chunk_tokens)
    return torch.full((need,), 255, dtype=torch.uint8, device="cuda")


def _check_full(lce, d, reduction=None, chunk_tokens=0, workspace=None, ref=None):
    reduction = reduction or d["reduction"]
    tol_loss = TOL[d["dtype"]][0]
    tol_dh, tol_dw = _grad_tol(d["dtype"], d["V"]), _grad_tol(d["dtype"], d["N"])
    X, W, y = _to_dev(d)
    plan = lce.plan_info(d["N"], d["H"], d["V"], X.dtype, True, chunk_tokens)
    print(f"case {d['name']} N={d['N']} H={d['H']} V={d['V']} {d['dtype']} {reduction} chunk={chunk_tokens} "
          f"plan {plan}", flush=True)
    loss, dH, dW = lce.forward_backward(X, W, y, d["ignore_index"], reduction, chunk_tokens=chunk_tokens,
                                        workspace=workspace)
    torch.cuda.synchronize()
    if ref is None:
        ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], reduction)
    L = loss.item()
    if ref["loss"] == 0.0:
        # Exactly zero in exact arithmetic (V = 1, or no valid token): fp32 rounding only.
        assert abs(L) <= 1e-5, L
    else:
        assert abs(L - ref["loss"]) <= tol_loss * abs(ref["loss"]), (L, ref["loss"])
    eh = _rel_max_err(dH.float().cpu().numpy(), ref["dH"])
    ew = _rel_max_err(dW.float().cpu().numpy(), ref["dW"])
    print(f"  loss {L:.7g} (oracle {ref['loss']:.7g}); dH err {eh:.3g} (bar {tol_dh:.3g}), "
          f"dW err {ew:.3g} (bar {tol_dw:.3g})", flush=True)
    assert eh <= tol_dh, f"dH rel max err {eh}"
    assert ew <= tol_dw, f"dW rel max err {ew}"
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


# The unsplit dH store (dh_splits == 1: the contraction writes dH rows straight from its epilogue,
# the path of the Llama-3-8B and Qwen2.5-7B workloads) against the whole oracle, with
# Llama-distributed inputs: one chunk (dW written), two chunks (dW written, then added to), and a
# ragged width and vocabulary (H = 4000: a 160-column last tile; V = 5000: a partial K-pair).
UNSPLIT = [
    # (N, H, V, dtype, chunk_tokens, chunks)
    (4096, 4096, 1024, "bf16", 4096, 1),
    (8192, 4096, 2048, "bf16", 4096, 2),
    (8192, 4000, 5000, "bf16", 4096, 2),
    (4096, 4096, 512, "fp32", 4096, 1),
    (8192, 4096, 512, "fp32", 4096, 2),
    (8192, 4096, 1024, "fp16", 4096, 2),
    (4096, 4096, 512, "fp16", 4096, 1),
]


@pytest.mark.parametrize("N,H,V,dtype,chunk,chunks", UNSPLIT)
def test_unsplit_dh_whole_oracle(lce, N, H, V, dtype, chunk, chunks):
    d = workloads.make_inputs("llama3_8b", seed=2, N=N, H=H, V=V, dtype=dtype)
    plan = lce.plan_info(N, H, V, d["hidden"].dtype, True, chunk)
    assert plan["dh_splits"] == 1 and plan["chunks"] == chunks and plan["dw_fp32_carry"] == 0, plan
    _check_full(lce, d, chunk_tokens=chunk, workspace=_nan_workspace(lce, d, chunk))


# The running dW sum over many chunks at Llama's width: carried in bf16 up to bf16's carry limit
# (4 chunks), in the fp32 accumulator beyond it (16 chunks); both against one whole-oracle result.
def test_many_chunks_llama_width(lce):
    d = workloads.make_inputs("llama3_8b", seed=3, N=16384, H=4096, V=4096)
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], d["reduction"])
    for chunk, chunks, carry in ((4096, 4, 0), (1024, 16, 1), (0, 4, 0)):
        plan = lce.plan_info(d["N"], d["H"], d["V"], torch.bfloat16, True, chunk)
        assert (plan["chunks"], plan["dw_fp32_carry"]) == (chunks, carry), plan
        _check_full(lce, d, chunk_tokens=chunk, ref=ref)


# fp16: its carry limit is 9 chunks; 8 chunks carry in fp16, 16 in the fp32 accumulator.
def test_many_chunks_fp16(lce):
    d = workloads.make_inputs("llama3_8b", seed=4, N=4096, H=1024, V=4096, dtype="fp16")
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], d["reduction"])
    for chunk, chunks, carry in ((512, 8, 0), (256, 16, 1)):
        plan = lce.plan_info(d["N"], d["H"], d["V"], torch.float16, True, chunk)
        assert (plan["chunks"], plan["dw_fp32_carry"]) == (chunks, carry), plan
        _check_full(lce, d, chunk_tokens=chunk, ref=ref, workspace=_nan_workspace(lce, d, chunk))


# A workspace full of NaN bytes: every byte a kernel reads must have been written earlier in the
# call. V % 8 in 1..4 leaves the last fp32 K-pair of 8 ids half inside the vocabulary; the dH
# contraction reads it whole, so its padding ids must be stored as zeros (V = 50257 is GPT-2's).
NAN_WS = [
    # (N, H, V, dtype, chunk_tokens)
    (200, 64, 50257, "fp32", 64),
    (150, 32, 1025, "fp32", 0),
    (130, 64, 4100, "fp32", 64),
    (300, 136, 4099, "bf16", 64),
    (300, 136, 4099, "fp16", 64),
    (64, 1024, 33000, "bf16", 0),
]


@pytest.mark.parametrize("N,H,V,dtype,chunk", NAN_WS)
def test_nan_filled_workspace(lce, N, H, V, dtype, chunk):
    d = workloads.random_case(N, H, V, dtype=dtype, seed=N + V, x_scale=1.0, w_std=0.5)
    loss, dH, dW = _check_full(lce, d, chunk_tokens=chunk, workspace=_nan_workspace(lce, d, chunk))
    assert torch.isfinite(dH.float()).all() and torch.isfinite(dW.float()).all()


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


# Confident tokens (target logit 20 above every other): S = sum_v exp(z_v - z_target) is 1 plus
# ~1e-5, and the GEMM's z_target differs from the reference dot product by a few fp32 roundings
# either way, so S falls slightly below 1 for about half of them. That is no reason to redo the
# chunk on the slice-maximum path: the flags must stay clear, and the results match the oracle.
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_confident_tokens_keep_the_fast_path(lce, dtype):
    d = workloads.random_case(256, 64, 3000, dtype=dtype, seed=13, w_std=0.02)
    d = _with_extreme_tokens(d, [(i, 20.0) for i in range(0, 256, 2)])
    chunk = 128
    plan = lce.plan_info(d["N"], d["H"], d["V"], d["hidden"].dtype, True, chunk)
    assert plan["target_referenced"] == 1
    ws = torch.zeros(plan["workspace_bytes"], dtype=torch.uint8, device="cuda")
    _check_full(lce, d, chunk_tokens=chunk, workspace=ws)
    off = plan["fallback_flags_offset"]
    flags = ws[off:off + 4 * plan["chunks"]].view(torch.int32).cpu().tolist()
    assert flags == [0] * plan["chunks"], flags


# And the converse: a chunk holding a token whose loss exceeds 60 is flagged (and redone), the
# others are not.
def test_high_loss_token_sets_its_chunks_flag(lce):
    d = workloads.random_case(300, 64, 300, dtype="bf16", seed=11, w_std=0.3)
    d = _with_extreme_tokens(d, [(200, -80.0)])
    plan = lce.plan_info(d["N"], d["H"], d["V"], torch.bfloat16, True, 64)
    ws = torch.zeros(plan["workspace_bytes"], dtype=torch.uint8, device="cuda")
    _check_full(lce, d, chunk_tokens=64, workspace=ws)
    off = plan["fallback_flags_offset"]
    flags = ws[off:off + 4 * plan["chunks"]].view(torch.int32).cpu().tolist()
    assert [f != 0 for f in flags] == [c == 200 // 64 for c in range(plan["chunks"])], flags


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


_FULL_INPUTS = {}


def _full_inputs(name):
    """The full-size workload's seed-0 draws, made once per test session (about a GB each)."""
    if name not in _FULL_INPUTS:
        _FULL_INPUTS[name] = workloads.make_inputs(name, seed=0)
    return _FULL_INPUTS[name]


def _golden(name):
    with open(os.path.join(GOLDEN, f"{name}_seed0.json")) as f:
        meta = json.load(f)
    arrs = np.load(os.path.join(GOLDEN, f"{name}_seed0.npz"))
    return meta, arrs["lse"], arrs["token_loss"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_sampled(lce, name):
    meta, lse_ref, tl_ref = _golden(name)
    d = _full_inputs(name)
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


def _max_abs_err_blocked(got, ref, rows=8192):
    """max |got - ref| over every element (got: device tensor, ref: float64 numpy), in row blocks so
    that no float64 copy of the whole device tensor is made."""
    err = 0.0
    for r0 in range(0, ref.shape[0], rows):
        g = got[r0:r0 + rows].float().cpu().numpy().astype(np.float64)
        err = max(err, float(np.max(np.abs(g - ref[r0:r0 + rows]))))
    return err


# Every element of loss, dH and dW at full size, against the whole float64 oracle on the host
# (tens of seconds of BLAS per workload), in the configuration bench.py times.
@pytest.mark.parametrize("name", FULL)
def test_full_size_every_element(lce, name):
    meta, lse_ref, tl_ref = _golden(name)
    d = _full_inputs(name)
    assert workloads.fingerprint(d) == meta["fingerprint"], "generator output changed"
    X, W, y = _to_dev(d)
    plan = lce.plan_info(d["N"], d["H"], d["V"], X.dtype, True, 0)
    print(f"full-size {name}, every element; plan {plan}", flush=True)
    loss, dH, dW = lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"])
    torch.cuda.synchronize()
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"], d["ignore_index"], d["reduction"],
                                  rows_per_block=256)
    print(f"  oracle done: loss {ref['loss']:.7g}", flush=True)
    assert abs(ref["loss"] - meta["loss"]) <= 1e-12 * abs(meta["loss"])
    assert abs(loss.item() - ref["loss"]) <= 1e-3 * abs(ref["loss"]), (loss.item(), ref["loss"])
    eh = _max_abs_err_blocked(dH, ref["dH"]) / np.max(np.abs(ref["dH"]))
    ew = _max_abs_err_blocked(dW, ref["dW"]) / np.max(np.abs(ref["dW"]))
    print(f"  dH err {eh:.3g}, dW err {ew:.3g} (bar 2e-2)", flush=True)
    assert eh <= 2e-2 and ew <= 2e-2, (eh, ew)


# Device memory of one call: the library allocates nothing (the caller's workspace and outputs are
# all it touches), and workspace + outputs are at least 80% below the peak of a step that
# materialises the logits (Section 3.3, paragraph "Optimized Triton Kernels", claims over 80% for
# the output layer of Llama3.1-8B).
def test_memory_bound_and_reduction(lce):
    d = _full_inputs("llama3_8b")
    X, W, y = _to_dev(d)
    ws = torch.empty(lce.workspace_size(d["N"], d["H"], d["V"], X.dtype, True, 0), dtype=torch.uint8,
                     device="cuda")
    out = (torch.empty(1, dtype=torch.float32, device="cuda"), torch.empty_like(X), torch.empty_like(W))
    lce_bytes = sum(t.numel() * t.element_size() for t in (ws,) + out)
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], 0, ws, out)
    torch.cuda.synchronize()
    inside = torch.cuda.max_memory_allocated() - base
    print(f"LCE: workspace {ws.numel() / 1e9:.3f} GB + outputs {(lce_bytes - ws.numel()) / 1e9:.3f} GB; "
          f"allocated inside the call: {inside} bytes", flush=True)
    assert inside == 0
    del ws, out
    torch.cuda.empty_cache()
    Xg, Wg = X.clone().requires_grad_(True), W.clone().requires_grad_(True)
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    logits = Xg @ Wg.T
    ref_loss = torch.nn.functional.cross_entropy(logits.float(), y, ignore_index=d["ignore_index"],
                                                 reduction=d["reduction"])
    gx, gw = torch.autograd.grad(ref_loss, [Xg, Wg])
    torch.cuda.synchronize()
    mat_peak = torch.cuda.max_memory_allocated() - base
    print(f"materialised peak {mat_peak / 1e9:.3f} GB: LCE is {100 * (1 - lce_bytes / mat_peak):.1f}% below",
          flush=True)
    assert lce_bytes <= 0.2 * mat_peak


@pytest.mark.parametrize("name", FULL)
def test_full_size_forward_lse(lce, name):
    meta, lse_ref, tl_ref = _golden(name)
    d = _full_inputs(name)
    X, W, y = _to_dev(d)
    tl, lse = lce.forward(X, W, y, d["ignore_index"], "none", return_lse=True)
    np.testing.assert_allclose(lse.cpu().numpy(), lse_ref, rtol=1e-4)
    np.testing.assert_allclose(tl.cpu().numpy(), tl_ref, rtol=2e-3, atol=2e-3)
    L = lce.forward(X, W, y, d["ignore_index"], d["reduction"]).item()
    assert abs(L - meta["loss"]) <= 1e-3 * abs(meta["loss"])
