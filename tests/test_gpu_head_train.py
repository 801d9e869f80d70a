"""The output-layer training step with host-resident weights (lce_head_train_step): the pipelined
schedule against the sequential one, the consistency of its host and device buffers, and the first
update's direction against the float64 oracle's gradient."""
import numpy as np
import pytest
import torch

import oracle
import workloads

pytestmark = pytest.mark.gpu

ADAM = dict(lr=1e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.01)


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return m


def _case(N, H, V, dtype, seed):
    d = workloads.make_inputs("llama3_8b", seed=seed, N=N, H=H, V=V, dtype=dtype)
    return d, d["hidden"].cuda(), d["labels"].cuda()


def _state(lce, d):
    return lce.HeadState(d["weight"].cuda())


@pytest.mark.parametrize("N,H,V,dtype,chunk,blocks", [
    (300, 136, 4099, "bf16", 128, 3),
    (513, 264, 2050, "fp16", 0, 4),
    (1024, 256, 9000, "bf16", 256, 8),
])
def test_pipelined_equals_sequential(lce, N, H, V, dtype, chunk, blocks):
    d, X, y = _case(N, H, V, dtype, seed=N + V)
    print(f"case N={N} H={H} V={V} {dtype} chunk={chunk} blocks={blocks}", flush=True)
    a, b = _state(lce, d), _state(lce, d)
    for _ in range(3):
        la, dha, _ = lce.head_train_step(a, X, y, chunk_tokens=chunk, vocab_blocks=blocks, overlap=True, **ADAM)
        lb, dhb, _ = lce.head_train_step(b, X, y, chunk_tokens=chunk, vocab_blocks=blocks, overlap=False, **ADAM)
        assert torch.equal(la, lb) and torch.equal(dha, dhb)
    torch.cuda.synchronize()
    for k in ("master", "exp_avg", "exp_avg_sq", "grad_host", "param_host"):
        assert torch.equal(getattr(a, k), getattr(b, k)), k
    assert torch.equal(a.weight, b.weight) and torch.equal(a.grad_weight, b.grad_weight)


# The last chunk's dW contraction in vocabulary blocks gives the same dW, bit for bit, as the plain
# step's single launch: with dW carried across chunks in its own type (2 chunks) and in the fp32
# accumulator (8 chunks, above bf16's carry limit of 4).
@pytest.mark.parametrize("chunk,carry", [(512, 0), (128, 1)])
def test_blocked_dw_equals_plain_step(lce, chunk, carry):
    N, H, V = 1024, 256, 9000
    d, X, y = _case(N, H, V, "bf16", seed=17)
    assert lce.plan_info(N, H, V, torch.bfloat16, True, chunk)["dw_fp32_carry"] == carry
    W = d["weight"].cuda()
    loss, dH, dW = lce.forward_backward(X, W, y, chunk_tokens=chunk)
    st = _state(lce, d)
    l2, dH2, _ = lce.head_train_step(st, X, y, chunk_tokens=chunk, vocab_blocks=6, **ADAM)
    torch.cuda.synchronize()
    assert torch.equal(loss, l2) and torch.equal(dH, dH2) and torch.equal(dW, st.grad_weight)


def test_buffers_and_first_update_against_oracle(lce):
    N, H, V = 400, 192, 5000
    d, X, y = _case(N, H, V, "bf16", seed=11)
    st = _state(lce, d)
    w0 = d["weight"].double().numpy()
    loss, dH, timing = lce.head_train_step(st, X, y, chunk_tokens=128, vocab_blocks=5, **ADAM)
    torch.cuda.synchronize()
    assert all(timing[k] >= 0 for k in timing) and timing["gpu_ms"] > 0
    # Host and device buffers agree: the copies moved every block.
    assert torch.equal(st.grad_host, st.grad_weight.cpu())
    assert torch.equal(st.param_host, st.master.to(torch.bfloat16))
    assert torch.equal(st.weight.cpu(), st.param_host)
    # The step's loss, dH and dW against the float64 oracle (the plain step's tolerances).
    ref = oracle.forward_backward(d["hidden"], d["weight"], d["labels"])
    assert abs(loss.item() - ref["loss"]) <= 1e-3 * abs(ref["loss"])
    scale = np.abs(ref["dW"]).max()
    assert np.abs(st.grad_weight.float().cpu().numpy() - ref["dW"]).max() <= 2e-2 * scale
    # First AdamW step: m_hat / sqrt(v_hat) = g / |g|, so every weight moves by lr (minus its decay)
    # against the gradient's sign wherever |g| dwarfs eps and the gradient's own error.
    delta = st.master.double().numpy() - (w0 - ADAM["lr"] * ADAM["weight_decay"] * w0)
    sure = np.abs(ref["dW"]) > 0.05 * scale
    assert sure.sum() > 100
    np.testing.assert_allclose(delta[sure], -ADAM["lr"] * np.sign(ref["dW"][sure]), rtol=1e-3, atol=1e-7)
    assert np.all(np.abs(delta) <= ADAM["lr"] * (1 + 1e-3))


def test_loss_decreases(lce):
    d, X, y = _case(512, 128, 3000, "bf16", seed=5)
    st = _state(lce, d)
    losses = [lce.head_train_step(st, X, y, vocab_blocks=4, lr=2e-3)[0].item() for _ in range(6)]
    assert all(b < a for a, b in zip(losses, losses[1:])), losses
