"""The host optimizer step of liblce.so (lce_host_adam_step; pure CPU code, so these run without a
GPU) against the float64 Adam oracle, for every gradient dtype and thread count, and its fused
16-bit copy against torch's own rounding of the fp32 result."""
import numpy as np
import pytest
import torch

from oracle import adam

DT = {"bf16": torch.bfloat16, "fp16": torch.float16, "fp32": torch.float32}


@pytest.fixture(scope="module")
def lce():
    import paper_2603_16428_amd as m
    m.load_library()
    return m


@pytest.mark.parametrize("dtype", ["bf16", "fp16", "fp32"])
@pytest.mark.parametrize("threads", [1, 3, 0])
@pytest.mark.parametrize("moment_offset", [0, 1])
def test_matches_oracle_over_steps(lce, dtype, threads, moment_offset):
    # moment_offset 0: every array 64-byte aligned (torch's host allocations), so bf16 takes the
    # streaming AVX-512 body where the host has it; 1: the moments start 4 bytes in, which keeps
    # every range on the generic body.
    n = 70001 if threads != 1 else 1003          # above the threading cut-off when threaded
    rng = np.random.default_rng(7)
    p = torch.empty(n)
    p.copy_(torch.from_numpy(rng.standard_normal(n).astype(np.float32)))
    m = torch.zeros(n + moment_offset)[moment_offset:]
    v = torch.zeros(n + moment_offset)[moment_offset:]
    assert p.data_ptr() % 64 == 0 and (m.data_ptr() % 64 == 0) == (moment_offset == 0)
    pr, mr, vr = p.double().numpy(), np.zeros(n), np.zeros(n)
    cfg = dict(lr=2e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.05)
    p16 = torch.empty(n, dtype=DT[dtype]) if dtype != "fp32" else None
    # The C ABI takes the settings as fp32: give the oracle the same values.
    f = lambda x: float(np.float32(x))
    b1, b2, lr, eps, wd = f(0.9), f(0.95), f(cfg["lr"]), f(cfg["eps"]), f(cfg["weight_decay"])
    u = 2.0 ** -24
    em = ev = ep = np.zeros(n)  # running bounds on |fp32 - float64| of m, v and the parameter
    for step in range(1, 5):
        g = torch.from_numpy(rng.standard_normal(n) * 10.0 ** rng.uniform(-6, 0, n)).to(DT[dtype])
        g64 = g.double().numpy()
        m_prev, v_prev = mr, vr
        lce.host_adam_step(p, g, m, v, step, param16=p16, threads=threads, **cfg)
        pr, mr, vr = adam.adamw_step(pr, g64, mr, vr, step, lr, b1, b2, eps, wd)
        # Error bounds of the fp32 arithmetic, propagated as the recurrences propagate them: each
        # moment's carried error decays by beta and gains a few roundings of this step's operands;
        # the parameter gains its own rounding and the update's sensitivity to the moments' errors.
        em = b1 * em + 4 * u * (b1 * np.abs(m_prev) + (1 - b1) * np.abs(g64))
        ev = b2 * ev + 4 * u * (b2 * v_prev + (1 - b2) * g64 * g64)
        c1, c2 = 1 / (1 - b1 ** step), 1 / (1 - b2 ** step)
        den = np.sqrt(vr * c2) + eps
        upd = np.abs(mr * c1) / den
        dupd = em * c1 / den + upd * (ev * c2) / (2 * np.sqrt(vr * c2) * den + 1e-300) + 8 * u * upd
        ep = ep + 2 * u * np.abs(pr) + lr * (dupd + wd * ep)
        assert np.all(np.abs(m.double().numpy() - mr) <= em + 1e-30)
        assert np.all(np.abs(v.double().numpy() - vr) <= ev + 1e-36)
        assert np.all(np.abs(p.double().numpy() - pr) <= ep + 1e-30)
        if p16 is not None:
            assert torch.equal(p16, p.to(DT[dtype]))   # round to nearest even of the fp32 master


def test_rejects_bad_arguments(lce):
    p, g = torch.zeros(8), torch.zeros(8, dtype=torch.bfloat16)
    for kw in (dict(lr=-1.0), dict(lr=1e-3, betas=(1.0, 0.9)), dict(lr=1e-3, eps=0.0),
               dict(lr=1e-3, weight_decay=-0.1), dict(lr=float("nan"))):
        with pytest.raises(lce.LCEError):
            lce.host_adam_step(p, g, torch.zeros(8), torch.zeros(8), 1, **kw)
    with pytest.raises(lce.LCEError):
        lce.host_adam_step(p, g, torch.zeros(8), torch.zeros(8), 0, lr=1e-3)


def test_bf16_rounding_of_ties_and_nan(lce):
    # Values exactly halfway between two bf16 numbers round to the even one; NaN stays NaN.
    p = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, float("nan"), -2.5], dtype=torch.float32)
    g = torch.zeros(4, dtype=torch.bfloat16)
    out = torch.empty(4, dtype=torch.bfloat16)
    lce.host_adam_step(p, g, torch.zeros(4), torch.zeros(4), 1, lr=0.0, param16=out, threads=1)
    assert out[0].item() == 1.0 and out[1].item() == 1.0 + 2 ** -6 and torch.isnan(out[2]) and out[3].item() == -2.5


def test_bf16_rounding_in_the_vector_body(lce):
    # 64 aligned parameters (the streaming AVX-512 body where the host has it): ties round to the
    # even neighbour, NaN stays NaN, and everything equals torch's own rounding of the fp32 result.
    vals = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, float("nan"), -2.5, 3.0e38, -1.0e-40, 0.0, -0.0]
    p = torch.empty(64)
    p.copy_(torch.tensor(vals * 8, dtype=torch.float32))
    g = torch.zeros(64, dtype=torch.bfloat16)
    out = torch.empty(64, dtype=torch.bfloat16)
    assert p.data_ptr() % 64 == 0 and out.data_ptr() % 64 == 0
    lce.host_adam_step(p, g, torch.zeros(64), torch.zeros(64), 1, lr=0.0, param16=out, threads=1)
    ref = p.to(torch.bfloat16)
    nan = torch.isnan(p)
    assert torch.equal(torch.isnan(out), nan)
    assert torch.equal(out[~nan].view(torch.int16), ref[~nan].view(torch.int16))
    assert out[0].item() == 1.0 and out[1].item() == 1.0 + 2 ** -6
