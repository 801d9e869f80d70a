"""Float64 CPU oracle for the host optimizer step of the output layer (Layer-Adam).

TEST INFRASTRUCTURE ONLY. Nothing in the product imports this module: only the
tests, the smoke check and the benchmark's CPU-baseline leg may call it.

The paper updates each layer's FP32 master parameters on the CPU with a variant
of DeepSpeed's CPU-Adam (Section 3.2, "Layer-Adam Optimizer"; schedule in
Section 3.1, "Asynchronous Parameter Updating"), from 16-bit gradients offloaded
to pinned host memory, and converts the updated parameters to 16 bits in a
shared buffer before the next h2d copy (Section 3.2, "Optimized CPU Memory
Layout with Shared Buffers"). It does not write the update out; the standard
Adam with decoupled weight decay (AdamW) and bias correction is used:

    m_t = b1 m_{t-1} + (1 - b1) g_t
    v_t = b2 v_{t-1} + (1 - b2) g_t^2
    p_t = p_{t-1} - lr ( (m_t / (1 - b1^t)) / (sqrt(v_t / (1 - b2^t)) + eps) + wd p_{t-1} )

with t counted from 1. Pinned by tests/test_oracle_adam.py against torch.optim.AdamW
in float64 (independent code) and closed forms.
"""
from __future__ import annotations

import numpy as np


def adamw_step(param, grad, exp_avg, exp_avg_sq, step: int, lr: float, beta1: float = 0.9,
               beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.0):
    """One step; returns new (param, exp_avg, exp_avg_sq) as float64 arrays (inputs untouched)."""
    if step < 1:
        raise ValueError("step counts from 1")
    p = np.asarray(param, dtype=np.float64)
    g = np.asarray(grad, dtype=np.float64)
    m = beta1 * np.asarray(exp_avg, dtype=np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(exp_avg_sq, dtype=np.float64) + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    p_new = p - lr * (m_hat / (np.sqrt(v_hat) + eps) + weight_decay * p)
    return p_new, m, v
