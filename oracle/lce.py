"""Float64 CPU oracle for the fused linear + cross-entropy (LCE) step.

TEST INFRASTRUCTURE ONLY. Nothing in the product imports this module: only the
tests, the smoke check and the benchmark's CPU-baseline leg may call it.

What it computes. The paper's fused LinearCrossEntropy kernel (Section 3.3,
"Integrated I/O and Compute Co-Design", paragraph "Optimized Triton Kernels")
fuses the output projection with the loss and produces the gradients in small
chunks so that the B x S x V logits tensor is never held in memory. Chunking
changes where the numbers live, not what they are: the result is the ordinary
linear + softmax cross-entropy with an ignore index. So this oracle is that
plain definition, written out in float64:

    z_i      = W x_i                                  (logits of token i, length V)
    lse_i    = log sum_v exp(z_iv)                    (log-sum-exp, max-shifted)
    l_i      = m_i (lse_i - z_i,y_i),   m_i = [y_i != ignore_index]
    loss     = sum_i l_i / n_valid (mean) | sum_i l_i (sum) | l (none)
    g_i      = d loss / d l_i = m_i / n_valid (mean) | m_i (sum)
    dZ_i     = g_i (softmax(z_i) - onehot(y_i))
    dH       = dZ W,       dW = dZ^T X

The operands are the workload's bf16/fp32 values upcast exactly to float64.
Rows (tokens) are independent in every formula above and the loss and dW are
sums over tokens, so the optional ``rows_per_block`` argument only bounds the
float64 logits buffer; tests check that it does not change the result.

Readings where the paper is silent (it gives the kernel one paragraph):
* mean divides by n_valid, the number of non-ignored tokens in the whole call;
* mean with n_valid == 0 returns loss 0 and zero gradients (not 0/0);
* a non-ignored label outside [0, V) raises ValueError;
* no bias, label smoothing, z-loss or soft-capping; upstream gradient is 1.

Every function here is pinned by tests/test_oracle_facts.py against facts that
do not come from this file (closed forms, finite differences, an independent
library routine, invariances).
"""
from __future__ import annotations

import math

import numpy as np

REDUCTIONS = ("none", "mean", "sum")


def _as_f64(a) -> np.ndarray:
    if hasattr(a, "detach"):  # a torch tensor: upcast exactly on the CPU
        a = a.detach().cpu()
        import torch
        a = a.to(torch.float64).numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _as_i64(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def token_weights(labels, ignore_index: int, reduction: str, V: int | None = None):
    """Per-token loss weights g_i = d loss / d l_i, and n_valid.

    Raises ValueError for a non-ignored label outside [0, V) when V is given.
    """
    if reduction not in REDUCTIONS:
        raise ValueError(f"unknown reduction {reduction!r}")
    y = _as_i64(labels)
    valid = y != ignore_index
    if V is not None and np.any((y[valid] < 0) | (y[valid] >= V)):
        raise ValueError("a non-ignored label lies outside [0, V)")
    n_valid = int(valid.sum())
    if reduction == "mean":
        g = valid / n_valid if n_valid > 0 else np.zeros(y.shape, dtype=np.float64)
    else:  # "sum"; for "none" these are the weights of each token's own loss
        g = valid.astype(np.float64)
    return g, n_valid


def log_sum_exp_rows(Z: np.ndarray) -> np.ndarray:
    """lse of each row of Z, shifted by the row maximum for stability."""
    M = Z.max(axis=1)
    return M + np.log(np.exp(Z - M[:, None]).sum(axis=1))


def forward_backward(hidden, weight, labels, ignore_index: int = -100,
                     reduction: str = "mean", want_grads: bool = True,
                     rows_per_block: int | None = None):
    """Loss (and dH, dW) of linear + softmax cross-entropy, in float64.

    Returns a dict with ``loss`` (a float, or the per-token vector for
    reduction="none"), ``lse`` [N], ``token_loss`` [N], ``n_valid``, and, when
    ``want_grads``, ``dH`` [N, H] and ``dW`` [V, H]. Gradients are those of
    the reduced loss with upstream gradient 1; they are not defined for
    reduction="none".
    """
    X = _as_f64(hidden)
    W = _as_f64(weight)
    y = _as_i64(labels)
    N, H = X.shape
    V, H2 = W.shape
    if H2 != H or y.shape != (N,):
        raise ValueError("shape mismatch")
    if want_grads and reduction == "none":
        raise ValueError("gradients are defined for mean or sum reduction only")
    g, n_valid = token_weights(y, ignore_index, reduction, V)
    valid = y != ignore_index

    lse = np.zeros(N)
    token_loss = np.zeros(N)
    dH = np.zeros((N, H)) if want_grads else None
    dW = np.zeros((V, H)) if want_grads else None
    r = N if rows_per_block is None else max(1, int(rows_per_block))
    for r0 in range(0, N, r):
        r1 = min(N, r0 + r)
        Z = X[r0:r1] @ W.T                          # logits of this block of tokens
        lse_b = log_sum_exp_rows(Z)
        lse[r0:r1] = lse_b
        rows = np.nonzero(valid[r0:r1])[0]
        z_target = Z[rows, y[r0:r1][rows]]          # only valid tokens index Z
        token_loss[r0 + rows] = lse_b[rows] - z_target
        if want_grads:
            P = np.exp(Z - lse_b[:, None])          # softmax
            P[rows, y[r0:r1][rows]] -= 1.0          # minus the one-hot target
            dZ = g[r0:r1, None] * P                 # ignored rows get g = 0
            dZ[~valid[r0:r1]] = 0.0
            dH[r0:r1] = dZ @ W
            dW += dZ.T @ X[r0:r1]

    if reduction == "none":
        loss = token_loss.copy()
    elif reduction == "sum":
        loss = math.fsum(token_loss)
    else:
        loss = math.fsum(token_loss) / n_valid if n_valid > 0 else 0.0
    out = {"loss": loss, "lse": lse, "token_loss": token_loss, "n_valid": n_valid}
    if want_grads:
        out["dH"] = dH
        out["dW"] = dW
    return out


def forward(hidden, weight, labels, ignore_index: int = -100, reduction: str = "mean",
            rows_per_block: int | None = None):
    """Forward only: the same definition without the gradients."""
    return forward_backward(hidden, weight, labels, ignore_index, reduction,
                            want_grads=False, rows_per_block=rows_per_block)


# --- sampled outputs, for shapes too large to run whole --------------------------------

def row_stats(hidden, weight, labels, rows, ignore_index: int = -100):
    """lse_i and l_i for the listed tokens only (one logits row each)."""
    X = _as_f64(hidden)
    W = _as_f64(weight)
    y = _as_i64(labels)
    rows = np.asarray(rows, dtype=np.int64)
    Z = X[rows] @ W.T
    lse = log_sum_exp_rows(Z)
    tl = np.zeros(len(rows))
    for j, i in enumerate(rows):
        if y[i] != ignore_index:
            tl[j] = lse[j] - Z[j, y[i]]
    return lse, tl


def grad_hidden_rows(hidden, weight, labels, rows, g, ignore_index: int = -100):
    """dH_i = g_i (softmax(z_i) - onehot(y_i)) W for the listed tokens."""
    X = _as_f64(hidden)
    W = _as_f64(weight)
    y = _as_i64(labels)
    g = np.asarray(g, dtype=np.float64)
    rows = np.asarray(rows, dtype=np.int64)
    Z = X[rows] @ W.T
    P = np.exp(Z - log_sum_exp_rows(Z)[:, None])
    for j, i in enumerate(rows):
        if y[i] == ignore_index:
            P[j] = 0.0
        else:
            P[j, y[i]] -= 1.0
            P[j] *= g[i]
    return P @ W


def grad_weight_rows(hidden, weight, labels, vocab_ids, lse, g, ignore_index: int = -100):
    """dW_v = sum_i g_i (p_iv - [y_i = v]) x_i for the listed vocabulary ids.

    ``lse`` is the per-token log-sum-exp over the whole vocabulary, as returned
    by this module (``forward`` or ``row_stats``), so that only the listed
    columns of the logits are formed here.
    """
    X = _as_f64(hidden)
    W = _as_f64(weight)
    y = _as_i64(labels)
    g = np.asarray(g, dtype=np.float64)
    lse = np.asarray(lse, dtype=np.float64)
    vocab_ids = np.asarray(vocab_ids, dtype=np.int64)
    valid = y != ignore_index
    Zc = X @ W[vocab_ids].T                        # [N, k]: the listed logit columns
    P = np.exp(Zc - lse[:, None])
    P -= ((y[:, None] == vocab_ids[None, :]) & valid[:, None]).astype(np.float64)
    P *= g[:, None]
    P[~valid] = 0.0
    return P.T @ X
