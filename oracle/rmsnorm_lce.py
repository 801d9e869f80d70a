"""Float64 CPU oracle for the final RMSNorm followed by the fused linear + cross-entropy step.

TEST INFRASTRUCTURE ONLY. Nothing in the product imports this module: only the
tests, the smoke check and the benchmark's CPU-baseline leg may call it.

The paper lists RMSNorm among the fused kernels of Section 3.3 ("Integrated I/O
and Compute Co-Design", paragraph "Optimized Triton Kernels") without writing
it out, and the normalisation right before the output projection is the one
that meets the LCE kernel. The standard definition is used (root-mean-square
normalisation with a learned per-feature gain; no mean subtraction, no bias):

    r_i   = 1 / sqrt(mean_j h_ij^2 + eps)            (per token)
    x_ij  = gamma_j h_ij r_i                          (the LCE step's hidden input)

and the loss is the LCE loss of x (``oracle.lce``). The gradients follow from
the chain rule, with dX = d loss / d x taken from the LCE oracle:

    d gamma_j = sum_i dX_ij h_ij r_i
    d h_ij    = r_i gamma_j dX_ij - r_i^3 h_ij (1/H) sum_k h_ik gamma_k dX_ik

(d r_i / d h_ij = -r_i^3 h_ij / H). Everything is float64 on the inputs upcast
exactly; rows are independent except through the LCE loss's sums.

Pinned by tests/test_oracle_rmsnorm.py: torch's own rms_norm with autograd in
float64, central finite differences, the scale invariance of the normalisation
(eps = 0), and the reduction to the plain LCE oracle on unit-RMS rows.
"""
from __future__ import annotations

import numpy as np

from . import lce


def rms_normalise(hidden, gamma, eps: float):
    """(x, r): the normalised rows and each row's 1 / rms."""
    h = lce._as_f64(hidden)
    g = lce._as_f64(gamma)
    if h.ndim != 2 or g.shape != (h.shape[1],):
        raise ValueError("hidden must be [N, H] and gamma [H]")
    r = 1.0 / np.sqrt(np.mean(h * h, axis=1) + float(eps))
    x = g[None, :] * h * r[:, None]
    return x, r


def forward_backward(hidden, gamma, weight, labels, eps: float = 1e-5, ignore_index: int = -100,
                     reduction: str = "mean", rows_per_block: int | None = None) -> dict:
    """Loss, lse and the gradients with respect to the pre-norm hidden, gamma and the weight."""
    h = lce._as_f64(hidden)
    g = lce._as_f64(gamma)
    x, r = rms_normalise(h, g, eps)
    out = lce.forward_backward(x, weight, labels, ignore_index, reduction, True, rows_per_block)
    dX = out["dH"]
    H = h.shape[1]
    dgamma = np.sum(dX * h * r[:, None], axis=0)
    s = np.sum(h * g[None, :] * dX, axis=1)              # sum_k h_ik gamma_k dX_ik
    dh = r[:, None] * g[None, :] * dX - (r ** 3)[:, None] * h * (s / H)[:, None]
    return {"loss": out["loss"], "lse": out["lse"], "token_loss": out["token_loss"],
            "n_valid": out["n_valid"], "x": x, "r": r, "dX": dX, "dh": dh, "dgamma": dgamma,
            "dW": out["dW"]}


def forward(hidden, gamma, weight, labels, eps: float = 1e-5, ignore_index: int = -100,
            reduction: str = "mean") -> dict:
    """Loss and per-token lse of the LCE step on the normalised rows."""
    x, r = rms_normalise(hidden, gamma, eps)
    out = lce.forward(x, weight, labels, ignore_index, reduction)
    out["x"], out["r"] = x, r
    return out


def grad_hidden_rows(hidden, gamma, weight, labels, rows, g, eps: float = 1e-5, ignore_index: int = -100):
    """d h_i for the listed tokens only (their dX rows from ``lce.grad_hidden_rows``, then the
    chain rule above); ``g`` are the token weights of ``lce.token_weights``."""
    h = lce._as_f64(hidden)
    gm = lce._as_f64(gamma)
    rows = np.asarray(rows, dtype=np.int64)
    x, r = rms_normalise(h[rows], gm, eps)
    xs = np.zeros_like(h)
    xs[rows] = x
    dX = lce.grad_hidden_rows(xs, weight, labels, rows, g, ignore_index)
    hr = h[rows]
    s = np.sum(hr * gm[None, :] * dX, axis=1)
    return r[:, None] * gm[None, :] * dX - (r ** 3)[:, None] * hr * (s / h.shape[1])[:, None]
