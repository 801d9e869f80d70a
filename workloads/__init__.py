"""Seeded synthetic workloads for the fused linear + cross-entropy step.

This module only draws inputs. It holds none of the step's arithmetic (no
logits, no softmax, no gradients), so the float64 oracle and the HIP path can
both consume it without sharing any part of the method.

The shapes follow the output layers of the models the paper fine-tunes
(Llama-3.1-8B, Qwen2.5-7B, Mistral-Large; Section 4.1, "Experimental Setup"),
with sequence length 1024 and synthetic data as in that section. The weights
are random: no checkpoint is needed or used.

Recipe (identical on every machine with the same numpy and torch):

* ``numpy.random.SeedSequence(seed).spawn(4)`` gives four independent PCG64
  streams, used for hidden, weight, labels and the ignore mask, in that order.
* Values are drawn in float64, shaped and normalised in float64, then rounded
  to the workload dtype by torch's float64 -> bfloat16 (or float16, float32) conversion
  (round to nearest even).
* "unit-RMS rows": each hidden row is g / sqrt(mean(g**2)) with g ~ N(0, 1),
  the shape of a post-RMSNorm activation.
* "zipf(s)": labels follow a Zipf law truncated to the vocabulary,
  p(k) proportional to k**-s over ranks k = 1..V, token id = k - 1.
* The ignore set is an exact count round(f * N) picked by a seeded permutation;
  the "prefix" recipe instead masks, for each sequence of 1024 tokens, a
  leading span whose length is uniform in [0, 307] (prompt masking).
"""
from __future__ import annotations

import dataclasses
import hashlib
import math

import numpy as np
import torch

IGNORE_INDEX = -100
TORCH_DTYPES = {"bf16": torch.bfloat16, "fp16": torch.float16, "fp32": torch.float32}

# Rows of W are drawn in blocks of this many rows so that the float64 staging
# buffer stays small; numpy's normal stream is sequential, so the values do not
# depend on the block size.
_W_BLOCK_ROWS = 8192


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    N: int            # tokens (batch x sequence)
    H: int            # hidden size
    V: int            # vocabulary size
    dtype: str        # "bf16", "fp16" or "fp32"
    hidden: str       # "normal", "normal_4_over_sqrt_h", "unit_rms"
    w_std: float
    labels: str       # "uniform" or "zipf"
    zipf_s: float
    ignore: str       # "count" or "prefix"
    ignore_frac: float
    reduction: str    # "mean" or "sum"
    seq_len: int = 1024

    @property
    def torch_dtype(self):
        return TORCH_DTYPES[self.dtype]


WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", 256, 256, 4096, "fp32", "normal", 0.02,
                          "uniform", 0.0, "count", 0.05, "mean", seq_len=256),
    "small_bf16": Workload("small_bf16", 2048, 2048, 32000, "bf16", "normal_4_over_sqrt_h", 0.02,
                           "zipf", 1.1, "count", 0.10, "mean"),
    "llama3_8b": Workload("llama3_8b", 8192, 4096, 128256, "bf16", "unit_rms", 0.02,
                          "zipf", 1.1, "count", 0.10, "mean"),
    "qwen25_7b": Workload("qwen25_7b", 16384, 3584, 152064, "bf16", "unit_rms", 0.02,
                          "zipf", 1.05, "prefix", 0.15, "sum"),
    "mistral_large": Workload("mistral_large", 4096, 12288, 32768, "bf16", "unit_rms", 0.01,
                              "uniform", 0.0, "count", 0.05, "mean"),
}


def _streams(seed: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(4)]


def _hidden(rng, w: Workload, N: int, H: int) -> np.ndarray:
    g = rng.standard_normal((N, H))
    if w.hidden == "normal":
        return g
    if w.hidden == "normal_4_over_sqrt_h":
        return g * (4.0 / math.sqrt(H))
    if w.hidden == "unit_rms":
        return g / np.sqrt(np.mean(g * g, axis=1, keepdims=True))
    raise ValueError(w.hidden)


def _weight(rng, w: Workload, V: int, H: int, tdtype) -> torch.Tensor:
    out = torch.empty((V, H), dtype=tdtype)
    for r0 in range(0, V, _W_BLOCK_ROWS):
        r1 = min(V, r0 + _W_BLOCK_ROWS)
        blk = rng.standard_normal((r1 - r0, H)) * w.w_std
        out[r0:r1] = torch.from_numpy(blk).to(tdtype)
    return out


def _labels(rng, w: Workload, N: int, V: int) -> np.ndarray:
    if w.labels == "uniform":
        return rng.integers(0, V, size=N, dtype=np.int64)
    if w.labels == "zipf":
        ranks = np.arange(1, V + 1, dtype=np.float64)
        p = ranks ** (-w.zipf_s)
        p /= p.sum()
        return rng.choice(V, size=N, p=p).astype(np.int64)
    raise ValueError(w.labels)


def _ignore_mask(rng, w: Workload, N: int) -> np.ndarray:
    mask = np.zeros(N, dtype=bool)
    if w.ignore == "count":
        k = int(round(w.ignore_frac * N))
        mask[rng.permutation(N)[:k]] = True
    elif w.ignore == "prefix":
        S = w.seq_len
        max_span = int(round(2 * w.ignore_frac * S))  # mean span = ignore_frac * S
        for b in range(0, N, S):
            L = int(rng.integers(0, max_span + 1))
            mask[b:b + min(L, N - b)] = True
    else:
        raise ValueError(w.ignore)
    return mask


def make_inputs(name: str, seed: int = 0, N: int | None = None, H: int | None = None,
                V: int | None = None, dtype: str | None = None):
    """Draw (hidden, weight, labels) for workload ``name`` as CPU torch tensors.

    ``N``/``H``/``V`` override the workload's sizes (same distributions), which
    the tests use for small ragged shapes; ``dtype`` overrides the element type
    (the same float64 draws, rounded to that type). Returns a dict with the
    tensors and the call parameters (ignore_index, reduction, dtype).
    """
    w = WORKLOADS[name]
    if dtype is not None:
        w = dataclasses.replace(w, dtype=dtype)
    N = w.N if N is None else N
    H = w.H if H is None else H
    V = w.V if V is None else V
    rx, rw, ry, rm = _streams(seed)
    tdtype = w.torch_dtype
    hidden = torch.from_numpy(_hidden(rx, w, N, H)).to(tdtype)
    weight = _weight(rw, w, V, H, tdtype)
    labels = _labels(ry, w, N, V)
    labels[_ignore_mask(rm, w, N)] = IGNORE_INDEX
    return {
        "name": name, "seed": seed, "N": N, "H": H, "V": V,
        "hidden": hidden, "weight": weight, "labels": torch.from_numpy(labels),
        "ignore_index": IGNORE_INDEX, "reduction": w.reduction, "dtype": w.dtype,
    }


def make_rmsnorm_inputs(name: str, seed: int = 0, N: int | None = None, H: int | None = None,
                        V: int | None = None, dtype: str | None = None, base: dict | None = None):
    """Inputs of the step with the final RMSNorm in front: ``make_inputs`` plus pre-norm rows and a gain.

    The pre-norm rows are the workload's hidden draws (before rounding) times a per-token scale
    drawn log-uniformly in [0.25, 16] (the residual stream's magnitude varies by token), rounded to
    the dtype; the gain is 1 + 0.1 N(0, 1) per feature. Both come from a fifth stream of the seed
    (child 4 of the same SeedSequence), so weight, labels and the mask are those of ``make_inputs``;
    ``base``, the result of that very ``make_inputs`` call, saves drawing them again.
    """
    d = dict(base) if base is not None else make_inputs(name, seed, N, H, V, dtype)
    w = WORKLOADS[name]
    rx = _streams(seed)[0]
    g = _hidden(rx, w, d["N"], d["H"])                   # the same float64 draws as d["hidden"]
    extra = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed).spawn(5)[4]))
    scale = np.exp(extra.uniform(np.log(0.25), np.log(16.0), size=(d["N"], 1)))
    gamma = 1.0 + 0.1 * extra.standard_normal(d["H"])
    tdtype = TORCH_DTYPES[d["dtype"]]
    d["hidden"] = torch.from_numpy(g * scale).to(tdtype)
    d["gamma"] = torch.from_numpy(gamma).to(tdtype)
    d["eps"] = 1e-5
    d["name"] = f"{name}_rmsnorm"
    return d


def fingerprint(inputs) -> str:
    """SHA-256 over the raw bytes of hidden, weight and labels."""
    h = hashlib.sha256()
    for key in ("hidden", "weight", "labels") + (("gamma",) if "gamma" in inputs else ()):
        t = inputs[key].contiguous()
        h.update(t.view(torch.uint8).numpy().tobytes() if t.dtype != torch.int64
                 else t.numpy().tobytes())
    return h.hexdigest()


def random_case(N: int, H: int, V: int, dtype: str = "bf16", seed: int = 0,
                ignore_frac: float = 0.1, x_scale: float = 1.0, w_std: float = 0.02,
                ignore_index: int = IGNORE_INDEX):
    """A small ad-hoc case: hidden ~ x_scale*N(0,1), W ~ w_std*N(0,1), uniform labels."""
    rx, rw, ry, rm = _streams(seed)
    tdtype = TORCH_DTYPES[dtype]
    hidden = torch.from_numpy(rx.standard_normal((N, H)) * x_scale).to(tdtype)
    weight = torch.from_numpy(rw.standard_normal((V, H)) * w_std).to(tdtype)
    labels = ry.integers(0, V, size=N, dtype=np.int64)
    k = int(round(ignore_frac * N))
    labels[rm.permutation(N)[:k]] = ignore_index
    return {"name": f"random_{N}x{H}x{V}", "seed": seed, "N": N, "H": H, "V": V,
            "hidden": hidden, "weight": weight, "labels": torch.from_numpy(labels),
            "ignore_index": ignore_index, "reduction": "mean", "dtype": dtype}
