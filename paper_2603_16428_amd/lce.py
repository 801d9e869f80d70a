"""Python binding of the C ABI in include/lce.h (argument marshalling only).

Every step of the fused linear + cross-entropy computation runs in the HIP
kernels of liblce.so; this module allocates the outputs and the workspace with
torch (device memory and streams are all torch is used for) and passes raw
pointers. There is no fallback: if the library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblce.so")

LCE_OK = 0
STATUS = {0: "LCE_OK", 1: "LCE_ERR_INVALID_ARGUMENT", 2: "LCE_ERR_UNSUPPORTED",
          3: "LCE_ERR_WORKSPACE_TOO_SMALL", 4: "LCE_ERR_HIP"}
DTYPES = {torch.float32: 0, torch.bfloat16: 1, torch.float16: 2}
REDUCTIONS = {"none": 0, "mean": 1, "sum": 2}
EXPORTED = ("lce_workspace_size", "lce_plan_info", "lce_auto_chunk_tokens", "lce_forward", "lce_forward_no_alloc",
            "lce_forward_backward",
            "lce_rmsnorm_workspace_size", "lce_rmsnorm_forward", "lce_rmsnorm_forward_backward",
            "lce_host_adam_step", "lce_head_train_step",
            "lce_timing_enable", "lce_timing_read", "lce_status_string")
TIMING_KINDS = ("logits_lse_gemm", "dh_gemm", "dw_gemm", "dlogits", "transpose", "other")

_lib = None


class HeadStepTiming(ctypes.Structure):
    """lce_head_step_timing_t (milliseconds)."""
    _fields_ = [("step_ms", ctypes.c_double), ("gpu_ms", ctypes.c_double), ("d2h_ms", ctypes.c_double),
                ("update_ms", ctypes.c_double), ("h2d_ms", ctypes.c_double), ("tail_ms", ctypes.c_double)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class PlanInfo(ctypes.Structure):
    """lce_plan_info_t."""
    _fields_ = [("chunk_tokens", ctypes.c_int64), ("chunks", ctypes.c_int64), ("dh_splits", ctypes.c_int32),
                ("target_referenced", ctypes.c_int32), ("dw_fp32_carry", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("workspace_bytes", ctypes.c_size_t),
                ("fallback_flags_offset", ctypes.c_size_t)]

    def as_dict(self):
        return {k: int(getattr(self, k)) for k, _ in self._fields_ if k != "reserved"}


class AdamConfig(ctypes.Structure):
    """lce_adam_config_t."""
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float)]


class LCEError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}")
        self.status = status


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load liblce.so and declare its signatures. Raises OSError if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise OSError(f"{path} is not built; run `python -m paper_2603_16428_amd.build`")
    lib = ctypes.CDLL(path)
    i64, vp, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
    lib.lce_workspace_size.argtypes = [i64, i64, i64, ctypes.c_int, ctypes.c_int, i64]
    lib.lce_workspace_size.restype = sz
    lib.lce_plan_info.argtypes = [i64, i64, i64, ctypes.c_int, ctypes.c_int, i64, ctypes.POINTER(PlanInfo)]
    lib.lce_plan_info.restype = ctypes.c_int
    lib.lce_auto_chunk_tokens.argtypes = [i64, i64, i64, ctypes.c_int]
    lib.lce_auto_chunk_tokens.restype = i64
    lib.lce_forward.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int, i64, ctypes.c_int, vp, vp, vp, sz, vp]
    lib.lce_forward.restype = ctypes.c_int
    lib.lce_forward_no_alloc.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int, i64, ctypes.c_int, vp, vp, vp]
    lib.lce_forward_no_alloc.restype = ctypes.c_int
    lib.lce_forward_backward.argtypes = [vp, vp, vp, i64, i64, i64, ctypes.c_int, i64, ctypes.c_int, vp, vp, vp,
                                         i64, vp, sz, vp]
    lib.lce_forward_backward.restype = ctypes.c_int
    f32 = ctypes.c_float
    lib.lce_rmsnorm_workspace_size.argtypes = [i64, i64, i64, ctypes.c_int, ctypes.c_int, i64]
    lib.lce_rmsnorm_workspace_size.restype = sz
    lib.lce_rmsnorm_forward.argtypes = [vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, f32, i64, ctypes.c_int,
                                        vp, vp, vp, vp, sz, vp]
    lib.lce_rmsnorm_forward.restype = ctypes.c_int
    lib.lce_rmsnorm_forward_backward.argtypes = [vp, vp, vp, vp, i64, i64, i64, ctypes.c_int, f32, i64,
                                                 ctypes.c_int, vp, vp, vp, vp, i64, vp, sz, vp]
    lib.lce_rmsnorm_forward_backward.restype = ctypes.c_int
    lib.lce_host_adam_step.argtypes = [vp, vp, ctypes.c_int, vp, vp, i64, ctypes.POINTER(AdamConfig), i64, vp,
                                       ctypes.c_int]
    lib.lce_host_adam_step.restype = ctypes.c_int
    lib.lce_head_train_step.argtypes = [vp, vp, i64, i64, i64, ctypes.c_int, i64, ctypes.c_int, i64, vp, vp, vp,
                                        vp, vp, vp, vp, vp, vp, ctypes.POINTER(AdamConfig), i64, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_int, vp, sz, vp, ctypes.POINTER(HeadStepTiming)]
    lib.lce_head_train_step.restype = ctypes.c_int
    lib.lce_timing_enable.argtypes = [ctypes.c_int]
    lib.lce_timing_enable.restype = ctypes.c_int
    lib.lce_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), ctypes.c_int]
    lib.lce_timing_read.restype = ctypes.c_int
    lib.lce_status_string.argtypes = [ctypes.c_int]
    lib.lce_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def timing_enable(enable: bool = True) -> None:
    """Start (and reset) or stop per-kernel event timing inside the library."""
    st = load_library().lce_timing_enable(int(enable))
    if st != LCE_OK:
        raise LCEError(st, "lce_timing_enable")


def timing_read() -> dict:
    """{kind: (total_ms, launches)} since the last timing_enable(True); waits for the events."""
    n = len(TIMING_KINDS)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    st = load_library().lce_timing_read(ms, cnt, n)
    if st != LCE_OK:
        raise LCEError(st, "lce_timing_read")
    return {k: (ms[i], int(cnt[i])) for i, k in enumerate(TIMING_KINDS)}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check_inputs(hidden, weight, labels):
    if not (hidden.is_cuda and weight.is_cuda and labels.is_cuda):
        raise ValueError("hidden, weight and labels must be device tensors")
    if hidden.dim() != 2 or weight.dim() != 2 or labels.dim() != 1:
        raise ValueError("expected hidden [N,H], weight [V,H], labels [N]")
    if hidden.dtype != weight.dtype or hidden.dtype not in DTYPES:
        raise ValueError("hidden and weight must have the same dtype, one of bfloat16, float16, float32")
    if labels.dtype != torch.int64:
        raise ValueError("labels must be int64")
    N, H = hidden.shape
    V, H2 = weight.shape
    if H2 != H or labels.shape[0] != N:
        raise ValueError("shape mismatch")
    if not (hidden.is_contiguous() and weight.is_contiguous() and labels.is_contiguous()):
        raise ValueError("inputs must be contiguous")
    return N, H, V


def workspace_size(N: int, H: int, V: int, dtype=torch.bfloat16, with_backward: bool = True,
                   chunk_tokens: int = 0) -> int:
    return int(load_library().lce_workspace_size(N, H, V, DTYPES[dtype], int(with_backward), chunk_tokens))


def plan_info(N: int, H: int, V: int, dtype=torch.bfloat16, with_backward: bool = True,
              chunk_tokens: int = 0) -> dict:
    """How a call with these sizes runs (lce_plan_info): chunking, dH splits, dW carry, flags offset."""
    info = PlanInfo()
    st = load_library().lce_plan_info(N, H, V, DTYPES[dtype], int(with_backward), chunk_tokens, ctypes.byref(info))
    if st != LCE_OK:
        raise LCEError(st, "lce_plan_info")
    return info.as_dict()


def auto_chunk_tokens(N: int, H: int, V: int, dtype=torch.bfloat16) -> int:
    return int(load_library().lce_auto_chunk_tokens(N, H, V, DTYPES[dtype]))


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def forward(hidden, weight, labels, ignore_index: int = -100, reduction: str = "mean",
            return_lse: bool = False, workspace: torch.Tensor | None = None):
    """Loss (scalar for mean/sum, [N] for none) and optionally each token's log-sum-exp."""
    lib = load_library()
    N, H, V = _check_inputs(hidden, weight, labels)
    dt = DTYPES[hidden.dtype]
    red = REDUCTIONS[reduction]
    need = lib.lce_workspace_size(N, H, V, dt, 0, 0)
    if need == 0:
        raise LCEError(2, "lce_workspace_size")
    ws = workspace if workspace is not None else _workspace(need, hidden.device)
    loss = torch.empty(N if red == 0 else 1, dtype=torch.float32, device=hidden.device)
    lse = torch.empty(N, dtype=torch.float32, device=hidden.device) if return_lse else None
    stream = ctypes.c_void_p(torch.cuda.current_stream(hidden.device).cuda_stream)
    st = lib.lce_forward(_ptr(hidden), _ptr(weight), _ptr(labels), N, H, V, dt, ignore_index, red,
                         _ptr(loss), _ptr(lse), _ptr(ws), ws.numel(), stream)
    if st != LCE_OK:
        raise LCEError(st, "lce_forward")
    loss = loss if red == 0 else loss[0]
    return (loss, lse) if return_lse else loss


def forward_no_alloc(hidden, weight, labels, ignore_index: int = -100, reduction: str = "mean",
                     return_lse: bool = False, loss=None, lse=None):
    """forward() through lce_forward_no_alloc: the library uses its static scratch, no workspace.
    `loss` / `lse` may be given (preallocated outputs) so that the call allocates nothing at all."""
    lib = load_library()
    N, H, V = _check_inputs(hidden, weight, labels)
    red = REDUCTIONS[reduction]
    if loss is None:
        loss = torch.empty(N if red == 0 else 1, dtype=torch.float32, device=hidden.device)
    if return_lse and lse is None:
        lse = torch.empty(N, dtype=torch.float32, device=hidden.device)
    stream = ctypes.c_void_p(torch.cuda.current_stream(hidden.device).cuda_stream)
    st = lib.lce_forward_no_alloc(_ptr(hidden), _ptr(weight), _ptr(labels), N, H, V, DTYPES[hidden.dtype],
                                  ignore_index, red, _ptr(loss), _ptr(lse if return_lse else None), stream)
    if st != LCE_OK:
        raise LCEError(st, "lce_forward_no_alloc")
    out = loss if red == 0 else loss[0]
    return (out, lse) if return_lse else out


def forward_backward(hidden, weight, labels, ignore_index: int = -100, reduction: str = "mean",
                     chunk_tokens: int = 0, workspace: torch.Tensor | None = None,
                     out: tuple | None = None):
    """(loss, grad_hidden, grad_weight) of the mean or sum loss, upstream gradient 1."""
    lib = load_library()
    N, H, V = _check_inputs(hidden, weight, labels)
    dt = DTYPES[hidden.dtype]
    red = REDUCTIONS[reduction]
    need = lib.lce_workspace_size(N, H, V, dt, 1, chunk_tokens)
    if need == 0:
        raise LCEError(2, "lce_workspace_size")
    ws = workspace if workspace is not None else _workspace(need, hidden.device)
    if out is None:
        loss = torch.empty(1, dtype=torch.float32, device=hidden.device)
        dH = torch.empty_like(hidden)
        dW = torch.empty_like(weight)
    else:
        loss, dH, dW = out
    stream = ctypes.c_void_p(torch.cuda.current_stream(hidden.device).cuda_stream)
    st = lib.lce_forward_backward(_ptr(hidden), _ptr(weight), _ptr(labels), N, H, V, dt, ignore_index, red,
                                  _ptr(loss), _ptr(dH), _ptr(dW), chunk_tokens, _ptr(ws), ws.numel(), stream)
    if st != LCE_OK:
        raise LCEError(st, "lce_forward_backward")
    return loss[0], dH, dW


class LinearCrossEntropy(torch.autograd.Function):
    """loss = cross_entropy(hidden @ weight.T, labels) without the logits tensor.

    The forward pass computes the gradients too (they come out of the same chunked pass) and the
    backward pass only scales them by the upstream gradient.
    """

    @staticmethod
    def forward(ctx, hidden, weight, labels, ignore_index=-100, reduction="mean"):
        if hidden.requires_grad or weight.requires_grad:
            loss, dH, dW = forward_backward(hidden, weight, labels, ignore_index, reduction)
            ctx.save_for_backward(dH, dW)
        else:
            loss = forward(hidden, weight, labels, ignore_index, reduction)
        return loss

    @staticmethod
    def backward(ctx, grad_out):
        dH, dW = ctx.saved_tensors
        g = grad_out.to(torch.float32)
        return (dH * g).to(dH.dtype), (dW * g).to(dW.dtype), None, None, None


def linear_cross_entropy(hidden, weight, labels, ignore_index: int = -100, reduction: str = "mean"):
    return LinearCrossEntropy.apply(hidden, weight, labels, ignore_index, reduction)


# ---- the final RMSNorm fused into the step --------------------------------------------------------

def _check_gamma(gamma, hidden):
    if gamma.dtype != hidden.dtype or gamma.dim() != 1 or gamma.shape[0] != hidden.shape[1]:
        raise ValueError("gamma must be [H] of the hidden dtype")
    if not gamma.is_contiguous() or gamma.device != hidden.device:
        raise ValueError("gamma must be contiguous and on the hidden's device")


def rmsnorm_workspace_size(N: int, H: int, V: int, dtype=torch.bfloat16, with_backward: bool = True,
                           chunk_tokens: int = 0) -> int:
    return int(load_library().lce_rmsnorm_workspace_size(N, H, V, DTYPES[dtype], int(with_backward), chunk_tokens))


def rmsnorm_forward(hidden, gamma, weight, labels, eps: float = 1e-5, ignore_index: int = -100,
                    reduction: str = "mean", return_lse: bool = False, return_normed: bool = False,
                    workspace: torch.Tensor | None = None):
    """Loss of the step on x = RMSNorm(hidden) * gamma; optionally each token's lse and x itself."""
    lib = load_library()
    N, H, V = _check_inputs(hidden, weight, labels)
    _check_gamma(gamma, hidden)
    dt = DTYPES[hidden.dtype]
    red = REDUCTIONS[reduction]
    need = lib.lce_rmsnorm_workspace_size(N, H, V, dt, 0, 0)
    if need == 0:
        raise LCEError(2, "lce_rmsnorm_workspace_size")
    ws = workspace if workspace is not None else _workspace(need, hidden.device)
    loss = torch.empty(N if red == 0 else 1, dtype=torch.float32, device=hidden.device)
    lse = torch.empty(N, dtype=torch.float32, device=hidden.device) if return_lse else None
    normed = torch.empty_like(hidden) if return_normed else None
    stream = ctypes.c_void_p(torch.cuda.current_stream(hidden.device).cuda_stream)
    st = lib.lce_rmsnorm_forward(_ptr(hidden), _ptr(gamma), _ptr(weight), _ptr(labels), N, H, V, dt, float(eps),
                                 ignore_index, red, _ptr(loss), _ptr(lse), _ptr(normed), _ptr(ws), ws.numel(), stream)
    if st != LCE_OK:
        raise LCEError(st, "lce_rmsnorm_forward")
    out = (loss if red == 0 else loss[0],)
    if return_lse:
        out += (lse,)
    if return_normed:
        out += (normed,)
    return out if len(out) > 1 else out[0]


def rmsnorm_forward_backward(hidden, gamma, weight, labels, eps: float = 1e-5, ignore_index: int = -100,
                             reduction: str = "mean", chunk_tokens: int = 0,
                             workspace: torch.Tensor | None = None):
    """(loss, grad_hidden, grad_gamma, grad_weight); grad_hidden is with respect to the pre-norm rows."""
    lib = load_library()
    N, H, V = _check_inputs(hidden, weight, labels)
    _check_gamma(gamma, hidden)
    dt = DTYPES[hidden.dtype]
    red = REDUCTIONS[reduction]
    need = lib.lce_rmsnorm_workspace_size(N, H, V, dt, 1, chunk_tokens)
    if need == 0:
        raise LCEError(2, "lce_rmsnorm_workspace_size")
    ws = workspace if workspace is not None else _workspace(need, hidden.device)
    loss = torch.empty(1, dtype=torch.float32, device=hidden.device)
    dh = torch.empty_like(hidden)
    dg = torch.empty_like(gamma)
    dW = torch.empty_like(weight)
    stream = ctypes.c_void_p(torch.cuda.current_stream(hidden.device).cuda_stream)
    st = lib.lce_rmsnorm_forward_backward(_ptr(hidden), _ptr(gamma), _ptr(weight), _ptr(labels), N, H, V, dt,
                                          float(eps), ignore_index, red, _ptr(loss), _ptr(dh), _ptr(dg), _ptr(dW),
                                          chunk_tokens, _ptr(ws), ws.numel(), stream)
    if st != LCE_OK:
        raise LCEError(st, "lce_rmsnorm_forward_backward")
    return loss[0], dh, dg, dW


class RMSNormLinearCrossEntropy(torch.autograd.Function):
    """loss = cross_entropy(rms_norm(hidden, gamma, eps) @ weight.T, labels), fused, without logits."""

    @staticmethod
    def forward(ctx, hidden, gamma, weight, labels, eps=1e-5, ignore_index=-100, reduction="mean"):
        if hidden.requires_grad or gamma.requires_grad or weight.requires_grad:
            loss, dh, dg, dW = rmsnorm_forward_backward(hidden, gamma, weight, labels, eps, ignore_index, reduction)
            ctx.save_for_backward(dh, dg, dW)
        else:
            loss = rmsnorm_forward(hidden, gamma, weight, labels, eps, ignore_index, reduction)
        return loss

    @staticmethod
    def backward(ctx, grad_out):
        dh, dg, dW = ctx.saved_tensors
        g = grad_out.to(torch.float32)
        return (dh * g).to(dh.dtype), (dg * g).to(dg.dtype), (dW * g).to(dW.dtype), None, None, None, None


def rmsnorm_linear_cross_entropy(hidden, gamma, weight, labels, eps: float = 1e-5, ignore_index: int = -100,
                                 reduction: str = "mean"):
    return RMSNormLinearCrossEntropy.apply(hidden, gamma, weight, labels, eps, ignore_index, reduction)


# ---- host optimizer step --------------------------------------------------------------------------

def host_adam_step(param, grad, exp_avg, exp_avg_sq, step: int, lr: float, betas=(0.9, 0.999), eps: float = 1e-8,
                   weight_decay: float = 0.0, param16=None, threads: int = 0) -> None:
    """AdamW on host fp32 tensors in place (grad: host bf16/fp16/fp32); optionally writes param16."""
    lib = load_library()
    for t in (param, exp_avg, exp_avg_sq):
        if t.device.type != "cpu" or t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("param and states must be contiguous host float32 tensors")
    n = param.numel()
    if grad.device.type != "cpu" or grad.numel() != n or not grad.is_contiguous() or grad.dtype not in DTYPES:
        raise ValueError("grad must be a contiguous host tensor of the same size")
    if exp_avg.numel() != n or exp_avg_sq.numel() != n:
        raise ValueError("state sizes differ from the parameter's")
    if param16 is not None and (param16.dtype != grad.dtype or param16.numel() != n or param16.device.type != "cpu"
                                or not param16.is_contiguous()):
        raise ValueError("param16 must be a contiguous host tensor of the gradient's dtype")
    cfg = AdamConfig(lr, betas[0], betas[1], eps, weight_decay)
    st = lib.lce_host_adam_step(_ptr(param), _ptr(grad), DTYPES[grad.dtype], _ptr(exp_avg), _ptr(exp_avg_sq), n,
                                ctypes.byref(cfg), step, _ptr(param16), threads)
    if st != LCE_OK:
        raise LCEError(st, "lce_host_adam_step")


# ---- a training step of the output layer with host-resident weights -------------------------------

class HeadState:
    """Host and device buffers of the output layer for lce_head_train_step.

    The FP32 master copy and the Adam states live in host memory; the 16-bit gradient and parameter
    buffers are pinned (torch's pin_memory allocates page-locked memory); `weight` is the device copy
    the step reads and refreshes.
    """

    def __init__(self, weight: torch.Tensor):
        if weight.dtype not in (torch.bfloat16, torch.float16) or not weight.is_cuda:
            raise ValueError("weight must be a bf16 or fp16 device tensor")
        self.weight = weight
        self.master = weight.detach().float().cpu()
        self.exp_avg = torch.zeros_like(self.master)
        self.exp_avg_sq = torch.zeros_like(self.master)
        self.grad_host = torch.empty(weight.shape, dtype=weight.dtype, pin_memory=True)
        self.param_host = torch.empty(weight.shape, dtype=weight.dtype, pin_memory=True)
        self.grad_weight = torch.empty_like(weight)
        self.step = 0


def head_train_step(state: HeadState, hidden, labels, lr: float, betas=(0.9, 0.999), eps: float = 1e-8,
                    weight_decay: float = 0.0, ignore_index: int = -100, reduction: str = "mean",
                    chunk_tokens: int = 0, vocab_blocks: int = 8, threads: int = 0, overlap: bool = True,
                    workspace: torch.Tensor | None = None):
    """One step: loss and dH on the device, W updated through the host; returns (loss, dH, timing)."""
    lib = load_library()
    W = state.weight
    N, H, V = _check_inputs(hidden, W, labels)
    dt = DTYPES[hidden.dtype]
    red = REDUCTIONS[reduction]
    need = lib.lce_workspace_size(N, H, V, dt, 1, chunk_tokens)
    if need == 0:
        raise LCEError(2, "lce_workspace_size")
    ws = workspace if workspace is not None else _workspace(need, hidden.device)
    loss = torch.empty(1, dtype=torch.float32, device=hidden.device)
    dH = torch.empty_like(hidden)
    state.step += 1
    cfg = AdamConfig(lr, betas[0], betas[1], eps, weight_decay)
    timing = HeadStepTiming()
    stream = ctypes.c_void_p(torch.cuda.current_stream(hidden.device).cuda_stream)
    st = lib.lce_head_train_step(_ptr(hidden), _ptr(labels), N, H, V, dt, ignore_index, red, chunk_tokens, _ptr(W),
                                 _ptr(dH), _ptr(state.grad_weight), _ptr(loss), _ptr(state.master),
                                 _ptr(state.exp_avg), _ptr(state.exp_avg_sq), _ptr(state.grad_host),
                                 _ptr(state.param_host), ctypes.byref(cfg), state.step, vocab_blocks, threads,
                                 int(overlap), _ptr(ws), ws.numel(), stream, ctypes.byref(timing))
    if st != LCE_OK:
        state.step -= 1
        raise LCEError(st, "lce_head_train_step")
    return loss[0], dH, timing.as_dict()
