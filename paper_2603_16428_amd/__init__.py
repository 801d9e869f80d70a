"""Fused linear + cross-entropy (output projection and loss) for MI355X, in HIP."""
from .lce import (AdamConfig, HeadState, HeadStepTiming, LCEError, LinearCrossEntropy, PlanInfo,
                  RMSNormLinearCrossEntropy, auto_chunk_tokens, forward, forward_backward, forward_no_alloc, head_train_step,
                  host_adam_step, linear_cross_entropy, load_library, plan_info, rmsnorm_forward,
                  rmsnorm_forward_backward, rmsnorm_linear_cross_entropy, rmsnorm_workspace_size, timing_enable,
                  timing_read, workspace_size)

__all__ = ["AdamConfig", "HeadState", "HeadStepTiming", "LCEError", "LinearCrossEntropy", "PlanInfo",
           "RMSNormLinearCrossEntropy", "auto_chunk_tokens", "forward", "forward_backward", "forward_no_alloc",
           "head_train_step",
           "host_adam_step", "linear_cross_entropy", "load_library", "plan_info", "rmsnorm_forward",
           "rmsnorm_forward_backward", "rmsnorm_linear_cross_entropy", "rmsnorm_workspace_size", "timing_enable",
           "timing_read", "workspace_size"]
