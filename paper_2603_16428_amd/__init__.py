"""Fused linear + cross-entropy (output projection and loss) for MI355X, in HIP."""
from .lce import (LCEError, LinearCrossEntropy, auto_chunk_tokens, forward, forward_backward,
                  linear_cross_entropy, load_library, timing_enable, timing_read, workspace_size)

__all__ = ["LCEError", "LinearCrossEntropy", "auto_chunk_tokens", "forward", "forward_backward",
           "linear_cross_entropy", "load_library", "timing_enable", "timing_read", "workspace_size"]
