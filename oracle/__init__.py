"""Float64 CPU oracle for the fused linear + cross-entropy step (test infrastructure only)."""
from .lce import (forward, forward_backward, grad_hidden_rows, grad_weight_rows,
                  log_sum_exp_rows, row_stats, token_weights)

__all__ = ["forward", "forward_backward", "grad_hidden_rows", "grad_weight_rows",
           "log_sum_exp_rows", "row_stats", "token_weights"]
