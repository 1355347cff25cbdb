"""Float64 CPU oracle (test infrastructure only; never imported by the library)."""
from .hdl_oracle import (allocate_continuations, bf16_bits_to_f64, branch_set_agrees, divergence,
                         full_logprobs, group_advantages, policy_loss_grad, select_branch_points,
                         select_by_value, select_constrained, token_entropy, token_logprobs,
                         token_logprobs_backward)

__all__ = ["allocate_continuations", "bf16_bits_to_f64", "branch_set_agrees", "divergence",
           "full_logprobs", "group_advantages", "policy_loss_grad", "select_branch_points",
           "select_by_value", "select_constrained", "token_entropy", "token_logprobs",
           "token_logprobs_backward"]
