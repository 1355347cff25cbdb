"""Float64 CPU oracle (test infrastructure only; never imported by the library)."""
from .hdl_oracle import (bf16_bits_to_f64, branch_set_agrees, divergence,
                         full_logprobs, select_branch_points, select_by_value,
                         token_entropy, token_logprobs)

__all__ = ["bf16_bits_to_f64", "branch_set_agrees", "divergence", "full_logprobs",
           "select_branch_points", "select_by_value", "token_entropy", "token_logprobs"]
