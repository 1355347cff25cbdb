"""Shared helpers for the GPU tests: move a workload to the device, run the
library, and compute oracle values for chosen rows.  The oracle side only
sees CPU copies of the generator's inputs."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import hdl_oracle as O


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_36864_amd as hdl
    hdl.load_library()   # raises (test fails) if the library is missing on a machine with a GPU
    return hdl


def as_f64(t: torch.Tensor) -> np.ndarray:
    """Exact float64 view of a CPU bf16/fp32 tensor, decoded by the oracle."""
    if t.dtype == torch.bfloat16:
        return O.bf16_bits_to_f64(t.contiguous().view(torch.int16).numpy().view(np.uint16))
    return t.double().numpy()


# Gradient tolerance (the backward pass rounds the logit gradient G once to
# bf16).  bf16 has 8 significant bits, so round-to-nearest moves an element
# by at most 2^-8 of itself, and an output element sum_v G W (or sum_n G h)
# by at most 2^-8 times the magnitude sum sum_v |G| |W| -- a worst case that
# is nearly reached where one term dominates the sum, as the sampled token's
# column g (1 - p_y) does in dL/dh.  The fp32 accumulation over K terms
# (error growing like sqrt(K) 2^-24, below 2^-15 of the magnitude sum for
# K <= 2^18) and the fp32 evaluation of p (a few ulps) come on top: the tests
# allow 2^-12 of the magnitude sum for them, and 1e-6 of the largest
# magnitude sum for outputs whose own sum is near zero.
GRAD_ROUND = 2.0 ** -8
GRAD_EXTRA = 2.0 ** -12


def grad_tol(mag: np.ndarray, extra=0.0) -> np.ndarray:
    """Allowed |GPU - oracle| of a gradient element with magnitude sum mag."""
    return (GRAD_ROUND + GRAD_EXTRA) * mag + extra + 1e-6 * mag.max()


def flat_inputs(w):
    """Row-major inputs of one call covering both contexts."""
    return w.rows_hidden(), w.W, w.rows_tokens(), w.rows_mask()


def run_logprobs(hdl, hidden, W, tokens, mask, device="cuda"):
    h = hidden.to(device)
    Wd = W.to(device)
    t = tokens.to(device=device, dtype=torch.int32)
    m = None if mask is None else mask.to(device=device, dtype=torch.uint8)
    logp, lse = hdl.token_logprobs(h, Wd, t, m)
    torch.cuda.synchronize()
    return logp.cpu().numpy(), lse.cpu().numpy()


def oracle_rows(hidden_cpu, W_cpu, tokens_cpu, rows, Wf64=None):
    """Oracle log p and lse for the listed rows only."""
    Wd = as_f64(W_cpu) if Wf64 is None else Wf64
    H = as_f64(hidden_cpu[torch.as_tensor(rows, dtype=torch.long)])
    y = tokens_cpu.numpy()[np.asarray(rows)]
    return O.token_logprobs(H, Wd, y)
