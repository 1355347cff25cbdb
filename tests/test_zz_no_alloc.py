"""The allocation-free entry point, hdl_token_logprobs_noalloc, through the C
ABI, against the workspace entry point hdl_token_logprobs on the same inputs,
on two calls in a row, the second with a smaller input:

1. 131,072 rows x V = 151,936 (d = 256, bf16): the default chunking's partials
   (38 chunks, about 60 MB) do not fit the library's 32 MiB array, so the call
   runs with fewer, longer chunks; log p and lse agree within the bf16
   tolerance (2e-3) with the workspace entry point and with the oracle on a
   seeded sample of rows;
2. 5,000 rows x V = 30,000 (d = 200, a K tail): the default chunking fits, so
   the results are bit-identical to the workspace entry point's although the
   array still holds the first call's data.

Outputs are pre-filled with NaN so that an element the call fails to write
shows up.  A call too large for the array is rejected before anything runs.
"""
import ctypes

import numpy as np
import pytest
import torch

from oracle import hdl_oracle as O
from tests.gpu_helpers import as_f64, require_gpu

pytestmark = pytest.mark.gpu

TOL = 2e-3
HDL_BF16 = 1


@pytest.fixture(scope="module")
def lib():
    hdl = require_gpu()
    return hdl.load_library()


def _inputs(n, d, V, seed):
    gen = torch.Generator(device="cuda").manual_seed(seed)
    H = torch.randn(n, d, device="cuda", generator=gen).to(torch.bfloat16)
    W = (torch.randn(V, d, device="cuda", generator=gen) * 0.05).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), device="cuda", dtype=torch.int32, generator=gen)
    m = (torch.rand(n, device="cuda", generator=gen) < 0.9).to(torch.uint8)
    return H, W, y, m


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _run_workspace(lib, H, W, y, m):
    n, d = H.shape
    V = W.shape[0]
    nbytes = lib.hdl_token_logprobs_workspace_size(n, d, V, HDL_BF16)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    logp = torch.full((n,), float("nan"), device="cuda")
    lse = torch.full((n,), float("nan"), device="cuda")
    st = lib.hdl_token_logprobs(H.data_ptr(), W.data_ptr(), y.data_ptr(), m.data_ptr(), n, d, V, HDL_BF16,
                                logp.data_ptr(), lse.data_ptr(), ws.data_ptr(), nbytes, _stream())
    assert st == 0, lib.hdl_last_hip_error()
    return logp, lse


def _run_noalloc(lib, H, W, y, m):
    n, d = H.shape
    V = W.shape[0]
    logp = torch.full((n,), float("nan"), device="cuda")
    lse = torch.full((n,), float("nan"), device="cuda")
    st = lib.hdl_token_logprobs_noalloc(H.data_ptr(), W.data_ptr(), y.data_ptr(), m.data_ptr(), n, d, V,
                                        HDL_BF16, logp.data_ptr(), lse.data_ptr(), _stream())
    assert st == 0, lib.hdl_last_hip_error()
    return logp, lse


def test_noalloc_matches_workspace_entry_point_on_two_calls(lib):
    # call 1: the array is too small for the default chunking
    H, W, y, m = _inputs(131072, 256, 151936, seed=21)
    ref_lp, ref_lse = _run_workspace(lib, H, W, y, m)
    lp, lse = _run_noalloc(lib, H, W, y, m)
    torch.cuda.synchronize()
    on = m.bool()
    assert torch.isfinite(lp).all() and torch.isfinite(lse).all()
    assert torch.all(lp[~on] == 0) and torch.all(lse[~on] == 0)
    err = (lp - ref_lp).abs().max().item()
    print(f"call 1: max |log p (noalloc) - log p (workspace)| = {err:.3g}")
    assert err <= TOL and (lse - ref_lse).abs().max().item() <= TOL
    rows = np.sort(np.random.default_rng(4).choice(np.nonzero(on.cpu().numpy())[0], 48, replace=False))
    idx = torch.as_tensor(rows, device="cuda")
    want, want_lse = O.token_logprobs(as_f64(H[idx].cpu()), as_f64(W.cpu()), y[idx].cpu().numpy())
    assert np.abs(lp[idx].cpu().numpy() - want).max() <= TOL
    assert np.abs(lse[idx].cpu().numpy() - want_lse).max() <= TOL
    del H, W, y, m

    # call 2: smaller; the default chunking fits, so bit-identical results
    H, W, y, m = _inputs(5000, 200, 30000, seed=22)
    ref_lp, ref_lse = _run_workspace(lib, H, W, y, m)
    lp, lse = _run_noalloc(lib, H, W, y, m)
    torch.cuda.synchronize()
    assert torch.equal(lp.view(torch.int32), ref_lp.view(torch.int32))
    assert torch.equal(lse.view(torch.int32), ref_lse.view(torch.int32))
    on = m.bool()
    rows = np.nonzero(on.cpu().numpy())[0][::50]
    idx = torch.as_tensor(rows, device="cuda")
    want, _ = O.token_logprobs(as_f64(H[idx].cpu()), as_f64(W.cpu()), y[idx].cpu().numpy())
    assert np.abs(lp[idx].cpu().numpy() - want).max() <= TOL


def test_noalloc_rejects_calls_beyond_the_array(lib):
    # d = 8 bf16: one launch could take 2^28 rows; 3 million rows need 48 MB
    # of the 32 MiB array, so the call is refused before anything runs
    n, d, V = 3_000_000, 8, 1000
    H = torch.zeros(n, d, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(V, d, dtype=torch.bfloat16, device="cuda")
    y = torch.zeros(n, dtype=torch.int32, device="cuda")
    logp = torch.full((n,), 7.0, device="cuda")
    st = lib.hdl_token_logprobs_noalloc(H.data_ptr(), W.data_ptr(), y.data_ptr(), None, n, d, V, HDL_BF16,
                                        logp.data_ptr(), None, _stream())
    torch.cuda.synchronize()
    assert st == -2 and b"scratch" in lib.hdl_last_hip_error()
    assert torch.all(logp == 7.0)
