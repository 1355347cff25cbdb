"""GPU parity of the Entropy localization baseline (Sec. 4.1, Table 4): the
next-token entropy accumulated by the fused lm-head kernel, and the per-root
top-k over a per-position value, against the float64 oracle through the C ABI.

Tolerances: |entropy error| <= 2e-3 nats for bf16 inputs and <= 1e-4 for fp32
inputs, the same bars as log p (entropy is lse minus an fp32-accumulated mean
logit, so its error is of the order of the lse error).  The top-k over values
is integer work and is compared bit-exactly on identical fp32 inputs.
"""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O
from tests.gpu_helpers import as_f64, flat_inputs, oracle_rows, require_gpu

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-3
TOL_F32 = 1e-4


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


def _run(hdl, hidden, W, tokens, mask, bitwise=False):
    h, Wd = hidden.cuda(), W.cuda()
    t = tokens.to(device="cuda", dtype=torch.int32)
    m = None if mask is None else mask.to(device="cuda", dtype=torch.uint8)
    lp, lse, ent = hdl.token_logprobs(h, Wd, t, m, want_entropy=True)
    lp0, lse0 = hdl.token_logprobs(h, Wd, t, m)
    torch.cuda.synchronize()
    if bitwise:
        # asking for the entropy leaves log p and lse bit-for-bit unchanged
        assert torch.equal(lp.view(torch.int32), lp0.view(torch.int32))
        assert torch.equal(lse.view(torch.int32), lse0.view(torch.int32))
    else:
        assert torch.equal(torch.isnan(lp), torch.isnan(lp0))
        ok = ~torch.isnan(lp)
        assert torch.allclose(lp[ok], lp0[ok], rtol=0, atol=1e-6)
    return lp.cpu().numpy(), lse.cpu().numpy(), ent.cpu().numpy()


def test_entropy_leaves_logp_bitwise_unchanged(hdl):
    w = workloads.make_workload("c4", R=2, T=700, d=128, V=20000)
    hidden, W, tokens, mask = flat_inputs(w)
    _run(hdl, hidden, W, tokens, mask, bitwise=True)
    g = torch.Generator().manual_seed(14)
    H = torch.randn(300, 72, generator=g).to(torch.bfloat16)       # K-tail instantiation
    Wt = (torch.randn(4133, 72, generator=g) * 0.05).to(torch.bfloat16)
    _run(hdl, H, Wt, torch.randint(0, 4133, (300,), generator=g, dtype=torch.int32), None, bitwise=True)


def _oracle_entropy(hidden, W, rows):
    return O.token_entropy(as_f64(hidden[torch.as_tensor(rows, dtype=torch.long)]), as_f64(W))


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("c2", dict(R=2, T=300, d=256)),                    # V = 151936: ragged last V-tile
    ("c4", dict(R=3, T=700, d=128, V=20000)),           # masked observation spans
])
def test_entropy_matches_oracle(hdl, name, over):
    w = workloads.make_workload(name, **over)
    hidden, W, tokens, mask = flat_inputs(w)
    tol = TOL_F32 if hidden.dtype == torch.float32 else TOL_BF16
    lp, lse, ent = _run(hdl, hidden, W, tokens, mask)
    m = mask.numpy().astype(bool)
    rows = np.nonzero(m)[0]
    want = _oracle_entropy(hidden, W, rows)
    err = np.abs(ent[rows] - want)
    assert err.max() <= tol, f"max |H err| {err.max():.3g} at row {rows[err.argmax()]}"
    assert np.all(ent[~m] == 0.0)
    assert np.all(ent >= 0.0) and np.all(ent <= math.log(w.cfg.V) + tol)
    want_lp, _ = oracle_rows(hidden, W, tokens, rows)
    assert np.abs(lp[rows] - want_lp).max() <= tol


@pytest.mark.parametrize("n_rows,d,V,dtype", [
    (257, 8, 1000, torch.bfloat16),      # K tail shorter than one slice
    (300, 72, 4133, torch.bfloat16),     # K tail after a slice, ragged vocab
    (1000, 2056, 2048, torch.bfloat16),  # long K with a tail
    (300, 40, 777, torch.float32),
    (513, 256, 4096, torch.float32),
])
def test_entropy_shape_edges(hdl, n_rows, d, V, dtype):
    g = torch.Generator().manual_seed(n_rows * 3 + d * 5 + V)
    W = (torch.randn(V, d, generator=g) * 0.05).to(dtype)
    H = torch.randn(n_rows, d, generator=g).to(dtype)
    y = torch.randint(0, V, (n_rows,), generator=g, dtype=torch.int32)
    _, _, ent = _run(hdl, H, W, y, None)
    want = _oracle_entropy(H, W, np.arange(n_rows))
    tol = TOL_F32 if dtype == torch.float32 else TOL_BF16
    assert np.abs(ent - want).max() <= tol


def test_entropy_closed_forms(hdl):
    # zero hidden state: uniform distribution, H = log V; a row whose logits
    # are one huge spike: H ~ 0; out-of-range token: log p is NaN but the
    # entropy of the row (which does not depend on the token) stays finite
    g = torch.Generator().manual_seed(12)
    V, d = 3001, 64
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(4, d, generator=g).to(torch.bfloat16)
    H[0] = 0
    W[123] = 0
    W[123, 0] = 64.0
    H[1] = 0
    H[1, 0] = 64.0                          # logit 4096 on token 123, others ~|0.05*64|
    y = torch.tensor([5, 123, -1, 7], dtype=torch.int32)
    lp, _, ent = _run(hdl, H, W, y, None)
    assert abs(ent[0] - math.log(V)) <= 1e-4
    assert ent[1] <= 1e-6
    assert math.isnan(lp[2]) and np.isfinite(ent[2])
    want = _oracle_entropy(H, W, [2, 3])
    assert np.abs(ent[2:] - want).max() <= TOL_BF16


def test_entropy_masked_rows_zero_and_empty_mask(hdl):
    g = torch.Generator().manual_seed(13)
    n, d, V = 600, 64, 2000
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    _, _, ent = _run(hdl, H, W, y, torch.zeros(n, dtype=torch.uint8))
    assert np.all(ent == 0.0)
    m = (torch.rand(n, generator=g) < 0.2).to(torch.uint8)
    _, _, ent = _run(hdl, H, W, y, m)
    rows = np.nonzero(m.numpy())[0]
    assert np.abs(ent[rows] - _oracle_entropy(H, W, rows)).max() <= TOL_BF16
    assert np.all(ent[m.numpy() == 0] == 0.0)


# ------------------------------------------------------ top-k over values
def _values_case(R, T, seed):
    rng = np.random.default_rng(seed)
    v = rng.gamma(2.0, 1.0, (R, T)).astype(np.float32)       # entropy-like, >= 0
    v[:, ::7] *= -1                                           # negatives too
    for r in range(R):                                        # exact ties and signed zeros
        a, b = rng.integers(0, T, (2, 6))
        v[r, b] = v[r, a]
        v[r, rng.integers(0, T, 3)] = 0.0
        v[r, rng.integers(0, T, 3)] = -0.0
        v[r, rng.integers(0, T, 2)] = np.nan
        v[r, rng.integers(0, T)] = np.inf
    mask = (rng.random((R, T)) < 0.85).astype(np.uint8)
    return v, mask


@pytest.mark.parametrize("R,T,k", [(1, 1, 1), (3, 257, 2), (8, 4096, 8), (2, 9000, 64),
                                   (5, 300, 1024), (2, 40000, 16), (1, 33000, 700)])
def test_select_top_k_bit_exact_vs_oracle(hdl, R, T, k):
    v, mask = _values_case(R, T, seed=R * 31 + T + k)
    for m in (mask, None):
        idx, score, count = hdl.select_top_k(torch.from_numpy(v).cuda(),
                                             None if m is None else torch.from_numpy(m).cuda(), k)
        torch.cuda.synchronize()
        oi, osc, oc = O.select_by_value(v, m, k)
        assert np.array_equal(count.cpu().numpy(), oc)
        assert np.array_equal(idx.cpu().numpy(), oi)
        # -0 ranks as +0 and is reported as +0
        assert np.array_equal(score.cpu().numpy().view(np.uint32),
                              (osc.astype(np.float32) + np.float32(0.0)).view(np.uint32))


def test_select_top_k_all_masked_and_boundary_errors(hdl):
    v = torch.ones(2, 50, device="cuda")
    idx, score, count = hdl.select_top_k(v, torch.zeros(2, 50, dtype=torch.uint8, device="cuda"), 3)
    torch.cuda.synchronize()
    assert count.tolist() == [0, 0] and torch.all(idx == -1) and torch.all(score == 0)
    with pytest.raises(hdl.HdlError):
        hdl.select_top_k(v, None, 0)
    with pytest.raises(hdl.HdlError):
        hdl.select_top_k(v, None, hdl.HDL_MAX_K + 1)


def test_entropy_baseline_end_to_end(hdl):
    # the Entropy baseline ranks positions of the ORIGINAL context by H; the
    # GPU branch set must agree with the oracle's under the tie-tolerant rule
    w = workloads.make_workload("c2", R=3, T=400, d=128, V=6000)
    c = w.cfg
    hidden, W, tokens, mask = flat_inputs(w)
    n0 = c.R * c.T
    _, _, ent = _run(hdl, hidden[:n0], W, tokens[:n0], mask[:n0])
    idx, score, count = hdl.select_top_k(torch.from_numpy(ent).cuda().view(c.R, c.T),
                                         w.mask.cuda(), c.k)
    torch.cuda.synchronize()
    m = w.mask.numpy().astype(bool)
    want = np.zeros(n0)
    rows = np.nonzero(m.reshape(-1))[0]
    want[rows] = _oracle_entropy(hidden[:n0], W, rows)
    want = want.reshape(c.R, c.T)
    for r in range(c.R):
        ok, why = O.branch_set_agrees(idx[r].cpu().numpy(), int(count[r]), want[r], m[r], c.k,
                                      gap=2 * TOL_BF16)
        assert ok, f"root {r}: {why}"
