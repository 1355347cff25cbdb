"""Seeded sweep of random shapes through the C ABI against the float64 oracle:
log p, lse and the next-token entropy for every scored row (Eq. 1; the
Entropy baseline of Sec. 4.1), and for bf16 inputs dL/dh and dL/dW of the
token-level loss (Sec. 3.3).  The shapes are drawn once from a fixed seed so
the cases are the same on every run (48 of them: 16 small, 32 wider, with
up to 3,000 rows, d up to 1,024 and vocabularies up to 40,000); together
they hit ragged row tiles,
ragged vocabulary tiles (down to V = 1), K tails (d not a multiple of 64)
and sparse or dense masks.

Tolerances as elsewhere: 2e-3 (bf16 inputs) and 1e-4 (fp32 inputs) for log p,
lse and entropy; for the gradients tests/gpu_helpers.grad_tol ((2^-8 +
2^-12) times the oracle's magnitude sums plus 1e-6 of the largest: G is
rounded to bf16 once).
"""
import numpy as np
import pytest
import torch

from oracle import hdl_oracle as O
from tests.gpu_helpers import as_f64, grad_tol, require_gpu

pytestmark = pytest.mark.gpu


def _cases():
    rng = np.random.default_rng(20261202)
    out = []
    for i in range(16):
        bf16 = i % 4 != 3
        n = int(rng.integers(1, 1500))
        d = 8 * int(rng.integers(1, 80))
        V = int(rng.choice([1, 2, int(rng.integers(3, 600)), int(rng.integers(600, 6000))],
                           p=[0.1, 0.1, 0.3, 0.5]))
        density = float(rng.choice([1.0, 0.7, 0.05]))
        out.append((i, bf16, n, d, V, density))
    # wider shapes: up to 3,000 rows, d up to 1,024, vocabularies up to 40,000
    rng = np.random.default_rng(20261203)
    for i in range(16, 48):
        bf16 = i % 5 != 4
        n = int(rng.integers(1, 3000))
        d = 8 * int(rng.integers(1, 129))
        V = int(rng.choice([int(rng.integers(1, 300)), int(rng.integers(300, 5000)), int(rng.integers(5000, 40000))]))
        density = float(rng.choice([1.0, 0.5, 0.02]))
        out.append((i, bf16, n, d, V, density))
    return out


CASES = _cases()


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


def _inputs(case):
    i, bf16, n, d, V, density = case
    g = torch.Generator().manual_seed(1000 + i)
    W = torch.randn(V, d, generator=g) * 0.05
    H = torch.randn(n, d, generator=g)
    if bf16:
        W, H = W.to(torch.bfloat16), H.to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    m = (torch.rand(n, generator=g) < density).to(torch.uint8)
    up = torch.randn(n, generator=g, dtype=torch.float32)
    return H, W, y, m, up


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{'bf16' if c[1] else 'f32'}-n{c[2]}-d{c[3]}-V{c[4]}"
                                              for c in CASES])
def test_random_shapes_against_oracle(hdl, case):
    _, bf16, n, d, V, _ = case
    tol = 2e-3 if bf16 else 1e-4
    H, W, y, m, up = _inputs(case)
    Hd, Wd, yd, md = H.cuda(), W.cuda(), y.cuda(), m.cuda()
    lp, lse, ent = hdl.token_logprobs(Hd, Wd, yd, md, want_entropy=True)
    torch.cuda.synchronize()
    lp, lse, ent = lp.cpu().numpy(), lse.cpu().numpy(), ent.cpu().numpy()
    keep = m.numpy() != 0
    rows = np.nonzero(keep)[0]
    assert np.all(lp[~keep] == 0.0) and np.all(ent[~keep] == 0.0)
    if rows.size:
        H64, W64 = as_f64(H), as_f64(W)
        want, want_lse = O.token_logprobs(H64[rows], W64, y.numpy()[rows])
        assert np.abs(lp[rows] - want).max() <= tol
        assert np.abs(lse[rows] - want_lse).max() <= tol
        want_ent = O.token_entropy(H64[rows], W64)
        assert np.abs(ent[rows] - want_ent).max() <= tol
    if not bf16 or n * V * d > 1.5e9:
        return
    _, lse_d = hdl.token_logprobs(Hd, Wd, yd, md)
    dh, dw = hdl.token_logprobs_backward(Hd, Wd, yd, md, lse_d, up.cuda())
    torch.cuda.synchronize()
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(as_f64(H), as_f64(W), y.numpy(),
                                                                 up.double().numpy(), m.numpy())
    got_dh, got_dw = dh.cpu().double().numpy(), dw.cpu().double().numpy()
    assert np.all(got_dh[~keep] == 0.0)
    # p = exp(z - lse) in fp32 is off by a few ulps of |z - lse| (< 2^-16
    # relative here), which moves G by |g| 2^-16 even where the exact G is 0
    # (V = 1): add that to the bf16 rounding bound
    ag = np.abs(up.double().numpy()) * keep
    fp_dh = 2.0 ** -16 * ag[:, None] * np.abs(as_f64(W)).sum(0)[None, :]
    fp_dw = 2.0 ** -16 * (ag[:, None] * np.abs(as_f64(H))).sum(0)[None, :]
    assert np.all(np.abs(got_dh - want_dh) <= grad_tol(mag_dh, fp_dh))
    assert np.all(np.abs(got_dw - want_dw) <= grad_tol(mag_dw, fp_dw))
