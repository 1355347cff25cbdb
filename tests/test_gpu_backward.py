"""GPU parity of the backward pass of the fused lm-head log-probability
(gradients of sum_n g_n log p_n(y_n), the token-level policy loss of Sec. 3.3)
against the float64 oracle, through the C ABI.

Tolerance (derived from the arithmetic, tests/gpu_helpers.grad_tol): the
library rounds the logit gradient G = g (1[v == y] - p) to bf16 (relative
error <= 2^-8 per element: 8 significant bits) and accumulates in fp32, so
each element of dH = G W and dW = G^T H may move by at most 2^-8 sum |G| |W|
(resp. sum |G| |h|) plus the fp32 accumulation error; the tests allow
(2^-8 + 2^-12) times the oracle's magnitude sums plus 1e-6 of the largest.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O
from tests.gpu_helpers import as_f64, grad_tol, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


def _case(n, d, V, seed, mask_p=0.7):
    g = torch.Generator().manual_seed(seed)
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    m = (torch.rand(n, generator=g) < mask_p).to(torch.uint8)
    up = torch.randn(n, generator=g, dtype=torch.float32)
    return H, W, y, m, up


def _gpu(hdl, H, W, y, m, up, **kw):
    Hd, Wd, yd = H.cuda(), W.cuda(), y.cuda()
    md = None if m is None else m.cuda()
    _, lse = hdl.token_logprobs(Hd, Wd, yd, md)
    dh, dw = hdl.token_logprobs_backward(Hd, Wd, yd, md, lse, up.cuda(), **kw)
    torch.cuda.synchronize()
    return dh.cpu().double().numpy(), dw.cpu().double().numpy()


def _check(got, want, mag, what):
    tol = grad_tol(mag)
    bad = np.abs(got - want) > tol
    assert not bad.any(), (f"{what}: {bad.sum()} elements out of bound, worst excess "
                           f"{(np.abs(got - want) - tol).max():.3g}")


@pytest.mark.parametrize("n,d,V", [
    (300, 64, 1000),     # one chunk, ragged last vocabulary tile
    (257, 72, 4133),     # K tail in the logit recompute, ragged GEMM edges
    (40, 8, 300),        # d smaller than one K-slice
    (700, 256, 20000),   # realistic vocabulary tail, several vocabulary splits
    (1, 16, 65),         # one row; one vocabulary entry past a 64-multiple
    (33, 200, 129),      # d not a multiple of 64 (K tail; clamped W columns in dH)
    (600, 64, 257),      # a last vocabulary tile with one live column; ragged scored-row count
])
def test_backward_matches_oracle(hdl, n, d, V):
    H, W, y, m, up = _case(n, d, V, seed=n + d + V)
    dh, dw = _gpu(hdl, H, W, y, m, up)
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(as_f64(H), as_f64(W), y.numpy(),
                                                                 up.double().numpy(), m.numpy())
    _check(dh, want_dh, mag_dh, "dH")
    _check(dw, want_dw, mag_dw, "dW")
    assert np.all(dh[m.numpy() == 0] == 0.0)


def test_backward_several_chunks(hdl):
    # more than 2 x 32768 scored rows: G is produced in three chunks and dW summed over them
    H, W, y, m, up = _case(80000, 64, 512, seed=31, mask_p=0.9)
    dh, dw = _gpu(hdl, H, W, y, m, up)
    assert int(m.sum()) > 2 * 32768
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(as_f64(H), as_f64(W), y.numpy(),
                                                                 up.double().numpy(), m.numpy())
    _check(dh, want_dh, mag_dh, "dH")
    _check(dw, want_dw, mag_dw, "dW")


def test_backward_trailing_chunks_empty(hdl):
    # 100,000 rows are planned as four chunks of 32,768 before the mask is
    # known (the host never reads the scored count); a sparse mask leaves
    # about 20,000 scored rows, so chunks 1-3 find no rows: their launches
    # must leave dH and the dW already accumulated from chunk 0 untouched
    H, W, y, m, up = _case(100000, 64, 300, seed=41, mask_p=0.2)
    assert int(m.sum()) < 32768
    dh, dw = _gpu(hdl, H, W, y, m, up)
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(as_f64(H), as_f64(W), y.numpy(),
                                                                 up.double().numpy(), m.numpy())
    _check(dh, want_dh, mag_dh, "dH")
    _check(dw, want_dw, mag_dw, "dW")
    assert np.all(dh[m.numpy() == 0] == 0.0)


def test_backward_workload_shapes(hdl):
    # reduced agent workload (observation spans masked), original context only
    w = workloads.make_workload("c4", R=2, T=600, d=128, V=9000)
    n0 = w.cfg.R * w.cfg.T
    H = w.rows_hidden()[:n0]
    y = w.rows_tokens()[:n0]
    m = w.rows_mask()[:n0]
    up = torch.from_numpy(np.random.default_rng(5).normal(size=n0).astype(np.float32))
    dh, dw = _gpu(hdl, H, w.W, y, m, up)
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(as_f64(H), as_f64(w.W), y.numpy(),
                                                                 up.double().numpy(), m.numpy())
    _check(dh, want_dh, mag_dh, "dH")
    _check(dw, want_dw, mag_dw, "dW")


def test_backward_accumulate_determinism_and_empty(hdl):
    H, W, y, m, up = _case(500, 64, 777, seed=7)
    dh1, dw1 = _gpu(hdl, H, W, y, m, up)
    dh2, dw2 = _gpu(hdl, H, W, y, m, up)
    assert np.array_equal(dh1, dh2) and np.array_equal(dw1, dw2)   # bitwise run to run
    # accumulate into an existing gradient
    Hd, Wd, yd, md = H.cuda(), W.cuda(), y.cuda(), m.cuda()
    _, lse = hdl.token_logprobs(Hd, Wd, yd, md)
    base = torch.full((777, 64), 0.25, dtype=torch.float32, device="cuda")
    _, acc = hdl.token_logprobs_backward(Hd, Wd, yd, md, lse, up.cuda(), grad_w=base, accumulate_w=True)
    torch.cuda.synchronize()
    assert np.allclose(acc.cpu().double().numpy(), dw1 + 0.25, rtol=0, atol=1e-6)
    # nothing scored: both gradients are zero
    dh0, dw0 = _gpu(hdl, H, W, y, torch.zeros_like(m), up)
    assert np.all(dh0 == 0.0) and np.all(dw0 == 0.0)


def test_backward_out_of_range_token_and_argument_errors(hdl):
    H, W, y, m, up = _case(64, 64, 300, seed=9, mask_p=1.1)
    y[5] = 300
    y[9] = -2
    dh, dw = _gpu(hdl, H, W, y, m, up)
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(as_f64(H), as_f64(W), y.numpy(),
                                                                 up.double().numpy(), m.numpy())
    _check(dh, want_dh, mag_dh, "dH")
    _check(dw, want_dw, mag_dw, "dW")
    with pytest.raises(ValueError):
        hdl.token_logprobs_backward(H.float().cuda(), W.float().cuda(), y.cuda(), None,
                                    torch.zeros(64, device="cuda"), up.cuda())


def test_backward_full_size_every_row_tile(hdl):
    # the benchmark's configuration (8 roots x 4096 tokens of the original
    # context, d = 2048, V = 151,936, one chunk of 32,512 trained rows):
    # dH of one seeded row from every 256-row tile of the trained rows (the
    # GEMM's M tiles, in the library's compaction order) and of the last
    # trained row, against the oracle; for dW a property that holds at any
    # size: the vocabulary rows of dW sum to sum_n (sum_v G_nv) h_n = 0, up
    # to the bf16 rounding of G, |sum_v dG_nv| <= 2^-8 sum_v |G_nv| <= 2^-7 |g_n|
    # (sum_v |G_nv| = 2 |g_n| (1 - p_n(y_n)))
    w = workloads.make_workload("c2")
    c = w.cfg
    n0 = c.R * c.T
    H = w.rows_hidden()[:n0]
    y = w.rows_tokens()[:n0]
    m = w.rows_mask()[:n0]
    up = torch.from_numpy(np.random.default_rng(11).normal(size=n0).astype(np.float32))
    dh, dw = _gpu(hdl, H, w.W, y, m, up)
    trained = np.nonzero(m.numpy())[0]
    rng = np.random.default_rng(c.seed + 7)
    pick = [int(rng.integers(t0, min(t0 + 256, len(trained)))) for t0 in range(0, len(trained), 256)]
    rows = trained[np.array(sorted(set(pick + [len(trained) - 1])))]
    want_dh, _, mag_dh, _ = O.token_logprobs_backward(as_f64(H[torch.as_tensor(rows)]), as_f64(w.W),
                                                      y.numpy()[rows], up.double().numpy()[rows])
    err = np.abs(dh[rows] - want_dh)
    print(f"\nc2 backward: dH of {len(rows)} rows (one per 256-row tile): max |error| {err.max():.3g}, "
          f"max |error| / bound {(err / grad_tol(mag_dh)).max():.3g}")
    _check(dh[rows], want_dh, mag_dh, "dH (one row per tile)")
    keep = m.numpy() != 0
    assert np.all(dh[~keep] == 0)
    bound = 2.0 ** -7 * (np.abs(up.double().numpy()[keep])[:, None] * np.abs(as_f64(H)[keep])).sum(0)
    colsum = dw.sum(axis=0)
    assert np.all(np.abs(colsum) <= bound + 1e-6 * np.abs(dw).max())
