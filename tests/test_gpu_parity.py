"""GPU parity of the fused lm-head log-probability path (Eq. 1) and of the
divergence / top-k selection (Eq. 2, Sec. 3.2) against the float64 oracle,
element by element, through the C ABI.

Tolerances: |log p error| <= 2e-3 for bf16 inputs (the stated bar) and
<= 1e-4 for fp32 inputs (fp32 accumulation over d <= 256 and a vocabulary
of 4096 errs by ~1e-6; 1e-4 leaves margin for the exp2/log2 hardware
approximations).  Selection is integer work and is compared bit-exactly on
identical fp32 inputs; end to end, branch sets follow the tie-tolerant rule.
"""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O
from tests.gpu_helpers import as_f64, flat_inputs, grad_tol, oracle_rows, require_gpu, run_logprobs

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-3
TOL_F32 = 1e-4


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


def _check_all_rows(hdl, w, tol):
    hidden, W, tokens, mask = flat_inputs(w)
    lp, lse = run_logprobs(hdl, hidden, W, tokens, mask)
    m = mask.numpy().astype(bool)
    rows = np.nonzero(m)[0]
    want, want_lse = oracle_rows(hidden, W, tokens, rows)
    err = np.abs(lp[rows] - want)
    assert err.max() <= tol, f"max |logp err| {err.max():.3g} at row {rows[err.argmax()]}"
    assert np.abs(lse[rows] - want_lse).max() <= tol
    assert np.all(lp[~m] == 0.0) and np.all(lse[~m] == 0.0)
    assert np.all(lp <= 0.0)
    return lp, want, rows


def test_tiny_full_parity_and_branch_points(hdl):
    w = workloads.make_workload("tiny")
    lp, want, rows = _check_all_rows(hdl, w, TOL_F32)
    T, k = w.cfg.T, w.cfg.k
    dev = "cuda"
    lp_t = torch.from_numpy(lp).to(dev)
    m = w.mask.to(dev)
    idx, score, count, delta = hdl.select_branch_points(lp_t[:T].view(1, T), lp_t[T:].view(1, T), m, k,
                                                        want_delta=True)
    torch.cuda.synchronize()
    # oracle ranking from oracle log-probs: the gap at k is huge here, so the
    # branch set and its order must match exactly
    full = np.zeros(2 * T)
    full[rows] = want
    oi, osc, oc = O.select_branch_points(full[:T][None], full[T:][None], w.mask.numpy(), k)
    assert idx.cpu().numpy().tolist() == oi.tolist()
    assert int(count[0]) == int(oc[0]) == k
    assert np.allclose(score.cpu().numpy(), osc, atol=2 * TOL_F32)
    assert sorted(idx[0].tolist()) == sorted(w.planted[0]["pos"].tolist())


@pytest.mark.parametrize("name,over", [
    ("c2", dict(R=2, T=300, d=256)),                    # V = 151936: ragged last V-tile
    ("c3", dict(R=1, T=520, d=256)),
    ("c4", dict(R=3, T=700, d=128, V=20000)),           # agent observation spans
    ("c5", dict(R=1, T=400, d=256)),                     # heavy-tailed, V = 152064
])
def test_bf16_reduced_configs_all_rows(hdl, name, over):
    w = workloads.make_workload(name, **over)
    _check_all_rows(hdl, w, TOL_BF16)


@pytest.mark.parametrize("n_rows,d,V", [
    (1, 64, 256),          # a single row, a single exact tile
    (257, 64, 257),        # ragged rows and one vocab row past a tile
    (511, 8, 1000),        # K tail: d smaller than one K-slice
    (300, 72, 4133),       # K tail after a full slice, ragged vocab
    (64, 136, 513),
    (1000, 2056, 2048),    # long K with a tail
])
def test_bf16_shape_edges(hdl, n_rows, d, V):
    g = torch.Generator().manual_seed(n_rows * 7 + d * 13 + V)
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n_rows, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n_rows,), generator=g, dtype=torch.int32)
    lp, lse = run_logprobs(hdl, H, W, y, None)
    want, want_lse = oracle_rows(H, W, y, np.arange(n_rows))
    assert np.abs(lp - want).max() <= TOL_BF16
    assert np.abs(lse - want_lse).max() <= TOL_BF16


@pytest.mark.parametrize("n_rows,d,V", [(300, 40, 777), (513, 256, 4096), (70, 24, 300)])
def test_f32_shape_edges(hdl, n_rows, d, V):
    g = torch.Generator().manual_seed(n_rows + d + V)
    W = torch.randn(V, d, generator=g) * 0.05
    H = torch.randn(n_rows, d, generator=g)
    y = torch.randint(0, V, (n_rows,), generator=g, dtype=torch.int32)
    lp, _ = run_logprobs(hdl, H, W, y, None)
    want, _ = oracle_rows(H, W, y, np.arange(n_rows))
    assert np.abs(lp - want).max() <= TOL_F32


def test_masks_empty_single_and_sparse(hdl):
    g = torch.Generator().manual_seed(5)
    n, d, V = 900, 64, 3000
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    # nothing eligible: every output is 0, no kernel work
    lp, lse = run_logprobs(hdl, H, W, y, torch.zeros(n, dtype=torch.uint8))
    assert np.all(lp == 0.0) and np.all(lse == 0.0)
    # one eligible row
    m = torch.zeros(n, dtype=torch.uint8); m[637] = 1
    lp, _ = run_logprobs(hdl, H, W, y, m)
    want, _ = oracle_rows(H, W, y, [637])
    assert abs(lp[637] - want[0]) <= TOL_BF16 and np.count_nonzero(lp) == 1
    # sparse random mask: compacted rows straddle several tiles
    m = (torch.rand(n, generator=g) < 0.3).to(torch.uint8)
    lp, _ = run_logprobs(hdl, H, W, y, m)
    rows = np.nonzero(m.numpy())[0]
    want, _ = oracle_rows(H, W, y, rows)
    assert np.abs(lp[rows] - want).max() <= TOL_BF16
    assert np.all(lp[m.numpy() == 0] == 0.0)


def test_out_of_range_tokens_give_nan(hdl):
    g = torch.Generator().manual_seed(6)
    n, d, V = 40, 64, 500
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    y[3] = -1; y[17] = V; y[30] = 2 ** 31 - 1
    lp, _ = run_logprobs(hdl, H, W, y, None)
    bad = [3, 17, 30]
    assert np.all(np.isnan(lp[bad]))
    good = [i for i in range(n) if i not in bad]
    want, _ = oracle_rows(H, W, y, good)
    assert np.abs(lp[good] - want).max() <= TOL_BF16


def test_probabilities_sum_to_one_by_sweep(hdl):
    # one hidden row repeated V times, tokens 0..V-1: sum_v p_v must be 1
    w = workloads.make_workload("tiny")
    V = w.cfg.V
    h = w.hidden[1, 0, 37].reshape(1, -1).repeat(V, 1)
    lp, _ = run_logprobs(hdl, h, w.W, torch.arange(V, dtype=torch.int32), None)
    assert abs(math.fsum(np.exp(lp.astype(np.float64))) - 1.0) < 1e-4


def test_identical_contexts_give_bitwise_zero_delta(hdl):
    w = workloads.make_workload("c2", R=2, T=300, d=256, V=5000)
    c = w.cfg
    h0 = w.hidden[0].reshape(c.R * c.T, c.d)
    hidden = torch.cat([h0, h0])           # hindsight := original
    tokens = w.rows_tokens()
    lp, _ = run_logprobs(hdl, hidden, w.W, tokens, w.rows_mask())
    n = c.R * c.T
    assert np.array_equal(lp[:n].view(np.uint32), lp[n:].view(np.uint32))
    lpt = torch.from_numpy(lp).cuda()
    idx, score, count, delta = hdl.select_branch_points(lpt[:n].view(c.R, c.T), lpt[n:].view(c.R, c.T),
                                                        w.mask.cuda(), c.k, want_delta=True)
    torch.cuda.synchronize()
    assert torch.all(delta == 0) and torch.all(score == 0)
    # all-zero scores: the first k eligible positions, in order
    first = [np.nonzero(w.mask[r].numpy())[0][:c.k].tolist() for r in range(c.R)]
    assert idx.cpu().numpy().tolist() == first


def test_duplicate_rows_bitwise_equal_across_tiles(hdl):
    g = torch.Generator().manual_seed(8)
    n, d, V = 1100, 128, 4100
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    for src, dst in [(3, 300), (10, 1099), (511, 512), (0, 767)]:
        H[dst] = H[src]; y[dst] = y[src]
    lp, lse = run_logprobs(hdl, H, W, y, None)
    for src, dst in [(3, 300), (10, 1099), (511, 512), (0, 767)]:
        assert lp[src].view(np.uint32) == lp[dst].view(np.uint32)
        assert lse[src].view(np.uint32) == lse[dst].view(np.uint32)


def test_run_to_run_determinism(hdl):
    w = workloads.make_workload("c4", R=2, T=1200, d=128, V=9000)
    hidden, W, tokens, mask = flat_inputs(w)
    a, _ = run_logprobs(hdl, hidden, W, tokens, mask)
    b, _ = run_logprobs(hdl, hidden, W, tokens, mask)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_vocab_permutation_invariance(hdl):
    g = torch.Generator().manual_seed(9)
    n, d, V = 300, 64, 3001
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    perm = torch.randperm(V, generator=g)
    inv = torch.argsort(perm)
    a, _ = run_logprobs(hdl, H, W, y, None)
    b, _ = run_logprobs(hdl, H, W[perm].contiguous(), inv[y.long()].to(torch.int32), None)
    assert np.abs(a - b).max() <= 1e-5


# ------------------------------------------------------------ selection alone
@pytest.mark.parametrize("R,T,k,nan_rows", [
    (1, 1, 1, 0), (3, 7, 4, 0), (2, 1023, 8, 1), (2, 1024, 32, 0), (4, 1025, 16, 2),
    (2, 32768, 32, 3), (1, 40000, 1024, 0), (32, 8192, 8, 1), (5, 300, 1024, 0),
])
def test_select_bit_exact_vs_oracle(hdl, R, T, k, nan_rows):
    lo, lh, mask = workloads.make_logp_pair(R, T, seed=R * 1000 + T + k, nan_rows=nan_rows)
    idx, score, count, delta = hdl.select_branch_points(torch.from_numpy(lo).cuda(), torch.from_numpy(lh).cuda(),
                                                        torch.from_numpy(mask).cuda(), k, want_delta=True)
    torch.cuda.synchronize()
    oi, osc, oc = O.select_branch_points(lo, lh, mask, k, precision="f32")
    sd, _, _ = O.divergence(lo, lh, mask, precision="f32")
    assert np.array_equal(count.cpu().numpy(), oc)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(score.cpu().numpy().view(np.uint32), osc.astype(np.float32).view(np.uint32))
    assert np.array_equal(delta.cpu().numpy().view(np.uint32), sd.view(np.uint32))


def test_select_ties_at_boundary_take_lower_index(hdl):
    T = 5000
    lo = np.full((2, T), -2.0, np.float32)
    lh = lo.copy()
    lh[:, [4000, 17, 2500, 3, 4999]] = -1.0        # five exact ties at s = 1
    lh[:, 1000] = 0.0                                # one clear winner, s = 2
    mask = np.ones((2, T), np.uint8)
    mask[1, 3] = 0
    idx, score, count, _ = hdl.select_branch_points(torch.from_numpy(lo).cuda(), torch.from_numpy(lh).cuda(),
                                                    torch.from_numpy(mask).cuda(), 4)
    torch.cuda.synchronize()
    assert idx[0].tolist() == [1000, 3, 17, 2500]
    assert idx[1].tolist() == [1000, 17, 2500, 4000]
    assert score[0].tolist() == [2.0, 1.0, 1.0, 1.0]


@pytest.mark.parametrize("R,T,k", [(3, 20000, 8), (2, 20000, 700), (2, 40000, 64), (2, 40000, 1024), (4, 777, 65)])
def test_select_many_ties_at_the_threshold(hdl, R, T, k):
    # scores from five levels only, so the k-th place falls inside a large
    # block of exact ties spread over every part of the root (staged roots
    # and, for T > 32768, roots read again from global memory)
    g = np.random.default_rng(T + k)
    lo = np.full((R, T), -3.0, np.float32)
    level = g.choice(5, size=(R, T), p=[0.4, 0.3, 0.2, 0.0998, 0.0002])   # s = level / 4
    lh = (lo + 0.25 * level).astype(np.float32)
    mask = (g.random((R, T)) < 0.9).astype(np.uint8)
    idx, score, count, _ = hdl.select_branch_points(torch.from_numpy(lo).cuda(), torch.from_numpy(lh).cuda(),
                                                    torch.from_numpy(mask).cuda(), k)
    torch.cuda.synchronize()
    oi, osc, oc = O.select_branch_points(lo, lh, mask, k, precision="f32")
    assert np.array_equal(count.cpu().numpy(), oc)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(score.cpu().numpy(), osc.astype(np.float32))


def test_select_fewer_candidates_than_k(hdl):
    lo = np.array([[-1.0, -2.0, -3.0, -4.0]], np.float32)
    lh = np.array([[-1.5, np.nan, -1.0, -9.0]], np.float32)
    mask = np.array([[1, 1, 1, 0]], np.uint8)
    idx, score, count, _ = hdl.select_branch_points(torch.from_numpy(lo).cuda(), torch.from_numpy(lh).cuda(),
                                                    torch.from_numpy(mask).cuda(), 6)
    torch.cuda.synchronize()
    assert int(count[0]) == 2
    assert idx[0].tolist() == [2, 0, -1, -1, -1, -1]
    assert score[0].tolist() == [2.0, 0.5, 0.0, 0.0, 0.0, 0.0]


def test_select_without_mask(hdl):
    lo, lh, _ = workloads.make_logp_pair(3, 2000, seed=3)
    idx, _, count, _ = hdl.select_branch_points(torch.from_numpy(lo).cuda(), torch.from_numpy(lh).cuda(), None, 10)
    torch.cuda.synchronize()
    oi, _, oc = O.select_branch_points(lo, lh, None, 10, precision="f32")
    assert np.array_equal(idx.cpu().numpy(), oi) and np.array_equal(count.cpu().numpy(), oc)


def test_boundary_errors(hdl):
    dev = "cuda"
    H = torch.zeros(4, 12, dtype=torch.bfloat16, device=dev)     # d = 12: not a multiple of 8
    W = torch.zeros(10, 12, dtype=torch.bfloat16, device=dev)
    y = torch.zeros(4, dtype=torch.int32, device=dev)
    with pytest.raises(hdl.HdlError) as e:
        hdl.token_logprobs(H, W, y)
    assert e.value.status == -2
    lo = torch.zeros(2, 5, device=dev)
    with pytest.raises(hdl.HdlError) as e:
        hdl.select_branch_points(lo, lo, None, 2000)
    assert e.value.status == -2
    H = torch.zeros(4, 16, dtype=torch.bfloat16, device=dev)
    W = torch.zeros(10, 16, dtype=torch.bfloat16, device=dev)
    small = torch.empty(16, dtype=torch.uint8, device=dev)
    with pytest.raises(hdl.HdlError) as e:
        hdl.token_logprobs(H, W, y, workspace=small)
    assert e.value.status == -3


def test_hidden_states_over_4gib_split_into_launches(hdl):
    # 525,065 rows of d = 4096 bf16 (4.3 GB): the library cuts the call into
    # launches of 2^32 / 8192 = 524,288 rows (32-bit DMA offsets); rows on
    # both sides of the cut must match the oracle and masked rows stay 0,
    # in the forward and in the backward pass
    n, d, V = 524288 + 777, 4096, 1000
    gen = torch.Generator(device="cuda").manual_seed(77)
    H = torch.randn(n, d, device="cuda", generator=gen).to(torch.bfloat16)
    W = (torch.randn(V, d, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), device="cuda", dtype=torch.int32, generator=gen)
    m = (torch.rand(n, device="cuda", generator=gen) < 0.9).to(torch.uint8)
    lp, lse = hdl.token_logprobs(H, W, y, m)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 1000, 524286, 524287, 524288, 524289, 524290, 524800, n - 1])
    mk = m[torch.as_tensor(rows, device="cuda")].cpu().numpy()
    Hs = H[torch.as_tensor(rows, device="cuda")].cpu()
    want, want_lse = O.token_logprobs(as_f64(Hs), as_f64(W.cpu()), y[torch.as_tensor(rows, device="cuda")].cpu().numpy())
    got = lp[torch.as_tensor(rows, device="cuda")].cpu().numpy()
    on = mk != 0
    assert np.abs(got[on] - want[on]).max() <= TOL_BF16
    assert np.all(got[~on] == 0.0)
    # the entropy output goes through the same row blocks
    lp2, _, ent = hdl.token_logprobs(H, W, y, m, want_entropy=True)
    torch.cuda.synchronize()
    assert torch.equal(lp2.view(torch.int32), lp.view(torch.int32))
    got_ent = ent[torch.as_tensor(rows, device="cuda")].cpu().numpy()
    want_ent = O.token_entropy(as_f64(Hs), as_f64(W.cpu()))
    assert np.abs(got_ent[on] - want_ent[on]).max() <= TOL_BF16
    assert np.all(got_ent[~on] == 0.0)
    del lp2, ent
    # the backward pass takes the same row blocks.  g is zero except on the
    # sampled rows, so dW = sum over those rows of G_n^T h_n is the oracle's
    # whole answer even though every row is processed; dH is zero elsewhere
    gs = np.random.default_rng(5).normal(size=rows.size).astype(np.float32)
    g = torch.zeros(n, device="cuda")
    g[torch.as_tensor(rows, device="cuda")] = torch.from_numpy(gs).cuda()
    prefill = torch.full((V, d), 1e3, device="cuda")       # overwritten: accumulate_w is off
    dh, dw = hdl.token_logprobs_backward(H, W, y, m, lse, g, grad_w=prefill)
    torch.cuda.synchronize()
    nz = torch.nonzero((dh != 0).any(dim=1)).flatten().cpu().numpy()
    assert set(nz.tolist()) <= set(rows[on].tolist())
    want_dh, want_dw, mag_dh, mag_dw = O.token_logprobs_backward(
        as_f64(Hs), as_f64(W.cpu()), y[torch.as_tensor(rows, device="cuda")].cpu().numpy(), gs, mk)
    got_dh = dh[torch.as_tensor(rows, device="cuda")].cpu().double().numpy()
    assert np.all(np.abs(got_dh - want_dh) <= grad_tol(mag_dh))
    got_dw = dw.cpu().double().numpy()
    assert np.all(np.abs(got_dw - want_dw) <= grad_tol(mag_dw))


def test_weight_over_4gib(hdl):
    # W of 262,400 x 8192 bf16 (4.3 GB): the DMA addresses W through a 64-bit
    # base per vocabulary tile and 32-bit offsets inside it.  W is zero except
    # a few random rows (the last row before the 4 GiB offset and three past
    # it among them), so every other
    # logit is exactly 0 and the log-sum-exp has a closed form:
    #     lse = log(sum_special exp(z_v) + (V - #special) * exp(0)).
    # The backward pass is checked the same way: dL/dh only sees the special
    # rows, and every zero row of W that is nobody's token gets the same
    # dL/dW = -sum_n g_n exp(-lse_n) h_n.
    d, V, n = 8192, 262400, 96
    assert V * d * 2 > 2 ** 32
    dev = "cuda"
    gen = torch.Generator().manual_seed(404)
    special = np.array([0, 1000, 131071, 262143, 262144, 262300, V - 1])
    assert np.sum(special * d * 2 >= 2 ** 32) == 3 and (262143 + 1) * d * 2 == 2 ** 32
    Ws = (torch.randn(len(special), d, generator=gen) * 0.05).to(torch.bfloat16)
    W = torch.zeros(V, d, dtype=torch.bfloat16, device=dev)
    W[torch.as_tensor(special, device=dev)] = Ws.to(dev)
    H = torch.randn(n, d, generator=gen).to(torch.bfloat16)
    rng = np.random.default_rng(404)
    y = special[rng.integers(0, len(special), n)]
    y[::7] = 262200                     # a zero row past 4 GiB as the sampled token
    y[3::11] = 5                        # and one before it
    y = y.astype(np.int32)
    Hd, yd = H.to(dev), torch.from_numpy(y).to(dev)
    lp, lse = hdl.token_logprobs(Hd, W, yd, None)
    torch.cuda.synchronize()
    z = as_f64(H) @ as_f64(Ws).T                          # [n, #special], exact products of the inputs
    m = np.maximum(z.max(axis=1), 0.0)
    want_lse = m + np.log(np.exp(z - m[:, None]).sum(axis=1) + (V - len(special)) * np.exp(-m))
    col = {int(v): j for j, v in enumerate(special)}
    z_y = np.array([z[i, col[int(t)]] if int(t) in col else 0.0 for i, t in enumerate(y)])
    assert np.abs(lp.cpu().numpy() - (z_y - want_lse)).max() <= TOL_BF16
    assert np.abs(lse.cpu().numpy() - want_lse).max() <= TOL_BF16

    up = torch.from_numpy(rng.normal(size=n).astype(np.float32))
    dh, dw = hdl.token_logprobs_backward(Hd, W, yd, None, lse, up.to(dev))
    torch.cuda.synchronize()
    g = up.double().numpy()
    p = np.exp(z - want_lse[:, None])                     # probabilities of the special rows
    G = -g[:, None] * p
    for i, t in enumerate(y):
        if int(t) in col:
            G[i, col[int(t)]] += g[i]
    want_dh = G @ as_f64(Ws)
    mag_dh = np.abs(G) @ np.abs(as_f64(Ws))
    got_dh = dh.cpu().double().numpy()
    assert np.all(np.abs(got_dh - want_dh) <= grad_tol(mag_dh))
    H64 = as_f64(H)
    p0 = np.exp(-want_lse)                                # probability of every zero row
    checks = {int(v): G[:, j] for j, v in enumerate(special)}
    checks[262350] = -g * p0                              # nobody's token, past 4 GiB
    checks[77] = -g * p0                                  # nobody's token, before it
    for t in (262200, 5):
        checks[t] = g * ((y == t).astype(np.float64) - p0)
    rows = np.array(sorted(checks))
    got_dw = dw[torch.as_tensor(rows, device=dev)].cpu().double().numpy()
    for r, got in zip(rows, got_dw):
        want = checks[int(r)] @ H64
        mag = np.abs(checks[int(r)]) @ np.abs(H64)
        assert np.all(np.abs(got - want) <= grad_tol(mag)), f"dW row {r}"


def test_non_finite_hidden_row_stays_local(hdl):
    # a NaN or Inf in one row's hidden state makes that row's log p NaN (its
    # logits are NaN); every other row of the same tile is unaffected, and
    # the selection never picks the poisoned position
    g = torch.Generator().manual_seed(15)
    R, T, d, V = 1, 600, 64, 3000
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(2 * T, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (2 * T,), generator=g, dtype=torch.int32)
    clean, _ = run_logprobs(hdl, H, W, y, None)
    Hbad = H.clone()
    Hbad[T + 17, 5] = float("nan")        # hindsight row of position 17
    Hbad[T + 300, 0] = float("inf")       # hindsight row of position 300
    lp, _ = run_logprobs(hdl, Hbad, W, y, None)
    bad = [T + 17, T + 300]
    assert np.all(np.isnan(lp[bad]))
    good = np.setdiff1d(np.arange(2 * T), bad)
    assert np.array_equal(lp[good].view(np.uint32), clean[good].view(np.uint32))
    lpt = torch.from_numpy(lp).cuda()
    idx, _, count, _ = hdl.select_branch_points(lpt[:T].view(1, T), lpt[T:].view(1, T), None, T)
    torch.cuda.synchronize()
    chosen = idx[0, : int(count[0])].tolist()
    assert int(count[0]) == T - 2 and 17 not in chosen and 300 not in chosen


def test_degenerate_vocabularies_and_large_logits(hdl):
    g = torch.Generator().manual_seed(16)
    n, d = 300, 64
    H = torch.randn(n, d, generator=g).to(torch.bfloat16)
    # V = 1: every log p is exactly 0; V = 2: the log-sigmoid, against the oracle
    for V in (1, 2):
        W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
        y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
        lp, lse = run_logprobs(hdl, H, W, y, None)
        want, want_lse = oracle_rows(H, W, y, np.arange(n))
        assert np.abs(lp - want).max() <= TOL_BF16 and np.abs(lse - want_lse).max() <= TOL_BF16
        if V == 1:
            assert np.all(lp == 0.0)
    # logits of a few hundred: the online max keeps exp in range and the
    # stated bar still holds (fp32 spacing at 1000 is 6e-5)
    V = 5000
    W = (torch.randn(V, d, generator=g) * 30.0).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, dtype=torch.int32)
    lp, lse = run_logprobs(hdl, H, W, y, None)
    want, want_lse = oracle_rows(H, W, y, np.arange(n))
    assert np.abs(want_lse).max() > 200
    assert np.all(np.isfinite(lp))
    err = np.abs(lp - want).max()
    assert err <= TOL_BF16, f"max |log p error| {err:.3g} at |lse| up to {np.abs(want_lse).max():.0f}"


@pytest.mark.parametrize("n_rows,d", [(8192, 256), (8192, 200), (65536, 256), (65536, 136)])
def test_work_items_spanning_several_vocab_tiles(hdl, n_rows, d):
    # The number of vocabulary tiles per work item follows the call's row
    # count, not its scored rows: 8,192 rows x 513 vocabulary tiles give 2
    # tiles per item, 65,536 rows give 16.  A sparse mask keeps the oracle's
    # share small while every scored row runs through items that carry their
    # DMA pipeline across vocabulary-tile boundaries (and, for d % 64 != 0,
    # zero-fill the K tail of every tile's last slice); the last chunk is
    # ragged (513 tiles, the last one with 77 live rows).
    V = 131072 + 77
    g = torch.Generator().manual_seed(n_rows + d)
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16)
    H = torch.randn(n_rows, d, generator=g).to(torch.bfloat16)
    y = torch.randint(0, V, (n_rows,), generator=g, dtype=torch.int32)
    y[::5] = torch.randint(V - 77, V, (len(y[::5]),), generator=g, dtype=torch.int32)   # last tile
    mask = (torch.rand(n_rows, generator=g) < 300.0 / n_rows).to(torch.uint8)
    mask[-1] = 1
    rows = np.nonzero(mask.numpy())[0]
    lp, lse = run_logprobs(hdl, H, W, y, mask)
    want, want_lse = oracle_rows(H, W, y, rows)
    err = np.abs(lp[rows] - want)
    print(f"n_rows={n_rows} d={d}: {len(rows)} scored rows, max |log p error| {err.max():.3g}")
    assert err.max() <= TOL_BF16
    assert np.abs(lse[rows] - want_lse).max() <= TOL_BF16
    off = np.ones(n_rows, bool)
    off[rows] = False
    assert np.all(lp[off] == 0.0)
    # entropy through the same items
    Hd, Wd = H.cuda(), W.cuda()
    _, _, ent = hdl.token_logprobs(Hd, Wd, y.cuda(), mask.cuda(), want_entropy=True)
    torch.cuda.synchronize()
    want_ent = O.token_entropy(as_f64(H[torch.as_tensor(rows)]), as_f64(W))
    assert np.abs(ent.cpu().numpy()[rows] - want_ent).max() <= TOL_BF16


def test_remainder_launch_keeps_the_call_chunking(hdl):
    # bf16, d = 5120, V = 32000: a launch takes at most 419,328 rows (4 GiB of
    # hidden states), so 446,208 rows run as 419,328 + 26,880.  The remainder
    # launch uses the call's vocabulary chunking; chunked on its own it would
    # need 125 chunks x 26,880 rows of partials, more than the workspace's
    # 8 x 419,328.  Every row of the remainder is scored, so the last chunk's
    # partials of its last compacted rows are exactly the ones that would not
    # fit; those rows and rows before the cut are checked against the oracle,
    # for log p and for the entropy (whose partial plane is the last one).
    n, d, V = 446208, 5120, 32000
    cut = 419328
    gen = torch.Generator(device="cuda").manual_seed(91)
    H = torch.empty(n, d, device="cuda", dtype=torch.bfloat16)
    for r0 in range(0, n, 65536):
        r1 = min(n, r0 + 65536)
        H[r0:r1] = torch.randn(r1 - r0, d, device="cuda", generator=gen).to(torch.bfloat16)
    W = (torch.randn(V, d, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), device="cuda", dtype=torch.int32, generator=gen)
    m = (torch.rand(n, device="cuda", generator=gen) < 0.01).to(torch.uint8)
    m[cut:] = 1
    lp, lse, ent = hdl.token_logprobs(H, W, y, m, want_entropy=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    before = np.nonzero(m[:cut].cpu().numpy())[0]
    rows = np.unique(np.concatenate([rng.choice(before, 40, replace=False),
                                     np.arange(cut, cut + 8), np.arange(n - 5400, n, 45), [n - 1]]))
    idx = torch.as_tensor(rows, device="cuda")
    Hs = as_f64(H[idx].cpu())
    Wd = as_f64(W.cpu())
    want, want_lse = O.token_logprobs(Hs, Wd, y[idx].cpu().numpy())
    err = np.abs(lp[idx].cpu().numpy() - want)
    print(f"remainder launch: max |log p error| {err.max():.3g} over {len(rows)} rows")
    assert err.max() <= TOL_BF16
    assert np.abs(lse[idx].cpu().numpy() - want_lse).max() <= TOL_BF16
    assert np.abs(ent[idx].cpu().numpy() - O.token_entropy(Hs, Wd)).max() <= TOL_BF16
