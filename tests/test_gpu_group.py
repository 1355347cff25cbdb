"""GPU parity of localized group construction (Sec. 3.3, Sec. 4.1, Sec. 4.3-4.4)
against the float64 oracle, through the C ABI: constrained branch-point
selection (index range, minimum spacing, with and without refill),
continuation allocation, group advantages and the per-token factor of the
clipped policy loss.

Selection and allocation are integer work and compared bit-exactly (the
selection on identical fp32 inputs, its difference taken in fp32 on both
sides).  Advantages: |error| <= 1e-6 * max|R| (fp32 mean in a fixed order).
Policy-loss factors: relative error <= 1e-5 (fp32 exp of the log-ratio).
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O
from tests.gpu_helpers import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


def _t(x, dtype=None):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if dtype is None else \
        torch.from_numpy(np.ascontiguousarray(x).astype(dtype)).cuda()


@pytest.mark.parametrize("R,T,k,gap,refill,ranged", [
    (4, 300, 2, 0, False, False),
    (4, 300, 2, 8, False, False),
    (4, 300, 2, 8, True, False),
    (8, 4096, 2, 64, False, True),
    (8, 4096, 2, 64, True, True),
    (3, 5000, 16, 100, True, True),
    (2, 2000, 300, 3, True, False),
    (2, 40000, 8, 500, True, True),    # longer than the LDS holds: read again from memory
    (2, 33000, 100, 10, False, True),
])
def test_constrained_selection_bit_exact(hdl, R, T, k, gap, refill, ranged):
    lo_, hi_, mask = workloads.make_logp_pair(R, T, seed=R * 7 + T + k + gap, nan_rows=1)
    rng = np.random.default_rng(T + k)
    L = rng.integers(0, T // 3, R).astype(np.int32) if ranged else None
    H = (L + rng.integers(T // 3, T, R)).astype(np.int32) if ranged else None
    idx, score, count = hdl.select_constrained(_t(lo_), _t(hi_), _t(mask), k,
                                               lo=None if L is None else _t(L), hi=None if H is None else _t(H),
                                               min_gap=gap, refill=refill)
    torch.cuda.synchronize()
    oi, osc, oc = O.select_constrained(lo_, hi_, mask, k, lo=L, hi=H, min_gap=gap, refill=refill,
                                       precision="f32")
    assert np.array_equal(count.cpu().numpy(), oc)
    assert np.array_equal(idx.cpu().numpy(), oi)
    assert np.array_equal(score.cpu().numpy().view(np.uint32), osc.astype(np.float32).view(np.uint32))


def test_constrained_value_mode_and_fixture(hdl):
    T = 60
    s = np.zeros((1, T), np.float32)
    for t, v in ((10, 0.9), (12, 0.8), (30, 0.7), (50, 0.6), (33, 0.65)):
        s[0, t] = v
    idx, _, cnt = hdl.select_constrained(_t(s), None, None, 2, min_gap=5)
    assert cnt.tolist() == [1] and idx[0].tolist() == [10, -1]
    idx, _, cnt = hdl.select_constrained(_t(s), None, None, 2, min_gap=5, refill=True)
    assert idx[0].tolist() == [10, 30]
    idx, _, cnt = hdl.select_constrained(_t(s), None, None, 3, lo=_t(np.array([11], np.int32)),
                                         hi=_t(np.array([40], np.int32)), min_gap=5, refill=True)
    assert idx[0].tolist() == [12, 30, 17]
    # entropy-like values with spacing, against the oracle
    rng = np.random.default_rng(4)
    v = rng.gamma(2.0, 1.0, (5, 3000)).astype(np.float32)
    m = (rng.random((5, 3000)) < 0.7).astype(np.uint8)
    idx, sc, cnt = hdl.select_constrained(_t(v), None, _t(m), 4, min_gap=50, refill=True)
    oi, osc, oc = O.select_constrained(v, None, m, 4, min_gap=50, refill=True)
    assert np.array_equal(idx.cpu().numpy(), oi) and np.array_equal(cnt.cpu().numpy(), oc)


def test_allocation_bit_exact(hdl):
    rng = np.random.default_rng(6)
    R, k = 300, 2
    idx = rng.integers(0, 8000, (R, k)).astype(np.int32)
    cnt = rng.integers(0, k + 1, R).astype(np.int32)
    idx[np.arange(k)[None, :] >= cnt[:, None]] = -1
    for alloc, fb in (((3, 4), 0), ((1, 2), 7), ((0, 5), 3)):
        pos, rank = hdl.allocate_continuations(_t(idx), _t(cnt), alloc, fallback_pos=fb)
        torch.cuda.synchronize()
        opos, orank = O.allocate_continuations(idx, cnt, alloc, fb)
        assert np.array_equal(pos.cpu().numpy(), opos) and np.array_equal(rank.cpu().numpy(), orank)
    # single-point configuration
    pos, _ = hdl.allocate_continuations(_t(idx[:, :1]), _t(np.minimum(cnt, 1)), (7,))
    opos, _ = O.allocate_continuations(idx[:, :1], np.minimum(cnt, 1), (7,))
    assert np.array_equal(pos.cpu().numpy(), opos)


def test_group_advantages(hdl):
    rng = np.random.default_rng(9)
    for n, G in ((128, 16), (3, 1), (5, 1000)):
        R = (rng.random((n, G)) < 0.4).astype(np.float32) + rng.normal(size=(n, G)).astype(np.float32) * 0.1
        A = hdl.group_advantages(_t(R)).cpu().double().numpy()
        want = O.group_advantages(R)
        assert np.abs(A - want).max() <= 1e-6 * max(1.0, np.abs(R).max())
    A = hdl.group_advantages(_t(np.array([[1, 0, 0, 1]], np.float32))).cpu().numpy()
    assert A.tolist() == [[0.5, -0.5, -0.5, 0.5]]


def test_policy_loss_grad(hdl):
    rng = np.random.default_rng(10)
    n_traj, n = 16, 50000
    adv = rng.normal(size=n_traj).astype(np.float32)
    traj = rng.integers(0, n_traj, n).astype(np.int32)
    traj[::997] = n_traj + 3                      # out of range: contributes nothing
    lo_ = (rng.normal(size=n) * 0.5 - 2).astype(np.float32)
    ln = (lo_ + rng.normal(size=n) * 0.3).astype(np.float32)
    mask = (rng.random(n) < 0.8).astype(np.uint8)
    pos = (np.arange(n) % 3000).astype(np.int32)
    start = rng.integers(0, 1500, n_traj).astype(np.int32)
    scale = 1.0 / mask.sum()
    g, l = hdl.policy_loss_grad(_t(adv), _t(traj), _t(ln), _t(lo_), loss_mask=_t(mask), pos=_t(pos),
                                start=_t(start), scale=scale)
    torch.cuda.synchronize()
    og, ol = O.policy_loss_grad(adv, traj, ln, lo_, mask, pos, start, 0.2, 0.28, scale)
    g, l = g.cpu().double().numpy(), l.cpu().double().numpy()
    # where fp32 and fp64 could disagree on the clip region (r within 1e-5 of
    # a boundary) only check that the GPU picked one of the two sides
    r = np.exp(ln.astype(np.float64) - lo_.astype(np.float64))
    near = (np.abs(r - 0.8) < 1e-5) | (np.abs(r - 1.28) < 1e-5)
    ok = ~near
    assert np.allclose(g[ok], og[ok], rtol=1e-5, atol=1e-12)
    assert np.allclose(l[ok], ol[ok], rtol=1e-5, atol=1e-12)
    assert np.all(g[(mask == 0) | (traj >= n_traj)] == 0.0)


def test_group_construction_full_size(hdl):
    # the benchmark's configuration (one training step at the paper's batch:
    # 128 groups of 2 roots + 14 continuations, T = 4096, spacing 64, range
    # excluding the first and last 32 positions): selection and allocation
    # bit-exact, advantages within 1e-6, and the per-token factors of a seeded
    # sample of the 8.4 million tokens against the oracle
    n_groups, rpg, alloc, T = 128, 2, (3, 4), 4096
    R = n_groups * rpg
    lo_, hi_, mask = workloads.make_logp_pair(R, T, seed=1002 + 11)
    L = np.full(R, 32, np.int32)
    H = np.full(R, T - 33, np.int32)
    idx, score, count = hdl.select_constrained(_t(lo_), _t(hi_), _t(mask), len(alloc), lo=_t(L), hi=_t(H),
                                               min_gap=64)
    bpos, brank = hdl.allocate_continuations(idx, count, alloc)
    torch.cuda.synchronize()
    oi, osc, oc = O.select_constrained(lo_, hi_, mask, len(alloc), lo=L, hi=H, min_gap=64, precision="f32")
    assert np.array_equal(count.cpu().numpy(), oc) and np.array_equal(idx.cpu().numpy(), oi)
    opos, orank = O.allocate_continuations(oi, oc, alloc)
    assert np.array_equal(bpos.cpu().numpy(), opos) and np.array_equal(brank.cpu().numpy(), orank)

    G = rpg * (1 + sum(alloc))
    n_traj = n_groups * G
    rng = np.random.default_rng(1002 + 12)
    rewards = (rng.random((n_groups, G)) < 0.5).astype(np.float32)
    adv = hdl.group_advantages(_t(rewards)).view(-1)
    oadv = O.group_advantages(rewards).reshape(-1)
    assert np.abs(adv.cpu().double().numpy() - oadv).max() <= 1e-6
    n_tok = n_traj * T
    traj = np.repeat(np.arange(n_traj, dtype=np.int32), T)
    pos = np.tile(np.arange(T, dtype=np.int32), n_traj)
    lo_old = (-rng.exponential(2.0, n_tok)).astype(np.float32)
    lo_new = (lo_old + rng.normal(size=n_tok).astype(np.float32) * 0.2).astype(np.float32)
    tmask = (rng.random(n_tok) < 0.9).astype(np.uint8)
    start = np.zeros((n_groups, G), np.int32)
    start[:, rpg:] = opos.reshape(n_groups, -1)
    start = start.reshape(-1)
    g, l = hdl.policy_loss_grad(adv, _t(traj), _t(lo_new), _t(lo_old), loss_mask=_t(tmask), pos=_t(pos),
                                start=_t(start), scale=1.0 / n_tok)
    torch.cuda.synchronize()
    s = np.sort(rng.choice(n_tok, 200000, replace=False))
    og, ol = O.policy_loss_grad(oadv, traj[s], lo_new[s], lo_old[s], tmask[s], pos[s], start,
                                0.2, 0.28, 1.0 / n_tok)
    gs, ls = g.cpu().double().numpy()[s], l.cpu().double().numpy()[s]
    r = np.exp(lo_new[s].astype(np.float64) - lo_old[s].astype(np.float64))
    ok = ~((np.abs(r - 0.8) < 1e-5) | (np.abs(r - 1.28) < 1e-5))
    assert np.allclose(gs[ok], og[ok], rtol=1e-5, atol=1e-15)
    assert np.allclose(ls[ok], ol[ok], rtol=1e-5, atol=1e-15)
    # a continuation's reused prefix trains nothing
    pre = pos[s] < start[traj[s]]
    assert pre.any() and np.all(gs[pre] == 0.0)


def test_policy_loss_grad_token_level_mean_on_device(hdl):
    # scale=None: the library counts the trained tokens on the device (in
    # the mask, of a known trajectory, at or after the trajectory's start)
    # and divides by that count, as the oracle's token-level mean does
    rng = np.random.default_rng(12)
    n_traj, n = 40, 70001
    adv = rng.normal(size=n_traj).astype(np.float32)
    traj = rng.integers(-2, n_traj + 2, n).astype(np.int32)
    lo_ = (rng.normal(size=n) * 0.5 - 2).astype(np.float32)
    ln = (lo_ + rng.normal(size=n) * 0.3).astype(np.float32)
    mask = (rng.random(n) < 0.7).astype(np.uint8)
    pos = (np.arange(n) % 4000).astype(np.int32)
    start = rng.integers(0, 3000, n_traj).astype(np.int32)
    cnt = torch.full((1,), -5, dtype=torch.int64, device="cuda")
    for args in ((_t(pos), _t(start)), (None, None)):   # with and without the suffix rule
        g, l = hdl.policy_loss_grad(_t(adv), _t(traj), _t(ln), _t(lo_), loss_mask=_t(mask), pos=args[0],
                                    start=args[1], n_trained=cnt)
        torch.cuda.synchronize()
        p_, s_ = (pos, start) if args[0] is not None else (None, None)
        want_n = O.trained_tokens(traj, n_traj, mask, p_, s_)
        assert int(cnt.item()) == want_n
        og, ol = O.policy_loss_grad(adv, traj, ln, lo_, mask, p_, s_, 0.2, 0.28, None)
        g, l = g.cpu().double().numpy(), l.cpu().double().numpy()
        r = np.exp(ln.astype(np.float64) - lo_.astype(np.float64))
        ok = ~((np.abs(r - 0.8) < 1e-5) | (np.abs(r - 1.28) < 1e-5))
        assert np.allclose(g[ok], og[ok], rtol=1e-5, atol=1e-14)
        assert np.allclose(l[ok], ol[ok], rtol=1e-5, atol=1e-14)
    # nothing trained: count 0, every factor 0
    g, _ = hdl.policy_loss_grad(_t(adv), _t(traj), _t(ln), _t(lo_), loss_mask=_t(np.zeros(n, np.uint8)),
                                n_trained=cnt)
    torch.cuda.synchronize()
    assert int(cnt.item()) == 0 and torch.all(g == 0)


def test_policy_loss_grad_tail_and_unaligned(hdl):
    # 1001 tokens: the four-per-thread path with a ragged tail; the same data
    # as views one element into their buffers (not 16-byte aligned): the
    # one-per-thread path.  Both against the oracle.
    rng = np.random.default_rng(21)
    n_traj, n = 7, 1001
    adv = rng.normal(size=n_traj).astype(np.float32)
    traj = rng.integers(0, n_traj, n + 1).astype(np.int32)
    lo_ = (rng.normal(size=n + 1) * 0.5 - 2).astype(np.float32)
    ln = (lo_ + rng.normal(size=n + 1) * 0.3).astype(np.float32)
    mask = (rng.random(n + 1) < 0.8).astype(np.uint8)
    pos = (np.arange(n + 1) % 300).astype(np.int32)
    start = rng.integers(0, 150, n_traj).astype(np.int32)
    for off in (0, 1):
        sl = slice(off, off + n)
        args = [_t(traj)[sl], _t(ln)[sl], _t(lo_)[sl]]
        g, l = hdl.policy_loss_grad(_t(adv), *args, loss_mask=_t(mask)[sl], pos=_t(pos)[sl], start=_t(start),
                                    scale=0.01)
        torch.cuda.synchronize()
        og, ol = O.policy_loss_grad(adv, traj[sl], ln[sl], lo_[sl], mask[sl], pos[sl], start, 0.2, 0.28, 0.01)
        r = np.exp(ln[sl].astype(np.float64) - lo_[sl].astype(np.float64))
        ok = ~((np.abs(r - 0.8) < 1e-5) | (np.abs(r - 1.28) < 1e-5))
        gg, ll = g.cpu().double().numpy(), l.cpu().double().numpy()
        assert np.allclose(gg[ok], og[ok], rtol=1e-5, atol=1e-12), f"offset {off}"
        assert np.allclose(ll[ok], ol[ok], rtol=1e-5, atol=1e-12), f"offset {off}"
