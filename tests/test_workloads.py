"""The seeded synthetic generator: determinism, recipe properties, and the
planted branch positions that the oracle must recover (end-to-end pin of the
oracle on the small fp32 workload)."""
import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O


def test_tiny_is_deterministic():
    a = workloads.make_workload("tiny")
    b = workloads.make_workload("tiny")
    assert torch.equal(a.W, b.W) and torch.equal(a.hidden, b.hidden)
    assert torch.equal(a.tokens, b.tokens) and torch.equal(a.mask, b.mask)
    c = workloads.make_workload("tiny", seed=77)
    assert not torch.equal(a.W, c.W)


def test_tiny_shapes_and_distributions():
    w = workloads.make_workload("tiny")
    c = w.cfg
    assert w.W.shape == (c.V, c.d) and w.W.dtype == torch.float32
    assert w.hidden.shape == (2, c.R, c.T, c.d)
    assert abs(float(w.W.std()) - 0.02) < 1e-3
    rms = w.hidden[0].pow(2).mean(-1).sqrt()
    assert torch.allclose(rms, torch.ones_like(rms), atol=1e-5)
    assert int(w.tokens.min()) >= 0 and int(w.tokens.max()) < c.V
    assert int(w.mask.sum()) == c.R * c.T


def test_planted_shift_moves_target_logit():
    w = workloads.make_workload("tiny")
    pl = w.planted[0]
    Wd = w.W.double()
    for t, a, s in zip(pl["pos"], pl["alpha"], pl["sign"]):
        y = int(w.tokens[0, t])
        dz = float((w.hidden[1, 0, t].double() - w.hidden[0, 0, t].double()) @ Wd[y])
        assert abs(dz - s * a) < 0.05


def test_oracle_recovers_planted_positions_tiny():
    w = workloads.make_workload("tiny")
    H = w.rows_hidden().double().numpy()
    Wd = w.W.double().numpy()
    y = w.rows_tokens().numpy()
    lp, _ = O.token_logprobs(H, Wd, y)
    T = w.cfg.T
    idx, sc, cnt = O.select_branch_points(lp[:T][None], lp[T:][None], w.mask.numpy(), w.cfg.k)
    assert sorted(idx[0].tolist()) == sorted(w.planted[0]["pos"].tolist())
    assert np.all(lp <= 0)
    # the k-th/(k+1)-th gap is huge here, so the set is unique
    _, s, el = O.divergence(lp[:T][None], lp[T:][None], w.mask.numpy())
    srt = np.sort(s[0])[::-1]
    assert srt[3] - srt[4] > 1.0


@pytest.mark.parametrize("name,over", [
    ("c2", dict(R=2, T=96, d=64, V=1000)),
    ("c3", dict(R=2, T=300, d=64, V=1000)),
    ("c4", dict(R=3, T=1500, d=64, V=1000)),
    ("c5", dict(R=2, T=400, d=64, V=1000)),
])
def test_reduced_recipes(name, over):
    w = workloads.make_workload(name, **over)
    c = w.cfg
    assert w.W.dtype == torch.bfloat16 and w.hidden.dtype == torch.bfloat16
    m = w.mask.numpy()
    for r in range(c.R):
        pos = w.planted[r]["pos"]
        assert np.all(m[r, pos] == 1), "planted positions must be policy tokens"
        assert len(np.unique(pos)) == len(pos)
    if name == "c2":
        assert np.all(m[:, :32] == 0) and np.all(m[:, 32:] == 1)
    if name == "c4":
        # at T = 1500, 5-20 spans of 64-512 tokens cover most of a root (the
        # full-shape fraction is checked below): some positions on, some off
        frac = m.mean()
        assert 0.0 < frac < 0.95
    if name == "c3":
        a = np.concatenate([p["alpha"] for p in w.planted])
        assert a.min() >= 0.05 - 1e-12 and a.max() <= 5.0 + 1e-12
    if name == "c5":
        for r in range(c.R):
            assert len(w.band[r]) == c.n_band
            for src, dst in w.dup_pairs[r]:
                assert torch.equal(w.hidden[:, r, src], w.hidden[:, r, dst])
                assert int(w.tokens[r, src]) == int(w.tokens[r, dst])


def test_c4_span_mask_full_shape_fraction():
    # The agent mask recipe alone (cheap at full T): ~56 % eligible.
    cfg = workloads.get_config("c4")
    from workloads.synth import _make_mask
    fr = np.mean([_make_mask(cfg, r).mean() for r in range(cfg.R)])
    assert 0.45 < fr < 0.7


def test_logp_pair_generator():
    lo, lh, mask = workloads.make_logp_pair(3, 500, seed=5, nan_rows=2)
    assert lo.dtype == np.float32 and lh.dtype == np.float32
    assert np.isnan(lh).sum() >= 1
    lo2, lh2, mask2 = workloads.make_logp_pair(3, 500, seed=5, nan_rows=2)
    assert np.array_equal(lo, lo2) and np.array_equal(mask, mask2)
