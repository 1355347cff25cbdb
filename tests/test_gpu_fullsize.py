"""Full-size parity of the re-scoring path on the four large workloads, in
the launch configuration the benchmark times (one call for both contexts of
all roots, then the per-root selection), checked on outputs the float64
oracle can compute row by row:

* log p of every planted position, every selected position and a seeded
  sample of other eligible positions, in both contexts (|error| <= 2e-3);
* the branch set of each checked root against the oracle's ranking of those
  positions under the tie-tolerant rule (identical wherever the k-th /
  (k+1)-th gap exceeds 1e-2), with the sampled unplanted positions scoring
  below the selected ones, and the selection drawn from the planted
  positions (the planted shifts are what the hindsight context changes).
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O
from tests.gpu_helpers import as_f64, require_gpu

pytestmark = pytest.mark.gpu

TOL = 2e-3


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


@pytest.mark.parametrize("name,roots_checked", [("c2", 8), ("c3", 4), ("c4", 6), ("c5", 2)])
def test_full_size_logprobs_and_branch_points(hdl, name, roots_checked):
    w = workloads.make_workload(name)
    c = w.cfg
    dev = "cuda"
    lp, idx, score, count = hdl.rescore(w.hidden.to(dev), w.W.to(dev), w.tokens.to(dev), w.mask.to(dev), c.k)
    torch.cuda.synchronize()
    lp = lp.cpu().numpy()
    idx = idx.cpu().numpy()
    count = count.cpu().numpy()
    mask = w.mask.numpy().astype(bool)
    assert np.all(lp[:, ~mask] == 0.0) and np.all(lp[:, mask] <= 0.0)

    rng = np.random.default_rng(c.seed + 99)
    roots = np.sort(rng.choice(c.R, size=roots_checked, replace=False))
    cand = {}
    for r in roots:
        elig = np.nonzero(mask[r])[0]
        sample = rng.choice(elig, size=8, replace=False)
        cand[r] = (np.unique(np.concatenate([w.planted[r]["pos"], idx[r, :count[r]], sample])), sample)
    rows, keys = [], []
    for r in roots:
        for t in cand[r][0]:
            for ctx in range(2):
                rows.append(ctx * c.R * c.T + r * c.T + int(t))
                keys.append((ctx, r, int(t)))
    rows = np.array(rows)
    H = as_f64(w.rows_hidden()[torch.as_tensor(rows)])
    want, _ = O.token_logprobs(H, as_f64(w.W), w.rows_tokens().numpy()[rows])
    got = np.array([lp[ctx, r, t] for ctx, r, t in keys])
    err = np.abs(got - want)
    assert err.max() <= TOL, f"{name}: max |log p error| {err.max():.3g}"

    ref = {key: v for key, v in zip(keys, want)}
    for r in roots:
        pos, sample = cand[r]
        s = np.zeros(c.T)
        elig = np.zeros(c.T, bool)
        for t in pos:
            s[t] = abs(ref[(1, r, int(t))] - ref[(0, r, int(t))])
            elig[t] = True
        ok, why = O.branch_set_agrees(idx[r], int(count[r]), s, elig, c.k)
        assert ok, f"{name} root {r}: {why}"
        sel = idx[r, :count[r]]
        kth = s[sel].min()
        unplanted = [t for t in sample if t not in set(w.planted[r]["pos"].tolist())]
        assert all(s[t] < kth - 1e-2 for t in unplanted), f"{name} root {r}: a sampled position outranks the selection"
        assert set(sel.tolist()) <= set(w.planted[r]["pos"].tolist()), f"{name} root {r}: unplanted point selected"
