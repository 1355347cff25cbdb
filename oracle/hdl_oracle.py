"""Float64 CPU oracle for hindsight-divergence localization (HDL) re-scoring.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously correct
definition of what the GPU library computes.  Only the test-suite, the smoke
check and the CPU-baseline leg of the benchmark may import it; the library
itself never calls it and shares no code with it.

What it follows (paper: "Where the Model Changes Its Mind: Hindsight-Divergence
Localization for Efficient RLVR"):

* Sec. 3.1, Eq. 1 -- for every policy-generated token y_i, the next-token
  distributions under the original context (x, y_<i) and the hindsight
  context (x, h, y_<i) come from the same parameters and the same prefix.
  Here each distribution is the softmax of the lm-head logits z = W h_i of the
  final hidden state h_i that predicts y_i; the teacher-forced log-likelihood
  of the sampled token is log p_i(y_i) = z_{y_i} - logsumexp_v z_v.
* Sec. 3.2, Eq. 2 -- the hindsight-divergence score
  s_i = | log p_i^H(y_i) - log p_i^0(y_i) |.
* Sec. 3.2 (last paragraph) and Sec. 4.1 ("Rollout protocols") -- positions
  are ranked within each root by s_i and the highest-scoring ones become the
  branch points (two per root in the paper's setting; k is a parameter here).

Readings where the paper is silent (each also listed in the design notes):

* row n of `hidden` is the state that predicts tokens[n] (the caller applies
  the teacher-forcing shift);
* only positions with mask != 0 are scored and are candidates; masked rows
  get log p = 0.0 and lse = 0.0 by convention;
* log p is plain log-softmax at temperature 1;
* ties in s are broken by the lower position index (order: s desc, t asc);
* a token outside [0, V) makes that row's log p NaN, and a NaN score is never
  a candidate;
* fewer than k candidates: count < k, idx padded with -1, score with 0.0.

Backward (training side, Sec. 3.3: roots and continuations are trained with
the same token-level policy loss): for L = sum_n g_n log p_n(y_n), where g_n
is whatever the loss puts on each token's log-likelihood, the gradients with
respect to the final hidden states and the lm-head weight follow from
d log p_n(y) / d z_n[v] = 1[v == y] - p_n(v).  Masked rows contribute
nothing and get a zero gradient; a token outside [0, V) has no indicator term.

Entropy baseline (Sec. 4.1, "Rollout protocols"; Table 4): the next-token
entropy -sum_v p(v) log p(v) of the same distributions under the original
context, ranked per root like s (`select_by_value`).

Group construction (Sec. 3 and 3.3, Sec. 4.1 "Training" and "Rollout
protocols", Sec. 4.3-4.4): selection under an allowed index range and a
minimum spacing (`select_constrained`), continuation slots per retained point
(`allocate_continuations`), mean-centred group advantages
(`group_advantages`), and the per-token derivative of the asymmetrically
clipped surrogate with suffix-only training of continuations
(`policy_loss_grad`).  Where the paper leaves values open (the constraint
values, which point gets more continuations, a root with no valid point)
they are parameters; the readings are listed in the design notes.

Pins: every function here is checked by tests that do not re-type its formula
(brute-force softmax with exact summation, closed forms, invariants, hand-worked
fixtures, brute-force sorting).  See tests/test_oracle_pins.py.
"""
from __future__ import annotations

import math
from typing import Optional, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# Input decoding
# ---------------------------------------------------------------------------
def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact decode of bfloat16 bit patterns (uint16) to float64.

    A bfloat16 value is the upper 16 bits of an IEEE-754 binary32 value, so
    placing the bits in the top half of a 32-bit word and widening is exact.
    """
    b = np.asarray(bits)
    if b.dtype != np.uint16:
        b = b.view(np.uint16) if b.dtype.itemsize == 2 else b.astype(np.uint16)
    u32 = b.astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return u32.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Eq. 1: teacher-forced log-likelihood of the sampled token
# ---------------------------------------------------------------------------
def token_logprobs(hidden: np.ndarray, W: np.ndarray, tokens: np.ndarray,
                   mask: Optional[np.ndarray] = None,
                   row_block: int = 256) -> Tuple[np.ndarray, np.ndarray]:
    """log p_n(tokens[n]) = z_n[tokens[n]] - logsumexp_v z_n[v],  z_n = W hidden[n].

    hidden: [N, d] float64; W: [V, d] float64; tokens: [N] int; mask: [N] or
    None (all rows scored).  Returns (logp [N], lse [N]) in float64; rows with
    mask == 0 get 0.0 in both.  Rows are processed in blocks of `row_block`
    only to bound memory; every row is independent.
    """
    hidden = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    tokens = np.asarray(tokens).astype(np.int64)
    N = hidden.shape[0]
    V = W.shape[0]
    logp = np.zeros(N, dtype=np.float64)
    lse = np.zeros(N, dtype=np.float64)
    rows = np.arange(N) if mask is None else np.nonzero(np.asarray(mask))[0]
    WT = W.T
    for b0 in range(0, len(rows), row_block):
        r = rows[b0:b0 + row_block]
        z = hidden[r] @ WT                                   # [b, V] logits
        m = z.max(axis=1)                                    # softmax shift
        l = m + np.log(np.exp(z - m[:, None]).sum(axis=1))   # log normaliser
        y = tokens[r]
        ok = (y >= 0) & (y < V)
        zy = np.where(ok, z[np.arange(len(r)), np.where(ok, y, 0)], np.nan)
        logp[r] = zy - l
        lse[r] = l
    return logp, lse


def full_logprobs(hidden: np.ndarray, W: np.ndarray) -> np.ndarray:
    """All-vocabulary log-softmax, [N, V] float64 (small inputs only)."""
    z = np.asarray(hidden, np.float64) @ np.asarray(W, np.float64).T
    m = z.max(axis=1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))


def token_entropy(hidden: np.ndarray, W: np.ndarray,
                  mask: Optional[np.ndarray] = None,
                  row_block: int = 256) -> np.ndarray:
    """Next-token entropy H_n = -sum_v p_n(v) log p_n(v) (Sec. 4.1, the
    Entropy localization baseline ranks positions by it).  float64 [N];
    masked rows get 0.0."""
    hidden = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    N = hidden.shape[0]
    out = np.zeros(N, dtype=np.float64)
    rows = np.arange(N) if mask is None else np.nonzero(np.asarray(mask))[0]
    for b0 in range(0, len(rows), row_block):
        r = rows[b0:b0 + row_block]
        z = hidden[r] @ W.T
        m = z.max(axis=1, keepdims=True)
        logq = z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))
        out[r] = -(np.exp(logq) * logq).sum(axis=1)
    return out


def token_logprobs_backward(hidden: np.ndarray, W: np.ndarray, tokens: np.ndarray,
                            grad_logp: np.ndarray, mask: Optional[np.ndarray] = None):
    """Gradients of L = sum_n g_n log p_n(tokens[n]) (Eq. 1's log-likelihood,
    weighted by the policy loss's per-token factor g_n, Sec. 3.3).

    With G[n, v] = g_n (1[v == y_n] - p_n(v)):
        dL/dhidden = G W        [N, d]
        dL/dW      = G^T hidden [V, d]
    Also returns the element-wise magnitudes sum_v |G| |W| and sum_n |G| |h|,
    which bound how far a result computed from a rounded G can move.
    Returns (dH, dW, mag_dH, mag_dW), all float64; masked rows of dH are 0.
    """
    H = np.asarray(hidden, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    y = np.asarray(tokens).astype(np.int64)
    g = np.asarray(grad_logp, dtype=np.float64)
    N, V = H.shape[0], W.shape[0]
    keep = np.ones(N, bool) if mask is None else (np.asarray(mask) != 0)
    z = H @ W.T
    m = z.max(axis=1, keepdims=True)
    P = np.exp(z - m)
    P /= P.sum(axis=1, keepdims=True)
    onehot = np.zeros((N, V))
    ok = (y >= 0) & (y < V)
    onehot[np.nonzero(ok)[0], y[ok]] = 1.0
    G = g[:, None] * (onehot - P)
    G[~keep] = 0.0
    return G @ W, G.T @ H, np.abs(G) @ np.abs(W), np.abs(G).T @ np.abs(H)


# ---------------------------------------------------------------------------
# Eq. 2: hindsight-divergence score and per-root ranking
# ---------------------------------------------------------------------------
def divergence(logp_orig: np.ndarray, logp_hind: np.ndarray,
               mask: Optional[np.ndarray] = None,
               precision: str = "f64") -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Signed change d = log p^H - log p^0, score s = |d|, and eligibility.

    Inputs [R, T].  precision="f64" evaluates in float64; precision="f32"
    evaluates the difference as one IEEE binary32 subtraction, which is the
    precision in which the GPU kernel takes its ranking decisions.
    Eligible = mask != 0 and the score is finite (NaN rows never qualify).
    Returns (signed [R,T], score [R,T], eligible bool [R,T]); signed and score
    are 0 where not eligible.
    """
    if precision == "f32":
        a = np.asarray(logp_orig, dtype=np.float32)
        b = np.asarray(logp_hind, dtype=np.float32)
        with np.errstate(invalid="ignore"):
            sd = (b - a).astype(np.float32)
    elif precision == "f64":
        a = np.asarray(logp_orig, dtype=np.float64)
        b = np.asarray(logp_hind, dtype=np.float64)
        with np.errstate(invalid="ignore"):
            sd = b - a
    else:
        raise ValueError(precision)
    m = np.ones(sd.shape, bool) if mask is None else (np.asarray(mask) != 0)
    elig = m & np.isfinite(sd)
    sd = np.where(elig, sd, 0.0).astype(sd.dtype)
    s = np.abs(sd)
    return sd, s, elig


def select_branch_points(logp_orig: np.ndarray, logp_hind: np.ndarray,
                         mask: Optional[np.ndarray], k: int,
                         precision: str = "f64"):
    """Per root, the k eligible positions with the largest score s, ordered by
    (s descending, position ascending).

    Returns (idx int32 [R,k], score [R,k], count int32 [R]); rows with fewer
    than k candidates are padded with idx -1 and score 0.
    """
    if k < 1:
        raise ValueError("k must be >= 1")
    _, s, elig = divergence(logp_orig, logp_hind, mask, precision)
    R, T = s.shape
    idx = np.full((R, k), -1, dtype=np.int32)
    score = np.zeros((R, k), dtype=s.dtype)
    count = np.zeros(R, dtype=np.int32)
    for r in range(R):
        cand = [t for t in range(T) if elig[r, t]]
        ranked = sorted(cand, key=lambda t: (-float(s[r, t]), t))[:k]
        count[r] = len(ranked)
        for j, t in enumerate(ranked):
            idx[r, j] = t
            score[r, j] = s[r, t]
    return idx, score, count


def select_by_value(values: np.ndarray, mask: Optional[np.ndarray], k: int):
    """Per-root top-k of an arbitrary per-position value (e.g. entropy for the
    Entropy baseline), ordered (value desc, position asc); NaN never selected."""
    v = np.asarray(values, dtype=np.float64)
    m = np.ones(v.shape, bool) if mask is None else (np.asarray(mask) != 0)
    elig = m & np.isfinite(v)
    R, T = v.shape
    idx = np.full((R, k), -1, dtype=np.int32)
    score = np.zeros((R, k), dtype=np.float64)
    count = np.zeros(R, dtype=np.int32)
    for r in range(R):
        cand = [t for t in range(T) if elig[r, t]]
        ranked = sorted(cand, key=lambda t: (-v[r, t], t))[:k]
        count[r] = len(ranked)
        for j, t in enumerate(ranked):
            idx[r, j] = t
            score[r, j] = v[r, t]
    return idx, score, count


# ---------------------------------------------------------------------------
# Group construction (Sec. 3.3, Sec. 4.1, Sec. 4.3-4.4)
# ---------------------------------------------------------------------------
def select_constrained(a: np.ndarray, b: Optional[np.ndarray], mask: Optional[np.ndarray], k: int,
                       lo=None, hi=None, min_gap: int = 0, refill: bool = False,
                       precision: str = "f64", pool_cap: int = 1024):
    """Per-root selection under the branch-point constraints.

    Score: |b - a| (Eq. 2; `precision="f32"` evaluates the difference as one
    binary32 subtraction) or, with b None, a's values.  Candidates: mask != 0,
    finite score, lo[r] <= t <= hi[r].  Ranked by (score desc, t asc).  A
    point is retained if it lies at least min_gap from every point retained
    before it (min_gap <= 1: always); without refill only the top k ranked
    candidates are considered (so fewer than k may remain), with refill the
    best `pool_cap` candidates are walked until k are retained.
    """
    a = np.asarray(a)
    R, T = a.shape
    if b is None:
        sc = a.astype(np.float64)
    elif precision == "f32":
        sc = np.abs((np.asarray(b, np.float32) - np.asarray(a, np.float32)).astype(np.float64))
    else:
        sc = np.abs(np.asarray(b, np.float64) - a.astype(np.float64))
    m = np.ones((R, T), bool) if mask is None else (np.asarray(mask) != 0)
    idx = np.full((R, k), -1, dtype=np.int32)
    score = np.zeros((R, k), dtype=np.float64)
    count = np.zeros(R, dtype=np.int32)
    for r in range(R):
        t_lo = 0 if lo is None else int(lo[r])
        t_hi = T - 1 if hi is None else int(hi[r])
        cand = [t for t in range(T) if m[r, t] and np.isfinite(sc[r, t]) and t_lo <= t <= t_hi]
        ranked = sorted(cand, key=lambda t: (-sc[r, t], t))
        pool = ranked[:pool_cap] if refill else ranked[:k]
        kept = []
        for t in pool:
            if len(kept) == k:
                break
            if min_gap <= 1 or all(abs(t - u) >= min_gap for u in kept):
                kept.append(t)
        count[r] = len(kept)
        for j, t in enumerate(kept):
            idx[r, j] = t
            score[r, j] = sc[r, t]
    return idx, score, count


def allocate_continuations(idx: np.ndarray, count: np.ndarray, alloc, fallback: int = 0):
    """Branch position (and rank, -1 for the fallback) of every continuation
    slot: rank j takes alloc[j] slots in rank order; a rank the root does not
    have sends its slots to the root's best point (Sec. 4.4: a root with one
    valid point takes all of its continuations there); a root with no point
    branches at `fallback`."""
    idx = np.asarray(idx)
    R, k = idx.shape
    if len(alloc) != k:
        raise ValueError("alloc needs one slot count per selected rank")
    total = int(sum(alloc))
    pos = np.zeros((R, total), dtype=np.int32)
    rank = np.zeros((R, total), dtype=np.int32)
    for r in range(R):
        c = max(0, min(int(count[r]), k))
        slot = 0
        for j in range(k):
            for _ in range(int(alloc[j])):
                if c == 0:
                    pos[r, slot], rank[r, slot] = fallback, -1
                else:
                    target = j if j < c else 0
                    pos[r, slot], rank[r, slot] = idx[r, target], target
                slot += 1
    return pos, rank


def group_advantages(rewards: np.ndarray) -> np.ndarray:
    """A_j = R_j - mean_k R_k within each group (row); no std normalisation
    (Sec. 3; Sec. 4.1 follows Dr. GRPO)."""
    R = np.asarray(rewards, dtype=np.float64)
    return R - R.mean(axis=1, keepdims=True)


def trained_tokens(traj, n_traj: int, loss_mask=None, pos=None, start=None) -> int:
    """Number of tokens the policy loss trains on: in the loss mask, with a
    trajectory index in [0, n_traj), and (given positions) at or after their
    trajectory's first trained position -- a continuation trains only its
    newly sampled suffix (Sec. 3.3)."""
    traj = np.asarray(traj).astype(np.int64)
    count = 0
    for i in range(traj.shape[0]):
        j = traj[i]
        if not (0 <= j < n_traj) or (loss_mask is not None and loss_mask[i] == 0):
            continue
        if pos is not None and pos[i] < start[j]:
            continue
        count += 1
    return count


def policy_loss_grad(adv, traj, logp_new, logp_old, loss_mask=None, pos=None, start=None,
                     eps_low: float = 0.2, eps_high: float = 0.28, scale: Optional[float] = 1.0):
    """Per-token loss l = -scale * min(r A, clip(r, 1 - eps_low, 1 + eps_high) A)
    with r = exp(logp_new - logp_old), and g = dl/dlogp_new (Sec. 4.1
    "Training"); tokens outside the loss mask, before their trajectory's
    first trained position (a continuation's reused prefix, Sec. 3.3) or
    with an out-of-range trajectory index give 0.  scale=None is the
    token-level aggregation of Sec. 4.1: the mean over the trained tokens,
    scale = 1 / max(1, trained_tokens(...)).  Returns (g, l)."""
    adv = np.asarray(adv, dtype=np.float64)
    traj = np.asarray(traj).astype(np.int64)
    if scale is None:
        scale = 1.0 / max(1, trained_tokens(traj, adv.shape[0], loss_mask, pos, start))
    n = traj.shape[0]
    g = np.zeros(n)
    loss = np.zeros(n)
    for i in range(n):
        j = traj[i]
        on = 0 <= j < adv.shape[0] and (loss_mask is None or loss_mask[i] != 0)
        if on and pos is not None:
            on = pos[i] >= start[j]
        if not on:
            continue
        r = math.exp(float(logp_new[i]) - float(logp_old[i]))
        a = adv[j]
        rc = min(max(r, 1.0 - eps_low), 1.0 + eps_high)
        unclipped, clipped = r * a, rc * a
        loss[i] = -scale * min(unclipped, clipped)
        g[i] = -scale * a * r if unclipped <= clipped else 0.0
    return g, loss


def branch_set_agrees(gpu_idx, gpu_count, oracle_scores, eligible, k,
                      gap: float = 1e-2) -> Tuple[bool, str]:
    """Acceptance rule for one root when several answers can be right.

    oracle_scores/eligible: [T] for one root (float64 scores from the oracle).
    Let s*_(k) be the k-th largest eligible oracle score.  If the gap between
    the k-th and (k+1)-th largest exceeds `gap`, the GPU set must equal the
    oracle set.  Otherwise every selected position must score at least
    s*_(k) - gap and every unselected eligible position at most s*_(k) + gap.
    """
    s = np.asarray(oracle_scores, np.float64)
    e = np.asarray(eligible, bool)
    cand = np.nonzero(e)[0]
    want = min(k, len(cand))
    sel = [int(t) for t in np.asarray(gpu_idx)[:int(gpu_count)]]
    if int(gpu_count) != want:
        return False, f"count {gpu_count} != {want}"
    if len(set(sel)) != len(sel):
        return False, "duplicate positions selected"
    if any((t < 0) or (t >= len(s)) or (not e[t]) for t in sel):
        return False, "ineligible position selected"
    if want == 0:
        return True, "empty"
    ranked = sorted(cand.tolist(), key=lambda t: (-s[t], t))
    sk = s[ranked[want - 1]]
    nxt = s[ranked[want]] if want < len(ranked) else -math.inf
    if sk - nxt > gap:
        ok = set(sel) == set(ranked[:want])
        return ok, "exact set" if ok else f"set differs: {sorted(sel)} vs {sorted(ranked[:want])}"
    for t in sel:
        if s[t] < sk - gap:
            return False, f"selected {t} scores {s[t]} < {sk} - gap"
    chosen = set(sel)
    for t in cand:
        if int(t) not in chosen and s[t] > sk + gap:
            return False, f"missed {t} scoring {s[t]} > {sk} + gap"
    return True, "tie-tolerant"
