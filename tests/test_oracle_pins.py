"""Pins for the float64 oracle: checks against facts fixed by the paper's
definitions and by mathematics, never against a re-typed copy of the oracle's
own formula.

Eq. 1 (teacher-forced log-softmax of the sampled token), Eq. 2 (absolute
log-likelihood change) and the per-root ranking of Sec. 3.2 are pinned by:
hand-worked fixtures, brute-force softmax with exact (fsum) summation,
closed forms (uniform, log-sigmoid, single-logit change), invariants
(normalisation, vocabulary permutation, logit shift, batching) and a
rank-counting brute force for the selection.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import workloads
from oracle import hdl_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")


# ---------------------------------------------------------------- decoding
def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x8000, 0x7F80, 0xFF80,
                     0x4049, 0x0080], dtype=np.uint16)
    got = O.bf16_bits_to_f64(bits)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 2.0 ** -133, -0.0, math.inf, -math.inf,
            3.140625, 2.0 ** -126]
    for g, w in zip(got, want):
        assert g == w
    assert math.copysign(1.0, got[4]) == -1.0
    assert np.isnan(O.bf16_bits_to_f64(np.array([0x7FC0], np.uint16)))[0]


def test_bf16_decode_matches_torch():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 1 << 16, 200000, dtype=np.uint32).astype(np.uint16)
    ours = O.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    fin = np.isfinite(ref)
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    assert np.array_equal(ours[fin], ref[fin])


# ---------------------------------------------------------------- Eq. 1
def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_golden_hand_worked_logprobs():
    for case in _golden()["logprob_cases"]:
        W = np.array(case["W"], dtype=np.float64)
        h = np.array(case["h"], dtype=np.float64)[None, :]
        for e in case["expected"]:
            lp, lse = O.token_logprobs(h, W, np.array([e["token"]]))
            assert abs(lp[0] - e["logp"]) < 1e-14, (case["name"], e)
            assert abs(lse[0] - case["lse"]["value"]) < 1e-14, case["name"]


def _brute_logp(h, W, y):
    """Direct definition: log( exp(z_y) / sum_v exp(z_v) ), exact sums, no shift."""
    z = [math.fsum(float(a) * float(b) for a, b in zip(h, w)) for w in W]
    denom = math.fsum(math.exp(zv) for zv in z)
    return math.log(math.exp(z[y]) / denom)


@pytest.mark.parametrize("V,d", [(2, 1), (7, 5), (64, 16), (33, 3)])
def test_bruteforce_softmax(V, d):
    rng = np.random.default_rng(V * 100 + d)
    W = rng.normal(0, 1.0, (V, d))
    H = rng.normal(0, 2.0, (9, d))
    y = rng.integers(0, V, 9)
    lp, _ = O.token_logprobs(H, W, y)
    for n in range(9):
        assert abs(lp[n] - _brute_logp(H[n], W, int(y[n]))) < 1e-12


def test_bruteforce_tiny_vocab_4096():
    rng = np.random.default_rng(7)
    W = rng.normal(0, 0.02, (4096, 8))
    H = rng.normal(0, 1.0, (3, 8))
    y = np.array([0, 4095, 1234])
    lp, _ = O.token_logprobs(H, W, y)
    for n in range(3):
        assert abs(lp[n] - _brute_logp(H[n], W, int(y[n]))) < 1e-12


@pytest.mark.parametrize("V", [4096, 151936, 152064])
def test_zero_hidden_is_minus_log_V(V):
    rng = np.random.default_rng(1)
    W = rng.normal(0, 0.02, (V, 4))
    lp, lse = O.token_logprobs(np.zeros((2, 4)), W, np.array([0, V - 1]))
    assert np.all(np.abs(lp + math.log(V)) < 1e-12)
    assert np.all(np.abs(lse - math.log(V)) < 1e-12)


def test_identical_W_rows_is_minus_log_V():
    V, d = 1000, 6
    rng = np.random.default_rng(2)
    W = np.tile(rng.normal(0, 1, (1, d)), (V, 1))
    H = rng.normal(0, 3, (4, d))
    lp, _ = O.token_logprobs(H, W, np.array([0, 5, 999, 500]))
    assert np.all(np.abs(lp + math.log(V)) < 1e-12)


def test_two_word_vocab_is_log_sigmoid():
    rng = np.random.default_rng(3)
    W = rng.normal(0, 1, (2, 5))
    H = rng.normal(0, 2, (20, 5))
    y = rng.integers(0, 2, 20)
    lp, _ = O.token_logprobs(H, W, y)
    for n in range(20):
        zy = float(H[n] @ W[y[n]])
        zo = float(H[n] @ W[1 - y[n]])
        x = zy - zo
        # log sigmoid(x) = -log(1 + e^-x), written in its overflow-safe form
        ls = -math.log1p(math.exp(-x)) if x >= 0 else x - math.log1p(math.exp(x))
        assert abs(lp[n] - ls) < 1e-13


def test_dominant_target_goes_to_zero():
    V, d = 50, 50
    W = np.eye(V, d) * 60.0
    H = np.zeros((1, d)); H[0, 7] = 1.0
    lp, _ = O.token_logprobs(H, W, np.array([7]))
    # log p = -log(1 + (V-1) e^-60)
    assert abs(lp[0] - (-math.log1p((V - 1) * math.exp(-60.0)))) < 1e-15
    assert lp[0] <= 0.0


def test_large_logits_do_not_overflow():
    # logits around 1000 overflow exp() without the max shift
    W = np.array([[1000.0], [999.0], [990.0]])
    lp, lse = O.token_logprobs(np.array([[1.0]]), W, np.array([1]))
    want = -1.0 - math.log(1.0 + math.exp(-1.0) + math.exp(-10.0))
    assert abs(lp[0] - want) < 1e-12
    assert abs(lse[0] - (1000.0 + math.log(1.0 + math.exp(-1.0) + math.exp(-10.0)))) < 1e-9


def test_probabilities_sum_to_one():
    rng = np.random.default_rng(4)
    V, d = 300, 12
    W = rng.normal(0, 0.5, (V, d))
    h = rng.normal(0, 2.0, (1, d))
    lp, _ = O.token_logprobs(np.repeat(h, V, 0), W, np.arange(V))
    assert abs(math.fsum(math.exp(x) for x in lp) - 1.0) < 1e-12
    assert np.all(lp < 0)
    full = O.full_logprobs(h, W)[0]
    assert np.allclose(full, lp, atol=1e-13, rtol=0)


def test_vocab_permutation_invariance():
    rng = np.random.default_rng(5)
    V, d, N = 257, 9, 11
    W = rng.normal(0, 1, (V, d))
    H = rng.normal(0, 1, (N, d))
    y = rng.integers(0, V, N)
    perm = rng.permutation(V)            # new row j holds old row perm[j]
    inv = np.argsort(perm)               # old token t sits at new row inv[t]
    a, _ = O.token_logprobs(H, W, y)
    b, _ = O.token_logprobs(H, W[perm], inv[y])
    assert np.allclose(a, b, atol=1e-12, rtol=0)


def test_logit_shift_invariance():
    # An extra feature equal to 1 in every hidden row with a constant weight c
    # in every vocab row adds c to every logit; log-softmax must not change.
    rng = np.random.default_rng(6)
    V, d, N = 120, 7, 6
    W = rng.normal(0, 1, (V, d))
    H = rng.normal(0, 1, (N, d))
    y = rng.integers(0, V, N)
    base, lse0 = O.token_logprobs(H, W, y)
    for c in (-50.0, 3.5, 400.0):
        W2 = np.hstack([W, np.full((V, 1), c)])
        H2 = np.hstack([H, np.ones((N, 1))])
        got, lse = O.token_logprobs(H2, W2, y)
        assert np.allclose(got, base, atol=1e-11, rtol=0)
        assert np.allclose(lse - lse0, c, atol=1e-10, rtol=0)


def test_row_blocking_and_order_invariance():
    rng = np.random.default_rng(8)
    V, d, N = 500, 10, 37
    W = rng.normal(0, 1, (V, d))
    H = rng.normal(0, 1, (N, d))
    y = rng.integers(0, V, N)
    a, _ = O.token_logprobs(H, W, y, row_block=256)
    b, _ = O.token_logprobs(H, W, y, row_block=1)
    p = rng.permutation(N)
    c, _ = O.token_logprobs(H[p], W, y[p], row_block=5)
    assert np.allclose(a, b, atol=1e-13, rtol=0)
    assert np.allclose(a[p], c, atol=1e-13, rtol=0)


def test_masked_rows_are_zero_and_unscored():
    rng = np.random.default_rng(9)
    W = rng.normal(0, 1, (40, 4))
    H = rng.normal(0, 1, (6, 4))
    y = rng.integers(0, 40, 6)
    mask = np.array([1, 0, 1, 0, 0, 1], np.uint8)
    lp, lse = O.token_logprobs(H, W, y, mask)
    full, _ = O.token_logprobs(H, W, y)
    assert np.all(lp[mask == 0] == 0.0) and np.all(lse[mask == 0] == 0.0)
    assert np.array_equal(lp[mask == 1], full[mask == 1])


def test_out_of_range_token_is_nan():
    rng = np.random.default_rng(10)
    W = rng.normal(0, 1, (40, 4))
    H = rng.normal(0, 1, (3, 4))
    lp, _ = O.token_logprobs(H, W, np.array([-1, 40, 3]))
    assert np.isnan(lp[0]) and np.isnan(lp[1]) and np.isfinite(lp[2])


# ---------------------------------------------------------------- Eq. 2
def test_single_logit_change_closed_form():
    """If hindsight raises only the sampled token's logit by delta, then
    log p^H - log p^0 = delta - log(1 - p + p e^delta), p = p^0(y)."""
    rng = np.random.default_rng(11)
    V, d = 90, 6
    W = rng.normal(0, 1, (V, d))
    y = 17
    # extra feature that only the sampled token's row reads
    W2 = np.hstack([W, np.zeros((V, 1))]); W2[y, -1] = 1.0
    h = rng.normal(0, 1, d)
    for delta in (-4.0, -0.3, 0.0, 0.7, 3.0):
        h0 = np.append(h, 0.0)[None, :]
        hH = np.append(h, delta)[None, :]
        l0, _ = O.token_logprobs(h0, W2, np.array([y]))
        lH, _ = O.token_logprobs(hH, W2, np.array([y]))
        p = math.exp(l0[0])
        want = delta - math.log(1.0 - p + p * math.exp(delta))
        sd, s, el = O.divergence(l0[None, :], lH[None, :], None)
        assert abs(sd[0, 0] - want) < 1e-12
        assert abs(s[0, 0] - abs(want)) < 1e-12 and el[0, 0]


def test_golden_selection_case():
    g = _golden()["selection_case"]
    W = np.array(g["W"], np.float64)
    l0, _ = O.token_logprobs(np.array(g["h_orig"]), W, np.array(g["tokens"]))
    lH, _ = O.token_logprobs(np.array(g["h_hind"]), W, np.array(g["tokens"]))
    sd, s, _ = O.divergence(l0[None], lH[None], None)
    assert np.allclose(sd[0], g["signed"], atol=1e-14, rtol=0)
    assert np.allclose(s[0], g["score"], atol=1e-14, rtol=0)
    for sel in g["selections"]:
        idx, sc, cnt = O.select_branch_points(l0[None], lH[None], np.array([sel["mask"]]), sel["k"])
        assert idx[0].tolist() == sel["idx"] and int(cnt[0]) == sel["count"]


def test_identical_contexts_give_zero_and_swap_negates():
    rng = np.random.default_rng(12)
    W = rng.normal(0, 0.3, (64, 8))
    H0 = rng.normal(0, 1, (10, 8)); HH = H0 + rng.normal(0, 0.2, (10, 8))
    y = rng.integers(0, 64, 10)
    a, _ = O.token_logprobs(H0, W, y)
    b, _ = O.token_logprobs(HH, W, y)
    sd, s, _ = O.divergence(a[None], a[None], None)
    assert np.all(sd == 0.0) and np.all(s == 0.0)
    sd1, s1, _ = O.divergence(a[None], b[None], None)
    sd2, s2, _ = O.divergence(b[None], a[None], None)
    assert np.array_equal(s1, s2) and np.array_equal(sd1, -sd2)


# ---------------------------------------------------------------- ranking
def _rank_count_select(s, elig, k):
    """Brute force: a candidate's rank is the number of candidates that beat
    it (higher score, or equal score at a lower position)."""
    T = len(s)
    cand = [t for t in range(T) if elig[t]]
    rank = {t: sum(1 for u in cand if (s[u] > s[t]) or (s[u] == s[t] and u < t)) for t in cand}
    chosen = sorted((rank[t], t) for t in cand if rank[t] < k)
    return [t for _, t in chosen]


def test_selection_matches_rank_counting():
    rng = np.random.default_rng(13)
    for trial in range(40):
        R, T = 3, int(rng.integers(1, 40))
        lo = -rng.exponential(2.0, (R, T))
        lh = lo + np.round(rng.normal(0, 1.0, (R, T)), 1)   # rounding makes ties
        mask = (rng.random((R, T)) < 0.7).astype(np.uint8)
        k = int(rng.integers(1, 12))
        idx, sc, cnt = O.select_branch_points(lo, lh, mask, k)
        _, s, el = O.divergence(lo, lh, mask)
        for r in range(R):
            want = _rank_count_select(s[r], el[r], k)
            assert idx[r, :cnt[r]].tolist() == want
            assert np.all(idx[r, cnt[r]:] == -1) and np.all(sc[r, cnt[r]:] == 0)
            assert cnt[r] == min(k, int(el[r].sum()))


def test_selection_all_zero_scores_takes_first_eligible():
    lo = np.full((2, 10), -1.0)
    mask = np.array([[0, 1, 1, 0, 1, 1, 1, 1, 1, 1], [1] * 10], np.uint8)
    idx, sc, cnt = O.select_branch_points(lo, lo.copy(), mask, 3)
    assert idx[0].tolist() == [1, 2, 4] and idx[1].tolist() == [0, 1, 2]
    assert np.all(sc == 0.0)


def test_selection_k_exceeds_candidates_and_nan():
    lo = np.array([[-1.0, -2.0, -3.0, -4.0, -5.0]])
    lh = np.array([[-1.5, np.nan, -1.0, -4.0, -9.0]])
    mask = np.array([[1, 1, 1, 0, 1]], np.uint8)
    idx, sc, cnt = O.select_branch_points(lo, lh, mask, 8)
    assert cnt[0] == 3
    assert idx[0, :3].tolist() == [4, 2, 0]     # scores 4.0, 2.0, 0.5
    assert np.all(idx[0, 3:] == -1)
    assert sc[0, :3].tolist() == [4.0, 2.0, 0.5]


def test_selection_exhaustive_tiny():
    # Every mask and every k on a 5-position root with ties: compare with
    # the rank-counting brute force.
    lo = np.array([[-1.0, -1.0, -2.0, -0.5, -3.0]])
    lh = np.array([[-2.0, 0.0, -1.0, -0.5, -1.0]])   # scores 1, 1, 1, 0, 2
    for bits in itertools.product([0, 1], repeat=5):
        mask = np.array([bits], np.uint8)
        for k in range(1, 7):
            idx, _, cnt = O.select_branch_points(lo, lh, mask, k)
            _, s, el = O.divergence(lo, lh, mask)
            assert idx[0, :cnt[0]].tolist() == _rank_count_select(s[0], el[0], k)


def test_f32_precision_mode_matches_binary32_subtraction():
    rng = np.random.default_rng(14)
    lo = (-rng.exponential(3, (2, 50))).astype(np.float32)
    lh = (lo + rng.normal(0, 1e-3, (2, 50))).astype(np.float32)
    sd, s, _ = O.divergence(lo, lh, None, precision="f32")
    assert sd.dtype == np.float32
    # the exact difference of two binary32 values, rounded once to binary32
    exact = lh.astype(np.float64) - lo.astype(np.float64)
    assert np.array_equal(sd, exact.astype(np.float32))


def test_branch_set_agreement_rule():
    s = np.array([5.0, 4.0, 1.0, 0.5, 0.0])
    e = np.ones(5, bool)
    assert O.branch_set_agrees([0, 1], 2, s, e, 2)[0]
    assert not O.branch_set_agrees([0, 2], 2, s, e, 2)[0]
    t = np.array([5.0, 1.004, 1.0, 0.2])          # k=2 boundary inside the gap
    assert O.branch_set_agrees([0, 2], 2, t, np.ones(4, bool), 2)[0]
    assert not O.branch_set_agrees([0, 3], 2, t, np.ones(4, bool), 2)[0]
    assert not O.branch_set_agrees([0], 1, s, e, 2)[0]


# ---------------------------------------------------------------- entropy
def test_entropy_closed_forms():
    rng = np.random.default_rng(15)
    V = 777
    W = rng.normal(0, 1, (V, 3))
    Hz = O.token_entropy(np.zeros((1, 3)), W)
    assert abs(Hz[0] - math.log(V)) < 1e-12
    W2 = np.eye(20, 20) * 80.0
    h = np.zeros((1, 20)); h[0, 3] = 1.0
    assert O.token_entropy(h, W2)[0] < 1e-25
    # brute force against exact sums
    W3 = rng.normal(0, 1, (30, 4)); h3 = rng.normal(0, 1, (1, 4))
    z = [math.fsum(a * b for a, b in zip(h3[0], w)) for w in W3]
    Z = math.fsum(math.exp(v) for v in z)
    want = -math.fsum((math.exp(v) / Z) * math.log(math.exp(v) / Z) for v in z)
    assert abs(O.token_entropy(h3, W3)[0] - want) < 1e-12
    # two words: the binary entropy of p = sigmoid(z0 - z1)
    W4 = np.array([[1.5, 0.0], [0.0, 1.0]])
    h4 = np.array([[0.8, -0.3]])
    p = 1.0 / (1.0 + math.exp(-(1.5 * 0.8 + 0.3)))
    assert abs(O.token_entropy(h4, W4)[0] - (-p * math.log(p) - (1 - p) * math.log(1 - p))) < 1e-14


# ------------------------------------------------------- top-k over values
def test_select_by_value_matches_rank_counting():
    # position t is in the top-k iff fewer than k eligible positions beat it,
    # where u beats t when v_u > v_t, or v_u == v_t and u < t (the ranking rule
    # of Sec. 3.2 applied to an arbitrary value); negatives, +-0, +-inf, NaN
    rng = np.random.default_rng(77)
    for trial in range(40):
        R, T, k = 3, int(rng.integers(1, 40)), int(rng.integers(1, 12))
        v = rng.choice([-3.0, -1.0, -0.0, 0.0, 0.5, 2.0, np.inf, -np.inf, np.nan], size=(R, T))
        fresh = rng.random((R, T)) < 0.5
        v[fresh] = np.round(rng.normal(size=int(fresh.sum())), 1)   # rounding makes ties
        mask = (rng.random((R, T)) < 0.8).astype(np.uint8)
        idx, score, count = O.select_by_value(v, mask, k)
        for r in range(R):
            elig = [t for t in range(T) if mask[r, t] and np.isfinite(v[r, t])]
            beats = {t: sum(1 for u in elig if v[r, u] > v[r, t] or (v[r, u] == v[r, t] and u < t))
                     for t in elig}
            want = sorted((t for t in elig if beats[t] < k), key=lambda t: beats[t])
            assert count[r] == len(want) == min(k, len(elig))
            assert idx[r, :count[r]].tolist() == want
            assert np.all(idx[r, count[r]:] == -1) and np.all(score[r, count[r]:] == 0.0)
            assert np.array_equal(score[r, :count[r]], v[r, want])


def test_select_by_value_on_abs_difference_is_branch_selection():
    # ranking |log p^H - log p^0| by value must reproduce the Eq. 2 selection
    lo, lh, mask = workloads.make_logp_pair(4, 300, seed=5, nan_rows=2)
    _, s, elig = O.divergence(lo, lh, mask)
    vals = np.where(elig, s, np.nan)
    a = O.select_by_value(vals, None, 9)
    b = O.select_branch_points(lo, lh, mask, 9)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_entropy_is_lse_minus_expected_logit():
    # H = lse - E_p[z]: the identity the fused kernel's third accumulator uses,
    # checked against the definition -sum p log p on random rows
    rng = np.random.default_rng(3)
    W = rng.normal(size=(700, 16))
    h = rng.normal(size=(5, 16)) * 2
    z = h @ W.T
    lse = np.log(np.exp(z - z.max(1, keepdims=True)).sum(1)) + z.max(1)
    p = np.exp(z - lse[:, None])
    assert np.allclose(O.token_entropy(h, W), lse - (p * z).sum(1), atol=1e-11)
    # masked rows are 0; entropy never exceeds log V
    m = np.array([1, 0, 1, 0, 1], np.uint8)
    H = O.token_entropy(h, W, m)
    assert np.all(H[m == 0] == 0.0) and np.all(H <= np.log(700) + 1e-12)


# ------------------------------------------------------------ backward pass
def _loss(H, W, y, g):
    # L = sum_n g_n log p_n(y_n), written with the library-free log-sum-exp
    z = H @ W.T
    out = 0.0
    for n in range(H.shape[0]):
        zn = z[n]
        m = max(zn)
        lse = m + math.log(math.fsum(math.exp(v - m) for v in zn))
        out += g[n] * (zn[y[n]] - lse)
    return out


def test_backward_matches_central_differences():
    # the gradient of L by central differences in every coordinate of H and W
    rng = np.random.default_rng(21)
    N, V, d = 4, 7, 3
    H = rng.normal(size=(N, d))
    W = rng.normal(size=(V, d))
    y = rng.integers(0, V, N)
    g = rng.normal(size=N)
    dH, dW, _, _ = O.token_logprobs_backward(H, W, y, g)
    h = 1e-6
    for arr, grad in ((H, dH), (W, dW)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + h
            lp = _loss(H, W, y, g)
            arr[idx] = old - h
            lm = _loss(H, W, y, g)
            arr[idx] = old
            num[idx] = (lp - lm) / (2 * h)
        assert np.allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_backward_closed_forms_and_invariants():
    rng = np.random.default_rng(22)
    N, V, d = 6, 9, 4
    H = rng.normal(size=(N, d))
    W = rng.normal(size=(V, d))
    y = rng.integers(0, V, N)
    g = rng.normal(size=N)
    dH, dW, mH, mW = O.token_logprobs_backward(H, W, y, g)
    # probabilities sum to one, so the vocabulary rows of dW sum to zero
    assert np.allclose(dW.sum(axis=0), 0.0, atol=1e-12)
    # identical W rows: uniform softmax, dH_n = g_n (W_y - mean W) = 0
    Wc = np.tile(rng.normal(size=(1, d)), (V, 1))
    dHc, _, _, _ = O.token_logprobs_backward(H, Wc, y, g)
    assert np.allclose(dHc, 0.0, atol=1e-12)
    # two words: d log sigmoid(z0 - z1) / d z0 = 1 - sigmoid(z0 - z1)
    W2 = np.array([[1.0, 0.0], [0.0, 1.0]])
    h2 = np.array([[0.7, -0.2]])
    sig = 1 / (1 + math.exp(-(0.7 + 0.2)))
    dH2, _, _, _ = O.token_logprobs_backward(h2, W2, np.array([0]), np.array([1.0]))
    assert np.allclose(dH2[0], [1 - sig, -(1 - sig)], atol=1e-15)
    # masked rows: zero dH, no contribution to dW; magnitudes dominate results
    mask = np.array([1, 0, 1, 1, 0, 1], np.uint8)
    dHm, dWm, _, _ = O.token_logprobs_backward(H, W, y, g, mask)
    assert np.all(dHm[mask == 0] == 0)
    keep = mask != 0
    _, dWk, _, _ = O.token_logprobs_backward(H[keep], W, y[keep], g[keep])
    assert np.allclose(dWm, dWk, atol=1e-13)
    assert np.all(np.abs(dH) <= mH + 1e-15) and np.all(np.abs(dW) <= mW + 1e-15)
    # an out-of-range token has no indicator term
    y_bad = y.copy(); y_bad[0] = V
    dHb, _, _, _ = O.token_logprobs_backward(H[:1], W, y_bad[:1], g[:1])
    z = H[0] @ W.T
    p = np.exp(z - z.max()); p /= p.sum()
    assert np.allclose(dHb[0], -g[0] * (p @ W), atol=1e-13)


# ------------------------------------------------------- group construction
def _greedy_by_repeated_argmax(sc, cand, k, min_gap):
    # independent formulation of the refill rule: each step takes the best
    # remaining candidate compatible with everything taken so far
    kept = []
    while len(kept) < k:
        ok = [t for t in cand if t not in kept and all(abs(t - u) >= min_gap for u in kept)]
        if not ok:
            break
        kept.append(max(ok, key=lambda t: (sc[t], -t)))
    return kept


def test_constrained_selection_fixture():
    T = 60
    s = np.zeros((1, T))
    for t, v in ((10, 0.9), (12, 0.8), (30, 0.7), (50, 0.6), (33, 0.65)):
        s[0, t] = v
    z = np.zeros_like(s)
    # drop mode: 12 is too close to 10 and is not replaced
    idx, sc, cnt = O.select_constrained(z, s, None, 2, min_gap=5)
    assert cnt.tolist() == [1] and idx[0].tolist() == [10, -1] and sc[0, 0] == 0.9
    # refill: the walk continues to 30
    idx, _, cnt = O.select_constrained(z, s, None, 2, min_gap=5, refill=True)
    assert cnt.tolist() == [2] and idx[0].tolist() == [10, 30]
    # index range [11, 40] removes 10 and 50; 33 is within 5 of 30; the third
    # point is the lowest zero-score position at least 5 from 12 and 30
    idx, _, cnt = O.select_constrained(z, s, None, 3, lo=[11], hi=[40], min_gap=5, refill=True)
    assert idx[0].tolist() == [12, 30, 17] and cnt.tolist() == [3]
    # value mode ranks the values themselves
    idx, _, _ = O.select_constrained(s, None, None, 2)
    assert idx[0].tolist() == [10, 12]


def test_constrained_selection_reduces_and_matches_repeated_argmax():
    lo_, hi_, mask = workloads.make_logp_pair(5, 200, seed=41, nan_rows=1)
    a = O.select_constrained(lo_, hi_, mask, 7)
    b = O.select_branch_points(lo_, hi_, mask, 7)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    _, s, elig = O.divergence(lo_, hi_, mask)
    rng = np.random.default_rng(42)
    for trial in range(30):
        k = int(rng.integers(1, 6))
        gap = int(rng.integers(2, 40))
        L = rng.integers(0, 100, 5)
        H = L + rng.integers(0, 120, 5)
        idx, _, cnt = O.select_constrained(lo_, hi_, mask, k, lo=L, hi=H, min_gap=gap, refill=True)
        for r in range(5):
            cand = [t for t in range(200) if elig[r, t] and L[r] <= t <= H[r]]
            want = _greedy_by_repeated_argmax(s[r], cand, k, gap)
            assert idx[r, :cnt[r]].tolist() == want
        # drop mode keeps a subset of the unconstrained top k, in rank order
        idx_d, _, cnt_d = O.select_constrained(lo_, hi_, mask, k, lo=L, hi=H, min_gap=gap)
        top, _, _ = O.select_constrained(lo_, hi_, mask, k, lo=L, hi=H)
        for r in range(5):
            kept = idx_d[r, :cnt_d[r]].tolist()
            order = [t for t in top[r].tolist() if t in kept]
            assert kept == order
            for t in top[r].tolist():
                if t >= 0 and t not in kept:
                    assert any(abs(t - u) < gap for u in kept)


def test_allocation_fixtures():
    idx = np.array([[17, 40], [5, -1], [-1, -1]], np.int32)
    pos, rank = O.allocate_continuations(idx, np.array([2, 1, 0]), (3, 4), fallback=0)
    assert pos[0].tolist() == [17] * 3 + [40] * 4 and rank[0].tolist() == [0] * 3 + [1] * 4
    assert pos[1].tolist() == [5] * 7 and rank[1].tolist() == [0] * 7
    assert pos[2].tolist() == [0] * 7 and rank[2].tolist() == [-1] * 7
    # 2 x 1 configuration (Table 5): all seven at the single point
    pos, _ = O.allocate_continuations(np.array([[9]], np.int32), np.array([1]), (7,))
    assert pos[0].tolist() == [9] * 7
    with pytest.raises(ValueError):   # one slot count per rank, as the C ABI requires
        O.allocate_continuations(np.array([[9]], np.int32), np.array([1]), (3, 4))


def test_group_advantages_closed_forms():
    R = np.array([[1.0, 0.0, 0.0, 1.0], [0.3, 0.3, 0.3, 0.3]])
    A = O.group_advantages(R)
    assert np.allclose(A[0], [0.5, -0.5, -0.5, 0.5]) and np.all(A[1] == 0)
    rng = np.random.default_rng(3)
    X = rng.normal(size=(5, 16))
    assert np.allclose(O.group_advantages(X).sum(axis=1), 0.0, atol=1e-14)
    assert np.allclose(O.group_advantages(X + 7.0), O.group_advantages(X), atol=1e-13)


def test_policy_loss_grad_by_finite_differences_and_clip_regions():
    rng = np.random.default_rng(8)
    n = 400
    adv = rng.normal(size=6)
    traj = rng.integers(0, 6, n)
    lo_ = rng.normal(size=n) * 0.1 - 2
    ln = lo_ + rng.normal(size=n) * 0.4
    g, l = O.policy_loss_grad(adv, traj, ln, lo_, scale=0.01)
    h = 1e-7
    for i in range(n):
        r = math.exp(ln[i] - lo_[i])
        if min(abs(r - 0.8), abs(r - 1.28)) < 1e-3:
            continue   # not differentiable at the clip boundaries
        lp = ln.copy(); lp[i] += h
        lm = ln.copy(); lm[i] -= h
        num = (O.policy_loss_grad(adv, traj[i:i+1], lp[i:i+1], lo_[i:i+1], scale=0.01)[1][0] -
               O.policy_loss_grad(adv, traj[i:i+1], lm[i:i+1], lo_[i:i+1], scale=0.01)[1][0]) / (2 * h)
        assert abs(num - g[i]) <= 1e-6 * max(1.0, abs(g[i]))
        # the clipped side carries no gradient
        if adv[traj[i]] > 0 and r > 1.28:
            assert g[i] == 0.0
        if adv[traj[i]] < 0 and r < 0.8:
            assert g[i] == 0.0
    # on-policy (r = 1): g = -scale * A
    g1, _ = O.policy_loss_grad(adv, traj, lo_, lo_, scale=0.5)
    assert np.allclose(g1, -0.5 * adv[traj])
    # a continuation's reused prefix and masked tokens carry nothing
    pos = np.arange(n) % 50
    start = np.array([0, 10, 0, 30, 0, 0])
    mask = (rng.random(n) < 0.8).astype(np.uint8)
    g2, _ = O.policy_loss_grad(adv, traj, ln, lo_, mask, pos, start)
    off = (mask == 0) | (pos < start[traj])
    assert np.all(g2[off] == 0.0)


def test_non_finite_hidden_row_gives_nan_for_that_row_only():
    rng = np.random.default_rng(16)
    W = rng.normal(size=(50, 6))
    H = rng.normal(size=(4, 6))
    y = rng.integers(0, 50, 4)
    clean, _ = O.token_logprobs(H, W, y)
    H[1, 2] = np.nan
    H[3, 0] = np.inf
    with np.errstate(invalid="ignore"):
        lp, lse = O.token_logprobs(H, W, y)
    assert np.isnan(lp[1]) and np.isnan(lp[3]) and np.isnan(lse[1])
    assert np.array_equal(lp[[0, 2]], clean[[0, 2]])


def test_token_level_aggregation_counts_trained_tokens():
    # Hand-worked (Sec. 4.1 "Training": token-level aggregation; Sec. 3.3: a
    # continuation trains only its suffix).  Two trajectories, the second a
    # continuation branched at position 2; token 1 is outside the loss mask,
    # tokens 2 and 3 are the continuation's reused prefix, token 5 names a
    # trajectory that does not exist: tokens 0 and 4 are trained, so the
    # token-level mean divides by 2.
    adv = np.array([0.5, -1.0])
    traj = np.array([0, 0, 1, 1, 1, 5])
    pos = np.array([0, 1, 0, 1, 2, 0])
    start = np.array([0, 2])
    mask = np.array([1, 0, 1, 1, 1, 1], np.uint8)
    lo_ = np.full(6, -1.0)
    assert O.trained_tokens(traj, 2, mask, pos, start) == 2
    g, l = O.policy_loss_grad(adv, traj, lo_, lo_, mask, pos, start, scale=None)
    # on policy (r = 1): g = -A / 2 on the trained tokens, 0 elsewhere
    assert g.tolist() == [-0.25, 0.0, 0.0, 0.0, 0.5, 0.0]
    assert l.tolist() == [-0.25, 0.0, 0.0, 0.0, 0.5, 0.0]
    # nothing trained: the divisor is 1, every factor 0
    assert O.trained_tokens(traj, 2, np.zeros(6, np.uint8), pos, start) == 0
    g0, _ = O.policy_loss_grad(adv, traj, lo_, lo_, np.zeros(6, np.uint8), pos, start, scale=None)
    assert np.all(g0 == 0.0)


def test_trained_token_count_per_trajectory():
    # Counted trajectory by trajectory (positions at or past the trajectory's
    # start among its masked-in tokens) instead of token by token; and the
    # scale=None factors are the scale=1 factors divided by that count.
    rng = np.random.default_rng(21)
    n, n_traj = 3000, 40
    traj = rng.integers(-3, n_traj + 3, n)
    pos = rng.integers(0, 200, n)
    start = rng.integers(0, 150, n_traj)
    mask = (rng.random(n) < 0.85).astype(np.uint8)
    want = 0
    for j in range(n_traj):
        mine = (traj == j) & (mask != 0)
        want += int(np.count_nonzero(pos[mine] >= start[j]))
    assert O.trained_tokens(traj, n_traj, mask, pos, start) == want
    assert O.trained_tokens(traj, n_traj, mask) == int(np.count_nonzero((traj >= 0) & (traj < n_traj) & (mask != 0)))
    adv = rng.normal(size=n_traj)
    lo_ = rng.normal(size=n) * 0.1 - 2
    ln = lo_ + rng.normal(size=n) * 0.3
    g1, l1 = O.policy_loss_grad(adv, traj, ln, lo_, mask, pos, start, scale=1.0)
    gm, lm = O.policy_loss_grad(adv, traj, ln, lo_, mask, pos, start, scale=None)
    assert np.allclose(gm, g1 / want, rtol=1e-15, atol=0) and np.allclose(lm, l1 / want, rtol=1e-15, atol=0)
