"""Seeded synthetic inputs for the hindsight re-scoring path.

This module only *makes inputs*: final hidden states for the original and the
hindsight context, the vocabulary projection, sampled tokens, the eligibility
mask and the planted branch positions.  It holds none of the method's
arithmetic (no log-softmax, no divergence, no ranking), so that both the HIP
path and the float64 oracle can be fed from it without sharing code.

Why these shapes: the paper re-scores sampled roots under two contexts that
differ only by the hindsight context (Sec. 3.1, Eq. 1) and ranks positions by
the absolute log-likelihood change (Sec. 3.2, Eq. 2).  It trains on responses
of up to 32,768 tokens and agent trajectories whose environment observations
are part of the sequence (Sec. 4.1, "Training").  The trained trunks and the
datasets are not available, so hidden states are drawn synthetically:

* W ~ N(0, 0.02^2), shape [V, d] (row-major, contiguous in d).
* original-context hidden rows h0 ~ N(0, 1) (Student-t, nu=3, for the
  heavy-tailed configuration), each row RMS-normalised.
* hindsight hidden rows hH = h0 + N(0, 0.01^2), plus, at planted positions, a
  shift sigma*alpha*w_y/||w_y||^2 that moves the target logit by sigma*alpha.
* tokens uniform in [0, V).
* mask: 1 for policy-generated tokens, 0 for excluded positions (a prefix, or
  seeded tool-observation spans).

Random streams are keyed by (seed, stream, chunk), so every chunk is
reproducible on its own and the result does not depend on thread counts.
Generation runs on the CPU with torch's generator; only operations whose
results are the same on every x86 host are used (square roots are taken with
NumPy: torch's CPU sqrt differs in the last bit between vendors); bf16 values
are produced by round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np
import torch

GENERATOR_VERSION = 2

# Stream identifiers (fixed order; never renumber).
_S_W, _S_H0, _S_NOISE, _S_TOK, _S_PLANT, _S_ALPHA, _S_MASK, _S_DUP = range(8)


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    R: int            # roots
    T: int            # response positions per root
    d: int            # hidden size
    V: int            # vocabulary size
    dtype: str        # "f32" or "bf16"
    seed: int
    k: int            # branch points per root
    mask: str         # "all" | "prefix" | "spans"
    mask_prefix: int = 0
    n_planted: int = 0
    alpha: str = "fixed"          # "fixed" | "loguniform" | "band"
    alpha_value: float = 3.0
    alpha_lo: float = 0.0
    alpha_hi: float = 0.0
    hidden_dist: str = "normal"   # "normal" | "student_t3"
    n_band: int = 0               # near-tie band size (heavy-tailed config)
    n_dup_pairs: int = 0          # bitwise-duplicate row pairs inside the band

    @property
    def n_rows(self) -> int:
        return 2 * self.R * self.T


CONFIGS: Dict[str, Config] = {
    "tiny": Config("tiny", R=1, T=256, d=256, V=4096, dtype="f32", seed=1001,
                   k=4, mask="all", n_planted=4, alpha="fixed", alpha_value=3.0),
    "c2": Config("c2", R=8, T=4096, d=2048, V=151936, dtype="bf16", seed=1002,
                 k=8, mask="prefix", mask_prefix=32, n_planted=16,
                 alpha="fixed", alpha_value=3.0),
    "c3": Config("c3", R=4, T=16384, d=4096, V=151936, dtype="bf16", seed=1003,
                 k=16, mask="all", n_planted=32, alpha="loguniform",
                 alpha_lo=0.05, alpha_hi=5.0),
    "c4": Config("c4", R=32, T=8192, d=4096, V=151936, dtype="bf16", seed=1004,
                 k=8, mask="spans", n_planted=16, alpha="fixed", alpha_value=3.0),
    "c5": Config("c5", R=2, T=32768, d=5120, V=152064, dtype="bf16", seed=1005,
                 k=32, mask="all", n_planted=16, alpha="loguniform",
                 alpha_lo=2.0, alpha_hi=5.0, hidden_dist="student_t3",
                 n_band=32, n_dup_pairs=4),
}

# Human-readable workload names (used in bench output and docs).
DESCRIPTIONS = {
    "tiny": "1 root x 2 contexts, T=256, d=256, V=4096, fp32",
    "c2": "8 roots x 2 contexts, T=4096, d=2048, V=151936, bf16",
    "c3": "4 roots x 2 contexts, T=16384, d=4096, V=151936, bf16",
    "c4": "32 roots x 2 contexts, T=8192, d=4096, V=151936, bf16, agent spans",
    "c5": "2 roots x 2 contexts, T=32768, d=5120, V=152064, bf16, heavy-tailed",
}


def get_config(name: str, **overrides) -> Config:
    """Named configuration, optionally with shape overrides for reduced runs."""
    cfg = CONFIGS[name]
    if overrides:
        cfg = dataclasses.replace(cfg, **overrides)
    return cfg


@dataclasses.dataclass
class Workload:
    cfg: Config
    W: torch.Tensor          # [V, d]  bf16 or f32 (CPU)
    hidden: torch.Tensor     # [2, R, T, d]; [0] original, [1] hindsight
    tokens: torch.Tensor     # [R, T] int32
    mask: torch.Tensor       # [R, T] uint8
    planted: List[dict]      # per root: {"pos", "alpha", "sign"} (numpy)
    band: List[np.ndarray]   # per root: near-tie band positions (may be empty)
    dup_pairs: List[list]    # per root: list of (src, dst) duplicated rows

    # Flattened views in the row order the library expects:
    # row n = c*R*T + r*T + t, c = 0 original, c = 1 hindsight.
    def rows_hidden(self) -> torch.Tensor:
        c = self.cfg
        return self.hidden.reshape(2 * c.R * c.T, c.d)

    def rows_tokens(self) -> torch.Tensor:
        return torch.cat([self.tokens.reshape(-1), self.tokens.reshape(-1)])

    def rows_mask(self) -> torch.Tensor:
        return torch.cat([self.mask.reshape(-1), self.mask.reshape(-1)])

    def n_eligible(self) -> int:
        return int(self.mask.sum())


def _seed(seed: int, stream: int, chunk: int = 0) -> int:
    ss = np.random.SeedSequence([seed, GENERATOR_VERSION, stream, chunk])
    return int(ss.generate_state(1, np.uint64)[0] & ((1 << 63) - 1))


def _gen(seed: int, stream: int, chunk: int = 0) -> torch.Generator:
    return torch.Generator().manual_seed(_seed(seed, stream, chunk))


def _np_rng(seed: int, stream: int, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, GENERATOR_VERSION, stream, chunk]))


def _to_dtype(x: torch.Tensor, dtype: str) -> torch.Tensor:
    # torch's float32 -> bfloat16 conversion rounds to nearest, ties to even.
    return x.to(torch.bfloat16) if dtype == "bf16" else x.contiguous()


def _make_W(cfg: Config) -> torch.Tensor:
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    W = torch.empty(cfg.V, cfg.d, dtype=tdt)
    rows = 8192
    for ci, v0 in enumerate(range(0, cfg.V, rows)):
        v1 = min(cfg.V, v0 + rows)
        blk = torch.empty(v1 - v0, cfg.d, dtype=torch.float32)
        blk.normal_(0.0, 0.02, generator=_gen(cfg.seed, _S_W, ci))
        W[v0:v1] = _to_dtype(blk, cfg.dtype)
    return W


def _make_mask(cfg: Config, r: int) -> np.ndarray:
    m = np.ones(cfg.T, dtype=np.uint8)
    if cfg.mask == "prefix":
        m[: min(cfg.mask_prefix, cfg.T)] = 0
    elif cfg.mask == "spans":
        # 5-20 tool-observation spans of 64-512 tokens each, uniform counts,
        # lengths and starts; overlaps allowed.
        g = _np_rng(cfg.seed, _S_MASK, r)
        n_spans = int(g.integers(5, 21))
        for _ in range(n_spans):
            ln = int(min(g.integers(64, 513), cfg.T))
            st = int(g.integers(0, cfg.T - ln + 1))
            m[st:st + ln] = 0
    elif cfg.mask != "all":
        raise ValueError(cfg.mask)
    return m


def _alphas(cfg: Config, g: np.random.Generator, n: int) -> np.ndarray:
    if cfg.alpha == "fixed":
        return np.full(n, cfg.alpha_value)
    if cfg.alpha == "loguniform":
        return np.exp(g.uniform(math.log(cfg.alpha_lo), math.log(cfg.alpha_hi), n))
    raise ValueError(cfg.alpha)


def _hidden0_rows(cfg: Config, r: int, t0: int, t1: int, chunk: int) -> torch.Tensor:
    n = t1 - t0
    g = _gen(cfg.seed, _S_H0, r * 100003 + chunk)
    if cfg.hidden_dist == "normal":
        x = torch.empty(n, cfg.d, dtype=torch.float32).normal_(generator=g)
    elif cfg.hidden_dist == "student_t3":
        # Student-t with 3 degrees of freedom: Z / sqrt(chi2_3 / 3), with
        # chi2_3 the sum of three squared standard normals.
        z = torch.empty(n, cfg.d, dtype=torch.float32).normal_(generator=g)
        c = torch.empty(3, n, cfg.d, dtype=torch.float32).normal_(generator=g)
        chi2 = (c * c).sum(0)
        x = z / _sqrt(chi2 / 3.0)
    else:
        raise ValueError(cfg.hidden_dist)
    rms = _sqrt((x * x).mean(dim=1, keepdim=True))
    return x / rms


def _sqrt(t: torch.Tensor) -> torch.Tensor:
    """Correctly rounded square root (NumPy's, the hardware instruction).
    torch's CPU sqrt gives different last bits on different x86 vendors, which
    would make the generated inputs depend on the host."""
    return torch.from_numpy(np.sqrt(t.contiguous().numpy()))


def make_workload(name: str, **overrides) -> Workload:
    """Build the seeded synthetic workload `name` (optionally reshaped)."""
    cfg = get_config(name, **overrides)
    R, T, d, V = cfg.R, cfg.T, cfg.d, cfg.V
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    W = _make_W(cfg)
    Wf = W.float()

    tokens = torch.empty(R, T, dtype=torch.int32)
    mask = torch.empty(R, T, dtype=torch.uint8)
    planted, bands, dups = [], [], []
    for r in range(R):
        gt = _gen(cfg.seed, _S_TOK, r)
        tokens[r] = torch.randint(0, V, (T,), generator=gt, dtype=torch.int64).to(torch.int32)
        m = _make_mask(cfg, r)
        mask[r] = torch.from_numpy(m)
        elig = np.nonzero(m)[0]
        gp = _np_rng(cfg.seed, _S_PLANT, r)
        n_pl = min(cfg.n_planted + cfg.n_band, len(elig))
        pos = np.sort(gp.choice(elig, size=n_pl, replace=False)) if n_pl else np.zeros(0, np.int64)
        ga = _np_rng(cfg.seed, _S_ALPHA, r)
        # The first n_planted (in a seeded shuffled order) get the configured
        # alphas; the remaining n_band form a near-tie band.
        order = ga.permutation(n_pl)
        main = np.sort(pos[order[: min(cfg.n_planted, n_pl)]])
        band = np.sort(pos[order[min(cfg.n_planted, n_pl):]])
        alpha = _alphas(cfg, ga, len(main))
        sign = ga.choice(np.array([-1.0, 1.0]), size=len(main))
        band_alpha = 1.0 + ga.uniform(0.0, 5e-3, len(band))
        band_sign = ga.choice(np.array([-1.0, 1.0]), size=len(band))
        allpos = np.concatenate([main, band])
        allalpha = np.concatenate([alpha, band_alpha])
        allsign = np.concatenate([sign, band_sign])
        srt = np.argsort(allpos, kind="stable")
        planted.append({"pos": allpos[srt].astype(np.int64),
                        "alpha": allalpha[srt], "sign": allsign[srt],
                        "main": main.astype(np.int64)})
        bands.append(band.astype(np.int64))
        gd = _np_rng(cfg.seed, _S_DUP, r)
        pairs = []
        if cfg.n_dup_pairs and len(band) >= 2 * cfg.n_dup_pairs:
            sel = gd.choice(len(band), size=2 * cfg.n_dup_pairs, replace=False)
            for i in range(cfg.n_dup_pairs):
                pairs.append((int(band[sel[2 * i]]), int(band[sel[2 * i + 1]])))
        dups.append(pairs)

    hidden = torch.empty(2, R, T, d, dtype=tdt)
    chunk_rows = max(1, (1 << 22) // d)
    for r in range(R):
        pl = planted[r]
        for ci, t0 in enumerate(range(0, T, chunk_rows)):
            t1 = min(T, t0 + chunk_rows)
            h0 = _to_dtype(_hidden0_rows(cfg, r, t0, t1, ci), cfg.dtype)
            hidden[0, r, t0:t1] = h0
            gn = _gen(cfg.seed, _S_NOISE, r * 100003 + ci)
            noise = torch.empty(t1 - t0, d, dtype=torch.float32).normal_(0.0, 0.01, generator=gn)
            hH = h0.float() + noise
            sel = (pl["pos"] >= t0) & (pl["pos"] < t1)
            for t, a, s in zip(pl["pos"][sel], pl["alpha"][sel], pl["sign"][sel]):
                w = Wf[int(tokens[r, t])]
                hH[t - t0] += (float(s) * float(a) / float((w.double() * w.double()).sum())) * w
            hidden[1, r, t0:t1] = _to_dtype(hH, cfg.dtype)
        for src, dst in dups[r]:
            hidden[:, r, dst] = hidden[:, r, src]
            tokens[r, dst] = tokens[r, src]
    return Workload(cfg, W, hidden, tokens, mask, planted, bands, dups)


def make_logp_pair(R: int, T: int, seed: int, mask_kind: str = "spans",
                   n_ties: int = 8, nan_rows: int = 0):
    """Synthetic fp32 log-probability pairs [R, T] for the selection step alone.

    Values are drawn like teacher-forced log-probabilities (negative, a few
    nats), with exact duplicates planted so that equal scores occur, and
    optionally NaN entries (rows whose token was out of range).
    """
    g = _np_rng(seed, 99, 0)
    lo = (-g.exponential(3.0, (R, T)) - 1e-3).astype(np.float32)
    lh = (lo + g.normal(0.0, 0.5, (R, T))).astype(np.float32)
    lh = np.minimum(lh, 0.0).astype(np.float32)
    mask = np.ones((R, T), np.uint8)
    for r in range(R):
        if mask_kind == "spans" and T > 8:
            for _ in range(int(g.integers(1, 6))):
                ln = int(g.integers(1, max(2, T // 8)))
                st = int(g.integers(0, T - ln + 1))
                mask[r, st:st + ln] = 0
        # exact ties: copy (orig, hind) pairs onto other positions
        for _ in range(min(n_ties, T // 2)):
            a, b = g.integers(0, T, 2)
            lo[r, b] = lo[r, a]
            lh[r, b] = lh[r, a]
        for _ in range(nan_rows):
            lh[r, int(g.integers(0, T))] = np.float32("nan")
    return lo, lh, mask


def input_digest(w: Workload) -> str:
    """SHA-256 over a workload's inputs (W, both contexts' hidden rows,
    tokens, mask), so that stored expected values can be tied to the exact
    inputs they were computed from."""
    import hashlib
    h = hashlib.sha256()
    h.update(f"{w.cfg.name} v{GENERATOR_VERSION} {tuple(w.hidden.shape)} {w.cfg.V} {w.cfg.dtype}".encode())
    for t in (w.W, w.hidden, w.tokens, w.mask):
        flat = t.contiguous().view(-1)
        step = 1 << 26   # elements per update (bounded temporary memory)
        for i in range(0, flat.numel(), step):
            h.update(flat[i:i + step].view(torch.uint8).numpy().tobytes() if t.dtype == torch.bfloat16
                     else flat[i:i + step].numpy().tobytes())
    return h.hexdigest()
