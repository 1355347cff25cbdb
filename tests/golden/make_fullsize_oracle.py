"""Write the float64 oracle's values for every scored row of the full-size
workloads: tests/golden/fullsize_oracle_<name>.npz.

Only the oracle (oracle/) and the seeded input generator (workloads/) are
used; nothing here touches the GPU library.  For each workload the file holds

* logp     float64 [n_scored]: log p of every scored row, in the library's row
           order (context, root, position) restricted to mask != 0 (Eq. 1);
* entropy  float64 [n_scored of the original context] (c2 only): the
           next-token entropy of every scored original-context row (the
           Entropy localization baseline, Sec. 4.1);
* digest   the SHA-256 of the generated inputs (workloads.input_digest), so a
           test can refuse values computed from other inputs.

The GPU parity tests compare the library's outputs element by element with
these values and re-compute a seeded sample of rows with the oracle on the
spot.  Run from the repository root (about an hour on 8 cores for all four):

    python tests/golden/make_fullsize_oracle.py c2 c3 c4 c5
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402
from oracle import hdl_oracle as O  # noqa: E402

BLOCK = 4096


def decode(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return O.bf16_bits_to_f64(t.contiguous().view(torch.int16).numpy().view(np.uint16))
    return t.double().numpy()


def path_for(name: str) -> str:
    return os.path.join(ROOT, "tests", "golden", f"fullsize_oracle_{name}.npz")


def make(name: str) -> None:
    t0 = time.time()
    w = workloads.make_workload(name)
    digest = workloads.input_digest(w)
    c = w.cfg
    Wd = decode(w.W)
    hidden = w.rows_hidden()
    tokens = w.rows_tokens().numpy()
    rows = np.nonzero(w.rows_mask().numpy())[0]
    logp = np.empty(len(rows), np.float64)
    for b0 in range(0, len(rows), BLOCK):
        r = rows[b0:b0 + BLOCK]
        logp[b0:b0 + len(r)], _ = O.token_logprobs(decode(hidden[torch.as_tensor(r)]), Wd, tokens[r])
        print(f"{name}: log p {b0 + len(r)}/{len(rows)} rows, {time.time() - t0:.0f} s", flush=True)
    out = {"logp": logp, "digest": np.array(digest)}
    if name == "c2":
        r0 = rows[rows < c.R * c.T]
        ent = np.empty(len(r0), np.float64)
        for b0 in range(0, len(r0), BLOCK):
            r = r0[b0:b0 + BLOCK]
            ent[b0:b0 + len(r)] = O.token_entropy(decode(hidden[torch.as_tensor(r)]), Wd)
            print(f"{name}: entropy {b0 + len(r)}/{len(r0)} rows, {time.time() - t0:.0f} s", flush=True)
        out["entropy"] = ent
    np.savez(path_for(name), **out)
    print(f"{name}: wrote {path_for(name)} in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    for n in sys.argv[1:] or ["c2", "c3", "c4", "c5"]:
        make(n)
