#!/usr/bin/env python
"""Throughput of the hindsight re-scoring hot path on one MI355X.

One step = the whole path over one batch of synthetic inputs already resident
in HBM: both contexts' teacher-forced log-probabilities of every eligible
token through the fused lm-head kernel (hdl_token_logprobs), then the
divergence score and per-root top-k (hdl_select_branch_points).

Default workload (the largest configuration that fits one GPU): the agent
multi-turn batch, 32 roots x 2 contexts, T=8192, d=4096, V=151936, bf16, with
seeded tool-observation spans masked out of every root (about 64 % of the
524,288 rows are scored), k=8.  --workload c2 | c3 | c5 | tiny selects the
other configurations.

Prints one JSON line:  value = scored tokens/s (both contexts), plus the
fused kernel's roofline (achieved TFLOP/s of algorithmic 2*d*V flops per
scored token over its HIP-event-timed duration, against the 2.5 PFLOP/s
dense bf16 MFMA peak; HBM traffic from the committed rocprofv3 counters;
for reference, this GPU's measured MFMA ceilings and the vendor GEMM on the
same contraction) and the float64 oracle timed on a bounded sample on the
host cores.

Other passes: --selector entropy (the Entropy baseline's pass over the
original context), --backward (gradients of a token-level loss through the
lm-head), --group (group construction at the paper's batch).  --gpus N with
N > 1 is refused: the path runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # MI355X dense MFMA (fp32: matrix fp32 peak)
METRIC = "scored tokens/sec (both contexts) + MFMA util of fused lm-head logprob kernel"
# The Entropy localization baseline (Sec. 4.1) scores the original context only.
METRIC_ENTROPY = "scored tokens/sec (original context) of fused lm-head entropy + top-k (Entropy baseline)"
# Training side: gradients of the token-level policy loss (Sec. 3.3) through the lm-head.
METRIC_BACKWARD = "trained tokens/sec of the lm-head backward (dL/dh, dL/dW) + MFMA util"
METRIC_GROUP = "trained tokens/sec of group construction (constrained selection, 3+4 allocation, advantages, policy-loss factors)"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Sources the fused kernel and its launch (work-item order, chunking) come from.
KERNEL_SOURCES = ("lmhead_logprob.hip", "tile_common.h", "hdl_internal.h", "plan.h")


def kernel_source_sha() -> str:
    """SHA-256 of the fused kernel's sources with comments and blank lines
    removed, so that a comment edit does not invalidate counters taken on
    the same code."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_36864_amd", "csrc", name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("\n".join(line.rstrip() for line in text.splitlines() if line.strip()).encode())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per launch of the fused kernel, from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, if it was taken on the current kernel
    sources (kernel_source_sha); otherwise None."""
    path = os.path.join(ROOT, "profiles", f"lmhead_logprob_{workload}_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha():
        return None
    return rec.get("hbm_bytes_per_launch")


def library_gemm_tflops(h, W, rows: int = 16384, reps: int = 3):
    """Reference point, not part of the path: the vendor library's plain bf16
    GEMM (torch.matmul -> hipBLASLt) on the same contraction, logits = h W^T
    for the scored rows, written as bf16 in row chunks into one reused
    buffer.  The fused kernel does this contraction plus the online
    log-sum-exp and never writes the logits."""
    import torch
    n = h.shape[0]
    out = torch.empty(min(rows, n), W.shape[0], dtype=torch.bfloat16, device=h.device)

    def run():
        for r0 in range(0, n, rows):
            r1 = min(n, r0 + rows)
            torch.matmul(h[r0:r1], W.t(), out=out[: r1 - r0])

    run()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del out
    return 2.0 * n * h.shape[1] * W.shape[0] / (ms / 1e3) / 1e12


def mfma_ceiling():
    """Run the built MFMA ceiling microbenchmark (paper_2609_36864_amd/mfma_ceiling)
    in a child process; returns its JSON record or None if it is not built."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2609_36864_amd", "mfma_ceiling")
    if not os.path.exists(exe):
        return None
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    if r.returncode != 0:
        log(f"mfma_ceiling failed: {r.stderr.strip()}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def host_cores():
    """(os.cpu_count(), threads of the BLAS pool the float64 oracle's matrix
    products run on): the oracle's exponentials and sums run on one thread,
    its products on the BLAS pool."""
    n = os.cpu_count() or 1
    try:
        from threadpoolctl import threadpool_info
        blas = max([int(i.get("num_threads", 1)) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover - informational only
        blas = n
    return n, blas


def cpu_baseline(w, budget_s: float = 15.0, max_rows: int = 32768, entropy: bool = False):
    """Time the float64 oracle on a seeded sample of eligible rows (both
    contexts; the original context only for the entropy selector) on the host
    cores; return oracle scored tokens/s."""
    import numpy as np
    import torch
    from oracle import hdl_oracle as O
    cores, blas_threads = host_cores()
    c = w.cfg
    if c.dtype == "bf16":
        Wd = O.bf16_bits_to_f64(w.W.view(torch.int16).numpy().view(np.uint16))
    else:
        Wd = w.W.double().numpy()
    hidden = w.rows_hidden()
    tokens = w.rows_tokens().numpy()
    elig = np.nonzero(w.rows_mask().numpy())[0]
    if entropy:
        elig = elig[elig < c.R * c.T]
    rng = np.random.default_rng(12345)
    sample = rng.permutation(elig)[:max_rows]
    done, t_total, blk = 0, 0.0, 64
    while done < len(sample) and t_total < budget_s:
        rows = np.sort(sample[done:done + blk])
        if c.dtype == "bf16":
            H = O.bf16_bits_to_f64(hidden[torch.as_tensor(rows)].view(torch.int16).numpy().view(np.uint16))
        else:
            H = hidden[torch.as_tensor(rows)].double().numpy()
        t0 = time.perf_counter()
        if entropy:
            O.token_entropy(H, Wd)
        else:
            O.token_logprobs(H, Wd, tokens[rows])
        t_total += time.perf_counter() - t0
        done += len(rows)
    return {"value": done / t_total, "unit": "scored tokens/s", "cores": blas_threads, "kind": "oracle",
            "host_cpus": cores, "blas_threads": blas_threads,
            "sample": f"{done} eligible rows drawn from "
                      f"{'the original context' if entropy else 'both contexts'} of this workload "
                      f"(float64 lm-head {'entropy' if entropy else 'log-softmax'}, {t_total:.1f} s)"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c4",
                    help="tiny | c2 | c3 | c4 | c5 (default c4, the largest single-GPU configuration)")
    ap.add_argument("--selector", default="hdl", choices=["hdl", "entropy"],
                    help="hdl: both contexts, |delta log p| top-k (default); entropy: the Entropy "
                         "baseline, next-token entropy of the original context and its top-k")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward pass (gradients with respect to the hidden states and the "
                         "lm-head weight) on the original-context rows instead of the re-scoring step")
    ap.add_argument("--group", action="store_true",
                    help="time localized group construction: constrained branch-point selection, "
                         "continuation allocation, group advantages and per-token policy-loss factors")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-mfma-ceiling", action="store_true",
                    help="skip measuring this GPU's ceilings of the kernel's main loop (MFMAs on "
                         "const/random operands, with LDS reads, with the per-slice DMA) and the "
                         "library GEMM reference")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="after timing, copy this many MiB device-to-device once (a known-size "
                         "kernel that calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(rows are independent; sharding is described in the design notes).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2609_36864_amd as hdl
    import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    hdl.load_library()
    dev = torch.device("cuda:0")

    t0 = time.time()
    w = workloads.make_workload(args.workload)
    c = w.cfg
    log(f"generated workload {args.workload} in {time.time() - t0:.1f} s")

    if args.backward:
        return bench_backward(args, w, hdl, dev)
    if args.group:
        return bench_group(args, w, hdl, dev)

    ent_sel = args.selector == "entropy"
    n_keep = c.R * c.T if ent_sel else 2 * c.R * c.T   # rows are [context][root][t]
    hidden = w.rows_hidden()[:n_keep].to(dev)
    W = w.W.to(dev)
    tokens = w.rows_tokens()[:n_keep].to(dev)
    mask = w.rows_mask()[:n_keep].to(dev)
    mask_rt = w.mask.to(dev)
    n_rows = hidden.shape[0]
    n_scored = int(mask.sum().item())
    dt = hdl.HDL_BF16 if c.dtype == "bf16" else hdl.HDL_F32
    ws = torch.empty(hdl.workspace_size(n_rows, c.d, c.V, dt), dtype=torch.uint8, device=dev)
    logp = torch.empty(n_rows, dtype=torch.float32, device=dev)
    ent = torch.empty(n_rows, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    props = torch.cuda.get_device_properties(0)
    log(f"inputs resident on {props.name or getattr(props, 'gcnArchName', 'cuda:0')}: {n_rows} rows, {n_scored} scored")

    def step():
        if ent_sel:
            hdl.token_logprobs(hidden, W, tokens, mask, logp=logp, want_lse=False,
                               want_entropy=True, entropy=ent, workspace=ws)
            return hdl.select_top_k(ent.view(c.R, c.T), mask_rt, c.k) + (None,)
        hdl.token_logprobs(hidden, W, tokens, mask, logp=logp, want_lse=False, workspace=ws)
        lp = logp.view(2, c.R, c.T)
        return hdl.select_branch_points(lp[0], lp[1], mask_rt, c.k)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    hdl.profile_enable(True)
    hdl.profile_read()   # reset the tally
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        out = step()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    kern_ms, launches = hdl.profile_read()
    hdl.profile_enable(False)
    step_ms = ev0.elapsed_time(ev1) / args.steps
    log(f"timed {args.steps} steps: {step_ms:.3f} ms/step (wall {wall / args.steps * 1e3:.3f} ms/step), "
        f"fused kernel {kern_ms / max(launches, 1):.3f} ms/launch")

    idx, score, count, _ = out
    counts = count.cpu().numpy()
    if not (np.all(counts == min(c.k, c.T)) or np.all(counts <= c.k)):
        raise RuntimeError("selection produced an invalid count")
    if not torch.isfinite(logp[mask.bool()]).all():
        raise RuntimeError("non-finite log-probabilities")
    if ent_sel and not torch.isfinite(ent[mask.bool()]).all():
        raise RuntimeError("non-finite entropies")

    value = n_scored / (step_ms / 1e3)
    flops = 2.0 * c.d * c.V * n_scored
    kern_avg_ms = kern_ms / max(launches, 1)
    achieved = flops / (kern_avg_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[c.dtype]
    result = {
        "metric": METRIC_ENTROPY if ent_sel else METRIC,
        "value": value,
        "unit": "scored tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": c.dtype,
        "data": "synthetic (seeded generator; random lm-head weights and hidden states)",
        "config": {"workload": f"{args.workload}: {workloads.DESCRIPTIONS[args.workload]}",
                   "selector": args.selector, "roots": c.R, "T": c.T, "d": c.d, "V": c.V, "k": c.k,
                   "scored_tokens_per_step": n_scored},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None,
                     "kernel": "lmhead_logprob_kernel", "kernel_ms": kern_avg_ms,
                     "flops_per_launch": flops},
    }
    if not ent_sel:
        # the divergence / top-k pass alone (a6-a7): HBM-bound in principle,
        # latency-bound at these sizes (one workgroup per root)
        lp = logp.view(2, c.R, c.T)
        hdl.select_branch_points(lp[0], lp[1], mask_rt, c.k)
        stream = torch.cuda.current_stream(dev)
        e2 = torch.cuda.Event(enable_timing=True)
        e3 = torch.cuda.Event(enable_timing=True)
        reps = 50
        torch.cuda.synchronize()
        hdl.profile_enable(True)
        hdl.profile_read(hdl.PROFILE_SELECT)   # reset the tally
        e2.record(stream)
        for _ in range(reps):
            hdl.select_branch_points(lp[0], lp[1], mask_rt, c.k)
        e3.record(stream)
        torch.cuda.synchronize()
        sel_kern_ms, sel_n = hdl.profile_read(hdl.PROFILE_SELECT)
        hdl.profile_enable(False)
        # the kernel's own time (HIP events around each launch on the
        # library's stream); back-to-back calls from Python can be bound by
        # the host instead, which call_ms shows
        sel_ms = sel_kern_ms / max(sel_n, 1)
        call_ms = e2.elapsed_time(e3) / reps
        sel_bytes = c.R * c.T * (4 + 4 + 1) + c.R * c.k * 8 + c.R * 4
        result["select_pass"] = {"kernel": "select_kernel", "bound": "latency (one workgroup per root)",
                                 "ms_per_call": sel_ms, "call_ms": call_ms, "bytes_per_call": sel_bytes,
                                 "achieved_GBps": sel_bytes / (sel_ms * 1e-3) / 1e9, "peak_GBps": 8000.0}
        log(f"divergence/top-k pass: {sel_ms * 1e3:.1f} us per call, {sel_bytes} bytes")
    if args.copy_probe_mb > 0:
        src = torch.empty(args.copy_probe_mb << 20, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: {args.copy_probe_mb} MiB device-to-device")
    if c.dtype == "bf16" and not args.no_mfma_ceiling:
        ceil = mfma_ceiling()
        if ceil is not None:
            ceil["frac_of_random_operand_ceiling"] = achieved / ceil["random_operands_tflops"]
            if ceil.get("slice_loop_dma_hbm_tflops"):
                ceil["frac_of_slice_loop_ceiling"] = achieved / ceil["slice_loop_dma_hbm_tflops"]
            result["roofline"]["measured_ceiling"] = ceil
            log(f"MFMA ceilings: {ceil}")
        lib = library_gemm_tflops(hidden[mask.bool()], W)
        result["roofline"]["library_gemm"] = {
            "what": "torch.matmul(scored hidden rows, W^T) -> bf16 logits (hipBLASLt), same contraction, "
                    "16384-row chunks; reference only",
            "tflops": lib, "fused_kernel_frac": achieved / lib}
        log(f"library GEMM on the same contraction: {lib:.0f} TFLOP/s (fused kernel: {achieved / lib:.3f} of it)")
    traffic = None if ent_sel else measured_traffic(args.workload)
    if traffic is not None:
        result["roofline"]["traffic"] = traffic
    if not args.no_cpu_baseline:
        log("timing the float64 oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(w, budget_s=args.cpu_budget, entropy=ent_sel)
    print(json.dumps(result), flush=True)
    return 0


def cpu_baseline_backward(w, budget_s: float = 15.0, max_rows: int = 2048):
    """Time the float64 oracle's backward on a seeded sample of eligible
    original-context rows; return oracle trained tokens/s."""
    import numpy as np
    import torch
    from oracle import hdl_oracle as O
    cores, blas_threads = host_cores()
    c = w.cfg
    Wd = O.bf16_bits_to_f64(w.W.view(torch.int16).numpy().view(np.uint16))
    n0 = c.R * c.T
    hidden = w.rows_hidden()[:n0]
    tokens = w.rows_tokens().numpy()[:n0]
    elig = np.nonzero(w.rows_mask().numpy()[:n0])[0]
    rng = np.random.default_rng(12346)
    sample = rng.permutation(elig)[:max_rows]
    done, t_total, blk = 0, 0.0, 32
    while done < len(sample) and t_total < budget_s:
        rows = np.sort(sample[done:done + blk])
        H = O.bf16_bits_to_f64(hidden[torch.as_tensor(rows)].view(torch.int16).numpy().view(np.uint16))
        g = rng.normal(size=len(rows))
        t0 = time.perf_counter()
        O.token_logprobs_backward(H, Wd, tokens[rows], g)
        t_total += time.perf_counter() - t0
        done += len(rows)
    return {"value": done / t_total, "unit": "trained tokens/s", "cores": blas_threads, "kind": "oracle",
            "host_cpus": cores, "blas_threads": blas_threads,
            "sample": f"{done} eligible original-context rows of this workload (float64 logits, "
                      f"softmax gradient, dL/dh and dL/dW, {t_total:.1f} s)"}


def bench_backward(args, w, hdl, dev) -> int:
    """Backward pass of the fused log-probability on the original-context rows:
    the logits are recomputed tile by tile, the logit gradient exists one chunk
    at a time as bf16, and dL/dh = G W and dL/dW = G^T H run as MFMA GEMMs."""
    import numpy as np
    import torch
    c = w.cfg
    if c.dtype != "bf16":
        print("the backward pass takes bf16 inputs", file=sys.stderr)
        return 2
    n0 = c.R * c.T
    hidden = w.rows_hidden()[:n0].to(dev)
    W = w.W.to(dev)
    tokens = w.rows_tokens()[:n0].to(dev)
    mask = w.rows_mask()[:n0].to(dev)
    n_scored = int(mask.sum().item())
    # per-token factor of a token-level policy loss: advantage-like, averaged over tokens
    g = torch.from_numpy(np.random.default_rng(c.seed + 7).normal(size=n0).astype(np.float32) / n_scored).to(dev)
    _, lse = hdl.token_logprobs(hidden, W, tokens, mask)
    ws = torch.empty(hdl.backward_workspace_size(n0, c.d, c.V), dtype=torch.uint8, device=dev)
    grad_w = torch.empty(c.V, c.d, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    log(f"backward: {n0} rows, {n_scored} trained, workspace {ws.numel() / 2**30:.2f} GiB")

    def step():
        return hdl.token_logprobs_backward(hidden, W, tokens, mask, lse, g, grad_w=grad_w, workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    hdl.profile_enable(True)
    for kind in (hdl.PROFILE_GRAD, hdl.PROFILE_GEMM):
        hdl.profile_read(kind)   # reset the tallies
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        dh, dw = step()
    ev1.record(stream)
    torch.cuda.synchronize()
    grad_ms, grad_n = hdl.profile_read(hdl.PROFILE_GRAD)
    gemm_ms, gemm_n = hdl.profile_read(hdl.PROFILE_GEMM)
    hdl.profile_enable(False)
    step_ms = ev0.elapsed_time(ev1) / args.steps
    log(f"timed {args.steps} backward steps: {step_ms:.3f} ms/step; gradient-mode kernel "
        f"{grad_ms / max(grad_n, 1):.3f} ms x {grad_n // args.steps}, GEMM {gemm_ms / max(gemm_n, 1):.3f} ms "
        f"x {gemm_n // args.steps} per step")
    if not (torch.isfinite(dh).all() and torch.isfinite(dw).all()):
        raise RuntimeError("non-finite gradients")
    # probabilities sum to one, so the vocabulary rows of dL/dW sum to ~0
    col = dw.double().sum(0).abs().max().item()
    log(f"max |sum_v dL/dW[v, :]| = {col:.3g} (max |dL/dW| = {dw.abs().max().item():.3g})")
    flops = 6.0 * c.d * c.V * n_scored   # logit recompute + two contractions
    achieved = flops / (step_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[c.dtype]
    # the dominant kernel is the GEMM (dH = G W and dW = G^T H): 4 d V n_scored
    # algorithmic flops per step over its launches
    gemm_launch_ms = gemm_ms / max(gemm_n, 1)
    gemm_flops = 4.0 * c.d * c.V * n_scored / max(gemm_n // args.steps, 1)
    gemm_tflops = gemm_flops / (gemm_launch_ms / 1e3) / 1e12
    grad_launch_ms = grad_ms / max(grad_n, 1)
    grad_tflops = (2.0 * c.d * c.V * n_scored / max(grad_n // args.steps, 1)) / (grad_launch_ms / 1e3) / 1e12
    result = {
        "metric": METRIC_BACKWARD,
        "value": n_scored / (step_ms / 1e3),
        "unit": "trained tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": c.dtype,
        "data": "synthetic (seeded generator; random lm-head weights, hidden states and upstream gradients)",
        "config": {"workload": f"{args.workload}: {workloads_description(args.workload)}, original context",
                   "pass": "backward", "roots": c.R, "T": c.T, "d": c.d, "V": c.V,
                   "trained_tokens_per_step": n_scored},
        "roofline": {"bound": "mfma", "achieved": gemm_tflops, "peak": peak, "unit": "TFLOP/s",
                     "frac": gemm_tflops / peak, "traffic": None,
                     "kernel": f"gemm_kernel (dH = G W, dW = G^T H; "
                               f"{100.0 * gemm_ms / args.steps / step_ms:.0f} % of the pass)",
                     "kernel_ms": gemm_launch_ms, "flops_per_launch": gemm_flops,
                     "gradient_mode_kernel": {"kernel_ms": grad_launch_ms, "achieved": grad_tflops,
                                              "frac": grad_tflops / peak},
                     "whole_pass": {"ms": step_ms, "flops": flops, "achieved": achieved,
                                    "frac": achieved / peak}},
    }
    if not args.no_mfma_ceiling:
        # reference only: the vendor GEMMs (torch.matmul -> hipBLASLt) on the
        # two contractions' shapes, with a bf16 logit gradient of the same size
        gref = torch.randn(n_scored, c.V, device=dev, dtype=torch.bfloat16)
        hs = hidden[mask.bool()]
        dh_ref = torch.empty(n_scored, c.d, device=dev, dtype=torch.bfloat16)
        dw_ref = torch.empty(c.V, c.d, device=dev, dtype=torch.bfloat16)
        ref = {}
        for name, fn in (("dH = G W", lambda: torch.matmul(gref, W, out=dh_ref)),
                         ("dW = G^T H", lambda: torch.matmul(gref.t(), hs, out=dw_ref))):
            fn()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(3):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ref[name] = 2.0 * n_scored * c.V * c.d / (e0.elapsed_time(e1) / 3 / 1e3) / 1e12
        del gref, dh_ref, dw_ref
        result["roofline"]["library_gemm"] = {
            "what": "torch.matmul (hipBLASLt) on the dH and dW shapes with a bf16 logit gradient, "
                    "bf16 outputs; reference only",
            "tflops": ref,
            # both GEMMs have the same flops: their combined rate is the harmonic mean
            "gemm_kernel_frac": gemm_tflops / (len(ref) / sum(1.0 / r for r in ref.values()))}
        log(f"library GEMMs on the same shapes: {ref}")
    if not args.no_cpu_baseline:
        log("timing the float64 oracle backward on a bounded sample")
        result["cpu_baseline"] = cpu_baseline_backward(w, budget_s=args.cpu_budget)
    print(json.dumps(result), flush=True)
    return 0


def bench_group(args, w, hdl, dev) -> int:
    """One training step's group construction at the paper's batch (128
    problems, 2 roots + 14 continuations each, Sec. 4.1) with the workload's
    trajectory length T: the 256 roots' log p pairs (synthetic, as the
    re-scoring step would leave them) are ranked under the branch-point
    constraints (spacing 64, index range excluding the first and last 32
    positions), 3 + 4 continuations are allocated per root, every group gets
    mean-centred advantages, and every token of every trajectory (T each; a
    continuation trains only its suffix) gets its clipped-loss factor."""
    import numpy as np
    import torch
    import workloads
    c = w.cfg
    n_groups, roots_per_group, alloc = 128, 2, (3, 4)
    R, T = n_groups * roots_per_group, c.T
    lo_, hi_, mask = workloads.make_logp_pair(R, T, seed=c.seed + 11)
    lo_t = torch.from_numpy(lo_).to(dev)
    hi_t = torch.from_numpy(hi_).to(dev)
    mask_t = torch.from_numpy(mask).to(dev)
    rlo = torch.full((R,), 32, dtype=torch.int32, device=dev)
    rhi = torch.full((R,), T - 33, dtype=torch.int32, device=dev)
    G = roots_per_group * (1 + sum(alloc))
    n_traj = n_groups * G
    rng = np.random.default_rng(c.seed + 12)
    rewards = torch.from_numpy((rng.random((n_groups, G)) < 0.5).astype(np.float32)).to(dev)
    n_tok = n_traj * T
    traj = torch.arange(n_traj, dtype=torch.int32, device=dev).repeat_interleave(T)
    pos = torch.arange(T, dtype=torch.int32, device=dev).repeat(n_traj)
    logp_old = torch.from_numpy((-rng.exponential(2.0, n_tok)).astype(np.float32)).to(dev)
    logp_new = logp_old + torch.from_numpy((rng.normal(size=n_tok) * 0.2).astype(np.float32)).to(dev)
    tmask = torch.from_numpy((rng.random(n_tok) < 0.9).astype(np.uint8)).to(dev)
    start = torch.zeros(n_traj, dtype=torch.int32, device=dev)
    grad = torch.empty(n_tok, dtype=torch.float32, device=dev)
    n_trained = torch.empty(1, dtype=torch.int64, device=dev)
    torch.cuda.synchronize()

    def step():
        idx, score, count = hdl.select_constrained(lo_t, hi_t, mask_t, len(alloc), lo=rlo, hi=rhi, min_gap=64)
        bpos, _ = hdl.allocate_continuations(idx, count, alloc)
        # trajectories of group g: its 2 roots, then their 7 continuations each;
        # a continuation trains from its branch position on
        st = start.view(n_groups, G)
        st[:, roots_per_group:] = bpos.view(n_groups, -1)
        adv = hdl.group_advantages(rewards).view(-1)
        # token-level mean over the trained tokens, counted on the device
        g, _ = hdl.policy_loss_grad(adv, traj, logp_new, logp_old, loss_mask=tmask, pos=pos, start=start,
                                    n_trained=n_trained)
        return idx, count, g

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        idx, count, g = step()
    ev1.record(stream)
    torch.cuda.synchronize()
    step_ms = ev0.elapsed_time(ev1) / args.steps
    cnt = count.cpu().numpy()
    log(f"timed {args.steps} group-construction steps: {step_ms:.3f} ms/step "
        f"({n_groups} groups of {G}, {n_tok} tokens; {cnt.mean():.3f} points per root, "
        f"{int((cnt < len(alloc)).sum())} roots keep fewer than {len(alloc)})")
    # the per-token factor pass dominates: 4 (traj) + 4 (pos) + 4 + 4 (log p) + 1 (mask)
    # bytes read and 8 written per token, plus the per-trajectory reads
    bytes_tok = 25.0 * n_tok
    ev2 = torch.cuda.Event(enable_timing=True)
    ev3 = torch.cuda.Event(enable_timing=True)
    adv = hdl.group_advantages(rewards).view(-1)
    ev2.record(stream)
    for _ in range(args.steps):
        hdl.policy_loss_grad(adv, traj, logp_new, logp_old, loss_mask=tmask, pos=pos, start=start,
                             scale=1.0 / n_tok)
    ev3.record(stream)
    torch.cuda.synchronize()
    k_ms = ev2.elapsed_time(ev3) / args.steps
    achieved = bytes_tok / (k_ms / 1e3) / 1e9
    result = {
        "metric": METRIC_GROUP,
        "value": n_tok / (step_ms / 1e3),
        "unit": "trained tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded log-probability pairs, rewards and policy log-probabilities)",
        "config": {"workload": f"{args.workload} trajectory length: {R} roots x T={T}, {n_groups} groups of "
                               f"{roots_per_group} roots + {G - roots_per_group} continuations (3+4 per root)",
                   "pass": "group", "min_gap": 64, "index_range": [32, T - 33], "tokens_per_step": n_tok},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": 8000.0, "unit": "GB/s",
                     "frac": achieved / 8000.0, "traffic": None, "kernel": "policy_grad_kernel",
                     "kernel_ms": k_ms, "bytes_per_launch": bytes_tok},
    }
    if not args.no_cpu_baseline:
        from oracle import hdl_oracle as O
        t0 = time.perf_counter()
        sample = 200000
        sl = slice(0, sample)
        O.policy_loss_grad(adv.cpu().numpy(), traj[sl].cpu().numpy(), logp_new[sl].cpu().numpy(),
                           logp_old[sl].cpu().numpy(), tmask[sl].cpu().numpy(), pos[sl].cpu().numpy(),
                           start.cpu().numpy(), 0.2, 0.28, 1.0 / n_tok)
        dt = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": sample / dt, "unit": "trained tokens/s", "cores": 1, "kind": "oracle",
                                  "sample": f"the oracle's per-token policy-loss factors for the first {sample} "
                                            f"tokens ({dt:.1f} s; selection and allocation excluded)"}
    print(json.dumps(result), flush=True)
    return 0


def workloads_description(name: str) -> str:
    import workloads
    return workloads.DESCRIPTIONS[name]


if __name__ == "__main__":
    sys.exit(main())
