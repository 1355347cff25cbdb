"""MI355X (gfx950) hindsight re-scoring path of Hindsight-Divergence Localization.

A thin ctypes binding over libhdl.so (C ABI in include/hdl.h).  Every step of
the path runs in the library's HIP kernels; this module only checks tensor
arguments, allocates outputs and workspace with torch, and passes device
pointers and the current HIP stream.  There is no CPU fallback: without the
built library or a GPU the calls raise.

    logp, lse = token_logprobs(hidden, w_vocab, tokens, mask)          # Eq. 1
    idx, score, count, delta = select_branch_points(lp0, lpH, mask, k)  # Eq. 2
"""
from __future__ import annotations

import ctypes
import functools
import os
from typing import Optional, Tuple

import torch

__all__ = ["HdlError", "HDL_F32", "HDL_BF16", "HDL_MAX_K", "library_path", "load_library",
           "workspace_size", "token_logprobs", "token_logprobs_noalloc", "token_logprobs_backward", "select_branch_points",
           "select_top_k", "select_constrained", "allocate_continuations", "group_advantages",
           "policy_loss_grad", "rescore",
           "profile_enable", "profile_read", "abi_version"]

HDL_F32 = 0
HDL_BF16 = 1
HDL_MAX_K = 1024

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
_LIB: Optional[ctypes.CDLL] = None


class HdlError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"libhdl status {status}: {message}")
        self.status = status


def library_path() -> str:
    return os.path.join(_PKG_DIR, "libhdl.so")


def load_library() -> ctypes.CDLL:
    """Load libhdl.so (built by paper_2609_36864_amd.build); raises if absent."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2609_36864_amd.build`")
    L = ctypes.CDLL(path)
    c_i64, c_vp, c_sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
    L.hdl_token_logprobs_workspace_size.argtypes = [c_i64, c_i64, c_i64, ctypes.c_int]
    L.hdl_token_logprobs_workspace_size.restype = c_sz
    L.hdl_token_logprobs.argtypes = [c_vp, c_vp, c_vp, c_vp, c_i64, c_i64, c_i64, ctypes.c_int,
                                     c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hdl_token_logprobs.restype = ctypes.c_int
    L.hdl_token_logprobs_entropy.argtypes = [c_vp, c_vp, c_vp, c_vp, c_i64, c_i64, c_i64, ctypes.c_int,
                                             c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hdl_token_logprobs_entropy.restype = ctypes.c_int
    L.hdl_token_logprobs_noalloc.argtypes = [c_vp, c_vp, c_vp, c_vp, c_i64, c_i64, c_i64, ctypes.c_int,
                                             c_vp, c_vp, c_vp]
    L.hdl_token_logprobs_noalloc.restype = ctypes.c_int
    L.hdl_select_top_k.argtypes = [c_vp, c_vp, c_i64, c_i64, ctypes.c_int32, c_vp, c_vp, c_vp, c_vp]
    L.hdl_select_top_k.restype = ctypes.c_int
    L.hdl_token_logprobs_backward_workspace_size.argtypes = [c_i64, c_i64, c_i64, ctypes.c_int]
    L.hdl_token_logprobs_backward_workspace_size.restype = c_sz
    L.hdl_token_logprobs_backward.argtypes = [c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_i64, c_i64, c_i64,
                                              ctypes.c_int, c_vp, c_vp, ctypes.c_int, c_vp, c_sz, c_vp]
    L.hdl_token_logprobs_backward.restype = ctypes.c_int
    L.hdl_select_constrained.argtypes = [c_vp, c_vp, c_vp, c_i64, c_i64, ctypes.c_int32, c_vp, c_vp,
                                         ctypes.c_int32, ctypes.c_int, c_vp, c_vp, c_vp, c_vp]
    L.hdl_select_constrained.restype = ctypes.c_int
    L.hdl_allocate_continuations.argtypes = [c_vp, c_vp, c_i64, ctypes.c_int32, c_vp, ctypes.c_int32, c_vp,
                                             c_vp, c_vp]
    L.hdl_allocate_continuations.restype = ctypes.c_int
    L.hdl_group_advantages.argtypes = [c_vp, c_i64, ctypes.c_int32, c_vp, c_vp]
    L.hdl_group_advantages.restype = ctypes.c_int
    L.hdl_policy_loss_grad.argtypes = [c_vp, c_i64, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_i64, ctypes.c_float,
                                       ctypes.c_float, ctypes.c_float, c_vp, c_vp, c_vp, c_vp]
    L.hdl_policy_loss_grad.restype = ctypes.c_int
    L.hdl_select_branch_points.argtypes = [c_vp, c_vp, c_vp, c_i64, c_i64, ctypes.c_int32,
                                           c_vp, c_vp, c_vp, c_vp, c_vp]
    L.hdl_select_branch_points.restype = ctypes.c_int
    L.hdl_status_string.argtypes = [ctypes.c_int]
    L.hdl_status_string.restype = ctypes.c_char_p
    L.hdl_last_hip_error.argtypes = []
    L.hdl_last_hip_error.restype = ctypes.c_char_p
    L.hdl_abi_version.argtypes = []
    L.hdl_abi_version.restype = ctypes.c_int
    L.hdl_profile_enable.argtypes = [ctypes.c_int]
    L.hdl_profile_enable.restype = ctypes.c_int
    L.hdl_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(c_i64)]
    L.hdl_profile_read.restype = ctypes.c_int
    L.hdl_profile_read_kind.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(c_i64)]
    L.hdl_profile_read_kind.restype = ctypes.c_int
    _LIB = L
    return L


def _check(status: int) -> None:
    if status != 0:
        L = load_library()
        msg = L.hdl_last_hip_error().decode() or L.hdl_status_string(status).decode()
        raise HdlError(status, msg)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _require_cuda(name: str, t: torch.Tensor) -> None:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _on_tensor_device(fn):
    """Run an entry point with its tensors' GPU as the current device (the
    library launches on the current device and the stream of that device);
    every GPU tensor argument must live on the same device."""
    @functools.wraps(fn)
    def wrapper(*args, **kwargs):
        devs = {a.device for a in list(args) + list(kwargs.values())
                if isinstance(a, torch.Tensor) and a.device.type == "cuda"}
        if len(devs) > 1:
            raise ValueError(f"{fn.__name__}: tensors on several devices {sorted(map(str, devs))}")
        if devs:
            with torch.cuda.device(devs.pop()):
                return fn(*args, **kwargs)
        return fn(*args, **kwargs)
    return wrapper


def abi_version() -> int:
    return int(load_library().hdl_abi_version())


def workspace_size(n_rows: int, d: int, vocab: int, dtype: int) -> int:
    return int(load_library().hdl_token_logprobs_workspace_size(n_rows, d, vocab, dtype))


_WS_CACHE: dict = {}


def _workspace(device: torch.device, nbytes: int) -> torch.Tensor:
    key = (device.index, str(torch.cuda.current_stream(device)))
    ws = _WS_CACHE.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        _WS_CACHE[key] = ws
    return ws


@_on_tensor_device
def token_logprobs(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor,
                   mask: Optional[torch.Tensor] = None, *, logp: Optional[torch.Tensor] = None,
                   lse: Optional[torch.Tensor] = None, want_lse: bool = True,
                   want_entropy: bool = False, entropy: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None):
    """Teacher-forced log p of each row's sampled token (Eq. 1), fused lm-head.

    hidden [n_rows, d] and w_vocab [vocab, d], both bf16 or both fp32;
    tokens [n_rows] int32; mask [n_rows] uint8/bool or None.
    Returns (logp [n_rows] fp32, lse [n_rows] fp32 or None), or, with
    want_entropy, (logp, lse, entropy [n_rows] fp32) where entropy is the
    next-token entropy computed in the same pass.
    """
    L = load_library()
    for name, t in (("hidden", hidden), ("w_vocab", w_vocab), ("tokens", tokens)):
        _require_cuda(name, t)
    if hidden.dim() != 2 or w_vocab.dim() != 2 or hidden.shape[1] != w_vocab.shape[1]:
        raise ValueError("hidden must be [n_rows, d] and w_vocab [vocab, d]")
    if hidden.dtype != w_vocab.dtype or hidden.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("hidden and w_vocab must both be bfloat16 or both float32")
    if tokens.dtype != torch.int32 or tokens.shape != (hidden.shape[0],):
        raise ValueError("tokens must be int32 [n_rows]")
    n_rows, d = hidden.shape
    vocab = w_vocab.shape[0]
    dev = hidden.device
    if mask is not None:
        _require_cuda("mask", mask)
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        if mask.dtype != torch.uint8 or mask.shape != (n_rows,):
            raise ValueError("mask must be uint8 [n_rows]")
    dt = HDL_BF16 if hidden.dtype == torch.bfloat16 else HDL_F32
    if logp is None:
        logp = torch.empty(n_rows, dtype=torch.float32, device=dev)
    if want_lse and lse is None:
        lse = torch.empty(n_rows, dtype=torch.float32, device=dev)
    if want_entropy and entropy is None:
        entropy = torch.empty(n_rows, dtype=torch.float32, device=dev)
    nbytes = workspace_size(n_rows, d, vocab, dt)
    if nbytes == 0:
        raise ValueError(f"invalid sizes n_rows={n_rows} d={d} vocab={vocab}")
    ws = workspace if workspace is not None else _workspace(dev, nbytes)
    if want_entropy:
        _check(L.hdl_token_logprobs_entropy(hidden.data_ptr(), w_vocab.data_ptr(), tokens.data_ptr(),
                                            _ptr(mask), n_rows, d, vocab, dt, logp.data_ptr(), _ptr(lse),
                                            entropy.data_ptr(), ws.data_ptr(),
                                            ws.numel() * ws.element_size(), _stream_handle(dev)))
        return logp, lse, entropy
    _check(L.hdl_token_logprobs(hidden.data_ptr(), w_vocab.data_ptr(), tokens.data_ptr(), _ptr(mask),
                                n_rows, d, vocab, dt, logp.data_ptr(), _ptr(lse), ws.data_ptr(),
                                ws.numel() * ws.element_size(), _stream_handle(dev)))
    return logp, lse


@_on_tensor_device
def select_branch_points(logp_orig: torch.Tensor, logp_hind: torch.Tensor,
                         mask: Optional[torch.Tensor], k: int, *, want_delta: bool = False):
    """|Delta log p| (Eq. 2) and the per-root top-k branch points (Sec. 3.2).

    logp_orig, logp_hind [R, T] fp32; mask [R, T] uint8 or None.
    Returns (idx [R,k] int32, score [R,k] fp32, count [R] int32, delta [R,T] or None).
    """
    L = load_library()
    _require_cuda("logp_orig", logp_orig)
    _require_cuda("logp_hind", logp_hind)
    if logp_orig.dtype != torch.float32 or logp_hind.dtype != torch.float32:
        raise ValueError("log-probabilities must be float32")
    if logp_orig.dim() != 2 or logp_orig.shape != logp_hind.shape:
        raise ValueError("logp_orig and logp_hind must both be [R, T]")
    R, T = logp_orig.shape
    dev = logp_orig.device
    if mask is not None:
        _require_cuda("mask", mask)
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        if mask.dtype != torch.uint8 or tuple(mask.shape) != (R, T):
            raise ValueError("mask must be uint8 [R, T]")
    kk = max(int(k), 1)
    idx = torch.empty(R, kk, dtype=torch.int32, device=dev)
    score = torch.empty(R, kk, dtype=torch.float32, device=dev)
    count = torch.empty(R, dtype=torch.int32, device=dev)
    delta = torch.empty(R, T, dtype=torch.float32, device=dev) if want_delta else None
    _check(L.hdl_select_branch_points(logp_orig.data_ptr(), logp_hind.data_ptr(), _ptr(mask), R, T,
                                      int(k), idx.data_ptr(), score.data_ptr(), count.data_ptr(),
                                      _ptr(delta), _stream_handle(dev)))
    return idx, score, count, delta


@_on_tensor_device
def select_top_k(values: torch.Tensor, mask: Optional[torch.Tensor], k: int):
    """Per-root top-k of a per-position value, e.g. next-token entropy for the
    Entropy localization baseline (Sec. 4.1).  values [R, T] fp32, mask
    [R, T] uint8 or None.  Returns (idx [R,k] int32, score [R,k] fp32, count [R] int32)."""
    L = load_library()
    _require_cuda("values", values)
    if values.dtype != torch.float32 or values.dim() != 2:
        raise ValueError("values must be float32 [R, T]")
    R, T = values.shape
    dev = values.device
    if mask is not None:
        _require_cuda("mask", mask)
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        if mask.dtype != torch.uint8 or tuple(mask.shape) != (R, T):
            raise ValueError("mask must be uint8 [R, T]")
    kk = max(int(k), 1)
    idx = torch.empty(R, kk, dtype=torch.int32, device=dev)
    score = torch.empty(R, kk, dtype=torch.float32, device=dev)
    count = torch.empty(R, dtype=torch.int32, device=dev)
    _check(L.hdl_select_top_k(values.data_ptr(), _ptr(mask), R, T, int(k), idx.data_ptr(),
                              score.data_ptr(), count.data_ptr(), _stream_handle(dev)))
    return idx, score, count


@_on_tensor_device
def token_logprobs_backward(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor,
                            mask: Optional[torch.Tensor], lse: torch.Tensor, grad_logp: torch.Tensor, *,
                            grad_w: Optional[torch.Tensor] = None, accumulate_w: bool = False,
                            workspace: Optional[torch.Tensor] = None):
    """Gradients of L = sum_n g_n log p_n(y_n) with respect to the hidden
    states and the lm-head weight (backward of token_logprobs; bf16 inputs).

    lse is the forward pass's log-sum-exp, grad_logp the per-row g_n (fp32).
    Returns (grad_hidden [n_rows, d] fp32, grad_w [vocab, d] fp32).
    """
    L = load_library()
    for name, t in (("hidden", hidden), ("w_vocab", w_vocab), ("tokens", tokens), ("lse", lse),
                    ("grad_logp", grad_logp)):
        _require_cuda(name, t)
    if hidden.dim() != 2 or w_vocab.dim() != 2 or hidden.shape[1] != w_vocab.shape[1]:
        raise ValueError("hidden must be [n_rows, d] and w_vocab [vocab, d]")
    if hidden.dtype != torch.bfloat16 or w_vocab.dtype != torch.bfloat16:
        raise ValueError("the backward pass takes bfloat16 hidden and w_vocab")
    n_rows, d = hidden.shape
    vocab = w_vocab.shape[0]
    if tokens.dtype != torch.int32 or tokens.shape != (n_rows,):
        raise ValueError("tokens must be int32 [n_rows]")
    for name, t in (("lse", lse), ("grad_logp", grad_logp)):
        if t.dtype != torch.float32 or t.shape != (n_rows,):
            raise ValueError(f"{name} must be float32 [n_rows]")
    dev = hidden.device
    if mask is not None:
        _require_cuda("mask", mask)
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        if mask.dtype != torch.uint8 or mask.shape != (n_rows,):
            raise ValueError("mask must be uint8 [n_rows]")
    grad_hidden = torch.empty(n_rows, d, dtype=torch.float32, device=dev)
    if grad_w is None:
        if accumulate_w:
            raise ValueError("accumulate_w needs grad_w")
        grad_w = torch.empty(vocab, d, dtype=torch.float32, device=dev)
    else:
        _require_cuda("grad_w", grad_w)
        if grad_w.dtype != torch.float32 or grad_w.shape != (vocab, d):
            raise ValueError("grad_w must be float32 [vocab, d]")
    nbytes = int(L.hdl_token_logprobs_backward_workspace_size(n_rows, d, vocab, HDL_BF16))
    if nbytes == 0:
        raise ValueError(f"unsupported sizes n_rows={n_rows} d={d} vocab={vocab}")
    ws = workspace if workspace is not None else torch.empty(nbytes, dtype=torch.uint8, device=dev)
    _check(L.hdl_token_logprobs_backward(hidden.data_ptr(), w_vocab.data_ptr(), tokens.data_ptr(), _ptr(mask),
                                         lse.data_ptr(), grad_logp.data_ptr(), n_rows, d, vocab, HDL_BF16,
                                         grad_hidden.data_ptr(), grad_w.data_ptr(), 1 if accumulate_w else 0,
                                         ws.data_ptr(), ws.numel() * ws.element_size(), _stream_handle(dev)))
    return grad_hidden, grad_w


def backward_workspace_size(n_rows: int, d: int, vocab: int) -> int:
    return int(load_library().hdl_token_logprobs_backward_workspace_size(n_rows, d, vocab, HDL_BF16))


def _dev_2d(name, t, dtype, shape=None):
    _require_cuda(name, t)
    if t.dtype != dtype or (shape is not None and tuple(t.shape) != tuple(shape)):
        raise ValueError(f"{name} must be {dtype} {list(shape) if shape else ''}")
    return t


@_on_tensor_device
def select_constrained(a: torch.Tensor, b: Optional[torch.Tensor], mask: Optional[torch.Tensor], k: int, *,
                       lo: Optional[torch.Tensor] = None, hi: Optional[torch.Tensor] = None, min_gap: int = 0,
                       refill: bool = False):
    """Per-root top-k under the branch-point constraints (index range
    [lo, hi] per root, minimum spacing).  b given: rank |b - a| (Eq. 2);
    b None: rank a's values.  Returns (idx [R,k], score [R,k], count [R])."""
    L = load_library()
    _dev_2d("a", a, torch.float32)
    if a.dim() != 2:
        raise ValueError("a must be [R, T]")
    R, T = a.shape
    if b is not None:
        _dev_2d("b", b, torch.float32, (R, T))
    if mask is not None:
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        _dev_2d("mask", mask, torch.uint8, (R, T))
    for name, t in (("lo", lo), ("hi", hi)):
        if t is not None:
            _dev_2d(name, t, torch.int32, (R,))
    dev = a.device
    kk = max(int(k), 1)
    idx = torch.empty(R, kk, dtype=torch.int32, device=dev)
    score = torch.empty(R, kk, dtype=torch.float32, device=dev)
    count = torch.empty(R, dtype=torch.int32, device=dev)
    _check(L.hdl_select_constrained(a.data_ptr(), _ptr(b), _ptr(mask), R, T, int(k), _ptr(lo), _ptr(hi),
                                    int(min_gap), 1 if refill else 0, idx.data_ptr(), score.data_ptr(),
                                    count.data_ptr(), _stream_handle(dev)))
    return idx, score, count


@_on_tensor_device
def allocate_continuations(idx: torch.Tensor, count: torch.Tensor, alloc=(3, 4), fallback_pos: int = 0):
    """Continuation slots per root: returns (branch_pos [R, sum(alloc)], branch_rank [R, sum(alloc)])."""
    L = load_library()
    _dev_2d("idx", idx, torch.int32)
    R, k = idx.shape
    _dev_2d("count", count, torch.int32, (R,))
    if len(alloc) != k:
        raise ValueError("alloc needs one entry per selected rank")
    total = int(sum(alloc))
    host = (ctypes.c_int32 * k)(*[int(x) for x in alloc])
    pos = torch.empty(R, max(total, 1), dtype=torch.int32, device=idx.device)
    rank = torch.empty_like(pos)
    _check(L.hdl_allocate_continuations(idx.data_ptr(), count.data_ptr(), R, k, ctypes.addressof(host),
                                        int(fallback_pos), pos.data_ptr(), rank.data_ptr(),
                                        _stream_handle(idx.device)))
    return pos, rank


@_on_tensor_device
def group_advantages(rewards: torch.Tensor) -> torch.Tensor:
    """A = R - mean over each group (rows of rewards [n_groups, G], fp32)."""
    L = load_library()
    _dev_2d("rewards", rewards, torch.float32)
    n, G = rewards.shape
    adv = torch.empty_like(rewards)
    _check(L.hdl_group_advantages(rewards.data_ptr(), n, G, adv.data_ptr(), _stream_handle(rewards.device)))
    return adv


@_on_tensor_device
def policy_loss_grad(adv: torch.Tensor, traj: torch.Tensor, logp_new: torch.Tensor, logp_old: torch.Tensor, *,
                     loss_mask: Optional[torch.Tensor] = None, pos: Optional[torch.Tensor] = None,
                     start: Optional[torch.Tensor] = None, eps_low: float = 0.2, eps_high: float = 0.28,
                     scale: Optional[float] = None, n_trained: Optional[torch.Tensor] = None):
    """Per-token g = dL/dlog pi of the clipped token-level policy loss and the
    per-token loss.  scale=None: the token-level mean over the trained tokens,
    counted on the device into n_trained (int64 [1], allocated if not given).
    Returns (grad, loss)."""
    L = load_library()
    _dev_2d("adv", adv, torch.float32)
    n = traj.numel()
    _dev_2d("traj", traj, torch.int32, (n,))
    _dev_2d("logp_new", logp_new, torch.float32, (n,))
    _dev_2d("logp_old", logp_old, torch.float32, (n,))
    if loss_mask is not None:
        if loss_mask.dtype == torch.bool:
            loss_mask = loss_mask.view(torch.uint8)
        _dev_2d("loss_mask", loss_mask, torch.uint8, (n,))
    if (pos is None) != (start is None):
        raise ValueError("pos and start go together")
    if pos is not None:
        _dev_2d("pos", pos, torch.int32, (n,))
        _dev_2d("start", start, torch.int32, (adv.numel(),))
    if scale is not None and not scale > 0:
        raise ValueError("scale must be positive (None: token-level mean)")
    if scale is None and n_trained is None:
        n_trained = torch.empty(1, dtype=torch.int64, device=traj.device)
    if n_trained is not None:
        _dev_2d("n_trained", n_trained, torch.int64, (1,))
    grad = torch.empty(n, dtype=torch.float32, device=traj.device)
    loss = torch.empty_like(grad)
    _check(L.hdl_policy_loss_grad(adv.data_ptr(), adv.numel(), traj.data_ptr(), _ptr(pos), _ptr(start),
                                  logp_new.data_ptr(), logp_old.data_ptr(), _ptr(loss_mask), n, float(eps_low),
                                  float(eps_high), 0.0 if scale is None else float(scale), grad.data_ptr(),
                                  loss.data_ptr(), _ptr(n_trained), _stream_handle(traj.device)))
    return grad, loss


@_on_tensor_device
def token_logprobs_noalloc(hidden: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor,
                           mask: Optional[torch.Tensor], logp: torch.Tensor,
                           lse: Optional[torch.Tensor] = None) -> None:
    """hdl_token_logprobs_noalloc: log p (and lse) into caller-given outputs,
    with the library's fixed device scratch instead of a workspace; nothing
    is allocated (usable under graph capture).  Calls on one GPU must not
    overlap.  Arguments as for token_logprobs; logp and lse are fp32 [n_rows]."""
    L = load_library()
    for name, t in (("hidden", hidden), ("w_vocab", w_vocab), ("tokens", tokens), ("logp", logp)):
        _require_cuda(name, t)
    n_rows, d = hidden.shape
    if hidden.dtype != w_vocab.dtype or hidden.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("hidden and w_vocab must both be bfloat16 or both float32")
    if tokens.dtype != torch.int32 or tokens.shape != (n_rows,):
        raise ValueError("tokens must be int32 [n_rows]")
    for name, t in (("logp", logp), ("lse", lse)):
        if t is not None and (t.dtype != torch.float32 or t.shape != (n_rows,)):
            raise ValueError(f"{name} must be float32 [n_rows]")
    if mask is not None:
        _require_cuda("mask", mask)
        if mask.dtype == torch.bool:
            mask = mask.view(torch.uint8)
        if mask.dtype != torch.uint8 or mask.shape != (n_rows,):
            raise ValueError("mask must be uint8 [n_rows]")
    dt = HDL_BF16 if hidden.dtype == torch.bfloat16 else HDL_F32
    _check(L.hdl_token_logprobs_noalloc(hidden.data_ptr(), w_vocab.data_ptr(), tokens.data_ptr(), _ptr(mask),
                                        n_rows, d, w_vocab.shape[0], dt, logp.data_ptr(), _ptr(lse),
                                        _stream_handle(hidden.device)))


def rescore(hidden_both: torch.Tensor, w_vocab: torch.Tensor, tokens: torch.Tensor,
            mask: Optional[torch.Tensor], k: int, *, workspace: Optional[torch.Tensor] = None):
    """The whole hot path for R roots: both contexts' log-probs in one fused
    call, then the divergence score and per-root top-k.

    hidden_both [2, R, T, d] (original context first), tokens [R, T] int32,
    mask [R, T] uint8 or None.  Returns (logp [2, R, T], idx, score, count).
    """
    _, R, T, d = hidden_both.shape
    rows = hidden_both.reshape(2 * R * T, d)
    tok2 = tokens.reshape(1, R * T).expand(2, R * T).reshape(-1)
    m2 = None if mask is None else mask.reshape(1, R * T).expand(2, R * T).reshape(-1)
    logp, _ = token_logprobs(rows, w_vocab, tok2.contiguous(), None if m2 is None else m2.contiguous(),
                             want_lse=False, workspace=workspace)
    lp = logp.view(2, R, T)
    idx, score, count, _ = select_branch_points(lp[0], lp[1], mask, k)
    return lp, idx, score, count


def profile_enable(on: bool = True) -> None:
    _check(load_library().hdl_profile_enable(1 if on else 0))


PROFILE_LMHEAD, PROFILE_GRAD, PROFILE_GEMM, PROFILE_SELECT = 0, 1, 2, 3


def profile_read(kind: int = PROFILE_LMHEAD) -> Tuple[float, int]:
    """(summed milliseconds, launches) of one kernel kind since its last read:
    the fused lm-head kernel (default), its gradient mode, the backward GEMMs,
    or the per-root selection kernel."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(load_library().hdl_profile_read_kind(int(kind), ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)
