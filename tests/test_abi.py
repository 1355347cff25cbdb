"""The C ABI without a GPU: the library loads, exports every function that
include/hdl.h declares, and rejects bad arguments synchronously (argument
checks run before any HIP call)."""
import ctypes
import os
import re

import pytest

import paper_2609_36864_amd as hdl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hdl.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hdl_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hdl.library_path()):
        pytest.fail("libhdl.so is not built (run __graft_entry__.build())")
    return hdl.load_library()


def test_header_declares_the_boundary():
    names = _declared_functions()
    for n in ("hdl_token_logprobs", "hdl_token_logprobs_entropy", "hdl_select_branch_points",
              "hdl_select_top_k", "hdl_token_logprobs_workspace_size", "hdl_status_string",
              "hdl_last_hip_error", "hdl_token_logprobs_backward", "hdl_token_logprobs_backward_workspace_size",
              "hdl_select_constrained", "hdl_allocate_continuations", "hdl_group_advantages",
              "hdl_policy_loss_grad", "hdl_profile_enable", "hdl_profile_read", "hdl_profile_read_kind"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for n in _declared_functions():
        assert hasattr(lib, n), f"{n} declared in hdl.h but not exported"


def test_status_strings(lib):
    assert lib.hdl_status_string(0) == b"ok"
    for s in (-1, -2, -3, -4):
        assert lib.hdl_status_string(s) not in (b"ok", b"unknown status")
    assert lib.hdl_abi_version() == 6


def test_workspace_size_rules(lib):
    f = lib.hdl_token_logprobs_workspace_size
    assert f(0, 64, 100, 1) == 0 and f(10, 0, 100, 1) == 0 and f(10, 64, 0, 1) == 0
    assert f(10, 64, 100, 7) == 0
    a = f(1000, 64, 151936, 1)
    b = f(100000, 64, 151936, 1)
    assert 0 < a < b
    assert f(65536, 2048, 151936, 1) % 256 == 0


def test_logprobs_argument_errors(lib):
    call = lib.hdl_token_logprobs
    p = ctypes.c_void_p(4096)       # never dereferenced: validation fails first
    assert call(None, p, p, None, 4, 64, 10, 1, p, None, p, 1 << 20, None) == -1
    assert b"null" in lib.hdl_last_hip_error()
    assert call(p, p, p, None, 0, 64, 10, 1, p, None, p, 1 << 20, None) == -1
    assert call(p, p, p, None, 4, 64, 10, 5, p, None, p, 1 << 20, None) == -2
    assert call(p, p, p, None, 4, 12, 10, 1, p, None, p, 1 << 20, None) == -2
    assert call(ctypes.c_void_p(4100), p, p, None, 4, 64, 10, 1, p, None, p, 1 << 20, None) == -1
    assert call(p, p, p, None, 4, 64, 10, 1, p, None, p, 16, None) == -3
    assert call(p, p, p, None, 4, 64, 10, 1, p, None, None, 1 << 20, None) == -3
    assert call(p, p, p, None, 4, 64, 10, 1, p, None, ctypes.c_void_p(4096 + 128), 1 << 20, None) == -1


def test_select_argument_errors(lib):
    call = lib.hdl_select_branch_points
    p = ctypes.c_void_p(4096)
    assert call(None, p, None, 1, 10, 2, p, p, p, None, None) == -1
    assert call(p, p, None, 0, 10, 2, p, p, p, None, None) == -1
    assert call(p, p, None, 1, 10, 0, p, p, p, None, None) == -1
    assert call(p, p, None, 1, 10, 1025, p, p, p, None, None) == -2
    assert b"1025" in lib.hdl_last_hip_error()


def test_entropy_and_value_topk_argument_errors(lib):
    p = ctypes.c_void_p(4096)
    f = lib.hdl_token_logprobs_entropy
    assert f(p, p, p, None, 4, 64, 10, 1, p, None, None, p, 1 << 20, None) == -1   # null entropy
    assert f(None, p, p, None, 4, 64, 10, 1, p, None, p, p, 1 << 20, None) == -1
    assert f(p, p, p, None, 4, 12, 10, 1, p, None, p, p, 1 << 20, None) == -2
    g = lib.hdl_select_top_k
    assert g(None, None, 1, 10, 2, p, p, p, None) == -1
    assert g(p, None, 1, 10, 0, p, p, p, None) == -1
    assert g(p, None, 1, 10, 1025, p, p, p, None) == -2


def test_backward_workspace_and_argument_errors(lib):
    ws = lib.hdl_token_logprobs_backward_workspace_size
    ws.restype = ctypes.c_size_t
    ws.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
    # one chunk of G dominates: 2 * round_up(rows, 256) * round_up(V, 64) bytes,
    # plus the gathered hidden rows (2 * 1024 * d) and the dH partials (4 * splits * 1024 * d)
    n, d, V = 1000, 64, 1000
    size = ws(n, d, V, 1)
    assert size >= 2 * 1024 * 1024 + 2 * 1024 * d and size < 2 * 1024 * 1024 + 40 * 1024 * d
    assert ws(n, d, 1 << 23, 1) > 0 and ws(n, d, (1 << 30) + 1, 1) == 0   # vocabulary limit
    # G is held for one chunk of at most 32768 rows: more rows only lengthen the row list
    assert 0 < ws(100000, d, V, 1) - ws(32768, d, V, 1) < 4 * 100000
    # rows are taken in blocks whose hidden states span at most 4 GiB, so the
    # row list stops growing at 2^32 / (2 d) rows
    assert ws(600000, 4096, V, 1) == ws(524288, 4096, V, 1) > ws(524287 - 32768, 4096, V, 1)
    assert ws(n, (1 << 23) + 8, V, 1) == 0
    assert ws(n, d, V, 0) == 0          # fp32 inputs are not supported
    assert ws(n, 12, V, 1) == 0         # d not a multiple of 8
    assert ws(0, d, V, 1) == 0
    f = lib.hdl_token_logprobs_backward
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p] * 6 + [ctypes.c_int64] * 3 + [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                                                 ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t,
                                                                 ctypes.c_void_p]
    p = ctypes.c_void_p(4096)
    assert f(p, p, p, None, p, None, n, d, V, 1, p, p, 0, p, size, None) == -1   # null grad_logp
    assert f(p, p, p, None, p, p, n, d, V, 0, p, p, 0, p, size, None) == -2      # fp32
    assert f(p, p, p, None, p, p, n, d, V, 1, p, p, 0, p, size - 256, None) == -3
    assert f(p, p, p, None, p, p, n, d, V, 1, p, p, 0, ctypes.c_void_p(4096 + 16), size, None) == -1


def test_group_construction_argument_errors(lib):
    p = ctypes.c_void_p(4096)
    sc = lib.hdl_select_constrained
    sc.restype = ctypes.c_int
    sc.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_int32, ctypes.c_int] + [ctypes.c_void_p] * 4
    assert sc(None, None, None, 1, 10, 2, None, None, 0, 0, p, p, p, None) == -1
    assert sc(p, None, None, 1, 10, 2000, None, None, 0, 0, p, p, p, None) == -2
    assert sc(p, None, None, 1, 10, 2, None, None, -1, 0, p, p, p, None) == -1
    al = lib.hdl_allocate_continuations
    al.restype = ctypes.c_int
    al.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                   ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    neg = (ctypes.c_int32 * 2)(3, -1)
    zero = (ctypes.c_int32 * 2)(0, 0)
    assert al(p, p, 4, 2, ctypes.addressof(neg), 0, p, None, None) == -1
    assert al(p, p, 4, 2, ctypes.addressof(zero), 0, p, None, None) == -1
    assert al(p, p, 4, 17, ctypes.addressof(zero), 0, p, None, None) == -2
    ga = lib.hdl_group_advantages
    ga.restype = ctypes.c_int
    ga.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    assert ga(p, 0, 16, p, None) == -1 and ga(None, 4, 16, p, None) == -1
    pg = lib.hdl_policy_loss_grad
    pg.restype = ctypes.c_int
    pg.argtypes = [ctypes.c_void_p, ctypes.c_int64] + [ctypes.c_void_p] * 6 + [ctypes.c_int64, ctypes.c_float,
                                                                                ctypes.c_float, ctypes.c_float,
                                                                                ctypes.c_void_p, ctypes.c_void_p,
                                                                                ctypes.c_void_p, ctypes.c_void_p]
    assert pg(p, 4, p, p, None, p, p, None, 10, 0.2, 0.28, 1.0, p, None, None, None) == -1   # pos without start
    assert pg(p, 4, p, None, None, p, p, None, 10, -0.2, 0.28, 1.0, p, None, None, None) == -1
    # the token-level mean (scale <= 0) needs the device count; NaN scale
    assert pg(p, 4, p, None, None, p, p, None, 10, 0.2, 0.28, 0.0, p, None, None, None) == -1
    assert b"n_trained" in lib.hdl_last_hip_error()
    assert pg(p, 4, p, None, None, p, p, None, 10, 0.2, 0.28, float("nan"), p, None, p, None) == -1
    assert pg(p, 4, p, None, None, p, p, None, 10, 0.2, 0.28, 0.0, p, None, ctypes.c_void_p(0x1004), None) == -1


def test_binding_rejects_host_tensors_before_any_launch():
    import torch
    import paper_2609_36864_amd as hdl
    h = torch.zeros(4, 64, dtype=torch.bfloat16)
    w = torch.zeros(10, 64, dtype=torch.bfloat16)
    y = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(ValueError):
        hdl.token_logprobs(h, w, y)
    with pytest.raises(ValueError):
        hdl.select_top_k(torch.zeros(2, 8), None, 2)
    with pytest.raises(ValueError):
        hdl.group_advantages(torch.zeros(2, 4))


def test_noalloc_argument_checks_before_any_hip_call(lib):
    f = lib.hdl_token_logprobs_noalloc
    p = 0x1000   # never dereferenced: every call below fails its checks first
    assert f(None, p, p, None, 10, 64, 100, 1, p, None, None) == -1
    assert f(p, p, p, None, 0, 64, 100, 1, p, None, None) == -1
    assert f(p, p, p, None, 10, 60, 100, 1, p, None, None) == -2
    assert f(p, p, p, None, 10, 64, 100, 9, p, None, None) == -2
    # 3 million rows of d = 8 would need 48 MB of the library's 32 MiB array
    assert f(p, p, p, None, 3_000_000, 8, 1000, 1, p, None, None) == -2
    assert b"scratch" in lib.hdl_last_hip_error()


def test_profile_kinds(lib):
    # every timing kind the header names reads back (nothing pending: zero
    # launches, no HIP call); kinds outside the enumeration are rejected
    ms = ctypes.c_double(-1.0)
    n = ctypes.c_int64(-1)
    for kind in (hdl.PROFILE_LMHEAD, hdl.PROFILE_GRAD, hdl.PROFILE_GEMM, hdl.PROFILE_SELECT):
        assert lib.hdl_profile_read_kind(kind, ctypes.byref(ms), ctypes.byref(n)) == 0
        assert n.value == 0 and ms.value == 0.0
    for kind in (-1, 4):
        assert lib.hdl_profile_read_kind(kind, ctypes.byref(ms), ctypes.byref(n)) < 0
