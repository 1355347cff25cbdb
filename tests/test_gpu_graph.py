"""The re-scoring path and the backward pass under HIP graph capture: the
library allocates, clears with memset and synchronises nothing inside a
call, so the fused lm-head kernel, the merge, the selection and the backward
kernels (gradient-mode lm-head, row gather, the two GEMMs, the split sum)
can be captured once and replayed.  Every replay (with other eager work and
synchronisations in between) must reproduce the eager result bit for bit,
including after the inputs change in place."""
import pytest
import torch

import workloads
from tests.gpu_helpers import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hdl():
    return require_gpu()


def test_graph_replays_match_eager(hdl):
    w = workloads.make_workload("c2", R=2, T=700, d=256, V=9000)
    c = w.cfg
    dev = "cuda"
    hidden = w.rows_hidden().to(dev)
    W = w.W.to(dev)
    tokens = w.rows_tokens().to(dev)
    mask = w.rows_mask().to(dev)
    mask_rt = w.mask.to(dev)
    n = hidden.shape[0]
    ws = torch.empty(hdl.workspace_size(n, c.d, c.V, hdl.HDL_BF16), dtype=torch.uint8, device=dev)
    logp = torch.empty(n, dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)

    def step():
        hdl.token_logprobs(hidden, W, tokens, mask, logp=logp, lse=lse, workspace=ws)
        lp = logp.view(2, c.R, c.T)
        return hdl.select_branch_points(lp[0], lp[1], mask_rt, c.k, want_delta=True)

    eager = [t.clone() for t in step()]
    eager_lp = logp.clone()
    torch.cuda.synchronize()

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                                  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = step()
    torch.cuda.synchronize()

    for rep in range(3):
        logp.fill_(123.0)                       # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(logp.view(torch.int32), eager_lp.view(torch.int32)), f"replay {rep}: log p"
        for a, b in zip(outs, eager):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), f"replay {rep}: selection"

    # new inputs written in place: the replay follows them
    hidden[: c.R * c.T].copy_(hidden[c.R * c.T:])            # original := hindsight
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    idx, score, count, delta = outs
    assert torch.all(delta == 0) and torch.all(score == 0)


def test_backward_graph_replays_match_eager(hdl):
    g = torch.Generator().manual_seed(77)
    n, d, V = 700, 128, 3000
    dev = "cuda"
    hidden = torch.randn(n, d, generator=g).to(torch.bfloat16).to(dev)
    W = (torch.randn(V, d, generator=g) * 0.05).to(torch.bfloat16).to(dev)
    tokens = torch.randint(0, V, (n,), generator=g, dtype=torch.int32).to(dev)
    mask = (torch.rand(n, generator=g) < 0.8).to(torch.uint8).to(dev)
    up = torch.randn(n, generator=g).to(dev)
    ws_f = torch.empty(hdl.workspace_size(n, d, V, hdl.HDL_BF16), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(hdl.backward_workspace_size(n, d, V), dtype=torch.uint8, device=dev)
    logp = torch.empty(n, dtype=torch.float32, device=dev)
    lse = torch.empty(n, dtype=torch.float32, device=dev)
    grad_w = torch.empty(V, d, dtype=torch.float32, device=dev)

    def step():
        hdl.token_logprobs(hidden, W, tokens, mask, logp=logp, lse=lse, workspace=ws_f)
        dh, _ = hdl.token_logprobs_backward(hidden, W, tokens, mask, lse, up, grad_w=grad_w, workspace=ws_b)
        return dh

    eager_dh = step().clone()
    eager_dw = grad_w.clone()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dh = step()
    torch.cuda.synchronize()
    for rep in range(3):
        grad_w.fill_(5.0)
        dh.fill_(-1.0)
        ws_b.fill_(0xFF)                        # stale workspace: NaN bit patterns everywhere
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(dh.view(torch.int32), eager_dh.view(torch.int32)), f"replay {rep}: dH"
        assert torch.equal(grad_w.view(torch.int32), eager_dw.view(torch.int32)), f"replay {rep}: dW"
    # new upstream gradient written in place: the replay follows it
    up.mul_(-2.0)
    graph.replay()
    torch.cuda.synchronize()
    want_dh, _ = hdl.token_logprobs_backward(hidden, W, tokens, mask, lse, up, workspace=ws_b)
    torch.cuda.synchronize()
    assert torch.equal(dh.view(torch.int32), want_dh.view(torch.int32))
