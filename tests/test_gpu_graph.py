"""The exact and the sampled SpMM captured in a HIP graph (through torch's
graph capture on the current stream): each replay must equal the eager call
bitwise, with eager work, new operand contents and a cache refresh between
replays. Only kernel launches are captured (no memset, no host sync)."""
import numpy as np
import pytest
import torch

import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


@pytest.mark.parametrize("name,d", [("tiny", 64), ("gcn2", 100)])
def test_graph_replays_match_eager(name, d):
    A = synth.make_graph(name, 0)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
    ws = torch.empty(rsc.spmm_workspace_bytes(X), dtype=torch.uint8, device="cuda")
    cache = rsc.Cache(X, X)
    H = torch.from_numpy(synth.dense_normal(A.n, d, seed=1)).cuda()
    Gm = torch.from_numpy(synth.dense_normal(A.n, d, seed=3)).cuda()
    k = A.n * 3 // 10
    cache.refresh(Gm, k, step=0)
    Y = rsc.spmm(X, H, ws=ws)
    Yb = cache.spmm_sampled(Gm)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        rsc.spmm(X, H, out=Y, ws=ws)          # warm-up on the capture stream
        cache.spmm_sampled(Gm, out=Yb)
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        rsc.spmm(X, H, out=Y, ws=ws)
        cache.spmm_sampled(Gm, out=Yb)
    for r in range(4):
        H.copy_(torch.from_numpy(synth.dense_normal(A.n, d, seed=10 + r)).cuda())
        Gm.mul_(1.5)                          # eager work between replays
        if r == 2:
            cache.refresh(Gm, k, step=10)     # new slice contents, same buffers and k
        g.replay()
        torch.cuda.synchronize()
        want_y = rsc.spmm(X, H)
        want_b = cache.spmm_sampled(Gm)
        torch.cuda.synchronize()
        assert torch.equal(Y, want_y), f"exact, replay {r}"
        assert torch.equal(Yb, want_b), f"sampled, replay {r}"
    del g
    cache.close()


def test_graph_replays_blocked_mode():
    """The column-blocked SpMM (forced to 4 ranges) captured and replayed:
    split, long-piece list, row and combine kernels, all launch-only."""
    import os
    old = os.environ.get("RSC_SPMM_BLOCKED")
    os.environ["RSC_SPMM_BLOCKED"] = "4"
    try:
        A = synth.make_graph("tiny", 0)
        X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
        ws = torch.empty(rsc.spmm_workspace_bytes(X), dtype=torch.uint8, device="cuda")
        H = torch.from_numpy(synth.dense_normal(A.n, 96, seed=2)).cuda()
        Y = rsc.spmm(X, H, ws=ws)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            rsc.spmm(X, H, out=Y, ws=ws)
        torch.cuda.current_stream().wait_stream(s)
        with torch.cuda.graph(g):
            rsc.spmm(X, H, out=Y, ws=ws)
        for r in range(3):
            H.copy_(torch.from_numpy(synth.dense_normal(A.n, 96, seed=20 + r)).cuda())
            g.replay()
            torch.cuda.synchronize()
            want = rsc.spmm(X, H)
            torch.cuda.synchronize()
            assert torch.equal(Y, want), f"replay {r}"
        del g
    finally:
        if old is None:
            del os.environ["RSC_SPMM_BLOCKED"]
        else:
            os.environ["RSC_SPMM_BLOCKED"] = old


def test_graph_replays_plan_run():
    """An SpMM plan's run (its own workspace, no allocation) captured and
    replayed, on an operand wide enough for the hinted column copy."""
    rng = np.random.default_rng(4)
    n_rows, n_cols = 4000, 300_000
    A = synth.bucket_csr(rng.integers(0, 400, n_rows), n_cols, seed=5)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    plan = rsc.SpmmPlan(X)
    H = torch.from_numpy(synth.dense_normal(n_cols, 512, seed=6)).cuda()
    Y = plan.run(H)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        plan.run(H, out=Y)
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        plan.run(H, out=Y)
    for r in range(3):
        H.mul_(-0.5)
        g.replay()
        torch.cuda.synchronize()
        want = rsc.spmm(X, H)
        torch.cuda.synchronize()
        assert torch.equal(Y, want), f"replay {r}"
    del g
    plan.close()
