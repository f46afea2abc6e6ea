"""Destroying a plan or a cache waits for that handle's own work only: work
queued on another stream is still running when the destroy call returns
(host-side check with an event query, no forced hang)."""
import numpy as np
import pytest
import torch

import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


def _busy_other_stream():
    """About a quarter second of matrix products on a second stream; returns
    the stream and an event recorded after them."""
    s2 = torch.cuda.Stream()
    M = torch.randn(8192, 8192, device="cuda")
    torch.cuda.synchronize()
    with torch.cuda.stream(s2):
        x = M
        for _ in range(20):
            x = torch.mm(M, x) * 1e-4
        ev = torch.cuda.Event()
        ev.record(s2)
    return s2, ev, x


def _graph():
    A = synth.erdos_renyi(3000, 12.0 / 2999, seed=4)
    B = torch.from_numpy(synth.dense_normal(3000, 64, seed=5)).cuda()
    return rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 3000), B


@pytest.mark.parametrize("kind", ["cache", "cache_torch_alloc", "plan"])
def test_destroy_leaves_other_streams_running(kind):
    X, B = _graph()
    if kind == "plan":
        h = rsc.SpmmPlan(X)
        Y = h.run(B)
    else:
        h = rsc.Cache(X, X, allocator="torch" if kind == "cache_torch_alloc" else None)
        h.refresh(B, 1500, step=0)
        Y = h.spmm_sampled(B)
    torch.cuda.current_stream().synchronize()
    _, ev, _ = _busy_other_stream()
    assert not ev.query()          # the other stream's products have not finished yet
    h.close()
    still_running = not ev.query()
    torch.cuda.synchronize()
    assert still_running, kind
    assert torch.isfinite(Y).all()


def test_destroy_waits_for_its_own_stream():
    # the handle's work on a side stream is complete once destroy returns
    X, B = _graph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        cache = rsc.Cache(X, X)
        cache.refresh(B, 1000, step=0)
        Y = cache.spmm_sampled(B)
        ev = torch.cuda.Event()
        ev.record(s)
        cache.close()
    assert ev.query()
    Y2 = rsc.spmm(X, B)
    torch.cuda.synchronize()
    assert Y.shape == Y2.shape
