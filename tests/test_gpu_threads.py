"""Host threads, each with its own stream, plan and cache, running exact
products, refreshes and sampled products at the same time (ctypes releases
the interpreter lock during each library call): every result equals, bit
for bit, the one the same calls give when run alone. The library's shared
state (the error text is per thread; the per-device free stream and the
pinned-word pool are taken under locks) must not mix the threads' work."""
import threading

import numpy as np
import pytest
import torch

import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


def _case(i):
    rng = np.random.default_rng(900 + i)
    n = 20_000 + 7_000 * i
    A = synth.bucket_csr(np.minimum(rng.integers(1, 120, n), n), n, seed=900 + i)
    B = synth.dense_normal(n, 64 + 32 * i, seed=950 + i)
    return A, B


def _run(A, B, n, steps, out):
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    Bd = torch.from_numpy(B).cuda()
    plan = rsc.SpmmPlan(X)
    cache = rsc.Cache(X, X, refresh_interval=2)
    res = []
    for s in range(steps):
        Y = plan.run(Bd)
        if cache.get(s, with_slice=False)["needs_refresh"]:
            cache.refresh(Bd * (1.0 + 0.25 * s), n // (3 + s % 2), step=s)
        Ys = cache.spmm_sampled(Bd)
        res.append((Y.clone(), Ys.clone()))
    torch.cuda.current_stream().synchronize()
    out.extend((a.cpu().numpy(), b.cpu().numpy()) for a, b in res)
    cache.close()
    plan.close()


def test_concurrent_threads_match_sequential_runs():
    cases = [_case(i) for i in range(4)]
    steps = 5
    alone = []
    for A, B in cases:
        out = []
        _run(A, B, len(A.rowptr) - 1, steps, out)
        alone.append(out)
    results = [[] for _ in cases]
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                A, B = cases[i]
                _run(A, B, len(A.rowptr) - 1, steps, results[i])
        except Exception as e:  # reported below, on the main thread
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker did not finish"
    assert not errors, errors
    for i in range(len(cases)):
        assert len(results[i]) == steps
        for (y, ys), (y0, ys0) in zip(results[i], alone[i]):
            assert np.array_equal(y.view(np.uint32), y0.view(np.uint32)), i
            assert np.array_equal(ys.view(np.uint32), ys0.view(np.uint32)), i
