"""CSR validation on the device (rsc_csr_validate, RSC_VALIDATE=1) and the
cache backed by torch's caching allocator (rsc_cache_create_ex).

Every malformed input keeps each row's reads inside the arrays (only values
are wrong), so the check itself never reads out of bounds; the
RSC_VALIDATE case uses unsorted columns, which no kernel could turn into an
out-of-bounds access even unchecked."""
import os

import numpy as np
import pytest
import torch

import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


def dev(rowptr, col, val, n_cols):
    return rsc.DeviceCsr.from_host(rowptr, col, val, n_cols)


def first_bad(A):
    with pytest.raises(rsc.RscError) as e:
        rsc.csr_validate(A)
    assert "INVALID_ARGUMENT" in str(e.value) or e.value.status == 1
    import re
    return int(re.search(r"row (\d+)", str(e.value)).group(1))


def base():
    return synth.random_csr(300, 200, 12, seed=3, hub_rows=2, hub_len=150, empty_frac=0.1)


def test_valid_inputs_pass():
    A = base()
    rsc.csr_validate(dev(A.rowptr, A.col, A.val, 200))
    G = synth.make_graph("tiny", 0)
    rsc.csr_validate(dev(G.rowptr, G.col, G.val, G.n))
    rsc.csr_validate(dev(np.zeros(1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), 5))
    rsc.csr_validate(dev(np.zeros(8, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), 5))


def nonempty_rows(A, start):
    return [r for r in range(start, A.n) if A.rowptr[r + 1] - A.rowptr[r] >= 2]


def test_each_malformation_names_its_row():
    A = base()
    r = nonempty_rows(A, 7)[0]
    col = A.col.copy(); col[A.rowptr[r]] = 200                      # column out of range
    assert first_bad(dev(A.rowptr, col, A.val, 200)) == r
    col = A.col.copy(); col[A.rowptr[r] + 1] = -3                   # negative column
    assert first_bad(dev(A.rowptr, col, A.val, 200)) == r
    r = nonempty_rows(A, 20)[0]
    col = A.col.copy(); a = A.rowptr[r]; col[a], col[a + 1] = col[a + 1], col[a]   # unsorted
    assert first_bad(dev(A.rowptr, col, A.val, 200)) == r
    col = A.col.copy(); col[a + 1] = col[a]                         # duplicate
    assert first_bad(dev(A.rowptr, col, A.val, 200)) == r
    r = nonempty_rows(A, 40)[0]
    rp = A.rowptr.copy(); rp[r + 1] = rp[r] - 1 if rp[r] > 0 else rp[r]   # decreasing row pointer
    if rp[r] > 0:
        assert first_bad(dev(rp, A.col, A.val, 200)) == r
    rp = A.rowptr.copy(); rp[0] = 1                                 # rowptr[0] != 0
    assert first_bad(dev(rp, A.col, A.val, 200)) == 0
    # rowptr[n] != nnz (the arrays are longer than rowptr says)
    assert first_bad(dev(A.rowptr, np.concatenate([A.col, [0]]).astype(np.int32),
                         np.concatenate([A.val, [1.0]]).astype(np.float32), 200)) == A.n - 1


def test_validate_env_stops_the_call():
    A = base()
    r = nonempty_rows(A, 30)[0]
    col = A.col.copy(); a = A.rowptr[r]; col[a], col[a + 1] = col[a + 1], col[a]
    bad = dev(A.rowptr, col, A.val, 200)
    B = torch.from_numpy(synth.dense_normal(200, 8, seed=4)).cuda()
    old = os.environ.get("RSC_VALIDATE")
    os.environ["RSC_VALIDATE"] = "1"
    try:
        with pytest.raises(rsc.RscError):
            rsc.spmm(bad, B)
        good = dev(A.rowptr, A.col, A.val, 200)
        Y1 = rsc.spmm(good, B)
    finally:
        if old is None:
            del os.environ["RSC_VALIDATE"]
        else:
            os.environ["RSC_VALIDATE"] = old
    assert torch.equal(Y1, rsc.spmm(good, B))


def test_cache_with_torch_allocator_matches_default():
    G = synth.make_graph("tiny", 0)
    X = dev(G.rowptr, G.col, G.val, G.n)
    B = torch.from_numpy(synth.dense_normal(G.n, 64, seed=5)).cuda()
    import gc
    gc.collect()            # no cyclic garbage from earlier tests may be freed inside the window
    gc.disable()
    try:
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        ct = rsc.Cache(X, X, allocator="torch")
        held = torch.cuda.memory_allocated() - before
        assert held >= G.nnz * 8            # the slice buffers at least
        cd = rsc.Cache(X, X)
        for c in (ct, cd):
            c.refresh(B, G.n // 2, step=0)
        st, sd = rsc.cache_snapshot(ct), rsc.cache_snapshot(cd)
        for key in ("idx", "rowptr", "col"):
            assert np.array_equal(st[key], sd[key])
        assert np.array_equal(st["val"].view(np.uint32), sd["val"].view(np.uint32))
        assert torch.equal(ct.spmm_sampled(B), cd.spmm_sampled(B))
        torch.cuda.synchronize()
        live = torch.cuda.memory_allocated()
        ct.close()                          # returns exactly what it took
        torch.cuda.synchronize()
        assert live - torch.cuda.memory_allocated() == held
        cd.close()
    finally:
        gc.enable()
