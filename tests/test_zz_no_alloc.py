"""rsc_spmm_noalloc: the exact SpMM with its scratch in a static device array
instead of a workspace. Checked through the C ABI against rsc_spmm (bitwise
where both take the same mode) and against the oracle, on consecutive calls
whose second input is smaller (the scratch keeps the previous call's
contents, so anything the call fails to clear would show up there)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu
FLT_MIN = np.float32(np.finfo(np.float32).tiny)


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


def rel_err(Y, Yo, S):
    return float(np.max(np.abs(np.asarray(Y, np.float64) - Yo) / np.maximum(S, FLT_MIN))) if Yo.size else 0.0


def _case(lens, n_cols, d, seed):
    A = synth.bucket_csr(lens, n_cols, seed=seed)
    B = synth.dense_normal(n_cols, d, seed=seed + 1)
    return A, B


def _both(A, B, n_cols):
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    Bd = torch.from_numpy(B).cuda()
    Yn = rsc.spmm_noalloc(X, Bd)
    Yw = rsc.spmm(X, Bd)
    torch.cuda.synchronize()
    return Yn.cpu().numpy(), Yw.cpu().numpy()


def test_consecutive_calls_match_rsc_spmm():
    rng = np.random.default_rng(77)
    # 1: long rows on average (length-class order, long-row blocks), d = 256
    lens1 = rng.integers(100, 300, 6000)
    lens1[rng.choice(6000, 60, replace=False)] = rng.integers(1100, 5000, 60)
    # 2: smaller, short rows only (no long-row pass), d = 64, a few empty rows
    lens2 = rng.integers(0, 40, 700)
    lens2[::50] = 0
    for lens, n_cols, d, seed in ((lens1, 6000, 256, 3), (lens2, 900, 64, 5)):
        A, B = _case(lens, n_cols, d, seed)
        Yn, Yw = _both(A, B, n_cols)
        assert np.array_equal(Yn.view(np.uint32), Yw.view(np.uint32)), (len(lens), d)
        Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
        assert rel_err(Yn, Yo, S) <= 1e-5, (len(lens), d)


def test_blocked_product_in_scratch_and_unblocked_fallback():
    # 100 rows x 10,000 entries over 40,000 columns: rsc_spmm takes 3 column
    # ranges, whose buffers fit the static scratch -> bitwise equal
    A, B = _case(np.full(100, 10_000), 40_000, 96, 31)
    Yn, Yw = _both(A, B, 40_000)
    assert np.array_equal(Yn.view(np.uint32), Yw.view(np.uint32))
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    assert rel_err(Yn, Yo, S) <= 1e-5
    # 70,000 rows over 20,000 columns: rsc_spmm takes 2 ranges, whose partial
    # rows (35.8 MB) exceed the scratch -> the unblocked product, same tolerance
    rng = np.random.default_rng(12)
    A, B = _case(rng.integers(150, 260, 70_000), 20_000, 128, 41)
    Yn, Yw = _both(A, B, 20_000)
    rows = np.arange(0, 70_000, 37, dtype=np.int32)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, rows=rows, with_mag=True)
    assert rel_err(Yn[rows], Yo, S) <= 1e-5
    assert rel_err(Yw[rows], Yo, S) <= 1e-5
    # a smaller call after it still matches
    A, B = _case(rng.integers(0, 30, 300), 300, 32, 43)
    Yn, Yw = _both(A, B, 300)
    assert np.array_equal(Yn.view(np.uint32), Yw.view(np.uint32))


def test_rejects_products_beyond_the_scratch():
    L = rsc.lib()
    s = rsc.CsrStruct(9_000_000, 1000, 0, 0x1000, 0, 0)   # 9M rows: 36 MB of row list
    Y = torch.empty((1, 4), device="cuda")
    B = torch.empty((1000, 4), device="cuda")
    st = L.rsc_spmm_noalloc(ctypes.byref(s), B.data_ptr(), 4, 4, Y.data_ptr(), 4, None)
    assert st == 4  # RSC_ERR_CAPACITY, nothing launched
    assert b"static scratch" in L.rsc_last_error()


def test_captured_in_a_graph_and_replayed():
    # the callers it is for: code under graph capture. Each replay (new
    # operand contents, eager work between) equals the eager rsc_spmm bitwise.
    A = synth.make_graph("gcn2", 0)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
    H = torch.from_numpy(synth.dense_normal(A.n, 100, seed=1)).cuda()
    Y = torch.empty((A.n, 100), device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        rsc.spmm_noalloc(X, H, out=Y)           # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        rsc.spmm_noalloc(X, H, out=Y)
    for r in range(3):
        H.copy_(torch.from_numpy(synth.dense_normal(A.n, 100, seed=20 + r)).cuda())
        H.mul_(1.0 + r)                          # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        want = rsc.spmm(X, H)
        torch.cuda.synchronize()
        assert torch.equal(Y, want), f"replay {r}"
    del g
