"""GPU parity: every hot-path step through the C ABI against the CPU oracle
on the same seeded inputs.

Bars: bit-exact for keys, selected indices, masks and slice structure
(integer work, and fp64 sums whose order is fixed); for fp32 SpMM outputs the
componentwise error relative to |A||B| (max |Y - Y_oracle| / max(S, FLT_MIN),
S = sum |a||b| in fp64) must be <= 1e-5 for exact and <= 1e-4 for sampled
SpMM. The kernel accumulates fp32 over runs of <= 64 entries and folds them
in fp64, so its error is about 64 * 2^-24 * S ~ 4e-6 S in the worst case.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu

FLT_MIN = np.float32(np.finfo(np.float32).tiny)
TOL_EXACT = 1e-5
TOL_SAMPLED = 1e-4


def to_dev(A: synth.Csr, n_cols=None):
    n_cols = A.n if n_cols is None else n_cols
    return rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)


def dense_dev(B: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(B)).cuda()


def rel_err(Y, Yo, S):
    Y = np.asarray(Y, np.float64)
    return float(np.max(np.abs(Y - Yo) / np.maximum(S, FLT_MIN))) if Y.size else 0.0


def padded(rows, d, seed, extra=4):
    ld = (d + 3) // 4 * 4 + extra
    return synth.dense_normal(rows, d, seed=seed, ld=ld), ld


def csr_with_lengths(lengths, n_cols, seed):
    rng = np.random.default_rng(seed)
    rowptr = np.zeros(len(lengths) + 1, np.int64)
    rowptr[1:] = np.cumsum(lengths)
    col = np.concatenate([np.sort(rng.choice(n_cols, size=L, replace=False)) if L else
                          np.zeros(0, np.int64) for L in lengths]).astype(np.int32)
    val = rng.standard_normal(len(col), dtype=np.float32)
    return synth.Csr(len(lengths), rowptr.astype(np.int32), col, val)


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


# ------------------------------------------------------------------ SpMM
SPMM_D = [1, 3, 4, 16, 17, 32, 48, 64, 65, 100, 128, 129, 256, 300, 512, 600, 1030]


@pytest.fixture(scope="module")
def gen_graph():
    # 3000 x 2500, rows 0..40 long, 10 % forced empty, 3 hub rows of 2400
    # entries (> 1024: the multi-wave long-row path)
    return synth.random_csr(3000, 2500, 40, seed=11, hub_rows=3, hub_len=2400, empty_frac=0.1)


@pytest.mark.parametrize("d", SPMM_D)
def test_spmm_general(gen_graph, d):
    A = gen_graph
    B, ld = padded(2500, d, seed=100 + d)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, d=d, with_mag=True)
    Bd = dense_dev(B)
    Y = torch.full((A.n, ld), 7.0, device="cuda")
    rsc.spmm(to_dev(A, 2500), Bd, d=d, out=Y)
    Yh = Y.cpu().numpy()
    assert rel_err(Yh[:, :d], Yo, S) <= TOL_EXACT
    assert np.all(Yh[:, d:] == 7.0)            # padding columns untouched
    empty = np.diff(A.rowptr) == 0
    assert np.all(Yh[empty, :d] == 0.0)


@pytest.fixture
def slice_env(request):
    """Forces the SpMM feature-slice width for one test (the library reads
    RSC_SPMM_SLICE on every call)."""
    import os
    old = os.environ.get("RSC_SPMM_SLICE")
    os.environ["RSC_SPMM_SLICE"] = str(request.param)
    yield request.param
    if old is None:
        del os.environ["RSC_SPMM_SLICE"]
    else:
        os.environ["RSC_SPMM_SLICE"] = old


@pytest.mark.parametrize("slice_env", [16, 32, 64, 128, 256], indirect=True)
@pytest.mark.parametrize("d", [1, 5, 64, 100, 256, 300])
def test_spmm_feature_slices(gen_graph, slice_env, d):
    A = gen_graph
    B, ld = padded(2500, d, seed=200 + d)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, d=d, with_mag=True)
    Y = torch.full((A.n, ld), 7.0, device="cuda")
    rsc.spmm(to_dev(A, 2500), dense_dev(B), d=d, out=Y)
    Yh = Y.cpu().numpy()
    assert rel_err(Yh[:, :d], Yo, S) <= TOL_EXACT
    assert np.all(Yh[:, d:] == 7.0)


@pytest.mark.parametrize("slice_env", [16, 32, 64, 128], indirect=True)
def test_spmm_slices_identity_and_thresholds(slice_env):
    lens = [5, 0, 1100, 64, 1, 1025, 300, 1023, 1024, 63, 65]
    A = csr_with_lengths(lens, 1100, seed=4)
    I = np.eye(1100, dtype=np.float32)
    Y = rsc.spmm(to_dev(A, 1100), dense_dev(I)).cpu().numpy()
    D = np.zeros((len(lens), 1100), np.float32)
    for i in range(len(lens)):
        s, e = A.rowptr[i], A.rowptr[i + 1]
        D[i, A.col[s:e]] = A.val[s:e]
    assert np.array_equal(Y, D)


@pytest.mark.parametrize("slice_env", [16, 32, 64, 128], indirect=True)
def test_sampled_full_budget_bitwise_per_slice(gen_graph, slice_env):
    X = to_dev(gen_graph, 2500)
    cache = rsc.Cache(X, to_dev(synth.transpose(gen_graph, 2500), gen_graph.n))
    B = dense_dev(synth.dense_normal(2500, 256, seed=13))
    cache.refresh(B, 2500, step=0)
    assert np.array_equal(cache.spmm_sampled(B).cpu().numpy().view(np.uint32),
                          rsc.spmm(X, B).cpu().numpy().view(np.uint32))
    cache.close()


def test_spmm_tiny_config():
    A = synth.make_graph("tiny", 0)
    B = synth.dense_normal(A.n, 64, seed=1)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    Y = rsc.spmm(to_dev(A), dense_dev(B)).cpu().numpy()
    assert rel_err(Y, Yo, S) <= TOL_EXACT


def test_spmm_row_length_thresholds():
    # lengths around the run size (64) and the long-row threshold (1024)
    lens = [0, 1, 7, 8, 9, 63, 64, 65, 127, 128, 1023, 1024, 1025, 1100, 2047, 0, 3]
    A = csr_with_lengths(lens, 2100, seed=3)
    for d in (4, 256, 512):
        B = synth.dense_normal(2100, d, seed=5)
        Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
        Y = rsc.spmm(to_dev(A, 2100), dense_dev(B)).cpu().numpy()
        assert rel_err(Y, Yo, S) <= TOL_EXACT


def test_spmm_identity_bitwise():
    # B = I: every output is one product a * 1 plus exact zeros -> dense(A)
    # bitwise, through the long-row path (rows of 1100 > 1024) and d > 512
    lens = [5, 0, 1100, 64, 1, 1025, 300]
    A = csr_with_lengths(lens, 1100, seed=4)
    I = np.eye(1100, dtype=np.float32)
    Y = rsc.spmm(to_dev(A, 1100), dense_dev(I)).cpu().numpy()
    D = np.zeros((len(lens), 1100), np.float32)
    for i in range(len(lens)):
        s, e = A.rowptr[i], A.rowptr[i + 1]
        D[i, A.col[s:e]] = A.val[s:e]
    assert np.array_equal(Y, D)


def test_spmm_permutation_bitwise():
    n = 5000
    p = np.random.default_rng(0).permutation(n).astype(np.int32)
    A = synth.Csr(n, np.arange(n + 1, dtype=np.int32), p, np.ones(n, np.float32))
    B = synth.dense_normal(n, 256, seed=8)
    Y = rsc.spmm(to_dev(A), dense_dev(B)).cpu().numpy()
    assert np.array_equal(Y, B[p])


def test_spmm_deterministic(gen_graph):
    B = dense_dev(synth.dense_normal(2500, 256, seed=9))
    A = to_dev(gen_graph, 2500)
    Y1 = rsc.spmm(A, B).cpu().numpy()
    Y2 = rsc.spmm(A, B).cpu().numpy()
    assert np.array_equal(Y1.view(np.uint32), Y2.view(np.uint32))


@pytest.mark.parametrize("d", [5, 64, 256, 300])
def test_spmm_processing_order_is_bitwise_neutral(gen_graph, d):
    """Taking rows longest class first (RSC_SPMM_ORDER=1) changes only which
    wave takes which row: the result equals the index-order schedule bit for
    bit, also with feature slices."""
    import os
    A = to_dev(gen_graph, 2500)
    Bh, _ = padded(2500, d, seed=19)
    B = dense_dev(Bh)
    old = os.environ.get("RSC_SPMM_ORDER")
    out = {}
    try:
        for mode in ("0", "1"):
            os.environ["RSC_SPMM_ORDER"] = mode
            out[mode] = [rsc.spmm(A, B, d=d).cpu().numpy()]
            for sl in ("32", "64"):
                os.environ["RSC_SPMM_SLICE"] = sl
                out[mode].append(rsc.spmm(A, B, d=d).cpu().numpy())
                del os.environ["RSC_SPMM_SLICE"]
    finally:
        os.environ.pop("RSC_SPMM_SLICE", None)
        if old is None:
            os.environ.pop("RSC_SPMM_ORDER", None)
        else:
            os.environ["RSC_SPMM_ORDER"] = old
    for y0, y1 in zip(out["0"], out["1"]):
        assert np.array_equal(y0.view(np.uint32), y1.view(np.uint32))
    Yo, S = oracle.spmm(gen_graph.rowptr, gen_graph.col, gen_graph.val, Bh, d=d, with_mag=True)
    assert rel_err(out["1"][0], Yo, S) <= TOL_EXACT


def test_spmm_empty():
    A = synth.Csr(5, np.zeros(6, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    Y = rsc.spmm(to_dev(A, 3), dense_dev(np.ones((3, 8), np.float32))).cpu().numpy()
    assert np.all(Y == 0)


def test_degenerate_shapes():
    """No rows; no columns (every row empty, B without rows), also in the
    column-blocked mode; one entry in one column through the cache at k = 0
    and k = 1."""
    A0 = synth.Csr(0, np.zeros(1, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    assert rsc.spmm(to_dev(A0, 5), dense_dev(np.ones((5, 8), np.float32))).shape == (0, 8)
    A1 = synth.Csr(4, np.zeros(5, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    B0 = torch.empty((0, 8), dtype=torch.float32, device="cuda")
    for blocks in (None, "3"):
        old = os.environ.get("RSC_SPMM_BLOCKED")
        if blocks:
            os.environ["RSC_SPMM_BLOCKED"] = blocks
        try:
            Y = torch.full((4, 8), 7.0, device="cuda")
            rsc.spmm(to_dev(A1, 0), B0, out=Y)
            assert not Y.any()
        finally:
            if old is None:
                os.environ.pop("RSC_SPMM_BLOCKED", None)
            else:
                os.environ["RSC_SPMM_BLOCKED"] = old
    A2 = synth.Csr(1, np.array([0, 1], np.int32), np.array([0], np.int32), np.array([0.5], np.float32))
    X = to_dev(A2, 1)
    B = dense_dev(np.full((1, 4), 3.0, np.float32))
    cache = rsc.Cache(X, X)
    cache.refresh(B, 0, step=0)
    assert not cache.spmm_sampled(B).any()
    cache.refresh(B, 1, step=1)
    assert torch.equal(cache.spmm_sampled(B), rsc.spmm(X, B))
    assert torch.equal(rsc.spmm(X, B), torch.full((1, 4), 1.5, device="cuda"))
    cache.close()


@pytest.mark.parametrize("d", [64, 256])
def test_spmm_nonfinite_operands_propagate(d):
    """NaN and +-Inf entries of B reach exactly the output elements whose
    sums contain them (IEEE: NaN spreads, Inf of one sign stays Inf, +Inf
    and -Inf meet as NaN, 0 * Inf is NaN), in the exact product (plan and
    plain call) and the sampled one; the finite elements stay within the
    usual tolerance."""
    n = 3000
    A = synth.random_csr(n, n, 60, seed=77, hub_rows=3, hub_len=2500)
    B = synth.dense_normal(n, d, seed=78)
    rng = np.random.default_rng(79)
    rows = rng.choice(n, 30, replace=False)
    B[rows[:10], rng.integers(0, d, 10)] = np.nan
    B[rows[10:20], rng.integers(0, d, 10)] = np.inf
    B[rows[20:], rng.integers(0, d, 10)] = -np.inf
    B[rows[12], 3] = np.inf                    # the same feature +Inf and -Inf in two rows
    B[rows[22], 3] = -np.inf
    X = to_dev(A)
    Bd = dense_dev(B)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    plan = rsc.SpmmPlan(X)
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    with np.errstate(invalid="ignore"):
        key = oracle.pair_keys(cn2, synth.dense_normal(n, d, seed=80))["key"]
    _, mask = oracle.topk(key, n // 2)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    Yso, Ss = oracle.spmm(ro, co, vo, B, with_mag=True)
    cache = rsc.Cache(X, X)
    cache.refresh(dense_dev(synth.dense_normal(n, d, seed=80)), n // 2, step=0)
    for Y, Yr, Sr, tol in ((rsc.spmm(X, Bd), Yo, S, 1e-5), (plan.run(Bd), Yo, S, 1e-5),
                           (cache.spmm_sampled(Bd), Yso, Ss, 1e-4)):
        Y = Y.cpu().numpy().astype(np.float64)
        assert np.array_equal(np.isnan(Y), np.isnan(Yr))
        assert np.array_equal(np.isposinf(Y), np.isposinf(Yr)) and np.array_equal(np.isneginf(Y), np.isneginf(Yr))
        fin = np.isfinite(Yr) & np.isfinite(Sr)
        assert fin.sum() > Y.size // 2
        assert np.max(np.abs(Y[fin] - Yr[fin]) / np.maximum(Sr[fin], FLT_MIN)) <= tol
    assert np.isnan(Yo).any() and np.isposinf(Yo).any() and np.isneginf(Yo).any()
    plan.close()
    cache.close()


# ------------------------------------------------------------------ scores
def test_col_sqnorms_bitwise(gen_graph):
    AT = synth.transpose(gen_graph, 2500)
    cn2_o, colnnz_o = oracle.col_sqnorms(AT.rowptr, AT.val)
    cn2, colnnz = rsc.col_sqnorms(to_dev(AT, gen_graph.n))
    assert np.array_equal(cn2.cpu().numpy().view(np.uint64), cn2_o.view(np.uint64))
    assert np.array_equal(colnnz.cpu().numpy(), colnnz_o)


@pytest.mark.parametrize("seed", range(4))
def test_col_sqnorms_both_paths_bitwise(seed):
    """Rows walked by their own lane (up to 2,048 entries: 16-byte alignment
    head of 0-3 values, 16-value steps, ragged tails) and rows taken by the
    whole wave (2,049 and more: 64-value loads, four in flight, ragged last
    block), mixed in one 64-row group and alone, with empty rows, values
    spanning many binades (so the sequential fp64 order shows in the last
    bits) and a row starting at every offset modulo 4."""
    rng = np.random.default_rng(100 + seed)
    lens = [0, 1, 2, 3, 4, 15, 16, 17, 31, 32, 33, 47, 48, 2047, 2048, 2049, 2050, 4095, 4096, 4097,
            255, 256, 257, 511, 512, 513, 70_001]
    lens += list(rng.integers(0, 3000, 200)) + [0] * 7 + [int(x) for x in rng.integers(2049, 9000, 5)]
    lens = np.array(lens if seed % 2 == 0 else lens[::-1], dtype=np.int64)
    if seed >= 2:
        lens = rng.permutation(lens)
    rowptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    nnz = int(rowptr[-1])
    val = (rng.standard_normal(nnz) * np.exp2(rng.integers(-40, 40, nnz))).astype(np.float32)
    val[rng.random(nnz) < 0.01] = 0.0
    n = len(lens)
    col = np.zeros(nnz, np.int32)          # cn2 reads rowptr and val only
    cn2_o, cnt_o = oracle.col_sqnorms(rowptr, val)
    AT = rsc.DeviceCsr.from_host(rowptr, col, val, 1)
    for shift in range(4):                # the rows' start offsets modulo 4
        buf = torch.zeros(nnz + 4, dtype=torch.float32, device="cuda")
        buf[shift:shift + nnz] = AT.val
        X = rsc.DeviceCsr(n, 1, AT.rowptr, AT.col, buf[shift:shift + nnz], nnz=nnz)
        cn2, cnt = rsc.col_sqnorms(X)
        assert np.array_equal(cn2.cpu().numpy().view(np.uint64), cn2_o.view(np.uint64)), (seed, shift)
        assert np.array_equal(cnt.cpu().numpy(), cnt_o)


@pytest.mark.parametrize("d", [1, 5, 32, 33, 256, 300])
def test_pair_scores_bitwise(d):
    n = 5000
    rng = np.random.default_rng(d)
    cn2 = rng.random(n) * 3.0
    cn2[::97] = 0.0
    B, ld = padded(n, d, seed=30 + d)
    B[3, 0] = np.nan
    B[4, d - 1] = np.inf
    cn2[5] = 0.0
    B[5, 0] = np.inf                 # 0 * inf -> NaN key
    o = oracle.pair_keys(cn2, B, d=d)
    key, score, rn2 = rsc.pair_scores(torch.from_numpy(cn2).cuda(), dense_dev(B), d=d, with_score=True,
                                      with_rn2=True)
    assert np.array_equal(key.cpu().numpy().view(np.uint64), o["key"])
    assert np.array_equal(rn2.cpu().numpy().view(np.uint64), o["rn2"].view(np.uint64))
    sc = score.cpu().numpy()
    fin = np.isfinite(o["score"])
    assert np.array_equal(np.isnan(sc), np.isnan(o["score"]))
    ulp = np.spacing(np.abs(o["score"][fin]))
    assert np.all(np.abs(sc[fin] - o["score"][fin]) <= ulp)


# ------------------------------------------------------------------ top-k
def _topk_case(key, k):
    idx_o, mask_o = oracle.topk(key, k)
    idx, mask = rsc.topk_select(torch.from_numpy(key.view(np.int64)).cuda(), k)
    assert np.array_equal(idx.cpu().numpy(), idx_o)
    assert np.array_equal(mask.cpu().numpy().view(np.uint32), mask_o)


@pytest.mark.parametrize("n", [1, 31, 32, 33, 4095, 4096, 4097, 50_001])
def test_topk_sizes(n):
    rng = np.random.default_rng(n)
    key = rng.integers(0, 2 ** 63, size=n, dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    for k in sorted({0, 1, n // 3, n // 2, max(n - 1, 0), n}):
        _topk_case(key, k)


def test_topk_ties_nan_inf():
    n = 20_000
    rng = np.random.default_rng(7)
    key = rng.integers(0, 6, size=n).astype(np.uint64) * np.uint64(1 << 52)  # heavy ties, some 0 (NaN)
    for k in (1, 777, 4096, 9999, 19_999):
        _topk_case(key, k)
    _topk_case(np.full(n, 42, np.uint64), 1234)                 # all equal -> [0, k)
    _topk_case(np.arange(n, 0, -1).astype(np.uint64), 500)       # decreasing -> [0, k)
    _topk_case(np.arange(1, n + 1).astype(np.uint64), 500)       # increasing -> [n-k, n)
    top = np.zeros(n, np.uint64)
    top[[5, 19_999, 77]] = np.uint64(0xFFFFFFFFFFFFFFFF)         # max keys first
    _topk_case(top, 3)
    _topk_case(top, 4)


@pytest.mark.parametrize("n", [16383, 16384, 16385])
def test_topk_single_block_boundary(n):
    """Both sides of the one-block path's size limit (16,384 keys), with
    heavy ties, NaN keys and the maximum key."""
    rng = np.random.default_rng(n)
    key = rng.integers(0, 5, size=n).astype(np.uint64) * np.uint64(1 << 60)
    key[::97] = np.uint64(0xFFFFFFFFFFFFFFFF)
    for k in (1, 170, n // 2, n - 1, n):
        _topk_case(key, k)
    _topk_case(np.arange(1, n + 1).astype(np.uint64), 777)


@pytest.mark.parametrize("m", [16384, 16385])
def test_topk_candidates_at_the_cap(m):
    """Keys crowded into the threshold's 22-bit bin after the first two
    radix passes, so the last four passes resolve T among them: exactly m
    keys share that prefix (with ties among them), the rest lie above and
    below it."""
    n = 100_000
    rng = np.random.default_rng(m)
    low = np.uint64((1 << 42) - 1)
    prefix = np.uint64(0x1234A5) << np.uint64(42)
    mid = prefix | (rng.integers(0, 1 << 20, size=m).astype(np.uint64) << np.uint64(22))  # ties in the low bits
    mid[: m // 4] = mid[0]
    rest = n - m
    above = (np.uint64(0x1234A6) + rng.integers(0, 1000, size=rest // 2).astype(np.uint64)) << np.uint64(42)
    below = (np.uint64(0x1234A4) - rng.integers(0, 1000, size=rest - rest // 2).astype(np.uint64)) << np.uint64(42)
    key = np.concatenate([above | (rng.integers(0, 1 << 40, size=rest // 2).astype(np.uint64) & low),
                          mid, below]).astype(np.uint64)
    key = key[rng.permutation(n)]
    for k in (rest // 2 + 1, rest // 2 + m // 8, rest // 2 + m // 2, rest // 2 + m):
        _topk_case(key, k)


def test_topk_on_real_keys():
    A = synth.make_graph("tiny", 0)
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    key = oracle.pair_keys(cn2, synth.dense_normal(A.n, 64, seed=1))["key"]
    _topk_case(key, 2048)


# ------------------------------------------------------------------ slice
def _slice_case(A, n_cols, idx):
    mask = np.zeros((n_cols + 31) // 32, np.uint32)
    for i in idx:
        mask[i >> 5] |= np.uint32(1 << (int(i) & 31))
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    S, nnz = rsc.slice_csr(to_dev(A, n_cols), torch.from_numpy(mask.view(np.int32)).cuda())
    m = int(nnz.item())
    assert m == len(co)
    assert np.array_equal(S.rowptr.cpu().numpy(), ro)
    assert np.array_equal(S.col[:m].cpu().numpy(), co)
    assert np.array_equal(S.val[:m].cpu().numpy().view(np.uint32), vo.view(np.uint32))


def test_slice_bitwise(gen_graph):
    rng = np.random.default_rng(2)
    for k in (0, 1, 100, 750, 2499, 2500):
        _slice_case(gen_graph, 2500, rng.choice(2500, size=k, replace=False))


def test_slice_tiles_and_empty_rows():
    # many empty rows, rows straddling 4096-entry tiles, trailing empty rows
    lens = ([0] * 50 + [4000, 5000, 1, 0, 0, 8191, 4097] + [0] * 20 + [3] * 2000 + [0] * 7)
    A = csr_with_lengths(lens, 9000, seed=6)
    rng = np.random.default_rng(3)
    for k in (0, 1, 4500, 9000):
        _slice_case(A, 9000, rng.choice(9000, size=k, replace=False))


def test_slice_capacity_error():
    A = csr_with_lengths([10, 20, 30], 100, seed=1)
    mask = np.full(4, 0xFFFFFFFF, np.uint32)
    with pytest.raises(rsc.RscError) as e:
        rsc.slice_csr(to_dev(A, 100), torch.from_numpy(mask.view(np.int32)).cuda(), capacity=59)
    assert e.value.status == 4
    S, nnz = rsc.slice_csr(to_dev(A, 100), torch.from_numpy(mask.view(np.int32)).cuda(), capacity=60)
    assert int(nnz.item()) == 60


def test_slice_nnz_zero():
    A = synth.Csr(4, np.zeros(5, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32))
    S, nnz = rsc.slice_csr(to_dev(A, 4), torch.zeros(1, dtype=torch.int32, device="cuda"))
    assert int(nnz.item()) == 0 and not S.rowptr.cpu().numpy().any()


# ------------------------------------------------------------------ cache + sampled SpMM
def test_cache_flow_and_sampled_spmm(gen_graph):
    A = gen_graph
    n_cols = 2500
    AT = synth.transpose(A, n_cols)
    X = to_dev(A, n_cols)
    XT = to_dev(AT, A.n)
    cache = rsc.Cache(X, XT, refresh_interval=10)
    g = cache.get(0)
    assert g["needs_refresh"] and g["version"] == 0
    cn2_o, colnnz_o = oracle.col_sqnorms(AT.rowptr, AT.val)
    B, ld = padded(n_cols, 100, seed=44)
    Bd = dense_dev(B)
    k = 750
    cache.refresh(Bd, k, step=0, d=100)
    snap = rsc.cache_snapshot(cache, step=3)
    assert snap["version"] == 1 and not snap["needs_refresh"] and snap["k"] == k
    assert cache.get(10)["needs_refresh"] and not cache.get(9)["needs_refresh"]
    key_o = oracle.pair_keys(cn2_o, B, d=100)["key"]
    idx_o, mask_o = oracle.topk(key_o, k)
    assert np.array_equal(snap["idx"], idx_o)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask_o)
    assert snap["nnz"] == len(co) == int(colnnz_o[idx_o].sum())
    assert np.array_equal(snap["rowptr"], ro) and np.array_equal(snap["col"], co)
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32))
    # the cached slice is reused with a different dense operand
    B2, _ = padded(n_cols, 100, seed=45)
    Ys = cache.spmm_sampled(dense_dev(B2), d=100).cpu().numpy()
    Yo, S = oracle.spmm(ro, co, vo, B2, d=100, with_mag=True)
    assert rel_err(Ys, Yo, S) <= TOL_SAMPLED
    cache.close()


def test_sampled_full_budget_equals_exact_bitwise(gen_graph):
    A = gen_graph
    X = to_dev(A, 2500)
    cache = rsc.Cache(X, to_dev(synth.transpose(A, 2500), A.n))
    B = dense_dev(synth.dense_normal(2500, 256, seed=12))
    cache.refresh(B, 2500, step=0)
    Ys = cache.spmm_sampled(B).cpu().numpy()
    Y = rsc.spmm(X, B).cpu().numpy()
    assert np.array_equal(Ys.view(np.uint32), Y.view(np.uint32))
    cache.refresh(B, 0, step=10)
    assert np.all(cache.spmm_sampled(B).cpu().numpy() == 0)
    cache.close()


# ------------------------------------------------------------------ full-size workloads
def full_rel_err(Yd, rowptr, col, val, Bh, chunk=250_000):
    """max |Y - Y_oracle| / max(S, FLT_MIN) over EVERY element of Y, the
    oracle run on row chunks (all host threads per chunk)."""
    n = len(rowptr) - 1
    worst = 0.0
    for r0 in range(0, n, chunk):
        rows = np.arange(r0, min(n, r0 + chunk), dtype=np.int32)
        Yo, S = oracle.spmm(rowptr, col, val, Bh, rows=rows, with_mag=True)
        got = Yd[r0:r0 + len(rows)].cpu().numpy()
        worst = max(worst, rel_err(got, Yo, S))
        del Yo, S, got
    return worst


@pytest.mark.parametrize("name,d,pcts", [("copurchase", 256, (10, 30, 50)), ("social", 256, (10, 30, 50)),
                                         ("protein", 256, (10, 30, 50)), ("gcn2", 100, (10, 30)),
                                         ("gcn2", 512, (10, 50)), ("protein", 32, (30,)),
                                         ("protein", 16, (30,)), ("social", 32, (30,))])
def test_full_workload(name, d, pcts):
    """The benchmark workloads at full size, in the configurations the
    benchmark times and at 10 / 30 / 50 % budgets (which change the sampled
    products' layouts: feature-slice width, column blocking; gcn2 also at the
    training step's d = 100; protein at d = 16 and 32, whose exact products
    run column-blocked in the 16- and 32-float layouts, and social at d = 32,
    which the blocking rule leaves unblocked): every element of the exact and the sampled products
    against the oracle; keys, selected indices, mask and slice bit-exact over
    the whole graph; the plan's product bitwise equal to rsc_spmm."""
    A = synth.make_graph(name, 0)
    n = A.n
    Bh = synth.dense_normal(n, d, seed=1)
    X = to_dev(A)
    Bd = dense_dev(Bh)
    Y = rsc.spmm(X, Bd)
    plan = rsc.SpmmPlan(X)      # hinted column copy on the wide operands (copurchase, gcn2)
    assert torch.equal(plan.run(Bd), Y)
    plan.close()
    err = full_rel_err(Y, A.rowptr, A.col, A.val, Bh)
    print(f"[full] {name} d={d} exact: max rel err {err:.3e} over {n * d} elements", flush=True)
    assert err <= TOL_EXACT
    del Y

    cn2, colnnz = oracle.col_sqnorms(A.rowptr, A.val)
    key_o = oracle.pair_keys(cn2, Bh)["key"]
    cache = rsc.Cache(X, X, refresh_interval=10)
    for pct in pcts:
        k = (n * pct) // 100
        cache.refresh(Bd, k, step=0)
        snap = rsc.cache_snapshot(cache)
        key_g = rsc.copy_to_host(cache.buffers()[2], n, np.uint64)
        assert np.array_equal(key_g, key_o)
        idx_o, mask_o = oracle.topk(key_o, k)
        assert np.array_equal(snap["idx"], idx_o)
        mask_g = rsc.copy_to_host(cache.buffers()[4], (n + 31) // 32, np.uint32)
        assert np.array_equal(mask_g, mask_o)
        ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask_o)
        assert snap["nnz"] == len(co)
        assert np.array_equal(snap["rowptr"], ro)
        assert np.array_equal(snap["col"], co)
        assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32))
        Ys = cache.spmm_sampled(Bd)
        err = full_rel_err(Ys, ro, co, vo, Bh)
        print(f"[full] {name} d={d} {pct}%: sampled max rel err {err:.3e}", flush=True)
        assert err <= TOL_SAMPLED
        del Ys
    cache.close()
