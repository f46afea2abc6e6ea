"""Seeded random shapes through the whole path against the oracle: CSR
sizes, row-length mixes (empty rows, rows around the 64-entry run and the
1024-entry long-row threshold, rows longer than the column count allows
are clipped), feature widths and leading dimensions, budgets including
k = 0 and k = n. Exact SpMM within 1e-5, keys / selection / slice bit for
bit, sampled SpMM within 1e-4."""
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


def case(seed):
    rng = np.random.default_rng(1000 + seed)
    n_rows = int(rng.integers(1, 3000))
    n_cols = int(rng.integers(1, 2600))
    kinds = rng.choice(["short", "runs", "long", "empty"], size=n_rows, p=[0.6, 0.25, 0.05, 0.1])
    lens = np.where(kinds == "short", rng.integers(0, 20, n_rows),
                    np.where(kinds == "runs", rng.integers(60, 200, n_rows),
                             np.where(kinds == "long", rng.integers(1000, 2600, n_rows), 0)))
    lens = np.minimum(lens, n_cols)
    A = synth.bucket_csr(lens, n_cols, seed=seed)
    d = int(rng.choice([1, 3, 4, 17, 64, 100, 256, 300, 513]))
    ld = (d + 3) // 4 * 4 + 4 * int(rng.integers(0, 3))
    k = int(rng.choice([0, 1, n_cols // 3, n_cols]))
    return A, n_cols, d, ld, k


@pytest.mark.parametrize("seed", range(24))
def test_random_shape(seed):
    A, n_cols, d, ld, k = case(seed)
    B = synth.dense_normal(n_cols, d, seed=seed + 7, ld=ld)
    Bd = torch.from_numpy(B).cuda()
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    Y = rsc.spmm(X, Bd, d=d).cpu().numpy()
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, d=d, with_mag=True)
    assert rel_err(Y, Yo, S) <= 1e-5, (seed, d, ld)
    AT = synth.transpose(A, n_cols)
    cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, A.n))
    cache.refresh(Bd, k, step=0, d=d)
    snap = rsc.cache_snapshot(cache)
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    idx, mask = oracle.topk(oracle.pair_keys(cn2, B, d=d)["key"], k)
    assert np.array_equal(snap["idx"], idx[:k]), seed
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    assert np.array_equal(snap["rowptr"], ro) and np.array_equal(snap["col"], co), seed
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32)), seed
    Ys = cache.spmm_sampled(Bd, d=d).cpu().numpy()
    Yso, Ss = oracle.spmm(ro, co, vo, B, d=d, with_mag=True)
    assert rel_err(Ys, Yso, Ss) <= 1e-4, seed
    if k == n_cols:
        assert np.array_equal(Ys.view(np.uint32), Y.view(np.uint32)), seed
    cache.close()
