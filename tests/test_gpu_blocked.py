"""Column-blocked SpMM mode (the columns cut into P index ranges processed
one after another, partial rows added in fixed range order). Forced with
RSC_SPMM_BLOCKED = 2..8 on seeded random shapes, and chosen automatically on
graphs whose B slice (16, 32 or 64 floats per row, by feature width) spans
2 to 9 (capped to 8) and 17 (not blocked) L2-sized ranges, with plans and
caches used at several widths: exact and sampled SpMM
against the oracle, a full-budget slice equal to the exact product bit for
bit, and the automatic choice equal to the forced one."""
import os

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


class blocked:
    """Sets RSC_SPMM_BLOCKED for the duration of a with-block."""

    def __init__(self, value):
        self.value = value

    def __enter__(self):
        self.old = os.environ.get("RSC_SPMM_BLOCKED")
        if self.value is None:
            os.environ.pop("RSC_SPMM_BLOCKED", None)
        else:
            os.environ["RSC_SPMM_BLOCKED"] = str(self.value)

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("RSC_SPMM_BLOCKED", None)
        else:
            os.environ["RSC_SPMM_BLOCKED"] = self.old


def rel_err(Y, Yo, S):
    return float(np.max(np.abs(np.asarray(Y, np.float64) - Yo) / np.maximum(S, FLT_MIN))) if Yo.size else 0.0


def shape(seed):
    rng = np.random.default_rng(5000 + seed)
    n_rows = int(rng.integers(1, 2500))
    n_cols = int(rng.integers(1, 3000))
    kinds = rng.choice(["short", "runs", "long", "empty"], size=n_rows, p=[0.5, 0.3, 0.1, 0.1])
    lens = np.where(kinds == "short", rng.integers(0, 20, n_rows),
                    np.where(kinds == "runs", rng.integers(60, 300, n_rows),
                             np.where(kinds == "long", rng.integers(1000, 3000, n_rows), 0)))
    lens = np.minimum(lens, n_cols)
    A = synth.bucket_csr(lens, n_cols, seed=seed)
    d = int(rng.choice([1, 5, 16, 64, 65, 100, 256, 300]))
    ld = (d + 3) // 4 * 4 + 4 * int(rng.integers(0, 3))
    k = int(rng.choice([0, 1, n_cols // 4, n_cols]))
    P = int(rng.choice([2, 3, 5, 8]))
    return A, n_cols, d, ld, k, P


@pytest.mark.parametrize("seed", range(12))
def test_forced_blocks_match_oracle(seed):
    A, n_cols, d, ld, k, P = shape(seed)
    B = synth.dense_normal(n_cols, d, seed=seed + 11, ld=ld)
    Bd = torch.from_numpy(B).cuda()
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, d=d, with_mag=True)
    AT = synth.transpose(A, n_cols)
    with blocked(P):
        Y = rsc.spmm(X, Bd, d=d).cpu().numpy()
        cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, A.n))
        cache.refresh(Bd, k, step=0, d=d)
        Ys = cache.spmm_sampled(Bd, d=d).cpu().numpy()
        snap = rsc.cache_snapshot(cache)
        cache.close()
    assert rel_err(Y, Yo, S) <= 1e-5, (seed, P, d, ld)
    # the oracle's own chain: column norms of X (rows of X^T), keys, top-k, slice
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    key = oracle.pair_keys(cn2, B, d=d)["key"]
    idx, mask = oracle.topk(key, k)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    assert np.array_equal(snap["idx"], idx), (seed, P)
    assert np.array_equal(snap["rowptr"], ro) and np.array_equal(snap["col"], co), (seed, P)
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32)), (seed, P)
    Yso, Ss = oracle.spmm(ro, co, vo, B, d=d, with_mag=True)
    assert rel_err(Ys, Yso, Ss) <= 1e-4, (seed, P)
    if k == n_cols:
        assert np.array_equal(Ys.view(np.uint32), Y.view(np.uint32)), (seed, P)
    with blocked(0):
        Y0 = rsc.spmm(X, Bd, d=d).cpu().numpy()
    assert rel_err(Y0, Yo, S) <= 1e-5


def test_blocked_is_reproducible_and_keeps_empty_rows_zero():
    lens = np.array([0, 700, 0, 1500, 64, 0, 2000], np.int64)
    A = synth.bucket_csr(lens, 2100, seed=3)
    Bh = synth.dense_normal(2100, 96, seed=4)
    B = torch.from_numpy(Bh).cuda()
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 2100)
    with blocked(8):
        Y1 = rsc.spmm(X, B)
        Y2 = rsc.spmm(X, B)
    assert torch.equal(Y1, Y2)
    assert torch.count_nonzero(Y1[torch.from_numpy(lens == 0).cuda()]) == 0
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, Bh, with_mag=True)
    assert rel_err(Y1.cpu().numpy(), Yo, S) <= 1e-5


def test_automatic_choice_on_long_rows():
    # 20,000 columns x 64 floats = 4.9 MiB of B per pass: two ranges; rows of
    # ~200 entries (>= 64 per range on average) switch the mode on.
    n = 20000
    rng = np.random.default_rng(9)
    lens = rng.integers(150, 260, n)
    A = synth.bucket_csr(lens, n, seed=12)
    B = synth.dense_normal(n, 128, seed=13)
    Bd = torch.from_numpy(B).cuda()
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    with blocked(None):
        Y = rsc.spmm(X, Bd)
        cache = rsc.Cache(X, X)
        cache.refresh(Bd, n, step=0)
        Yk = cache.spmm_sampled(Bd)
        cache.close()
    with blocked(2):
        Y2 = rsc.spmm(X, Bd)
    assert torch.equal(Y, Y2)                  # the automatic mode took P = 2
    assert torch.equal(Yk, Y)                  # full budget == exact, bitwise
    rows = np.arange(0, n, 97, dtype=np.int32)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, rows=rows, with_mag=True)
    assert rel_err(Y.cpu().numpy()[rows], Yo, S) <= 1e-5


@pytest.mark.parametrize("n_cols,d,row_len,P", [
    (160_000, 96, 500, 8),    # 64-float passes: 9 ranges of 4.5 MiB, capped to 8
    (160_000, 32, 1000, 5),   # the 32-float layout: 4.3 ranges
    (160_000, 16, 1000, 3),   # the 16-float layout: 2.2 ranges
    (300_000, 96, 500, 0),    # 17 ranges, beyond the cap of 16: not blocked
    (300_000, 32, 1000, 8),   # 8.1 ranges at 32 floats: capped to 8 (125 entries per piece)
    (300_000, 16, 1200, 5),   # 240 entries per piece, at least 224 in the 16-float layout
    (300_000, 16, 500, 0),    # 100 entries per piece: too short for it, not blocked
])
def test_automatic_range_count(n_cols, d, row_len, P):
    # The range count follows the slice of B one pass gathers from (the
    # blocked layout's 16, 32 or 64 floats of each row), and the pieces must
    # hold 56, 112 or 224 entries on average. The automatic choice equals
    # the forced one bit for bit; a plan and a full-budget slice reproduce it.
    n_rows = 2000
    A = synth.bucket_csr(np.full(n_rows, row_len), n_cols, seed=31)
    AT = synth.transpose(A, n_cols)
    B = synth.dense_normal(n_cols, d, seed=32)
    Bd = torch.from_numpy(B).cuda()
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    XT = rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, n_rows)
    with blocked(None):
        Y = rsc.spmm(X, Bd)
        plan = rsc.SpmmPlan(X)
        Yp = plan.run(Bd)
        plan.close()
        cache = rsc.Cache(X, XT)
        cache.refresh(Bd, n_cols, step=0)
        Yk = cache.spmm_sampled(Bd)
        cache.close()
    with blocked(P):
        Yf = rsc.spmm(X, Bd)
    with blocked(0 if P else 8):
        Yo_mode = rsc.spmm(X, Bd)
    torch.cuda.synchronize()
    assert torch.equal(Y, Yf), P               # the automatic mode took this P
    assert not torch.equal(Y, Yo_mode), P      # and not the other mode
    assert torch.equal(Yp, Y) and torch.equal(Yk, Y)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    assert rel_err(Y.cpu().numpy(), Yo, S) <= 1e-5


def test_plan_and_cache_across_feature_widths():
    # A plan prepares for 64-float passes (8 ranges here); a run at d = 16
    # takes 3 ranges (d = 32: 5) and prepares for itself, and later runs at
    # any width still equal rsc_spmm bit for bit. A cache refreshed at one
    # width and used at another does the same.
    n_rows, n_cols = 2000, 160_000
    A = synth.bucket_csr(np.full(n_rows, 1000), n_cols, seed=33)
    AT = synth.transpose(A, n_cols)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    XT = rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, n_rows)
    Bs = {d: torch.from_numpy(synth.dense_normal(n_cols, d, seed=34 + d)).cuda() for d in (16, 32, 96)}
    with blocked(None):
        ref = {d: rsc.spmm(X, B) for d, B in Bs.items()}
        plan = rsc.SpmmPlan(X)
        for d in (96, 16, 96, 32, 16):
            assert torch.equal(plan.run(Bs[d]), ref[d]), d
        plan.close()
        cache = rsc.Cache(X, XT)
        for d_ref, order in ((16, (16, 96, 32)), (96, (96, 16))):
            cache.refresh(Bs[d_ref], n_cols, step=0)
            for d in order:
                assert torch.equal(cache.spmm_sampled(Bs[d]), ref[d]), (d_ref, d)
        cache.close()
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, Bs[16].cpu().numpy(), with_mag=True)
    assert rel_err(ref[16].cpu().numpy(), Yo, S) <= 1e-5


@pytest.mark.parametrize("n_rows,n_cols,row_len,d", [
    (100, 40_000, 10_000, 96),     # P = 3: 300 long pieces from 100 rows
    (20_000, 20_000, 2_200, 64),   # P = 2: 40,000 pieces of 1,100 entries from 20,000 rows
])
def test_long_pieces_outnumber_rows(n_rows, n_cols, row_len, d):
    # Regression: the long-piece list of the column-blocked mode must hold up
    # to P pieces per row (not one per row) when rows average over 1,024
    # entries per range. The automatic rule picks the blocked mode here.
    A = synth.bucket_csr(np.full(n_rows, row_len), n_cols, seed=21)
    B = synth.dense_normal(n_cols, d, seed=22)
    Bd = torch.from_numpy(B).cuda()
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    with blocked(None):
        Y = rsc.spmm(X, Bd)
        plan = rsc.SpmmPlan(X)
        Yp = plan.run(Bd)
        plan.close()
    with blocked(0):
        Yu = rsc.spmm(X, Bd)
    torch.cuda.synchronize()
    assert not torch.equal(Y, Yu)              # the blocked mode ran (different partial rounding)
    assert torch.equal(Y, Yp)                  # the plan's prepared list gives the same product
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    assert rel_err(Y.cpu().numpy(), Yo, S) <= 1e-5
    assert rel_err(Yu.cpu().numpy(), Yo, S) <= 1e-5
