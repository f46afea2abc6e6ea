"""The single-pass CSR column slice (count, decoupled look-back scan over
ticketed tiles, compaction in one kernel; taken with RSC_SLICE_FUSED=1)
against the default multi-launch form and the oracle: rowptr', col', val' and nnz'
byte for byte, with the mask in LDS (up to 1,179,648 columns) and in global
memory (above that), with a per-column scale, ragged tails, empty rows,
k = 0 and k = n, and the capacity error."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2210_10737_amd as rsc
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


class fused:
    def __init__(self, value):
        self.value = value

    def __enter__(self):
        self.old = os.environ.get("RSC_SLICE_FUSED")
        os.environ["RSC_SLICE_FUSED"] = str(self.value)

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("RSC_SLICE_FUSED", None)
        else:
            os.environ["RSC_SLICE_FUSED"] = self.old


def _mask(n, keep, rng):
    m = np.zeros((n + 31) // 32, np.uint32)
    idx = rng.choice(n, keep, replace=False) if keep else np.zeros(0, np.int64)
    for i in idx:
        m[i >> 5] |= np.uint32(1 << (int(i) & 31))
    return m


def _slice(X, mask_d, cap=None, colw=None):
    S, nnz = rsc.slice_csr(X, mask_d, capacity=cap, colw=colw)
    torch.cuda.synchronize()
    k = int(nnz.item())
    m = min(k, S.col.numel())
    return S.rowptr.cpu().numpy(), S.col[:m].cpu().numpy(), S.val[:m].cpu().numpy(), k


@pytest.mark.parametrize("seed", range(10))
def test_fused_equals_three_launch_and_oracle(seed):
    rng = np.random.default_rng(700 + seed)
    n_rows = int(rng.integers(1, 6000))
    n_cols = int(rng.choice([1, 37, 3000, 100_000, 1_179_648]))
    lens = np.minimum(rng.integers(0, 200, n_rows) * (rng.random(n_rows) < 0.8), n_cols)
    A = synth.bucket_csr(lens, n_cols, seed=seed)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    keep = int(rng.choice([0, 1, n_cols // 3, n_cols]))
    mask = _mask(n_cols, keep, rng)
    mask_d = torch.from_numpy(mask.view(np.int32)).cuda()
    colw = rng.random(n_cols) * 3
    colw_d = torch.from_numpy(colw).cuda()
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    ros, cos_, vos = oracle.slice_scaled(A.rowptr, A.col, A.val, mask, colw)
    for w in (None, colw_d):
        with fused(1):
            f = _slice(X, mask_d, colw=w)
        with fused(0):
            t = _slice(X, mask_d, colw=w)
        for a, b in zip(f[:3], t[:3]):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), (seed, w is None)
        assert f[3] == t[3]
        r, c, v = (ro, co, vo) if w is None else (ros, cos_, vos)
        assert f[3] == len(c)
        assert np.array_equal(f[0], r) and np.array_equal(f[1], c)
        assert np.array_equal(f[2].view(np.uint32), v.view(np.uint32))


@pytest.mark.parametrize("n_cols", [1_179_649, 2_449_029])
def test_fused_with_the_mask_in_global_memory(n_cols):
    # more columns than the LDS mask holds: forced fused takes the global-memory variant
    rng = np.random.default_rng(n_cols % 97)
    n_rows = 50_000
    lens = rng.integers(0, 60, n_rows)
    A = synth.bucket_csr(lens, n_cols, seed=3)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    mask = _mask(n_cols, n_cols // 3, rng)
    mask_d = torch.from_numpy(mask.view(np.int32)).cuda()
    with fused(1):
        f = _slice(X, mask_d)
    with fused(0):
        t = _slice(X, mask_d)
    for a, b in zip(f[:3], t[:3]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    assert f[3] == len(co) and np.array_equal(f[0], ro) and np.array_equal(f[1], co)


def test_fused_capacity_error():
    rng = np.random.default_rng(5)
    A = synth.bucket_csr(rng.integers(0, 300, 3000), 5000, seed=5)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 5000)
    mask = _mask(5000, 2500, rng)
    mask_d = torch.from_numpy(mask.view(np.int32)).cuda()
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    with fused(1):
        with pytest.raises(rsc.RscError) as e:
            rsc.slice_csr(X, mask_d, capacity=len(co) // 2)
        assert e.value.status == 4
        f = _slice(X, mask_d, cap=len(co))              # exactly enough room
    assert f[3] == len(co) and np.array_equal(f[0], ro) and np.array_equal(f[1], co)
    assert np.array_equal(f[2].view(np.uint32), vo.view(np.uint32))


def test_fused_full_size_copurchase_against_three_launch():
    # the largest graph (2.45M columns: global-memory mask) at its 30 % budget
    A = synth.make_graph("copurchase", 0)
    n = A.n
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    key = oracle.pair_keys(cn2, synth.dense_normal(n, 256, seed=1))["key"]
    _, mask = oracle.topk(key, (n * 30) // 100)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    mask_d = torch.from_numpy(mask.view(np.int32)).cuda()
    with fused(1):
        f = _slice(X, mask_d)
    with fused(0):
        t = _slice(X, mask_d)
    for a, b in zip(f[:3], t[:3]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert f[3] == t[3]


def _tile_edge_lengths(case):
    """Row lengths whose row boundaries sit on 4096-entry tile edges (both
    slice forms cut the entries into such tiles): rows ending exactly on an
    edge, runs of empty rows at an edge and at both ends, rows spanning
    several tiles, and nnz a whole number of tiles or one entry past it."""
    T = 4096
    if case == "edges":
        return [0, 0, T, 0, 0, 0, T - 1, 1, 0, 2 * T, 0, T, 0, 0]
    if case == "spans":
        return [1, 5 * T + 7, 0, T - 8, 3, 0, 0, 3 * T, 0]
    if case == "one_past":
        return [T] * 5 + [0, 1, 0]
    if case == "all_empty_tail":
        return [2 * T - 1, 1] + [0] * 9000
    raise ValueError(case)


@pytest.mark.parametrize("case", ["edges", "spans", "one_past", "all_empty_tail"])
@pytest.mark.parametrize("form", [0, 1])
def test_rows_on_tile_edges(case, form):
    rng = np.random.default_rng(["edges", "spans", "one_past", "all_empty_tail"].index(case) + 900)
    lens = np.array(_tile_edge_lengths(case), dtype=np.int64)
    n_cols = int(max(lens.max(), 1)) + 3
    A = synth.bucket_csr(lens, n_cols, seed=11)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    for keep in (0, n_cols // 2, n_cols):
        mask = _mask(n_cols, keep, rng)
        mask_d = torch.from_numpy(mask.view(np.int32)).cuda()
        ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
        with fused(form):
            r, c, v, k = _slice(X, mask_d)
        assert k == len(co), (case, form, keep)
        assert np.array_equal(r, ro), (case, form, keep)
        assert np.array_equal(c, co) and np.array_equal(v.view(np.uint32), vo.view(np.uint32)), (case, form, keep)


class paired:
    def __init__(self, value):
        self.value = value

    def __enter__(self):
        self.old = os.environ.get("RSC_SLICE_PAIRED")
        os.environ["RSC_SLICE_PAIRED"] = str(self.value)

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("RSC_SLICE_PAIRED", None)
        else:
            os.environ["RSC_SLICE_PAIRED"] = self.old


@pytest.mark.parametrize("n_rows,mean_len", [(60_000, 40), (500, 20)])
def test_two_piece_mask_paired_and_unpaired(n_rows, mean_len):
    """A mask of two LDS pieces (2,000,003 columns): the count pass by pairs
    of blocks (one piece each; the default when the tiles fill 16 blocks)
    and by one block per CU walking col twice give the same bytes as the
    oracle; the small case has too few tiles to pair."""
    n_cols = 2_000_003
    rng = np.random.default_rng(n_rows)
    A = synth.bucket_csr(rng.integers(0, 2 * mean_len, n_rows), n_cols, seed=21)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    mask = np.zeros((n_cols + 31) // 32, np.uint32)
    keep = rng.choice(n_cols, n_cols * 3 // 10, replace=False)
    np.bitwise_or.at(mask, keep >> 5, (np.uint32(1) << (keep & 31).astype(np.uint32)))
    mask_d = torch.from_numpy(mask.view(np.int32)).cuda()
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    for p in (1, 0):
        with paired(p):
            r, c, v, k = _slice(X, mask_d)
        assert k == len(co), p
        assert np.array_equal(r, ro) and np.array_equal(c, co), p
        assert np.array_equal(v.view(np.uint32), vo.view(np.uint32)), p
