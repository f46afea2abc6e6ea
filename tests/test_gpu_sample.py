"""Randomized column-row sampling on the GPU (Eq. 2 with Eq. 3's
probabilities, scale 1/(k p)) against the oracle: draw counts, per-column
scales and masks bit for bit, the scaled slice bit for bit, the sampled
product within fp32 tolerance, and unbiasedness over seeds."""
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


def keys_for(name, d, seed):
    A = synth.make_graph(name, 0)
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    return A, oracle.pair_keys(cn2, synth.dense_normal(A.n, d, seed=seed))["key"]


def _check(key, k, seed):
    o = oracle.sample_columns(key, k, seed)
    cnt, colw, mask = rsc.sample_columns(torch.from_numpy(key.view(np.int64)).cuda(), k, seed)
    assert np.array_equal(cnt.cpu().numpy(), o["count"])
    assert np.array_equal(colw.cpu().numpy().view(np.uint64), o["colw"].view(np.uint64))
    assert np.array_equal(mask.cpu().numpy().view(np.uint32), o["mask"])
    return o


@pytest.mark.parametrize("k,seed", [(0, 1), (1, 2), (2048, 3), (20_000, 4)])
def test_sample_columns_bitwise_tiny(k, seed):
    _, key = keys_for("tiny", 64, 1)
    key = key.copy()
    key[::37] = 0
    _check(key, k, seed)


def test_sample_columns_bitwise_full_size():
    _, key = keys_for("gcn2", 100, 5)
    o = _check(key, 215_054, 11)
    assert o["count"].sum() == 215_054


def test_sample_draw_on_a_cdf_boundary():
    """The first draw's u equals the CDF boundary W_0 (the case constructed in
    the oracle's pins): the device draw lands on column 1, as the oracle's."""
    from test_oracle_pins import boundary_case
    key, seed, _ = boundary_case()
    o = _check(key, 1, seed)
    assert list(o["count"]) == [0, 1]


def test_sample_columns_degenerate():
    n = 5000
    _check(np.zeros(n, np.uint64), 100, 1)                      # nothing to draw
    key = np.arange(1, n + 1, dtype=np.uint64) << np.uint64(40)
    inf_key = np.uint64(0x7FF0000000000000 + 1)
    key[[10, 4000]] = inf_key                                   # infinite scores share the mass
    o = _check(key, 999, 7)
    assert o["count"][[10, 4000]].sum() == 999


def test_sample_columns_reduced_weight_resolution():
    """Above 2^24 pairs the weights keep fewer bits (the CDF stays below
    2^63); draws still match the oracle bit for bit."""
    n = (1 << 24) + 1000
    key = np.full(n, np.uint64(0x3FF0000000000001), np.uint64)      # q = 1
    key[::7] = np.uint64(0x4010000000000001)                        # q = 4
    key[5::11] = 0
    o = _check(key, 300_000, 21)
    assert np.all(o["w"][::7][o["w"][::7] > 0] == 1 << 37)


def test_cache_random_refresh_and_sampled_product():
    A = synth.random_csr(3000, 2500, 40, seed=51, hub_rows=2, hub_len=2200, empty_frac=0.1)
    AT = synth.transpose(A, 2500)
    cache = rsc.Cache(rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 2500),
                      rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, 3000), refresh_interval=10)
    B = synth.dense_normal(2500, 96, seed=52)
    Bd = torch.from_numpy(B).cuda()
    cache.refresh_random(Bd, 1500, seed=9, step=0)
    snap = rsc.cache_snapshot(cache)
    assert snap["k"] == 1500 and snap["idx_ptr"] is None
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    o = oracle.sample_columns(oracle.pair_keys(cn2, B)["key"], 1500, 9)
    ro, co, vo = oracle.slice_scaled(A.rowptr, A.col, A.val, o["mask"], o["colw"])
    assert np.array_equal(snap["rowptr"], ro) and np.array_equal(snap["col"], co)
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32))
    Ys = cache.spmm_sampled(Bd).cpu().numpy()
    Yo, S = oracle.spmm(ro, co, vo, B, with_mag=True)
    assert np.max(np.abs(Ys.astype(np.float64) - Yo) / np.maximum(S, FLT_MIN)) <= 1e-4
    cache.close()


def test_sampled_product_unbiased_on_gpu():
    A = synth.random_csr(400, 300, 20, seed=61)
    AT = synth.transpose(A, 300)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 300)
    cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, 400))
    B = synth.dense_normal(300, 32, seed=62)
    Bd = torch.from_numpy(B).cuda()
    exact = rsc.spmm(X, Bd).double()
    acc = torch.zeros_like(exact)
    first = None
    seeds = 300
    for s in range(seeds):
        cache.refresh_random(Bd, 60, seed=1000 + s, step=s)
        Y = cache.spmm_sampled(Bd).double()
        acc += Y
        first = Y.clone() if first is None else first
    assert float(torch.linalg.norm(acc / seeds - exact)) < 0.2 * float(torch.linalg.norm(first - exact))
    cache.close()


def test_cache_random_zero_draws_and_unrefreshed_cache():
    A = synth.random_csr(500, 400, 20, seed=71)
    AT = synth.transpose(A, 400)
    cache = rsc.Cache(rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 400),
                      rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, 500))
    B = torch.from_numpy(synth.dense_normal(400, 16, seed=72)).cuda()
    with pytest.raises(rsc.RscError):          # never refreshed
        cache.spmm_sampled(B)
    cache.refresh_random(B, 0, seed=1, step=0)  # no draws: empty slice, zero product
    snap = rsc.cache_snapshot(cache)
    assert snap["nnz"] == 0 and not snap["rowptr"].any()
    assert not cache.spmm_sampled(B).any()
    cache.close()


def test_cache_switches_between_random_and_topk_slices():
    """A top-k refresh after a randomized one reports its index list again;
    selecting before anything was scored is an error."""
    A = synth.random_csr(600, 500, 25, seed=81)
    AT = synth.transpose(A, 500)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 500)
    cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, 600))
    with pytest.raises(rsc.RscError):
        cache.select(10, step=0)
    B = synth.dense_normal(500, 24, seed=82)
    Bd = torch.from_numpy(B).cuda()
    cache.refresh_random(Bd, 100, seed=3, step=0)
    assert rsc.cache_snapshot(cache)["idx_ptr"] is None
    cache.refresh(Bd, 120, step=1)
    snap = rsc.cache_snapshot(cache, 1)
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    idx, mask = oracle.topk(oracle.pair_keys(cn2, B)["key"], 120)
    assert snap["idx_ptr"] is not None and np.array_equal(snap["idx"], idx)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32))
    cache.close()


def test_full_size_randomized_refresh_copurchase():
    """The bench's randomized-selector configuration at full size
    (copurchase, 734,708 draws): draws, scales, mask and the scaled slice bit
    for bit against the oracle, and every element of the sampled product."""
    A = synth.make_graph("copurchase", 0)
    n = A.n
    G = synth.dense_normal(n, 256, seed=3)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    cache = rsc.Cache(X, X, refresh_interval=10)
    Gd = torch.from_numpy(G).cuda()
    k, seed = (n * 30) // 100, 12345
    cache.refresh_random(Gd, k, seed=seed, step=0)
    snap = rsc.cache_snapshot(cache)
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    o = oracle.sample_columns(oracle.pair_keys(cn2, G)["key"], k, seed)
    mask_g = rsc.copy_to_host(cache.buffers()[4], (n + 31) // 32, np.uint32)
    assert np.array_equal(mask_g, o["mask"])
    ro, co, vo = oracle.slice_scaled(A.rowptr, A.col, A.val, o["mask"], o["colw"])
    assert snap["nnz"] == len(co)
    assert np.array_equal(snap["rowptr"], ro) and np.array_equal(snap["col"], co)
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32))
    Ys = cache.spmm_sampled(Gd)
    worst = 0.0
    for r0 in range(0, n, 250_000):
        rows = np.arange(r0, min(n, r0 + 250_000), dtype=np.int32)
        Yo, S = oracle.spmm(ro, co, vo, G, rows=rows, with_mag=True)
        got = Ys[r0:r0 + len(rows)].cpu().numpy().astype(np.float64)
        worst = max(worst, float(np.max(np.abs(got - Yo) / np.maximum(S, FLT_MIN))))
    print(f"[full] randomized sampled: max rel err {worst:.3e}", flush=True)
    assert worst <= 1e-4
    cache.close()
