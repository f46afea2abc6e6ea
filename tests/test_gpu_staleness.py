"""The cache's staleness record (section 3.3.1, Fig. 4; rsc_cache_staleness)
against the oracle's: the AUC of the selection a refresh replaced under a
new ranking, bit for bit, and the overlap of the two selections exactly.
Both selections and the ranking the oracle uses come from the oracle's own
keys (col_sqnorms, pair_keys, topk / sample_columns, rank_order); the GPU
side makes its own from the same operands."""
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


def _graph(n, seed):
    rng = np.random.default_rng(seed)
    A = synth.bucket_csr(np.minimum(rng.integers(1, 9, n), n), n, seed=seed)
    return A, synth.transpose(A, n)


def _same(a, b):
    return (np.isnan(a) and np.isnan(b)) or a == b


@pytest.mark.parametrize("n,k1,k2,seed", [(1, 1, 0, 0), (31, 7, 9, 1), (32, 16, 16, 2), (33, 0, 5, 3),
                                          (33, 33, 4, 4), (4097, 1000, 2000, 5), (100_003, 30_000, 30_000, 6),
                                          (716_847, 71_684, 358_423, 7)])
def test_staleness_matches_oracle(n, k1, k2, seed):
    A, AT = _graph(n, seed)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    XT = rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, n)
    cache = rsc.Cache(X, XT)
    B1 = synth.dense_normal(n, 24, seed=seed + 10)
    B2 = synth.dense_normal(n, 24, seed=seed + 11)
    B2[: n // 2] = B1[: n // 2]            # half the rows unchanged: the two rankings overlap
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    key1 = oracle.pair_keys(cn2, B1)["key"]
    key2 = oracle.pair_keys(cn2, B2)["key"]
    _, m1 = oracle.topk(key1, k1)
    _, m2 = oracle.topk(key2, k2)
    orders = {"ranking": oracle.rank_order(key2),
              "random": np.random.default_rng(seed).permutation(n).astype(np.int32)}
    cache.refresh(torch.from_numpy(B1).cuda(), k1, step=0)
    with pytest.raises(rsc.RscError):          # one selection: nothing replaced yet
        cache.staleness(torch.from_numpy(orders["random"]).cuda())
    cache.refresh(torch.from_numpy(B2).cuda(), k2, step=10)
    for name, order in orders.items():
        auc, both, kp = cache.staleness(torch.from_numpy(order).cuda())
        want_auc, want_ov = oracle.selection_staleness(order, m1, m2)
        assert _same(auc, want_auc), (name, auc, want_auc)
        assert kp == k1
        assert (want_ov is None and k1 == 0) or both == round(want_ov * k1), (name, both, want_ov)
    cache.close()


def test_staleness_after_a_randomized_refresh_and_bad_orders():
    n = 5000
    A, AT = _graph(n, 20)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    XT = rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, n)
    cache = rsc.Cache(X, XT)
    B1 = synth.dense_normal(n, 16, seed=21)
    B2 = synth.dense_normal(n, 16, seed=22)
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    _, m1 = oracle.topk(oracle.pair_keys(cn2, B1)["key"], 1200)
    key2 = oracle.pair_keys(cn2, B2)["key"]
    m2 = oracle.sample_columns(key2, 900, 77)["mask"]
    cache.refresh(torch.from_numpy(B1).cuda(), 1200, step=0)
    cache.refresh_random(torch.from_numpy(B2).cuda(), 900, seed=77, step=1)
    order = oracle.rank_order(key2)
    auc, both, kp = cache.staleness(torch.from_numpy(order).cuda())
    want_auc, want_ov = oracle.selection_staleness(order, m1, m2)
    assert _same(auc, want_auc) and kp == 1200 and both == round(want_ov * 1200)
    bad = order.copy()
    bad[17] = n                                   # an entry outside [0, n)
    with pytest.raises(rsc.RscError, match="not a ranking"):
        cache.staleness(torch.from_numpy(bad).cuda())
    dup = order.copy()
    sel = np.flatnonzero(np.unpackbits(m1.view(np.uint8), bitorder="little")[:n])
    dup[np.flatnonzero(~np.isin(order, sel))[0]] = sel[0]   # a selected pair ranked twice
    with pytest.raises(rsc.RscError, match="not a ranking"):
        cache.staleness(torch.from_numpy(dup).cuda())
    cache.close()
