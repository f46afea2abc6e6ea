"""Full-size exact and sampled SpMM against an independent implementation: the vendor
library's SpMM (rocSPARSE's rocsparse_spmm, not an oracle and sharing
nothing with this library) on the same operands, compared on every output
element. The oracle checks sampled rows at these sizes; this covers all of
them. Both sides accumulate in fp32 in their own orders, so the bound is
relative to S = |A| |B| (computed by rocSPARSE on the absolute values):
1e-5, the exact product's parity bound (measured: at most 4.2e-7); a wrong
column, a dropped or doubled entry or run, a misplaced row or a garbled
tile exceeds it."""
import pytest
import torch

import paper_2210_10737_amd as rsc
import synth
from bench import RocsparseSpmm

pytestmark = pytest.mark.gpu
FLT_MIN = torch.finfo(torch.float32).tiny


@pytest.fixture(scope="module", autouse=True)
def _gpu(gpu):
    yield


@pytest.mark.parametrize("name", ["copurchase", "social", "protein", "gcn2"])
def test_exact_spmm_matches_the_vendor_library_everywhere(name):
    w = synth.WORKLOADS[name]
    A = synth.make_graph(name, 0)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
    H = torch.from_numpy(synth.dense_normal(A.n, w.d, seed=1)).cuda()
    plan = rsc.SpmmPlan(X)
    Y = plan.run(H)
    Y_plain = rsc.spmm(X, H)
    try:
        v = RocsparseSpmm(X, H)
    except OSError:
        pytest.skip("rocSPARSE cannot be loaded")
    try:
        C = v.run("csr_nnz_split").clone()
    finally:
        v.close()
    Xa = rsc.DeviceCsr(X.n_rows, X.n_cols, X.rowptr, X.col, X.val.abs())
    Ha = H.abs()
    va = RocsparseSpmm(Xa, Ha)
    try:
        S = va.run("csr_nnz_split").clone()
    finally:
        va.close()
    torch.cuda.synchronize()
    err = float(((Y - C).abs() / S.clamp_min(FLT_MIN)).max())
    print(f"{name}: max |ours - rocSPARSE| / (|A||B|) = {err:.2e}", flush=True)
    assert err <= 1e-5
    assert torch.equal(Y, Y_plain)      # the plan's product is rsc_spmm's, bit for bit
    plan.close()


@pytest.mark.parametrize("name,pct", [("copurchase", 30), ("social", 30), ("protein", 30), ("gcn2", 50)])
def test_sampled_spmm_matches_the_vendor_library_everywhere(name, pct):
    """The sampled product on the cached slice (whose keys, selection and
    CSR slice the full-workload parity test checks bit for bit against the
    oracle) against rocSPARSE's product with the same slice, every element."""
    w = synth.WORKLOADS[name]
    A = synth.make_graph(name, 0)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
    G = torch.from_numpy(synth.dense_normal(A.n, w.d, seed=3)).cuda()
    cache = rsc.Cache(X, X, refresh_interval=10)
    cache.refresh(G, (A.n * pct) // 100, step=0)
    Ys = cache.spmm_sampled(G)
    snap = rsc.cache_snapshot(cache)
    cache.close()
    Xs = rsc.DeviceCsr.from_host(snap["rowptr"], snap["col"], snap["val"], A.n)
    try:
        v = RocsparseSpmm(Xs, G)
    except OSError:
        pytest.skip("rocSPARSE cannot be loaded")
    try:
        C = v.run("csr_nnz_split").clone()
    finally:
        v.close()
    va = RocsparseSpmm(rsc.DeviceCsr(Xs.n_rows, Xs.n_cols, Xs.rowptr, Xs.col, Xs.val.abs()), G.abs())
    try:
        S = va.run("csr_nnz_split").clone()
    finally:
        va.close()
    torch.cuda.synchronize()
    err = float(((Ys - C).abs() / S.clamp_min(FLT_MIN)).max())
    print(f"{name} {pct}%: max |ours - rocSPARSE| / (|A'||B|) = {err:.2e}", flush=True)
    assert err <= 1e-5
