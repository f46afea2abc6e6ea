"""SpMM plans (rsc_spmm_plan_*) and the column cache hint: a plan's product
equals rsc_spmm bitwise, on small operands (no hinted copy) and on operands
with more than 262,144 columns (hinted copy; the hint active when a pass
gathers from more than 512 MiB of B rows), also with the hint switched off
and with the column-blocked mode forced; and it matches the oracle. Plans
and caches prepare their row lists once; runs under changed environment
switches rebuild their own and stay correct."""
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


class env:
    def __init__(self, **kv):
        self.kv = kv

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in self.kv}
        for k, v in self.kv.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = str(v)

    def __exit__(self, *exc):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def rel_err(Y, Yo, S):
    return float(np.max(np.abs(np.asarray(Y, np.float64) - Yo) / np.maximum(S, FLT_MIN))) if Yo.size else 0.0


def wide_graph(seed=1):
    """20,000 rows over 300,000 columns, power-law-like row lengths, columns
    drawn with a skewed popularity (so there are hub columns)."""
    rng = np.random.default_rng(seed)
    n_rows, n_cols = 20_000, 300_000
    lens = np.minimum((rng.pareto(1.5, n_rows) * 40 + 5).astype(np.int64), 3000)
    w = 1.0 / (np.arange(n_cols) + 10.0) ** 0.8
    w = w[rng.permutation(n_cols)]
    w /= w.sum()
    draws = rng.choice(n_cols, size=int(lens.sum()), p=w)
    cols = [np.unique(c) for c in np.split(draws, np.cumsum(lens)[:-1])]
    rowptr = np.zeros(n_rows + 1, np.int64)
    rowptr[1:] = np.cumsum([len(c) for c in cols])
    col = np.concatenate(cols).astype(np.int32)
    val = rng.uniform(-1, 1, len(col)).astype(np.float32)
    return synth.Csr(n_rows, rowptr.astype(np.int32), col, val), n_cols


@pytest.mark.parametrize("d", [1, 64, 100, 256, 300, 512])
def test_plan_equals_spmm_small(d):
    A = synth.make_graph("tiny", 0)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
    B = torch.from_numpy(synth.dense_normal(A.n, d, seed=d, ld=(d + 3) // 4 * 4)).cuda()
    plan = rsc.SpmmPlan(X)
    for _ in range(2):
        assert torch.equal(plan.run(B, d=d), rsc.spmm(X, B, d=d))
    plan.close()


@pytest.fixture(scope="module")
def wide():
    return wide_graph()


@pytest.mark.parametrize("d,mode", [(512, None), (256, None), (512, "nohint"), (64, "blocked"), (300, "ordered")])
def test_plan_equals_spmm_wide(wide, d, mode):
    A, n_cols = wide
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    Bh = synth.dense_normal(n_cols, d, seed=7)
    B = torch.from_numpy(Bh).cuda()
    kv = {"RSC_SPMM_HINT": 0 if mode == "nohint" else None, "RSC_SPMM_BLOCKED": 3 if mode == "blocked" else None,
          "RSC_SPMM_ORDER": 1 if mode == "ordered" else None}
    with env(**kv):
        plan = rsc.SpmmPlan(X)
        Yp = plan.run(B)
        Yp2 = plan.run(B)
        Ys = rsc.spmm(X, B)
        plan.close()
    assert torch.equal(Yp, Ys) and torch.equal(Yp, Yp2)
    rows = np.arange(0, A.n, 13, dtype=np.int32)
    Yo, S = oracle.spmm(A.rowptr, A.col, A.val, Bh, rows=rows, with_mag=True)
    assert rel_err(Yp.cpu().numpy()[rows], Yo, S) <= 1e-5


def test_plan_keeps_split_bounds():
    """A product that runs column-blocked (20,000 columns, ~200 entries per
    row: two ranges): the plan's precomputed split bounds give rsc_spmm's
    result. Switched off later, the plan runs unblocked like rsc_spmm; asked
    for more ranges than its workspace was sized for, it runs unblocked too
    (rsc_spmm would size a larger workspace), so that result only agrees
    within rounding."""
    n = 20000
    rng = np.random.default_rng(9)
    A = synth.bucket_csr(rng.integers(150, 260, n), n, seed=12)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    B = torch.from_numpy(synth.dense_normal(n, 128, seed=13)).cuda()
    with env(RSC_SPMM_BLOCKED=None):
        plan = rsc.SpmmPlan(X)
        assert torch.equal(plan.run(B), rsc.spmm(X, B))
    for blocks in (0, 2):
        with env(RSC_SPMM_BLOCKED=blocks):
            assert torch.equal(plan.run(B), rsc.spmm(X, B)), blocks
    with env(RSC_SPMM_BLOCKED=4):
        Y4 = plan.run(B)
    with env(RSC_SPMM_BLOCKED=0):
        assert torch.equal(Y4, rsc.spmm(X, B))
    plan.close()


def test_plan_row_list_survives_switches(wide):
    """The plan builds its long-row list (or the length-class order) once;
    runs under a different row-order switch rebuild it themselves, and every
    run equals rsc_spmm."""
    A, n_cols = wide
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    B = torch.from_numpy(synth.dense_normal(n_cols, 64, seed=21)).cuda()
    want = rsc.spmm(X, B)
    for first in (0, 1):
        with env(RSC_SPMM_ORDER=first):
            plan = rsc.SpmmPlan(X)
        for order in (first, 1 - first, first):
            with env(RSC_SPMM_ORDER=order):
                assert torch.equal(plan.run(B), want), (first, order)
        plan.close()


@pytest.mark.parametrize("switch", ["RSC_SPMM_ORDER", "RSC_SPMM_BLOCKED", "RSC_SPMM_SLICE"])
def test_cache_prepared_list_survives_switches(switch):
    """The cache prepares each slice's row list at refresh; sampled products
    run under other switch settings rebuild their own, and every product
    stays within tolerance of the oracle (and bitwise stable per setting)."""
    rng = np.random.default_rng(77)
    n = 3000
    lens = np.minimum(np.where(rng.random(n) < 0.05, rng.integers(1100, 2900, n), rng.integers(0, 300, n)), n)
    A = synth.bucket_csr(lens, n, seed=31)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    AT = synth.transpose(A, n)
    Bh = synth.dense_normal(n, 96, seed=32)
    B = torch.from_numpy(Bh).cuda()
    values = {"RSC_SPMM_ORDER": (1, 0, 1), "RSC_SPMM_BLOCKED": (2, 0, 3, 2), "RSC_SPMM_SLICE": (32, 256, 32)}[switch]
    with env(**{switch: values[0]}):
        cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, n))
        cache.refresh(B, n // 2, step=0)
        snap = rsc.cache_snapshot(cache)
        first = cache.spmm_sampled(B)
    # the oracle's own chain (column norms, keys, top-k, slice), then its product
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    _, mask = oracle.topk(oracle.pair_keys(cn2, Bh)["key"], n // 2)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    assert np.array_equal(snap["rowptr"], ro) and np.array_equal(snap["col"], co)
    assert np.array_equal(snap["val"].view(np.uint32), vo.view(np.uint32))
    Yo, S = oracle.spmm(ro, co, vo, Bh, with_mag=True)
    seen = {}
    for v in values:
        with env(**{switch: v}):
            Ys = cache.spmm_sampled(B)
        assert rel_err(Ys.cpu().numpy(), Yo, S) <= 1e-4, (switch, v)
        if v in seen:
            assert torch.equal(Ys, seen[v]), (switch, v)
        seen[v] = Ys
    assert torch.equal(seen[values[0]], first)
    cache.close()


def test_whole_chain_on_a_side_stream_matches_the_current_stream():
    """Every call enqueues on the stream it is given: plan creation and runs,
    the cache's creation, refresh, slice read-back and sampled product, all
    issued inside a side stream, give the same bits as on the default stream
    (a launch or copy on another stream would race with the producer of B
    here, which is enqueued just before on the same stream)."""
    A = synth.make_graph("tiny", 0)
    d, k = 64, 1500

    def chain():
        X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
        H0 = torch.from_numpy(synth.dense_normal(A.n, d, seed=4)).cuda()
        plan = rsc.SpmmPlan(X)
        cache = rsc.Cache(X, X, refresh_interval=10)
        H = H0 * 2.0 - 1.0                 # produced on this stream right before use
        Y = plan.run(H)
        cache.refresh(H, k, step=0)
        nnz = cache.get(0)["slice"].nnz
        Yb = cache.spmm_sampled(H)
        out = (Y.cpu().numpy(), Yb.cpu().numpy(), nnz)
        plan.close()
        cache.close()
        return out

    ref = chain()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        got = chain()
    torch.cuda.current_stream().wait_stream(side)
    assert got[2] == ref[2]
    assert np.array_equal(got[0].view(np.uint32), ref[0].view(np.uint32))
    assert np.array_equal(got[1].view(np.uint32), ref[1].view(np.uint32))


def test_binding_refuses_tensors_off_the_current_device():
    """The binding hands the kernels raw addresses on the current device's
    stream; a host tensor is refused before anything is launched."""
    A = synth.make_graph("tiny", 0)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, A.n)
    H = torch.from_numpy(synth.dense_normal(A.n, 8, seed=1))        # host memory
    with pytest.raises(ValueError, match="current device"):
        rsc.spmm(X, H)
    plan = rsc.SpmmPlan(X)
    with pytest.raises(ValueError, match="current device"):
        plan.run(H)
    Y = plan.run(H.cuda())
    with pytest.raises(ValueError, match="current device"):
        plan.run(H.cuda(), out=torch.empty_like(Y).cpu())
    plan.close()
    Xh = rsc.DeviceCsr(A.n, A.n, torch.from_numpy(A.rowptr), torch.from_numpy(A.col), torch.from_numpy(A.val))
    with pytest.raises(ValueError, match="current device"):
        rsc.spmm(Xh, H.cuda())


@pytest.mark.parametrize("d", [64, 100, 256, 512])
@pytest.mark.parametrize("wide", [False, True])
def test_gather_probe_gathers_the_plan_rows(d, wide):
    # The gather-ceiling probe loads exactly the B rows of the column stream:
    # the float it writes per 64 entries equals the sum of those rows' last
    # feature pass (the sink is rewritten by every pass).
    if wide:
        A, n_cols = wide_graph(3)
    else:
        A = synth.random_csr(3000, 2500, 400, seed=8, hub_rows=5, hub_len=2400)
        n_cols = 2500
    B = synth.dense_normal(n_cols, d, seed=9)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n_cols)
    plan = rsc.SpmmPlan(X)
    Bd = torch.from_numpy(B).cuda()
    nnz = int(A.rowptr[-1])
    chunks = (nnz + 63) // 64
    for inflight in (4, 8, 16):
        sink = torch.full((chunks,), float("nan"), device="cuda")
        slice_w = plan.gather_probe(Bd, inflight=inflight, sink=sink)
        got = sink.cpu().numpy().astype(np.float64)
        f_last = ((d - 1) // slice_w) * slice_w
        part = B[:, f_last:d].astype(np.float64)
        pad = np.zeros(chunks * 64 - nnz)
        want = np.concatenate([part.sum(axis=1)[A.col], pad]).reshape(chunks, 64).sum(axis=1)
        mag = np.concatenate([np.abs(part).sum(axis=1)[A.col], pad]).reshape(chunks, 64).sum(axis=1)
        assert np.all(np.abs(got - want) <= 1e-4 * mag + 1e-30), (d, wide, inflight, slice_w)
    plan.close()


@pytest.mark.parametrize("d", [64, 256])
def test_cache_gather_probe_gathers_the_slice_rows(d):
    # the sampled product's probe streams the cached slice's columns (the
    # oracle's slice of the same selection) and loads exactly those rows
    A = synth.random_csr(3000, 2500, 400, seed=18, hub_rows=5, hub_len=2400)
    AT = synth.transpose(A, 2500)
    B = synth.dense_normal(2500, d, seed=19)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 2500)
    cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, 3000))
    Bd = torch.from_numpy(B).cuda()
    cache.refresh(Bd, 900, step=0)
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    _, mask = oracle.topk(oracle.pair_keys(cn2, B)["key"], 900)
    _, co, _ = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    nnz = len(co)
    chunks = (nnz + 63) // 64
    for inflight in (4, 8, 16):
        sink = torch.full((max(chunks, 1),), float("nan"), device="cuda")
        slice_w = cache.gather_probe(Bd, inflight=inflight, sink=sink)
        got = sink[:chunks].cpu().numpy().astype(np.float64)
        f_last = ((d - 1) // slice_w) * slice_w
        part = B[:, f_last:d].astype(np.float64)
        pad = np.zeros(chunks * 64 - nnz)
        want = np.concatenate([part.sum(axis=1)[co], pad]).reshape(chunks, 64).sum(axis=1)
        mag = np.concatenate([np.abs(part).sum(axis=1)[co], pad]).reshape(chunks, 64).sum(axis=1)
        assert np.all(np.abs(got - want) <= 1e-4 * mag + 1e-30), (d, inflight, slice_w)
    cache.close()


def _probe_out_expected(B, col, n_rows, d, slice_w):
    # row r of the probe's output, pass [f0, f0 + slice_w): the sum over the
    # 64-entry chunk w(r) of the gathered rows' slice, w(r) the chunk whose
    # share [w n_rows / W, (w + 1) n_rows / W) holds r
    nnz = len(col)
    W = (nnz + 63) // 64
    starts = (np.arange(W, dtype=np.int64) * n_rows) // W
    owner = np.searchsorted(starts, np.arange(n_rows), side="right") - 1
    want = np.empty((n_rows, d))
    mag = np.empty((n_rows, d))
    pad = np.zeros(W * 64 - nnz)
    for f0 in range(0, d, slice_w):
        part = B[:, f0:f0 + slice_w].astype(np.float64)
        s = np.concatenate([part.sum(axis=1)[col], pad]).reshape(W, 64).sum(axis=1)
        m = np.concatenate([np.abs(part).sum(axis=1)[col], pad]).reshape(W, 64).sum(axis=1)
        want[:, f0:f0 + slice_w] = s[owner][:, None]
        mag[:, f0:f0 + slice_w] = m[owner][:, None]
    return want, mag


@pytest.mark.parametrize("d", [66, 100, 256, 512])
@pytest.mark.parametrize("n_rows", [3000, 40])
def test_gather_probe_output_stream(d, n_rows):
    # With an output, the probe writes every element of the n_rows x d rows
    # (each its chunk's pass sum, so the stores follow the gathers), into a
    # padded view, leaving the padding alone; fewer rows than 64-entry chunks
    # (40 rows) leaves some chunks without rows.
    A = synth.random_csr(n_rows, 2500, 60000 // n_rows, seed=28, hub_rows=2, hub_len=2000)
    B = synth.dense_normal(2500, d, seed=29)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 2500)
    plan = rsc.SpmmPlan(X)
    ld = (d + 3) // 4 * 4 + 8
    Bd = torch.zeros((2500, ld), device="cuda")
    Bd[:, :d] = torch.from_numpy(B).cuda()
    Bd = Bd[:, :d]
    for inflight in (4, 16):
        wide = torch.full((n_rows, ld), 7777.0, device="cuda")
        out = wide[:, :d]
        slice_w = plan.gather_probe(Bd, inflight=inflight, out=out)
        got = wide.cpu().numpy()
        assert np.all(got[:, d:] == 7777.0)
        want, mag = _probe_out_expected(B, A.col, n_rows, d, slice_w)
        g = got[:, :d].astype(np.float64)
        assert np.all(np.abs(g - want) <= 1e-4 * mag + 1e-30), (d, n_rows, inflight, slice_w)
    with pytest.raises(ValueError, match="holds less"):   # refused before any launch
        plan.gather_probe(Bd, out=torch.empty((n_rows - 1, d), device="cuda"))
    with pytest.raises(rsc.RscError):                        # ld not a multiple of 4
        plan.gather_probe(Bd, out=torch.empty((n_rows, d + 1), device="cuda")[:, :d])
    plan.close()


@pytest.mark.parametrize("d", [64, 256])
def test_cache_gather_probe_output_stream(d):
    A = synth.random_csr(3000, 2500, 400, seed=38, hub_rows=5, hub_len=2400)
    AT = synth.transpose(A, 2500)
    B = synth.dense_normal(2500, d, seed=39)
    X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, 2500)
    cache = rsc.Cache(X, rsc.DeviceCsr.from_host(AT.rowptr, AT.col, AT.val, 3000))
    Bd = torch.from_numpy(B).cuda()
    cache.refresh(Bd, 700, step=0)
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    _, mask = oracle.topk(oracle.pair_keys(cn2, B)["key"], 700)
    _, co, _ = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    out = torch.full((3000, d), float("nan"), device="cuda")
    slice_w = cache.gather_probe(Bd, inflight=8, out=out)
    want, mag = _probe_out_expected(B, co, 3000, d, slice_w)
    g = out.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(g - want) <= 1e-4 * mag + 1e-30), (d, slice_w)
    cache.close()
