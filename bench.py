"""Benchmark of the RSC aggregation hot path on one MI355X.

One step = one pass of the whole hot path over the workload, in the order a
GCN training step uses it (sections 3.1 and 3.3): the exact forward SpMM
Y = A_hat H (through an SpMM plan of the static A_hat, made once before
timing); the cache lookup, and every `refresh_interval` steps a cache
refresh (pair scores of A_hat^T and the backward operand G, top-k at the
column budget, CSR column slice); then the sampled backward SpMM
G' = A_hat^T[:, S] G on the cached slice. H and G are resident in HBM before
timing starts. The column budget k = floor(n * pct / 100) is computed once.

Prints ONE JSON line. `value` is the step's algorithmic HBM bytes (exact +
sampled SpMM compulsory traffic, plus one tenth of a refresh) divided by the
measured step time, in GB/s. `roofline` describes the dominant kernel (the
exact SpMM): algorithmic bytes per launch over its average duration measured
with HIP events on the stream the kernels run on, against the 8 TB/s HBM
peak. `cpu_baseline` times the oracle (all its OpenMP threads) on a bounded
sample of the same step. `vendor_baseline` times rocSPARSE's SpMM on the
exact product's operands beside the library's (context only).

usage: python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload copurchase]
                       [--budget-pct 30] [--features D] [--aggregator gcn|mean] [--selector topk|random]
                       [--no-cpu-baseline] [--no-vendor-baseline]
       python bench.py --workload gcn2-train [--budget-pct 10]   (training-step comparison)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def counters_path(workload: str) -> str:
    """The committed rocprofv3 counter record of a workload's SpMM calls."""
    return os.path.join(ROOT, "profiles", f"spmm_{workload}_counters.json")


def spmm_bytes(n: int, nnz: int, n_src: int, d: int) -> int:
    """Compulsory HBM bytes of one SpMM launch: rowptr (4(n+1)), col + val
    (8 per entry), each referenced B row once (4 d per source row), and Y
    written once (4 n d)."""
    return 4 * (n + 1) + 8 * nnz + 4 * n_src * d + 4 * n * d


def refresh_bytes(n: int, nnz: int, nnz_kept: int, k: int, d: int) -> int:
    """Algorithmic bytes of one cache refresh: B row norms (4nd) with cn2 in
    (8n) and keys out (8n); six histogram passes and two tile passes over the
    keys (8 * 8n); the slice's count pass over col (4 nnz) and compaction
    pass over col + val (8 nnz), rowptr in/out (8(n+1)), kept entries out
    (8 nnz'); idx and mask out (4k + n/8)."""
    return (4 * n * d + 16 * n + 64 * n + 12 * nnz + 8 * (n + 1) + 8 * nnz_kept
            + 4 * k + n // 8)


def refresh_random_bytes(n: int, nnz: int, nnz_kept: int, k: int, d: int) -> int:
    """Algorithmic bytes of one randomized refresh: B row norms with cn2 in and
    keys out (4nd + 16n); key max and weight passes (16n), w out and back in
    (16n), the prefix W out (8n); k draws (one 8-byte CDF read and one 4-byte
    count update each); count zeroing, the per-column pass over count, w and W
    writing colw (4n + 20n + 8n) and the mask (n/8); the slice as for top-k
    (12 nnz + 8(n+1) + 8 nnz') plus one 8-byte scale per kept entry."""
    return (4 * n * d + 16 * n + 16 * n + 16 * n + 8 * n + 12 * k + 32 * n + n // 8
            + 12 * nnz + 8 * (n + 1) + 16 * nnz_kept)


# The paper's own speedups (one RTX 3090, PyG/torch_sparse operators, the
# real datasets): context beside this run's `sampled_speedup`, not a target
# and not the same metric, so `vs_baseline` stays null.
PAPER_CONTEXT = {
    "hardware": "RTX 3090 (PyG / torch_sparse operators, real datasets)",
    "bwd_spmm_speedup_max": {"value": 11.6, "dataset": "Reddit", "source": "Table 2"},
    "bwd_spmm_speedup_copurchase": {"value": 8.98, "dataset": "ogbn-products", "source": "Table 2"},
    "end_to_end_speedup_max": {"value": 1.60, "model": "GraphSAGE", "dataset": "ogbn-proteins",
                               "source": "Table 3"},
    "note": "context only",
}

COUNTED_SOURCES = ("spmm.hip", "probe.hip", "scores.hip", "topk.hip", "slice.hip")


def kernel_source_digest() -> str:
    """Digest of the kernel sources the counter records measure (the SpMM,
    the gather probe and the refresh's scores, top-k and slice), with
    comments and blank lines removed (a comment edit does not invalidate a
    counter record)."""
    import re
    code = []
    for name in COUNTED_SOURCES:
        with open(os.path.join(ROOT, "paper_2210_10737_amd", "csrc", name)) as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        lines = [re.sub(r"//.*", "", line).rstrip() for line in src.splitlines()]
        code.append("\n".join(line for line in lines if line.strip()))
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


COUNTER_CONFIG_KEYS = ("workload", "n", "nnz", "d", "budget_pct", "aggregator", "selector")


def load_traffic(config: dict, digest: str, op_bytes: dict):
    """Bytes past L2 per call of each operation (FETCH_SIZE + WRITE_SIZE,
    scaled by a 1 GiB copy) and L2 hit rates, from the workload's committed
    rocprofv3 counter record, if it was taken on the current kernel source
    and the same configuration; else None."""
    path = counters_path(config["workload"])
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_src_digest") != digest:
        return None
    if any(rec.get("config", {}).get(k_) != config.get(k_) for k_ in COUNTER_CONFIG_KEYS):
        return None
    out = {"source": os.path.relpath(path, ROOT), "ops": {}}
    for op, r in rec["ops"].items():
        tot = r["fetch_bytes"] + r["write_bytes"]
        out["ops"][op] = {"fetch_bytes": round(r["fetch_bytes"]), "write_bytes": round(r["write_bytes"]),
                          "total_bytes": round(tot), "l2_hit_rate": r.get("l2_hit_rate"),
                          "over_algorithmic": round(tot / op_bytes[op], 3) if op_bytes.get(op) else None}
    return out


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_ops(A, Hh, Gh, k, rows):
    """One pass of the hot path through the oracle, each operation timed on
    its own (seconds): the exact SpMM, the column square-norms cn2, the pair
    keys (row norms of the backward operand), the top-k selection (full
    sort), the CSR slice, and the sampled SpMM on the slice. With `rows` the
    two SpMMs compute only those rows."""
    import oracle
    t = {}
    t0 = time.perf_counter()
    oracle.spmm(A.rowptr, A.col, A.val, Hh, rows=rows)
    t["exact_spmm"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)   # A_hat is symmetric: its transpose's CSR is its own
    t["cn2"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    key = oracle.pair_keys(cn2, Gh)["key"]
    t["keys"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    idx, mask = oracle.topk(key, k)
    t["select"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    t["slice"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.spmm(ro, co, vo, Gh, rows=rows)
    t["sampled_spmm"] = time.perf_counter() - t0
    return t


def cpu_baseline(A, Hh, Gh, k, pct, refresh_interval, step_bytes_full, n_rows_sample,
                 min_s: float = 10.0, max_reps: int = 5):
    """Oracle timing on the host cores of the machine the bench runs on:
    every operation of the hot path timed separately (exact SpMM, cn2, keys,
    select, slice, sampled SpMM), repeated until about min_s seconds of CPU
    work (at most max_reps), median per operation, with all the oracle's
    threads; the SpMMs on the
    first n_rows_sample rows (scaled linearly to the whole graph when that is
    fewer than all). The step time is exact + sampled SpMM plus one refresh
    (keys, select, slice) per refresh_interval steps; cn2 is computed once per
    graph and reported apart. Then the tiny workload (4,096 nodes) the same
    way on one thread and on all of them, in this process."""
    import numpy as np

    import oracle
    import synth
    n = A.n
    rows = None if n_rows_sample >= n else np.arange(n_rows_sample, dtype=np.int32)
    scale = 1.0 if rows is None else n / n_rows_sample
    cores = oracle.num_threads()
    reps = []
    t_all = time.perf_counter()
    while len(reps) < max_reps and (time.perf_counter() - t_all < min_s or not reps):
        reps.append(_oracle_ops(A, Hh, Gh, k, rows))
    measured = time.perf_counter() - t_all
    med = {op: float(np.median([r[op] for r in reps])) for op in reps[0]}
    for op in ("exact_spmm", "sampled_spmm"):
        med[op] *= scale
    refresh_s = med["keys"] + med["select"] + med["slice"]
    step_s = med["exact_spmm"] + med["sampled_spmm"] + refresh_s / refresh_interval

    # the tiny workload on one core and on all of them (same process)
    w = synth.WORKLOADS["tiny"]
    At = synth.make_graph("tiny", 0)
    Ht = synth.dense_normal(At.n, w.d, seed=1)
    Gt = synth.dense_normal(At.n, w.d, seed=3)
    kt = (At.n * w.budgets_pct[0]) // 100
    tiny = {}
    try:
        for label, threads in (("one_core", 1), ("all_cores", cores)):
            oracle.set_num_threads(threads)
            rt = [_oracle_ops(At, Ht, Gt, kt, None) for _ in range(5)]
            tiny[label] = {"threads": oracle.num_threads(),
                           "ms": {op: round(float(np.median([r[op] for r in rt])) * 1e3, 3) for op in rt[0]}}
    finally:
        oracle.set_num_threads(cores)
    return {
        "value": round(step_bytes_full / step_s / 1e9, 3),
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (("exact and sampled SpMM over every row" if rows is None else
                    f"exact and sampled SpMM on rows [0, {n_rows_sample}) of {n} (x{scale:.1f} to the full graph)")
                   + f"; cn2, keys, top-k at {pct}% and slice on the whole graph, the refresh amortised over "
                   f"{refresh_interval} steps; {len(reps)} repetitions, median per operation"),
        "ms_per_step": round(step_s * 1e3, 1),
        "ops_ms": {op: round(v * 1e3, 2) for op, v in med.items()},
        "exact_spmm_ms": round(med["exact_spmm"] * 1e3, 1),
        "sampled_spmm_ms": round(med["sampled_spmm"] * 1e3, 1),
        "refresh_ms": round(refresh_s * 1e3, 1),
        "tiny_workload": {"n": At.n, "nnz": At.nnz, "d": w.d, "budget_pct": w.budgets_pct[0], **tiny},
        "cpu_model": _cpu_model(),
        "measured_s": round(measured, 2),
    }


ROCSPARSE = "/opt/rocm/lib/librocsparse.so"


class RocsparseSpmm:
    """rocSPARSE's generic SpMM (rocsparse_spmm) set up on one CSR operand X
    (int32 indices, fp32) and one row-major dense B: run(alg) writes
    C = X B into a row-major n_rows x d tensor, after the algorithm's
    preprocess stage. The vendor library, used as a timing baseline and a
    cross-check only; raises OSError when the library cannot be loaded and
    RuntimeError on a rocSPARSE error status."""

    # enumerator values of the rocSPARSE C API
    OP_NONE, IDX_I32, BASE_ZERO, F32, ORDER_ROW = 111, 2, 0, 151, 0
    STAGE_BUFFER, STAGE_PREPROCESS, STAGE_COMPUTE = 1, 2, 3
    ALGS = {"default": 0, "csr_nnz_split": 5}

    def __init__(self, X, B):
        import ctypes

        import torch
        self.ct, self.torch = ctypes, torch
        self.X, self.B = X, B   # the descriptors hold raw pointers: keep the tensors alive
        self.L = ctypes.CDLL(ROCSPARSE)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        self.h, self.mA, self.mB, self.mC = vp(), vp(), vp(), vp()
        self.C = torch.empty((X.n_rows, B.shape[1]), dtype=torch.float32, device=B.device)
        self._check(self.L.rocsparse_create_handle(ctypes.byref(self.h)), "create handle")
        try:
            ver = ctypes.c_int(0)
            self.L.rocsparse_get_version(self.h, ctypes.byref(ver))
            self.version = f"{ver.value // 100000}.{ver.value // 100 % 1000}.{ver.value % 100}"
            self._check(self.L.rocsparse_set_stream(self.h, vp(torch.cuda.current_stream().cuda_stream)), "stream")
            self._check(self.L.rocsparse_create_csr_descr(
                ctypes.byref(self.mA), i64(X.n_rows), i64(X.n_cols), i64(X.nnz), vp(X.rowptr.data_ptr()),
                vp(X.col.data_ptr()), vp(X.val.data_ptr()), self.IDX_I32, self.IDX_I32, self.BASE_ZERO, self.F32),
                "CSR descriptor")
            self._check(self.L.rocsparse_create_dnmat_descr(
                ctypes.byref(self.mB), i64(X.n_cols), i64(B.shape[1]), i64(B.stride(0)), vp(B.data_ptr()), self.F32,
                self.ORDER_ROW), "B descriptor")
            self._check(self.L.rocsparse_create_dnmat_descr(
                ctypes.byref(self.mC), i64(X.n_rows), i64(B.shape[1]), i64(B.shape[1]), vp(self.C.data_ptr()),
                self.F32, self.ORDER_ROW), "C descriptor")
        except RuntimeError:
            self.close()
            raise
        self.alpha, self.beta = ctypes.c_float(1.0), ctypes.c_float(0.0)
        self.bufs, self.sizes = {}, {}

    @staticmethod
    def _check(status, what):
        if status != 0:
            raise RuntimeError(f"rocSPARSE {what}: status {status}")

    def _call(self, alg, stage, buf):
        ct = self.ct
        size = ct.c_size_t(0)
        st = self.L.rocsparse_spmm(self.h, self.OP_NONE, self.OP_NONE, ct.byref(self.alpha), self.mA, self.mB,
                                   ct.byref(self.beta), self.mC, self.F32, self.ALGS[alg], stage, ct.byref(size),
                                   buf)
        return st, size.value

    def prepare(self, alg):
        """Buffer and preprocess stages of one algorithm (once per algorithm)."""
        if alg not in self.bufs:
            st, size = self._call(alg, self.STAGE_BUFFER, None)
            self._check(st, "buffer size")
            buf = self.torch.empty(max(size, 256), dtype=self.torch.uint8, device=self.C.device)
            self._check(self._call(alg, self.STAGE_PREPROCESS, self.ct.c_void_p(buf.data_ptr()))[0], "preprocess")
            self.bufs[alg], self.sizes[alg] = buf, size
        return self.sizes[alg]

    def run(self, alg="csr_nnz_split"):
        self.prepare(alg)
        self._check(self._call(alg, self.STAGE_COMPUTE, self.ct.c_void_p(self.bufs[alg].data_ptr()))[0], "compute")
        return self.C

    def close(self):
        self.torch.cuda.synchronize()
        if self.mA.value:
            self.L.rocsparse_destroy_spmat_descr(self.mA)
        for m in (self.mB, self.mC):
            if m.value:
                self.L.rocsparse_destroy_dnmat_descr(m)
        if self.h.value:
            self.L.rocsparse_destroy_handle(self.h)
        self.h, self.mA, self.mB, self.mC = (self.ct.c_void_p() for _ in range(4))
        self.bufs.clear()
        self.X = self.B = None


def vendor_baseline(X, H, Y, plan, reps: int = 10):
    """The vendor library's sparse-dense product on the same operands as the
    exact SpMM, timed beside it (context, like the CPU baseline; the product
    path never calls it): rocsparse_spmm on the CSR (int32 indices, fp32),
    row-major B and C, the preprocess stage run before timing, with the
    library's default CSR algorithm and its nnz-split one. Returns None when
    the library cannot be loaded."""
    import statistics

    import torch

    def median_ms(fn):
        for _ in range(2):
            fn()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return statistics.median(ts)

    ours = median_ms(lambda: plan.run(H, out=Y))
    try:
        v = RocsparseSpmm(X, H)
    except OSError:
        return None
    except RuntimeError as e:
        return {"library": "rocSPARSE", "error": str(e)}
    out = {"library": "rocSPARSE", "version": v.version,
           "call": "rocsparse_spmm, CSR int32 / fp32, row-major B and C", "ours_ms": round(ours, 4),
           "algorithms": {}}
    try:
        for alg in RocsparseSpmm.ALGS:
            try:
                buf_bytes = v.prepare(alg)
                C = v.run(alg)
                torch.cuda.synchronize()
                diff = float((C - Y).abs().max() / Y.abs().max().clamp_min(1e-30))
                ms = median_ms(lambda: v.run(alg))
            except RuntimeError as e:
                out["algorithms"][alg] = {"error": str(e)}
                continue
            out["algorithms"][alg] = {"ms": round(ms, 4), "buffer_bytes": buf_bytes,
                                      "max_abs_diff_over_max_abs": diff}
    finally:
        v.close()
    best = min((a["ms"] for a in out["algorithms"].values() if "ms" in a), default=None)
    out["vendor_best_over_ours"] = None if best is None else round(best / ours, 3)
    return out


def gather_ceiling(handle, B, d, n_entries, reps: int = 5, out=None):
    """Times a gather probe (rsc_spmm_plan_gather_probe for a plan, the exact
    product's B-row gathers alone; rsc_cache_gather_probe for a cache, the
    sampled product's) at 4, 8 and 16 loads in flight per wave, median of
    `reps` each after one untimed run; the fastest setting is the ceiling.
    With `out` (a scratch tensor of the product's output shape) the probe
    also writes the product's output stream. HIP events on the current
    stream, which the library launches on."""
    import statistics

    import torch
    sink = torch.empty(max((n_entries + 63) // 64, 1), dtype=torch.float32, device=B.device)
    per, slice_w = {}, None
    for inflight in (4, 8, 16):
        slice_w = handle.gather_probe(B, d=d, inflight=inflight, sink=sink, out=out)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            handle.gather_probe(B, d=d, inflight=inflight, sink=sink, out=out)
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        per[inflight] = statistics.median(ts)
    best = min(per, key=per.get)
    ms = per[best]
    return {"ms": round(ms, 4), "inflight": best, "slice_floats": slice_w,
            "ms_by_inflight": {str(k_): round(v, 4) for k_, v in per.items()},
            "logical_gather_GBs": round(4.0 * n_entries * d / (ms * 1e-3) / 1e9, 1),
            "what": ("the product's B-row gathers alone: same column stream (a plan's hinted copy), "
                     "feature passes and cache policy; no values, row walk or output") if out is None else
                    ("the product's B-row gathers and its output stream (each wave writes an even share "
                     "of the output rows after its gathers); no values or row walk")}


def parity_check(A, Hh, Gh, k, Y, Yb, kept, n_rows, seed):
    """The benchmarked outputs against the oracle: the kept columns bit for
    bit, and the exact and sampled products on a seeded sample of rows
    (max |Y - Y_oracle| / max(S, FLT_MIN), S = sum |a||b|)."""
    import numpy as np
    import torch

    import oracle
    rng = np.random.Generator(np.random.PCG64(seed + 11))
    rows = np.sort(rng.choice(A.n, size=min(A.n, n_rows), replace=False)).astype(np.int32)
    tiny = np.float32(np.finfo(np.float32).tiny)

    def err(Yd, rowptr, col, val, Bh):
        Yo, S = oracle.spmm(rowptr, col, val, Bh, rows=rows, with_mag=True)
        got = Yd[torch.from_numpy(rows.astype(np.int64)).to(Yd.device)].cpu().numpy().astype(np.float64)
        return float(np.max(np.abs(got - Yo) / np.maximum(S, tiny)))

    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    idx_o, mask_o = oracle.topk(oracle.pair_keys(cn2, Gh)["key"], k)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask_o)
    return {"rows_checked": int(len(rows)),
            "kept_columns_equal": bool(np.array_equal(np.asarray(kept), idx_o[:k])),
            "exact_max_rel_err": err(Y, A.rowptr, A.col, A.val, Hh),
            "sampled_max_rel_err": err(Yb, ro, co, vo, Gh),
            "tolerance": {"exact": 1e-5, "sampled": 1e-4}}


def train_bench(args) -> int:
    """Two-layer GCN training on the gcn2 workload (716,847 nodes, 300 input
    features, hidden 512, 100 labels, multi-label BCE, Adam): exact training
    against RSC training (exact forward, cached top-k backward, greedy
    allocation and refresh every `refresh` steps, FLOPs budget C). Every
    timed step includes forward, backward and the optimizer update; RSC steps
    include the greedy and refreshes."""
    import numpy as np
    import torch

    import paper_2210_10737_amd as rsc
    import synth
    from paper_2210_10737_amd.gcn import GCN, RscConfig

    torch.cuda.set_device(0)
    torch.backends.cuda.matmul.allow_tf32 = False
    w = synth.WORKLOADS["gcn2"]
    p = w.params
    pct = args.budget_pct if args.budget_pct is not None else 10
    A = synth.make_graph("gcn2", args.seed)
    n = A.n
    X = torch.from_numpy(synth.dense_normal(n, p["in_features"], seed=args.seed + 1)).cuda()
    rng = np.random.Generator(np.random.PCG64(args.seed + 4))
    Y = torch.from_numpy((rng.random((n, p["classes"]), dtype=np.float32) < 0.5).astype(np.float32)).cuda()
    Ad = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)
    print(f"[bench] gcn2 training: n={n} nnz={A.nnz} hidden={p['hidden']} classes={p['classes']} "
          f"C={pct}%", file=sys.stderr, flush=True)
    results = {}
    for name, enabled in (("exact", False), ("rsc", True)):
        cfg = RscConfig(budget=(pct, 100), alpha=(2, 100), refresh_interval=args.refresh, enabled=enabled)
        model = GCN(Ad, p["in_features"], p["hidden"], p["classes"], cfg, seed=args.seed + 2)
        opt = torch.optim.Adam(model.parameters(), lr=0.01)
        for s in range(args.warmup):
            model.train_step(X, Y, opt, s)
        torch.cuda.synchronize()
        for layer in (model.agg1, model.agg2):
            layer.timings = []   # events around each SpMM: its share of the step (Fig. 1)
        t0 = time.perf_counter()
        losses = []
        for s in range(args.warmup, args.warmup + args.steps):
            losses.append(model.train_step(X, Y, opt, s).detach())
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        spmm_ms = {"forward": 0.0, "backward": 0.0}
        for layer in (model.agg1, model.agg2):
            for kind, a, b in layer.timings:
                spmm_ms[kind] += a.elapsed_time(b) / args.steps
            layer.timings = None
        hist = model.controller.history[args.warmup:]
        greedy = [r.greedy_s * 1e3 for r in hist if r.mode == "score"]
        results[name] = {"ms_per_step": round(ms, 3), "final_loss": round(float(losses[-1]), 5),
                         "refresh_steps": sum(r.mode == "score" for r in hist),
                         "greedy_ms_per_call": round(float(np.mean(greedy)), 2) if greedy else None,
                         "k_per_layer": hist[-1].k,
                         "spmm_fwd_ms_per_step": round(spmm_ms["forward"], 3),
                         "spmm_bwd_ms_per_step": round(spmm_ms["backward"], 3),
                         "spmm_share": round((spmm_ms["forward"] + spmm_ms["backward"]) / ms, 4)}
        model.close()
        del model, opt
        torch.cuda.empty_cache()
    ablation = None
    if args.ablation_steps > 0:
        # caching / switching ablation (Table 4's layout): a whole run of
        # `ablation_steps` steps per setting, timed end to end; "no cache"
        # selects and slices against each step's own gradient (k_l still
        # allocated every `refresh` steps), "switch" runs the last 20 % of
        # the steps exact
        def run(enabled, cache_on, total):
            cfg = RscConfig(budget=(pct, 100), alpha=(2, 100), refresh_interval=args.refresh, enabled=enabled,
                            total_steps=total, cache=cache_on)
            model = GCN(Ad, p["in_features"], p["hidden"], p["classes"], cfg, seed=args.seed + 2)
            opt = torch.optim.Adam(model.parameters(), lr=0.01)
            model.train_step(X, Y, opt, 0)    # untimed: first-call costs
            model.controller.last_refresh = None
            model.controller.history.clear()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for s_ in range(args.ablation_steps):
                model.train_step(X, Y, opt, s_)
            torch.cuda.synchronize()
            ms_ = (time.perf_counter() - t0) * 1e3 / args.ablation_steps
            model.close()
            del model, opt
            torch.cuda.empty_cache()
            return ms_
        T = args.ablation_steps
        base = run(False, True, None)
        ablation = {"steps": T, "exact_ms_per_step": round(base, 3)}
        for cache_on in (False, True):
            for switch_on in (False, True):
                ms_ = run(True, cache_on, T if switch_on else None)
                ablation[f"cache={'yes' if cache_on else 'no'},switch={'yes' if switch_on else 'no'}"] = {
                    "ms_per_step": round(ms_, 3), "speedup": round(base / ms_, 3)}
    staleness = None
    if args.staleness_steps > 0:
        # untimed diagnostic run: AUC / overlap of each layer's selection
        # between consecutive refreshes, and the k_l trace (Figs. 4 and 7)
        cfg = RscConfig(budget=(pct, 100), alpha=(2, 100), refresh_interval=args.refresh,
                        track_staleness=True)
        model = GCN(Ad, p["in_features"], p["hidden"], p["classes"], cfg, seed=args.seed + 2)
        opt = torch.optim.Adam(model.parameters(), lr=0.01)
        for s_ in range(args.staleness_steps):
            model.train_step(X, Y, opt, s_)
        recs = [r for r in model.controller.history if r.mode == "score"]
        staleness = {"steps": args.staleness_steps,
                     "refresh_steps": [r.step for r in recs],
                     "k_trace": [r.k for r in recs],
                     "auc": [[round(a, 5) for a in r.auc] for r in recs[1:]],
                     "overlap": [[round(o, 5) for o in r.overlap] for r in recs[1:]]}
        model.close()
        del model, opt
    out = {
        "metric": "GCN training step ms (exact vs RSC) on 1 MI355X",
        "value": round(results["exact"]["ms_per_step"] / results["rsc"]["ms_per_step"], 3),
        "unit": "x speedup (exact step / RSC step)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": results["rsc"]["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "gcn2-train", "n": n, "nnz": A.nnz, "in_features": p["in_features"],
                   "hidden": p["hidden"], "classes": p["classes"], "budget_pct": pct,
                   "refresh_interval": args.refresh, "alpha_pct": 2, "seed": args.seed},
        "exact": results["exact"], "rsc": results["rsc"],
        "ablation": ablation,
        "staleness": staleness,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="copurchase")
    ap.add_argument("--budget-pct", type=int, default=None)
    ap.add_argument("--features", type=int, default=None,
                    help="feature width d of the dense operands (default: the workload's)")
    ap.add_argument("--refresh", type=int, default=10)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=None,
                    help="rows of the CPU-baseline SpMM sample (default: all rows)")
    ap.add_argument("--aggregator", choices=("gcn", "mean"), default="gcn",
                    help="gcn: A_hat = D^-1/2 (A+I) D^-1/2 (symmetric); mean: the MEAN aggregator "
                         "D^-1 (A+I) forward, its transpose (A+I) D^-1 in the backward")
    ap.add_argument("--selector", choices=("topk", "random"), default="topk",
                    help="topk: the k pairs with the largest scores, unscaled (section 2.2.1); random: k "
                         "i.i.d. draws with p_i proportional to the pair score, scaled by 1/(k p_i) "
                         "(Eq. 2 with Eq. 3)")
    ap.add_argument("--ablation-steps", type=int, default=50,
                    help="gcn2-train only: steps per setting of the caching / switching ablation (0 = skip)")
    ap.add_argument("--staleness-steps", type=int, default=60,
                    help="gcn2-train only: steps of the untimed selection-staleness run (0 = skip)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the exact + sampled SpMM of each step from one captured HIP graph "
                         "(refreshes stay eager)")
    ap.add_argument("--parity-rows", type=int, default=2000,
                    help="after timing, check this many sampled output rows and the kept columns against "
                         "the oracle (0 = skip)")
    ap.add_argument("--cold-reps", type=int, default=5,
                    help="after the timed steps, repetitions of each op that follow a 1 GiB cache flush")
    ap.add_argument("--no-vendor-baseline", action="store_true",
                    help="skip timing the vendor library's SpMM (rocSPARSE) on the exact product's operands")
    ap.add_argument("--marked-ops", type=int, default=0,
                    help="after timing, run this many rounds of exact SpMM, refresh, sampled SpMM and gather "
                         "probe, each operation between two launches of a 3-byte uint8 fill (markers for "
                         "attributing profiler counters to operations)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after timing, copy a buffer of this many MiB once (a plain copy of known "
                         "size, so hardware byte counters can be scaled)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        return 2

    if args.workload == "gcn2-train":
        return train_bench(args)

    import numpy as np
    import torch

    import paper_2210_10737_amd as rsc
    import synth

    torch.cuda.set_device(0)
    w = synth.WORKLOADS[args.workload]
    pct = args.budget_pct if args.budget_pct is not None else w.budgets_pct[-1 if args.workload != "social" else 1]
    d = args.features if args.features else w.d
    if d < 1:
        raise SystemExit("--features must be at least 1")
    t_gen = time.perf_counter()
    A = synth.make_graph(args.workload, args.seed)
    Hh = synth.dense_normal(A.n, d, seed=args.seed + 1)
    Gh = synth.dense_normal(A.n, d, seed=args.seed + 3)
    t_gen = time.perf_counter() - t_gen
    n, nnz = A.n, A.nnz
    deg_all = np.diff(A.rowptr)
    deg_stats = {"max": int(deg_all.max()), "p50": float(np.percentile(deg_all, 50)),
                 "p99": float(np.percentile(deg_all, 99)), "mean": round(float(deg_all.mean()), 2)}
    print(f"[bench] {args.workload}: n={n} nnz={nnz} d={d} budget={pct}% seed={args.seed} "
          f"row lengths max/p50/p99 {deg_stats['max']}/{deg_stats['p50']:.0f}/{deg_stats['p99']:.0f} "
          f"(inputs {t_gen:.1f}s)",
          file=sys.stderr, flush=True)

    if args.aggregator == "gcn":
        X = rsc.DeviceCsr.from_host(A.rowptr, A.col, A.val, n)  # A_hat is symmetric: A_hat^T = A_hat
        XB = XT = X
    else:
        # MEAN aggregator on the same (symmetric) structure with unit values:
        # forward D^-1 A, backward operand A^T D^-1 (whose column norms come
        # from its transpose, D^-1 A)
        ones = rsc.DeviceCsr.from_host(A.rowptr, A.col, np.ones_like(A.val), n)
        X = rsc.degree_scale(ones)
        XB = rsc.degree_scale(ones, by_column=True, deg_rowptr=ones.rowptr)
        XT = X
    H = torch.from_numpy(Hh).cuda()
    G = torch.from_numpy(Gh).cuda()
    Y = torch.empty((n, d), dtype=torch.float32, device="cuda")
    Yb = torch.empty((n, d), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    tp = time.perf_counter()
    plan = rsc.SpmmPlan(X)   # the static forward operand: prepared once, as a training run would
    plan_create_ms = (time.perf_counter() - tp) * 1e3
    k = rsc.k_from_fraction(n, pct, 100)
    cache = rsc.Cache(XB, XT, refresh_interval=args.refresh)
    torch.cuda.synchronize()

    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    records = []   # (kind, start_event, end_event)

    def step(s: int, timed: bool):
        e0, e1 = ev(), ev()
        e0.record()
        plan.run(H, out=Y)                     # forward, exact
        e1.record()
        if timed:
            records.append(("exact", e0, e1))
        if cache.get(s, with_slice=False)["needs_refresh"]:
            r0, r1 = ev(), ev()
            r0.record()
            if args.selector == "topk":
                cache.refresh(G, k, step=s)
            else:
                cache.refresh_random(G, k, seed=args.seed * 1_000_003 + s, step=s)
            r1.record()
            if timed:
                records.append(("refresh", r0, r1))
        s0, s1 = ev(), ev()
        s0.record()
        cache.spmm_sampled(G, out=Yb)                    # backward, sampled on the cached slice
        s1.record()
        if timed:
            records.append(("sampled", s0, s1))

    for s in range(args.warmup):
        step(s, False)
    torch.cuda.synchronize()
    if args.graph:
        # in graph mode, per-op times come from eager steps run before capture
        for s in range(args.warmup, args.warmup + args.steps):
            step(s, True)
        torch.cuda.synchronize()
    eager_records = records[:]
    records.clear()
    graph = None
    if args.graph:
        # one HIP graph holds the exact and the sampled SpMM of a step (kernel
        # launches only); refreshes stay eager, every `refresh` steps
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            plan.run(H, out=Y)
            cache.spmm_sampled(G, out=Yb)
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(graph):
            plan.run(H, out=Y)
            cache.spmm_sampled(G, out=Yb)
        torch.cuda.synchronize()

        def step(s: int, timed: bool):  # noqa: F811
            if cache.get(s, with_slice=False)["needs_refresh"]:
                r0, r1 = ev(), ev()
                r0.record()
                if args.selector == "topk":
                    cache.refresh(G, k, step=s)
                else:
                    cache.refresh_random(G, k, seed=args.seed * 1_000_003 + s, step=s)
                r1.record()
                if timed:
                    records.append(("refresh", r0, r1))
            graph.replay()

        for s in range(args.warmup):
            step(s, False)
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    g0, g1 = ev(), ev()
    g0.record()
    for s in range(args.warmup, args.warmup + args.steps):
        step(s, True)
    g1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = g0.elapsed_time(g1)
    if graph is not None:
        # per-op times of the eager steps that preceded capture stand for the ops
        records.extend(eager_records)

    per = {"exact": [], "refresh": [], "sampled": []}
    for kind, a, b in records:
        per[kind].append(a.elapsed_time(b))
    snap = cache.get(args.warmup + args.steps)
    nnz_kept = int(snap["slice"].nnz)
    mask_words = rsc.copy_to_host(cache.buffers()[4], (n + 31) // 32, np.uint32)
    idx = np.flatnonzero(np.unpackbits(mask_words.view(np.uint8), bitorder="little")[:n])
    # approximation quality of the last backward (a diagnostic outside the
    # timed region): relative Frobenius error of the sampled product
    Yx = rsc.spmm(XB, G)
    approx_err = float(torch.linalg.norm((Yb - Yx).double()) / torch.linalg.norm(Yx.double()))
    del Yx
    deg = np.diff(A.rowptr)
    exact_ms = float(np.mean(per["exact"]))
    sampled_ms = float(np.mean(per["sampled"]))
    refresh_ms = float(np.mean(per["refresh"])) if per["refresh"] else None

    def stats(v):
        if not v:
            return None
        q = np.percentile(v, [10, 50, 90])
        return {"mean": round(float(np.mean(v)), 4), "p10": round(float(q[0]), 4),
                "p50": round(float(q[1]), 4), "p90": round(float(q[2]), 4), "n": len(v)}

    # the gather ceiling: the exact product's gathers alone (same column
    # stream, feature passes and cache policy; no values, rows or output),
    # at 4, 8 and 16 loads in flight per wave; the fastest is the ceiling
    probe = gather_ceiling(plan, H, d, nnz)
    nnz_s = int(cache.get(args.warmup + args.steps)["slice"].nnz)
    probe_sampled = gather_ceiling(cache, G, d, nnz_s)
    # the same with each product's output stream (into scratch of its shape)
    scratch_out = torch.empty_like(Y)
    probe_out = gather_ceiling(plan, H, d, nnz, out=scratch_out)
    probe_sampled_out = gather_ceiling(cache, G, d, nnz_s, out=scratch_out)
    del scratch_out

    # cold-cache repetitions, outside the timed steps: before each, write a
    # 1 GiB scratch buffer (more than the 4 MB L2s and the 256 MB MALL)
    scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    cold = {"exact": [], "sampled": [], "refresh": []}
    for r in range(args.cold_reps):
        for kind in ("exact", "refresh", "sampled"):
            scratch.fill_(float(r))
            e0, e1 = ev(), ev()
            e0.record()
            if kind == "exact":
                plan.run(H, out=Y)
            elif kind == "refresh":
                if args.selector == "topk":
                    cache.refresh(G, k, step=args.warmup + args.steps)
                else:
                    cache.refresh_random(G, k, seed=args.seed * 1_000_003 + args.warmup + args.steps,
                                         step=args.warmup + args.steps)
            else:
                cache.spmm_sampled(G, out=Yb)
            e1.record()
            cold[kind].append((e0, e1))
    # the measured copy ceiling: device-to-device copy of the 1 GiB buffer
    dst = torch.empty_like(scratch)
    copies = []
    for _ in range(5):
        e0, e1 = ev(), ev()
        e0.record()
        dst.copy_(scratch)
        e1.record()
        copies.append((e0, e1))
    torch.cuda.synchronize()
    cold = {kk: [a.elapsed_time(b) for a, b in v] for kk, v in cold.items()}
    copy_ms = float(np.median([a.elapsed_time(b) for a, b in copies]))
    copy_gbs = 2.0 * scratch.numel() * 4 / (copy_ms * 1e-3) / 1e9
    del scratch, dst
    ms_per_step = max(wall * 1e3, gpu_ms) / args.steps

    b_exact = spmm_bytes(n, nnz, n, d)
    b_sampled = spmm_bytes(n, nnz_kept, len(idx), d)
    b_refresh = (refresh_bytes(n, nnz, nnz_kept, k, d) if args.selector == "topk"
                 else refresh_random_bytes(n, nnz, nnz_kept, k, d))
    step_bytes = b_exact + b_sampled + b_refresh / args.refresh
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    achieved = b_exact / (exact_ms * 1e-3) / 1e9
    digest = kernel_source_digest()

    out = {
        "metric": "SpMM ms + achieved HBM GB/s (exact vs top-k sampled) on 1 MI355X; % of roofline",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "aggregator": args.aggregator, "graph": w.description,
                   "row_lengths": deg_stats,
                   "n": n, "nnz": nnz, "d": d,
                   "budget_pct": pct, "k": k, "selector": args.selector, "hip_graph": bool(args.graph), "exact_spmm": "plan",
                   "refresh_interval": args.refresh,
                   "seed": args.seed},
        "exact_spmm_ms": round(exact_ms, 4),
        "plan_create_ms": round(plan_create_ms, 2),   # one-time, outside the timed steps
        "sampled_spmm_ms": round(sampled_ms, 4),
        "refresh_ms": None if refresh_ms is None else round(refresh_ms, 4),
        "sampled_speedup": round(exact_ms / sampled_ms, 3),
        "backward_amortised_ms": round(sampled_ms + (refresh_ms or 0.0) / args.refresh, 4),
        "amortised_speedup": round(exact_ms / (sampled_ms + (refresh_ms or 0.0) / args.refresh), 3),
        "columns_kept": int(len(idx)),
        "nnz_kept": nnz_kept,
        "approx_rel_fro_error": round(approx_err, 5),
        "kept_nnz_frac": round(nnz_kept / nnz, 4),
        "mean_degree_selected": round(float(deg[idx].mean()), 2) if len(idx) else None,
        "mean_degree_all": round(float(deg.mean()), 2),
        "exact_logical_gather_GBs": round(4.0 * nnz * d / (exact_ms * 1e-3) / 1e9, 1),
        "ops_ms": {"warm": {kk: stats(v) for kk, v in per.items()},
                   "cold": {kk: stats(v) for kk, v in cold.items()}},
        "copy_ceiling_GBs": round(copy_gbs, 1),
        # each op's algorithmic bytes over its p50 time, against the HBM peak
        "ops_roofline": {
            kind: {"bytes": int(b), "p50_ms": round(float(np.median(per[kind])), 4),
                   "GBs": round(b / (float(np.median(per[kind])) * 1e-3) / 1e9, 1),
                   "frac": round(b / (float(np.median(per[kind])) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
            for kind, b in (("exact", b_exact), ("sampled", b_sampled), ("refresh", b_refresh)) if per[kind]},
        # the sampled product against its own gathers alone (the cache's probe)
        "sampled_gather_ceiling": dict(
            probe_sampled,
            frac_of_gather_ceiling=round(probe_sampled["ms"] / float(np.median(per["sampled"])), 4),
            with_output_stream=probe_sampled_out,
            frac_of_gather_output_ceiling=round(probe_sampled_out["ms"] / float(np.median(per["sampled"])), 4)),
        "roofline": {
            "bound": "hbm",
            "kernel": "spmm_long_kernel + spmm_rows_kernel (the exact SpMM, one plan run)",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "frac_of_copy_ceiling": round(achieved / copy_gbs, 4),
            # the same algorithmic bytes over the gather probe's time: the rate
            # the product would reach if it took no longer than its gathers
            "gather_ceiling_GBs": round(b_exact / (probe["ms"] * 1e-3) / 1e9, 2),
            "frac_of_gather_ceiling": round(probe["ms"] / exact_ms, 4),
            "gather_ceiling": probe,
            # gathers plus the product's output stream
            "frac_of_gather_output_ceiling": round(probe_out["ms"] / exact_ms, 4),
            "gather_output_ceiling": probe_out,
            "algorithmic_bytes_per_launch": b_exact,
            "avg_launch_ms": round(exact_ms, 4),
            "traffic": None,
            "kernel_src_digest": digest,
        },
    }
    if args.parity_rows > 0 and args.aggregator == "gcn" and args.selector == "topk":
        out["parity"] = parity_check(A, Hh, Gh, k, Y, Yb, idx, args.parity_rows, args.seed)
    cfg = {"workload": args.workload, "n": n, "nnz": nnz, "d": d, "budget_pct": pct,
           "aggregator": args.aggregator, "selector": args.selector}
    traffic = load_traffic(cfg, digest, {"exact": b_exact, "sampled": b_sampled, "refresh": b_refresh,
                                         "probe": b_exact})
    if traffic is not None and "exact" in traffic["ops"]:
        ex = traffic["ops"]["exact"]
        out["roofline"]["traffic"] = ex["total_bytes"]
        out["roofline"]["l2_hit_rate"] = ex["l2_hit_rate"]
        out["roofline"]["traffic_detail"] = traffic
    out["vendor_baseline"] = None if args.no_vendor_baseline else vendor_baseline(X, H, Y, plan)
    out["paper_context"] = PAPER_CONTEXT
    if args.marked_ops > 0:
        # for per-dispatch profiler counters: each operation's kernels between
        # two launches of a 3-byte uint8 fill, in the order exact SpMM,
        # refresh, sampled SpMM, gather probe
        mk = torch.zeros(3, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        for r in range(args.marked_ops):
            mk.fill_(1)
            plan.run(H, out=Y)
            mk.fill_(2)
            cache.refresh(G, k, step=args.warmup + args.steps) if args.selector == "topk" else \
                cache.refresh_random(G, k, seed=args.seed * 1_000_003 + r, step=args.warmup + args.steps)
            mk.fill_(3)
            cache.spmm_sampled(G, out=Yb)
            mk.fill_(4)
            plan.gather_probe(H, d=d, inflight=probe["inflight"])
            mk.fill_(5)
        torch.cuda.synchronize()
        out["marked_ops"] = args.marked_ops
    cache.close()
    plan.close()
    del X, XB, XT, H, G, Y, Yb, plan
    torch.cuda.empty_cache()
    if args.copy_probe_mib > 0:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_probe_bytes"] = src.numel() * 4
        del src, dst
    if not args.no_cpu_baseline and args.aggregator == "gcn" and args.selector == "topk":
        rows = args.cpu_rows or n
        print(f"[bench] gpu done ({ms_per_step:.3f} ms/step); timing the oracle on {rows} rows",
              file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(A, Hh, Gh, k, pct, args.refresh, step_bytes, rows)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
