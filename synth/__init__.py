"""Seeded synthetic inputs shaped like the paper's GCN workloads.

Shared by the GPU path's tests/bench and by the CPU oracle's tests; holds the
input recipe only (graph structure, the GCN normalisation that defines the
operand, and dense N(0,1) matrices), none of the aggregation, scoring,
selection or slicing arithmetic.

Workloads (structure stand-ins for the datasets of the paper's Table 6; the
datasets themselves are not used):

* ``tiny``        Erdos-Renyi G(4096, 16/(n-1)), d = 64, 50 % column budget.
* ``social``      Chung-Lu power law (exponent 2.1), n = 232,965, mean degree
                  ~490 (~114M nnz), d = 256, budgets 10/30/50 %.
* ``copurchase``  Chung-Lu power law (exponent 2.1), n = 2,449,029, mean ~50
                  (~126M nnz), d = 256, 30 % budget, slice reused 10 steps.
* ``protein``     Chung-Lu with weights ~U[450, 750], n = 132,534, mean ~600
                  (~79M nnz), d = 256, 30 % budget.
* ``gcn2``        Chung-Lu power law (exponent 2.1), n = 716,847, mean ~20
                  (~14.7M nnz); 2-layer GCN with 300 input features, hidden
                  512, 100 outputs.

Seeds: graph ``seed``, dense operand ``seed + 1``, weights ``seed + 2``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(verbose: bool = False) -> str:
    import subprocess
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", _LIB_PATH,
           os.path.join(_HERE, "gen.c"), "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        i32p = ctypes.POINTER(ctypes.c_int32)
        lib.syn_dense_normal.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_void_p]
        lib.syn_bucket_csr.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p]
        lib.syn_gcn_values.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.syn_er.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_double, ctypes.c_void_p,
                               ctypes.POINTER(i32p)]
        lib.syn_er.restype = ctypes.c_int64
        lib.syn_chung_lu_powerlaw.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_double,
                                              ctypes.c_double, ctypes.c_double, ctypes.c_int64,
                                              ctypes.c_void_p, ctypes.POINTER(i32p)]
        lib.syn_chung_lu_powerlaw.restype = ctypes.c_int64
        lib.syn_chung_lu_uniform.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_double,
                                             ctypes.c_double, ctypes.c_int64, ctypes.c_void_p,
                                             ctypes.POINTER(i32p)]
        lib.syn_chung_lu_uniform.restype = ctypes.c_int64
        lib.syn_copy_free.argtypes = [i32p, ctypes.c_int64, ctypes.c_void_p]
        _lib = lib
    return _lib


@dataclass
class Csr:
    """Host CSR: rowptr int32[n+1], col int32[nnz], val float32[nnz]."""
    n: int
    rowptr: np.ndarray
    col: np.ndarray
    val: np.ndarray

    @property
    def nnz(self) -> int:
        return int(self.rowptr[-1])

    def degrees(self) -> np.ndarray:
        return np.diff(self.rowptr)


def _finish(n: int, rowptr: np.ndarray, colp, nnz: int) -> Csr:
    lib = _load()
    col = np.empty(nnz, dtype=np.int32)
    lib.syn_copy_free(colp, nnz, col.ctypes.data)
    val = np.empty(nnz, dtype=np.float32)
    lib.syn_gcn_values(n, rowptr.ctypes.data, col.ctypes.data, val.ctypes.data)
    return Csr(n, rowptr, col, val)


def erdos_renyi(n: int, p: float, seed: int) -> Csr:
    """Symmetric G(n, p) with self-loops, GCN-normalised fp32 values."""
    lib = _load()
    rowptr = np.empty(n + 1, dtype=np.int32)
    colp = ctypes.POINTER(ctypes.c_int32)()
    nnz = lib.syn_er(seed, n, p, rowptr.ctypes.data, ctypes.byref(colp))
    return _finish(n, rowptr, colp, nnz)


def chung_lu_powerlaw(n: int, mean: float, gamma: float, wmax: float, draws: int, seed: int) -> Csr:
    lib = _load()
    rowptr = np.empty(n + 1, dtype=np.int32)
    colp = ctypes.POINTER(ctypes.c_int32)()
    nnz = lib.syn_chung_lu_powerlaw(seed, n, mean, gamma, wmax, draws, rowptr.ctypes.data,
                                    ctypes.byref(colp))
    return _finish(n, rowptr, colp, nnz)


def chung_lu_uniform(n: int, wlo: float, whi: float, draws: int, seed: int) -> Csr:
    lib = _load()
    rowptr = np.empty(n + 1, dtype=np.int32)
    colp = ctypes.POINTER(ctypes.c_int32)()
    nnz = lib.syn_chung_lu_uniform(seed, n, wlo, whi, draws, rowptr.ctypes.data, ctypes.byref(colp))
    return _finish(n, rowptr, colp, nnz)


def dense_normal(rows: int, cols: int, seed: int, ld: int | None = None) -> np.ndarray:
    """rows x cols fp32 ~ N(0,1) (Box-Muller on counter-based draws). With
    ``ld > cols`` the returned array is rows x ld with zero padding."""
    lib = _load()
    ld = cols if ld is None else ld
    out = np.zeros((rows, ld), dtype=np.float32)
    lib.syn_dense_normal(seed, rows, cols, ld, out.ctypes.data)
    return out


def random_csr(n: int, n_cols: int, row_len_max: int, seed: int, hub_rows: int = 0,
               hub_len: int = 0, empty_frac: float = 0.0) -> Csr:
    """Small general (non-symmetric) CSR with sorted unique columns and
    N(0,1)-ish values, for edge-case tests: random row lengths in
    [0, row_len_max], optional hub rows of length ``hub_len`` and a fraction
    of forced-empty rows."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(0, row_len_max + 1, size=n)
    if empty_frac > 0:
        lens[rng.random(n) < empty_frac] = 0
    if hub_rows:
        hubs = rng.choice(n, size=min(hub_rows, n), replace=False)
        lens[hubs] = min(hub_len, n_cols)
    lens = np.minimum(lens, n_cols)
    rowptr = np.zeros(n + 1, dtype=np.int64)
    rowptr[1:] = np.cumsum(lens)
    cols = []
    for i in range(n):
        if lens[i]:
            cols.append(np.sort(rng.choice(n_cols, size=int(lens[i]), replace=False)))
    col = (np.concatenate(cols) if cols else np.zeros(0, dtype=np.int64)).astype(np.int32)
    val = rng.standard_normal(int(rowptr[-1]), dtype=np.float32)
    return Csr(n, rowptr.astype(np.int32), col, val)


def bucket_csr(lens, n_cols: int, seed: int) -> Csr:
    """CSR with the given row lengths (each <= n_cols, total < 2^31): row r
    takes one uniform random column from each of len_r near-equal buckets of
    [0, n_cols) (strictly increasing columns), values uniform in [-1, 1).
    Generated in C in O(nnz), for inputs up to the int32 index limit."""
    lens = np.asarray(lens, dtype=np.int64)
    if lens.size and (lens.min() < 0 or lens.max() > n_cols):
        raise ValueError("row lengths must lie in [0, n_cols]")
    rowptr = np.zeros(len(lens) + 1, dtype=np.int64)
    np.cumsum(lens, out=rowptr[1:])
    nnz = int(rowptr[-1])
    if nnz > np.iinfo(np.int32).max:
        raise ValueError("nnz exceeds the int32 index range")
    col = np.empty(max(nnz, 1), dtype=np.int32)
    val = np.empty(max(nnz, 1), dtype=np.float32)
    _load().syn_bucket_csr(seed, len(lens), n_cols, rowptr.ctypes.data, col.ctypes.data, val.ctypes.data)
    return Csr(len(lens), rowptr.astype(np.int32), col[:nnz], val[:nnz])


def transpose(A: Csr, n_cols: int | None = None) -> Csr:
    """CSR of A^T (columns become rows; entries keep ascending order)."""
    n_cols = A.n if n_cols is None else n_cols
    rows = np.repeat(np.arange(A.n, dtype=np.int32), np.diff(A.rowptr))
    order = np.lexsort((rows, A.col))
    rowptr = np.zeros(n_cols + 1, dtype=np.int64)
    np.add.at(rowptr, A.col.astype(np.int64) + 1, 1)
    rowptr = np.cumsum(rowptr).astype(np.int32)
    return Csr(n_cols, rowptr, rows[order].astype(np.int32), A.val[order].copy())


@dataclass
class Workload:
    name: str
    n: int
    d: int
    budgets_pct: tuple
    kind: str
    params: dict = field(default_factory=dict)
    description: str = ""


WORKLOADS = {
    "tiny": Workload("tiny", 4096, 64, (50,), "er", {"p": 16.0 / 4095.0},
                     "Erdos-Renyi G(4096, 16/(n-1)), symmetric, self-loops, d=64"),
    "social": Workload("social", 232_965, 256, (10, 30, 50), "powerlaw",
                       {"mean": 490.0, "gamma": 2.1, "wmax": 49_000.0, "draws": 66_400_000},
                       "Chung-Lu power law 2.1, n=232,965, mean degree ~490, d=256"),
    "copurchase": Workload("copurchase", 2_449_029, 256, (30,), "powerlaw",
                           {"mean": 50.0, "gamma": 2.1, "wmax": 5_000.0, "draws": 62_140_000},
                           "Chung-Lu power law 2.1, n=2,449,029, mean degree ~50, d=256"),
    "protein": Workload("protein", 132_534, 256, (30,), "uniform",
                        {"wlo": 450.0, "whi": 750.0, "draws": 39_680_000},
                        "Chung-Lu weights ~U[450,750], n=132,534, mean degree ~600, d=256"),
    "gcn2": Workload("gcn2", 716_847, 512, (10, 30, 50), "powerlaw",
                     {"mean": 20.0, "gamma": 2.1, "wmax": 2_000.0, "draws": 7_000_000,
                      "in_features": 300, "hidden": 512, "classes": 100},
                     "Chung-Lu power law 2.1, n=716,847, mean degree ~20; GCN 300-512-100"),
}


def make_graph(name: str, seed: int = 0) -> Csr:
    w = WORKLOADS[name]
    p = w.params
    if w.kind == "er":
        return erdos_renyi(w.n, p["p"], seed)
    if w.kind == "powerlaw":
        return chung_lu_powerlaw(w.n, p["mean"], p["gamma"], p["wmax"], p["draws"], seed)
    if w.kind == "uniform":
        return chung_lu_uniform(w.n, p["wlo"], p["whi"], p["draws"], seed)
    raise ValueError(name)

