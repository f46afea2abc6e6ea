"""CPU oracle for the RSC aggregation hot path.

TEST INFRASTRUCTURE ONLY: the plain, slow, fp64 reference that the GPU
library is checked against. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path never
does. It shares no code with the GPU library (its arithmetic lives in
``orc.c``, compiled with gcc, plus the small cache-policy class below).

Every function takes and returns numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liborc.so")
_lib = None

CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared"]


def build(verbose: bool = False) -> str:
    cmd = ["gcc", *CFLAGS, "-o", _LIB_PATH, os.path.join(_HERE, "orc.c"), "-lm"]
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
        vp, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.orc_check_csr.argtypes = [i32, i32, vp, vp]
        lib.orc_check_csr.restype = ctypes.c_int
        lib.orc_check_gcn_values.argtypes = [i32, vp, vp, vp]
        lib.orc_check_gcn_values.restype = i64
        lib.orc_spmm.argtypes = [i32, vp, vp, vp, vp, i32, i64, vp, i64, vp, i64, vp, i32]
        lib.orc_col_sqnorms.argtypes = [i32, vp, vp, vp, vp]
        lib.orc_pair_keys.argtypes = [i32, vp, vp, i32, i64, vp, vp, vp, vp]
        lib.orc_rank_order.argtypes = [i32, vp, vp]
        lib.orc_topk.argtypes = [i32, vp, i32, vp, vp]
        lib.orc_slice.argtypes = [i32, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_slice.restype = i64
        lib.orc_k_from_fraction.argtypes = [i32, i32, i32]
        lib.orc_k_from_fraction.restype = i32
        lib.orc_greedy.argtypes = [i32, i32, i64, vp, vp, vp, f64, vp, i32, i32, i32, i32, vp]
        lib.orc_greedy.restype = i64
        lib.orc_num_threads.restype = i32
        lib.orc_set_num_threads.argtypes = [i32]
        lib.orc_set_num_threads.restype = i32
        lib.orc_sum_sequential.argtypes = [i64, vp]
        lib.orc_sum_sequential.restype = f64
        lib.orc_selection_auc.argtypes = [i32, vp, vp, vp, vp]
        lib.orc_selection_auc.restype = f64
        lib.orc_spmm_mean.argtypes = [i32, vp, vp, vp, vp, i32, i64, vp, i64]
        lib.orc_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        lib.orc_splitmix64.restype = ctypes.c_uint64
        lib.orc_sample_columns.argtypes = [i32, vp, i32, ctypes.c_uint64, vp, vp, vp, vp]
        lib.orc_slice_scaled.argtypes = [i32, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_slice_scaled.restype = i64
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def check_csr(rowptr, col, n_rows, n_cols) -> int:
    rowptr, col = _c(rowptr, np.int32), _c(col, np.int32)
    return _load().orc_check_csr(n_rows, n_cols, _p(rowptr), _p(col))


def check_gcn_values(rowptr, col, val) -> int:
    rowptr, col, val = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    return _load().orc_check_gcn_values(len(rowptr) - 1, _p(rowptr), _p(col), _p(val))


def spmm(rowptr, col, val, B, d=None, rows=None, with_mag=False):
    """Y = A B (fp64 accumulation, fp32 result). B is a 2-D fp32 array whose
    leading dimension is its row stride; ``d`` defaults to B.shape[1].
    With ``rows`` only those rows are computed (output row r = rows[r]).
    Returns Y, or (Y, S) with S the fp64 magnitude sum |A| |B|."""
    rowptr, col, val = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    B = _c(B, np.float32)
    d = B.shape[1] if d is None else d
    n_rows = len(rowptr) - 1
    sel = None if rows is None else _c(rows, np.int32)
    m = n_rows if sel is None else len(sel)
    Y = np.zeros((m, d), dtype=np.float32)
    S = np.zeros((m, d), dtype=np.float64) if with_mag else None
    _load().orc_spmm(n_rows, _p(rowptr), _p(col), _p(val), _p(B), d, B.shape[1], _p(Y), d,
                     _p(S), d, _p(sel), 0 if sel is None else len(sel))
    return (Y, S) if with_mag else Y


def spmm_mean(rowptr, col, val, B, d=None):
    """SpMM_MEAN: D^-1 A B with D_ii = stored entries of row i (fp64 sum,
    one division, one fp32 rounding)."""
    rowptr, col, val = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    B = _c(B, np.float32)
    d = B.shape[1] if d is None else d
    n_rows = len(rowptr) - 1
    Y = np.zeros((n_rows, d), dtype=np.float32)
    _load().orc_spmm_mean(n_rows, _p(rowptr), _p(col), _p(val), _p(B), d, B.shape[1], _p(Y), d)
    return Y


def col_sqnorms(rowptr_t, val_t):
    """cn2 (fp64) and colnnz (int32) from the CSR of X^T."""
    rowptr_t, val_t = _c(rowptr_t, np.int32), _c(val_t, np.float32)
    n = len(rowptr_t) - 1
    cn2 = np.zeros(n, dtype=np.float64)
    colnnz = np.zeros(n, dtype=np.int32)
    _load().orc_col_sqnorms(n, _p(rowptr_t), _p(val_t), _p(cn2), _p(colnnz))
    return cn2, colnnz


def pair_keys(cn2, B, d=None):
    """Returns dict with rn2, q (fp64), key (uint64), score (fp32)."""
    cn2, B = _c(cn2, np.float64), _c(B, np.float32)
    n = len(cn2)
    d = B.shape[1] if d is None else d
    out = {"rn2": np.zeros(n, np.float64), "q": np.zeros(n, np.float64),
           "key": np.zeros(n, np.uint64), "score": np.zeros(n, np.float32)}
    _load().orc_pair_keys(n, _p(cn2), _p(B), d, B.shape[1], _p(out["rn2"]), _p(out["q"]),
                          _p(out["key"]), _p(out["score"]))
    return out


def rank_order(key):
    key = _c(key, np.uint64)
    order = np.zeros(len(key), dtype=np.int32)
    _load().orc_rank_order(len(key), _p(key), _p(order))
    return order


def topk(key, k):
    """(idx ascending int32[k], mask uint32[ceil(n/32)])."""
    key = _c(key, np.uint64)
    n = len(key)
    idx = np.zeros(max(k, 1), dtype=np.int32)
    mask = np.zeros((n + 31) // 32, dtype=np.uint32)
    _load().orc_topk(n, _p(key), k, _p(idx), _p(mask))
    return idx[:k].copy(), mask


def slice_csr(rowptr, col, val, mask):
    """(rowptr', col', val') of A[:, S] with global column ids."""
    rowptr, col, val = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    mask = _c(mask, np.uint32)
    n = len(rowptr) - 1
    ro = np.zeros(n + 1, dtype=np.int32)
    co = np.zeros(max(len(col), 1), dtype=np.int32)
    vo = np.zeros(max(len(col), 1), dtype=np.float32)
    nnz2 = _load().orc_slice(n, _p(rowptr), _p(col), _p(val), _p(mask), _p(ro), _p(co), _p(vo))
    return ro, co[:nnz2].copy(), vo[:nnz2].copy()


def k_from_fraction(n, num, den) -> int:
    return _load().orc_k_from_fraction(n, num, den)


def greedy(keys, colnnz, nnz, d, fro_a2, fro_b2, C, alpha):
    """Greedy layer-wise allocation. keys: list of uint64 arrays (one per
    layer); d: list of widths; fro_b2: list of ||grad H||_F^2; C and alpha
    are (num, den) pairs. Returns (k list, final budget)."""
    L = len(keys)
    keys = [_c(k, np.uint64) for k in keys]
    n = len(keys[0])
    ptrs = (ctypes.c_void_p * L)(*[k.ctypes.data for k in keys])
    colnnz = _c(colnnz, np.int32)
    d_arr = _c(d, np.int32)
    fb = _c(fro_b2, np.float64)
    k_out = np.zeros(L, dtype=np.int32)
    bud = _load().orc_greedy(L, n, nnz, ctypes.cast(ptrs, ctypes.c_void_p), _p(colnnz), _p(d_arr),
                             float(fro_a2), _p(fb), C[0], C[1], alpha[0], alpha[1], _p(k_out))
    return [int(x) for x in k_out], int(bud)


def splitmix64(seed: int, t: int) -> int:
    return int(_load().orc_splitmix64(seed, t))


def sample_columns(key, k, seed):
    """Randomized column-row sampling: dict(count, colw, mask, w)."""
    key = _c(key, np.uint64)
    n = len(key)
    out = {"count": np.zeros(n, np.int32), "colw": np.zeros(n, np.float64),
           "mask": np.zeros((n + 31) // 32, np.uint32), "w": np.zeros(n, np.int64)}
    _load().orc_sample_columns(n, _p(key), k, seed, _p(out["count"]), _p(out["colw"]), _p(out["mask"]),
                               _p(out["w"]))
    return out


def slice_scaled(rowptr, col, val, mask, colw):
    rowptr, col, val = _c(rowptr, np.int32), _c(col, np.int32), _c(val, np.float32)
    mask, colw = _c(mask, np.uint32), _c(colw, np.float64)
    n = len(rowptr) - 1
    ro = np.zeros(n + 1, dtype=np.int32)
    co = np.zeros(max(len(col), 1), dtype=np.int32)
    vo = np.zeros(max(len(col), 1), dtype=np.float32)
    m = _load().orc_slice_scaled(n, _p(rowptr), _p(col), _p(val), _p(mask), _p(colw), _p(ro), _p(co), _p(vo))
    return ro, co[:m].copy(), vo[:m].copy()


def num_threads() -> int:
    return int(_load().orc_num_threads())


def set_num_threads(t: int) -> int:
    """Thread count of the oracle's row loops from now on; returns it."""
    return int(_load().orc_set_num_threads(int(t)))


def sum_sequential(x) -> float:
    """Plain sequential fp64 sum (Eq. 4a's Frobenius normalisers)."""
    x = _c(x, np.float64)
    return float(_load().orc_sum_sequential(len(x), _p(x)))


def selection_staleness(order, prev_mask, new_mask=None):
    """(AUC of the previous selection under the new ranking `order`, overlap
    |S_prev & S_new| / |S_prev|) for masks of ceil(n/32) words; AUC NaN for an
    empty or full selection, overlap None without new_mask or for an empty
    previous selection."""
    order = _c(order, np.int32)
    n = len(order)
    prev_mask = _c(prev_mask, np.uint32)
    nm = None if new_mask is None else _c(new_mask, np.uint32)
    both = ctypes.c_int64(0)
    auc = _load().orc_selection_auc(n, _p(order), _p(prev_mask), _p(nm), ctypes.byref(both))
    k = int(np.unpackbits(prev_mask.view(np.uint8), bitorder="little")[:n].sum())
    overlap = None if (nm is None or k == 0) else both.value / k
    return float(auc), overlap


class CachePolicy:
    """Refresh policy of the sampled-matrix cache (section 3.3.1; refresh
    every R = 10 steps per section 5.1): refresh at the first request and
    whenever step - last_refresh >= R; in between, the same slice is reused
    even though the dense operand changes."""

    def __init__(self, interval: int = 10):
        self.interval = interval
        self.last = None

    def needs_refresh(self, step: int) -> bool:
        return self.last is None or step - self.last >= self.interval

    def refreshed(self, step: int) -> None:
        self.last = step
