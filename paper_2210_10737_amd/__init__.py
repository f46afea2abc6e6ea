"""Python binding of librsc.so (the MI355X RSC hot-path library).

Argument marshalling only: each function takes torch tensors that live on the
GPU, passes their data pointers and the current HIP stream to the C ABI of
include/rsc.h, and returns torch tensors. Every step of the computation runs
in the library's HIP kernels; there is no fallback. If librsc.so has not been
built, every call raises.

Paper: Liu et al., "RSC: Accelerate Graph Neural Networks Training via
Randomized Sparse Computations", ICML 2023 (arXiv 2210.10737).

Typical use (A_hat symmetric, so it serves as its own transpose):

    A = DeviceCsr.from_host(rowptr, col, val, n_cols)   # int32 / int32 / float32
    Y = spmm(A, H)                                       # exact forward (one-off)
    plan = SpmmPlan(A)                                   # or: prepare the static operand once,
    Y = plan.run(H)                                      # same Y bit for bit, every step
    cache = Cache(A, A, refresh_interval=10)
    k = k_from_fraction(A.n_cols, 30, 100)
    if cache.get(step, with_slice=False)["needs_refresh"]:
        cache.refresh(G, k, step)                        # scores, top-k, slice
    G_back = cache.spmm_sampled(G)                       # sampled backward

`gcn.GCN` wires these into a training step with the layer-wise allocation.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librsc.so")

RSC_OK = 0
STATUS = {0: "RSC_OK", 1: "RSC_ERR_INVALID_ARGUMENT", 2: "RSC_ERR_UNSUPPORTED",
          3: "RSC_ERR_OUT_OF_MEMORY", 4: "RSC_ERR_CAPACITY", 5: "RSC_ERR_NO_DEVICE",
          6: "RSC_ERR_HIP", 7: "RSC_ERR_INTERNAL"}

EXPORTED = [
    "rsc_status_string", "rsc_last_error", "rsc_abi_version", "rsc_csr_validate",
    "rsc_spmm_workspace_bytes", "rsc_spmm", "rsc_spmm_noalloc", "rsc_degree_scale",
    "rsc_spmm_plan_create", "rsc_spmm_plan_run", "rsc_spmm_plan_destroy", "rsc_spmm_plan_gather_probe",
    "rsc_col_sqnorms", "rsc_pair_scores",
    "rsc_topk_workspace_bytes", "rsc_topk_select",
    "rsc_slice_workspace_bytes", "rsc_slice_csr",
    "rsc_sample_workspace_bytes", "rsc_sample_columns",
    "rsc_cache_create", "rsc_cache_create_ex", "rsc_cache_refresh", "rsc_cache_score", "rsc_cache_select",
    "rsc_cache_refresh_random",
    "rsc_cache_get", "rsc_spmm_sampled",
    "rsc_cache_buffers", "rsc_cache_norms", "rsc_cache_staleness", "rsc_cache_gather_probe", "rsc_cache_destroy",
    "rsc_k_from_fraction", "rsc_greedy_allocate",
    "rsc_greedy_profile_workspace_bytes", "rsc_greedy_blocks", "rsc_greedy_profile",
    "rsc_greedy_allocate_profiles",
]


class RscError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


_ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
_FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p)


class Allocator(ctypes.Structure):
    _fields_ = [("alloc", _ALLOC_FN), ("free", _FREE_FN), ("ctx", ctypes.c_void_p)]


def _torch_allocator() -> Allocator:
    """rsc_allocator_t backed by torch's caching allocator on the current
    device (its blocks are 512-byte aligned)."""
    dev = torch.cuda.current_device()

    def alloc(nbytes, stream, ctx):
        try:
            return torch.cuda.caching_allocator_alloc(int(nbytes), device=dev, stream=stream)
        except Exception:  # out of memory: the library reports RSC_ERR_OUT_OF_MEMORY
            return None

    def free(ptr, stream, ctx):
        torch.cuda.caching_allocator_delete(ptr)

    return Allocator(_ALLOC_FN(alloc), _FREE_FN(free), None)


class CsrStruct(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int32), ("n_cols", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("rowptr", ctypes.c_void_p), ("col", ctypes.c_void_p), ("val", ctypes.c_void_p)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2210_10737_amd.build` (or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        csrp = ctypes.POINTER(CsrStruct)
        sig = {
            "rsc_status_string": ([ctypes.c_int], ctypes.c_char_p),
            "rsc_last_error": ([], ctypes.c_char_p),
            "rsc_abi_version": ([], i32),
            "rsc_spmm_workspace_bytes": ([csrp], sz),
            "rsc_spmm": ([csrp, vp, i32, i64, vp, i64, vp, sz, vp], ctypes.c_int),
            "rsc_spmm_noalloc": ([csrp, vp, i32, i64, vp, i64, vp], ctypes.c_int),
            "rsc_spmm_plan_create": ([csrp, vp, ctypes.POINTER(vp)], ctypes.c_int),
            "rsc_spmm_plan_run": ([vp, vp, i32, i64, vp, i64, vp], ctypes.c_int),
            "rsc_spmm_plan_destroy": ([vp], ctypes.c_int),
            "rsc_spmm_plan_gather_probe": ([vp, vp, i32, i64, i32, vp, i64, vp, i64, ctypes.POINTER(i32), vp],
                                          ctypes.c_int),
            "rsc_col_sqnorms": ([csrp, vp, vp, vp], ctypes.c_int),
            "rsc_degree_scale": ([csrp, vp, i32, vp, vp], ctypes.c_int),
            "rsc_pair_scores": ([vp, vp, i32, i32, i64, vp, vp, vp, vp], ctypes.c_int),
            "rsc_topk_workspace_bytes": ([i32], sz),
            "rsc_topk_select": ([vp, i32, i32, vp, vp, vp, sz, vp], ctypes.c_int),
            "rsc_slice_workspace_bytes": ([csrp], sz),
            "rsc_slice_csr": ([csrp, vp, vp, vp, vp, vp, i64, vp, vp, sz, vp], ctypes.c_int),
            "rsc_sample_workspace_bytes": ([i32], sz),
            "rsc_sample_columns": ([vp, i32, i32, ctypes.c_uint64, vp, vp, vp, vp, sz, vp], ctypes.c_int),
            "rsc_cache_refresh_random": ([vp, vp, i32, i64, i32, ctypes.c_uint64, i64, vp], ctypes.c_int),
            "rsc_cache_create": ([csrp, csrp, i32, vp, ctypes.POINTER(vp)], ctypes.c_int),
            "rsc_cache_create_ex": ([csrp, csrp, i32, ctypes.POINTER(Allocator), vp, ctypes.POINTER(vp)],
                                    ctypes.c_int),
            "rsc_csr_validate": ([csrp, ctypes.POINTER(i64), vp], ctypes.c_int),
            "rsc_cache_refresh": ([vp, vp, i32, i64, i32, i64, vp], ctypes.c_int),
            "rsc_cache_score": ([vp, vp, i32, i64, vp], ctypes.c_int),
            "rsc_cache_select": ([vp, i32, i64, vp], ctypes.c_int),
            "rsc_cache_get": ([vp, i64, csrp, ctypes.POINTER(vp), ctypes.POINTER(i32),
                               ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_uint64)], ctypes.c_int),
            "rsc_spmm_sampled": ([vp, vp, i32, i64, vp, i64, vp], ctypes.c_int),
            "rsc_cache_buffers": ([vp, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                   ctypes.POINTER(vp), ctypes.POINTER(vp)], ctypes.c_int),
            "rsc_cache_destroy": ([vp], ctypes.c_int),
            "rsc_cache_gather_probe": ([vp, vp, i32, i64, i32, vp, i64, vp, i64, ctypes.POINTER(i32), vp],
                                      ctypes.c_int),
            "rsc_cache_norms": ([vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), vp],
                                ctypes.c_int),
            "rsc_cache_staleness": ([vp, vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64),
                                     ctypes.POINTER(i64), vp], ctypes.c_int),
            "rsc_k_from_fraction": ([i32, i32, i32], i32),
            "rsc_greedy_allocate": ([i32, i32, i64, vp, vp, vp, ctypes.c_double, vp, i32, i32, i32,
                                     i32, vp, vp], ctypes.c_int),
            "rsc_greedy_profile_workspace_bytes": ([i32], sz),
            "rsc_greedy_blocks": ([i32, i32, i32], i32),
            "rsc_greedy_profile": ([vp, vp, i32, i32, i32, vp, vp, vp, vp, sz, vp], ctypes.c_int),
            "rsc_greedy_allocate_profiles": ([i32, i32, i64, i32, i32, vp, vp, vp, ctypes.c_double, vp,
                                              i32, i32, vp, vp], ctypes.c_int),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def csr_validate(A: "DeviceCsr") -> None:
    """Device check that A is a well-formed CSR with sorted unique columns
    (rsc_csr_validate); raises RscError naming the first bad row."""
    bad = ctypes.c_int64(-1)
    _check(lib().rsc_csr_validate(ctypes.byref(A.struct()), ctypes.byref(bad), _stream()))


def _check(status: int) -> None:
    if status != RSC_OK:
        raise RscError(status, lib().rsc_last_error().decode())


def _stream() -> int:
    """The current HIP stream of the current device, as a raw handle. torch's
    raw-stream getter costs ~0.1 us per call against ~3 us for building a
    torch.cuda.Stream object, which matters for launch-bound products."""
    try:
        return torch._C._cuda_getCurrentRawStream(torch._C._cuda_getDevice())
    except AttributeError:
        return torch.cuda.current_stream().cuda_stream


def _device_index() -> int:
    try:
        return torch._C._cuda_getDevice()
    except AttributeError:
        return torch.cuda.current_device()


def _dp(t: torch.Tensor) -> int:
    """Device address of a tensor that lives on the current GPU (the library
    launches on the current device's stream, so a host tensor or one on
    another GPU would hand the kernels an address they cannot use)."""
    if t.get_device() != _device_index():   # -1 for host tensors
        raise ValueError(f"tensor on {t.device}: the library runs on the current device cuda:{_device_index()}")
    return t.data_ptr()


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else _dp(t)


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("dense operands must be 2-D with unit column stride")
    return t.stride(0)


def _dense(t: torch.Tensor, rows: int, d: int, name: str) -> tuple[int, int]:
    """(device address, leading dimension) of a float32 operand that holds at
    least rows x d elements: the library reads or writes that many through
    the pointer, so a smaller or differently typed tensor is refused here."""
    if t.dtype != torch.float32:
        raise ValueError(f"{name}: dtype {t.dtype}, float32 expected")
    ld = _ld(t)
    if t.shape[0] < rows or t.shape[1] < d:
        raise ValueError(f"{name}: shape {tuple(t.shape)} holds less than {rows} x {d}")
    return _dp(t), ld


def _vec_check(t: torch.Tensor, count: int, dtype, name: str) -> None:
    if t.dtype != dtype or not t.is_contiguous() or t.numel() < count:
        raise ValueError(f"{name}: {t.dtype}[{t.numel()}], contiguous {dtype}[>= {count}] expected")


def _vec(t: torch.Tensor | None, count: int, dtype, name: str) -> int | None:
    """Device address of an optional contiguous array of at least count
    elements of dtype."""
    if t is None:
        return None
    _vec_check(t, count, dtype, name)
    return _dp(t)


def _new_out(rows: int, d: int, device) -> torch.Tensor:
    """rows x d output view with a leading dimension rounded up to 4 floats."""
    ld = (d + 3) // 4 * 4
    return torch.empty((rows, ld), dtype=torch.float32, device=device)[:, :d]


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns 256-byte (or larger) aligned blocks
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


@dataclass
class DeviceCsr:
    """CSR on the GPU: rowptr int32[n_rows+1], col int32[nnz], val float32[nnz]."""
    n_rows: int
    n_cols: int
    rowptr: torch.Tensor
    col: torch.Tensor
    val: torch.Tensor
    nnz: int | None = None

    def __post_init__(self):
        if self.nnz is None:
            self.nnz = int(self.col.numel())

    @classmethod
    def from_host(cls, rowptr, col, val, n_cols, device="cuda"):
        rp = torch.as_tensor(rowptr, dtype=torch.int32).to(device)
        c = torch.as_tensor(col, dtype=torch.int32).to(device)
        v = torch.as_tensor(val, dtype=torch.float32).to(device)
        return cls(len(rowptr) - 1, int(n_cols), rp, c, v)

    def struct(self) -> CsrStruct:
        _vec_check(self.rowptr, self.n_rows + 1, torch.int32, "rowptr")
        if self.nnz:
            _vec_check(self.col, self.nnz, torch.int32, "col")
            _vec_check(self.val, self.nnz, torch.float32, "val")
        return CsrStruct(self.n_rows, self.n_cols, self.nnz,
                         _vec(self.rowptr, self.n_rows + 1, torch.int32, "rowptr"),
                         _vec(self.col, self.nnz, torch.int32, "col") if self.nnz else None,
                         _vec(self.val, self.nnz, torch.float32, "val") if self.nnz else None)


# ---------------------------------------------------------------- A1
def spmm_workspace_bytes(A: DeviceCsr) -> int:
    return lib().rsc_spmm_workspace_bytes(ctypes.byref(A.struct()))


def spmm(A: DeviceCsr, B: torch.Tensor, d: int | None = None, out: torch.Tensor | None = None,
         ws: torch.Tensor | None = None) -> torch.Tensor:
    """Y = A @ B[:, :d] (exact SpMM)."""
    d = B.shape[1] if d is None else d
    Y = _new_out(A.n_rows, d, B.device) if out is None else out
    s = A.struct()
    need = lib().rsc_spmm_workspace_bytes(ctypes.byref(s))
    ws = _workspace(need, B.device) if ws is None else ws
    pb, ldb = _dense(B, A.n_cols, d, "B")
    py, ldy = _dense(Y, A.n_rows, d, "Y")
    _check(lib().rsc_spmm(ctypes.byref(s), pb, d, ldb, py, ldy, _dp(ws), ws.numel(), _stream()))
    return Y


def spmm_noalloc(A: DeviceCsr, B: torch.Tensor, d: int | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """Y = A @ B[:, :d] through rsc_spmm_noalloc: no workspace, no device
    allocation inside the library (its scratch is static). With ``out`` given
    nothing is allocated here either."""
    d = B.shape[1] if d is None else d
    Y = _new_out(A.n_rows, d, B.device) if out is None else out
    pb, ldb = _dense(B, A.n_cols, d, "B")
    py, ldy = _dense(Y, A.n_rows, d, "Y")
    _check(lib().rsc_spmm_noalloc(ctypes.byref(A.struct()), pb, d, ldb, py, ldy, _stream()))
    return Y


class SpmmPlan:
    """Repeated exact products with one sparse operand (rsc_spmm_plan_*):
    the same result as spmm(A, B) bit for bit, with the plan's own workspace
    and, on large operands, the column cache hint. A's tensors must outlive
    the plan."""

    def __init__(self, A: DeviceCsr):
        self.A = A
        h = ctypes.c_void_p()
        _check(lib().rsc_spmm_plan_create(ctypes.byref(A.struct()), _stream(), ctypes.byref(h)))
        self._h = h

    def run(self, B: torch.Tensor, d: int | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
        d = B.shape[1] if d is None else d
        Y = _new_out(self.A.n_rows, d, B.device) if out is None else out
        pb, ldb = _dense(B, self.A.n_cols, d, "B")
        py, ldy = _dense(Y, self.A.n_rows, d, "Y")
        _check(lib().rsc_spmm_plan_run(self._h, pb, d, ldb, py, ldy, _stream()))
        return Y

    def gather_probe(self, B: torch.Tensor, d: int | None = None, inflight: int = 8,
                     sink: torch.Tensor | None = None, out: torch.Tensor | None = None) -> int:
        """The gather-only pass of this plan's product (rsc_spmm_plan_gather_probe,
        a measurement helper), with `out` (n_rows x d) also the product's
        output stream (out's contents are then unspecified); returns the
        feature-pass width it used."""
        d = B.shape[1] if d is None else d
        need = (self.A.nnz + 63) // 64
        sink = torch.empty(max(need, 1), dtype=torch.float32, device=B.device) if sink is None else sink
        sl = ctypes.c_int32(0)
        pb, ldb = _dense(B, self.A.n_cols, d, "B")
        py, ldy = _dense(out, self.A.n_rows, d, "out") if out is not None else (None, 0)
        _check(lib().rsc_spmm_plan_gather_probe(self._h, pb, d, ldb, inflight, _vec(sink, 0, torch.float32, "sink"),
                                                sink.numel(), py, ldy, ctypes.byref(sl), _stream()))
        return sl.value

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            _check(lib().rsc_spmm_plan_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def degree_scale(A: DeviceCsr, by_column: bool = False, deg_rowptr: torch.Tensor | None = None) -> DeviceCsr:
    """MEAN-aggregator operand: D^-1 A (by_column=False) or, for A = CSR of
    M^T and deg_rowptr = M's rowptr, M^T D^-1 (by_column=True)."""
    out = torch.empty_like(A.val)
    _check(lib().rsc_degree_scale(ctypes.byref(A.struct()), _ptr(deg_rowptr), 1 if by_column else 0,
                                  _dp(out) if A.nnz else None, _stream()))
    return DeviceCsr(A.n_rows, A.n_cols, A.rowptr, A.col, out, nnz=A.nnz)


# ---------------------------------------------------------------- A2 / A3
def col_sqnorms(XT: DeviceCsr):
    """(cn2 float64[n], colnnz int32[n]) from the CSR of X^T."""
    cn2 = torch.empty(XT.n_rows, dtype=torch.float64, device=XT.rowptr.device)
    colnnz = torch.empty(XT.n_rows, dtype=torch.int32, device=XT.rowptr.device)
    _check(lib().rsc_col_sqnorms(ctypes.byref(XT.struct()), _dp(cn2), _dp(colnnz), _stream()))
    return cn2, colnnz


def pair_scores(cn2: torch.Tensor, B: torch.Tensor, d: int | None = None, with_score: bool = False,
                with_rn2: bool = False):
    """Keys (uint64 bit patterns stored in an int64 tensor) for the
    n = B.shape[0] column-row pairs; with_score / with_rn2 also return the
    fp32 scores and the fp64 row square-norms."""
    n = B.shape[0]
    d = B.shape[1] if d is None else d
    key = torch.empty(n, dtype=torch.int64, device=B.device)
    score = torch.empty(n, dtype=torch.float32, device=B.device) if with_score else None
    rn2 = torch.empty(n, dtype=torch.float64, device=B.device) if with_rn2 else None
    pb, ldb = _dense(B, n, d, "B")
    _check(lib().rsc_pair_scores(_vec(cn2, n, torch.float64, "cn2"), pb, n, d, ldb, _dp(key),
                                 _ptr(score), _ptr(rn2), _stream()))
    out = [key] + ([score] if with_score else []) + ([rn2] if with_rn2 else [])
    return out[0] if len(out) == 1 else tuple(out)


# ---------------------------------------------------------------- A4
def topk_select(key: torch.Tensor, k: int, ws: torch.Tensor | None = None):
    """(idx int32[k] ascending, mask int32[ceil(n/32)] holding uint32 words)."""
    n = key.numel()
    idx = torch.empty(max(k, 1), dtype=torch.int32, device=key.device)
    mask = torch.empty(max((n + 31) // 32, 1), dtype=torch.int32, device=key.device)
    need = lib().rsc_topk_workspace_bytes(n)
    ws = _workspace(need, key.device) if ws is None else ws
    _check(lib().rsc_topk_select(_dp(key), n, k, _dp(idx), _dp(mask), _dp(ws),
                                 ws.numel(), _stream()))
    return idx[:k], mask[: (n + 31) // 32]


# ---------------------------------------------------------------- A5
def slice_csr(A: DeviceCsr, mask: torch.Tensor, capacity: int | None = None,
              ws: torch.Tensor | None = None, colw: torch.Tensor | None = None):
    """(DeviceCsr slice with capacity-sized col/val, nnz' as a device int64
    tensor). The slice's nnz field is left as None-equivalent (capacity)
    until the caller reads nnz'."""
    cap = A.nnz if capacity is None else capacity
    dev = A.rowptr.device
    rp = torch.empty(A.n_rows + 1, dtype=torch.int32, device=dev)
    co = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    vo = torch.empty(max(cap, 1), dtype=torch.float32, device=dev)
    nnz_out = torch.empty(1, dtype=torch.int64, device=dev)
    s = A.struct()
    need = lib().rsc_slice_workspace_bytes(ctypes.byref(s))
    ws = _workspace(need, dev) if ws is None else ws
    pm = _vec(mask, (A.n_cols + 31) // 32, torch.int32, "mask")
    pw = _vec(colw, A.n_cols, torch.float64, "colw")
    _check(lib().rsc_slice_csr(ctypes.byref(s), pm, pw, _dp(rp), _dp(co),
                               _dp(vo), cap, _dp(nnz_out), _dp(ws), ws.numel(), _stream()))
    return DeviceCsr(A.n_rows, A.n_cols, rp, co, vo, nnz=cap), nnz_out


def sample_columns(key: torch.Tensor, k: int, seed: int, ws: torch.Tensor | None = None):
    """Randomized column-row sampling: (count int32[n], colw float64[n],
    mask int32[ceil(n/32)] holding uint32 words)."""
    n = key.numel()
    count = torch.empty(max(n, 1), dtype=torch.int32, device=key.device)
    colw = torch.empty(max(n, 1), dtype=torch.float64, device=key.device)
    mask = torch.empty(max((n + 31) // 32, 1), dtype=torch.int32, device=key.device)
    need = lib().rsc_sample_workspace_bytes(n)
    ws = _workspace(need, key.device) if ws is None else ws
    _check(lib().rsc_sample_columns(_dp(key), n, k, seed, _dp(count), _dp(colw),
                                    _dp(mask), _dp(ws), ws.numel(), _stream()))
    return count[:n], colw[:n], mask[: (n + 31) // 32]


# ---------------------------------------------------------------- A6 / A7
class Cache:
    """Sampled-matrix cache (section 3.3.1): rsc_cache_create / refresh /
    get / spmm_sampled / destroy."""

    def __init__(self, X: DeviceCsr, XT: DeviceCsr | None = None, refresh_interval: int = 10,
                 allocator: str | None = None):
        """allocator: None (the library's hipMalloc) or "torch" (torch's
        caching allocator, through rsc_cache_create_ex)."""
        self.X = X
        self.XT = X if XT is None else XT
        h = ctypes.c_void_p()
        self._alloc = None
        if allocator is None:
            _check(lib().rsc_cache_create(ctypes.byref(X.struct()), ctypes.byref(self.XT.struct()),
                                          refresh_interval, _stream(), ctypes.byref(h)))
        elif allocator == "torch":
            self._alloc = _torch_allocator()  # kept alive until destroy
            _check(lib().rsc_cache_create_ex(ctypes.byref(X.struct()), ctypes.byref(self.XT.struct()),
                                             refresh_interval, ctypes.byref(self._alloc), _stream(),
                                             ctypes.byref(h)))
        else:
            raise ValueError(f"unknown allocator {allocator!r}")
        self._h = h

    def refresh(self, B: torch.Tensor, k: int, step: int, d: int | None = None) -> None:
        d = B.shape[1] if d is None else d
        _check(lib().rsc_cache_refresh(self._h, *self._b(B, d), k, step, _stream()))

    def score(self, B: torch.Tensor, d: int | None = None) -> None:
        d = B.shape[1] if d is None else d
        _check(lib().rsc_cache_score(self._h, *self._b(B, d), _stream()))

    def _b(self, B: torch.Tensor, d: int):
        # (pointer, d, ld) of an operand with a row per column of X
        pb, ldb = _dense(B, self.X.n_cols, d, "B")
        return pb, d, ldb

    def select(self, k: int, step: int) -> None:
        _check(lib().rsc_cache_select(self._h, k, step, _stream()))

    def refresh_random(self, B: torch.Tensor, k_draws: int, seed: int, step: int, d: int | None = None) -> None:
        d = B.shape[1] if d is None else d
        _check(lib().rsc_cache_refresh_random(self._h, *self._b(B, d), k_draws, seed, step, _stream()))

    def get(self, step: int, with_slice: bool = True):
        """dict(slice=CsrStruct or None, idx_ptr, k, needs_refresh, version).
        Asking for the slice waits (once per refresh) for its nnz."""
        s = CsrStruct()
        idx = ctypes.c_void_p()
        k = ctypes.c_int32()
        nr = ctypes.c_int32()
        ver = ctypes.c_uint64()
        _check(lib().rsc_cache_get(self._h, step, ctypes.byref(s) if with_slice else None,
                                   ctypes.byref(idx), ctypes.byref(k), ctypes.byref(nr),
                                   ctypes.byref(ver)))
        return {"slice": s if with_slice else None, "idx_ptr": idx.value, "k": k.value,
                "needs_refresh": bool(nr.value), "version": ver.value}

    def spmm_sampled(self, B: torch.Tensor, d: int | None = None, out: torch.Tensor | None = None):
        d = B.shape[1] if d is None else d
        Y = _new_out(self.X.n_rows, d, B.device) if out is None else out
        py, ldy = _dense(Y, self.X.n_rows, d, "Y")
        _check(lib().rsc_spmm_sampled(self._h, *self._b(B, d), py, ldy, _stream()))
        return Y

    def gather_probe(self, B: torch.Tensor, d: int | None = None, inflight: int = 8,
                     sink: torch.Tensor | None = None, out: torch.Tensor | None = None) -> int:
        """The gather-only pass of spmm_sampled on the cached slice
        (rsc_cache_gather_probe, a measurement helper), with `out` also the
        product's output stream; returns the feature-pass width it used."""
        d = B.shape[1] if d is None else d
        if sink is None:
            nnz = self.get(0)["slice"].nnz
            sink = torch.empty(max((nnz + 63) // 64, 1), dtype=torch.float32, device=B.device)
        sl = ctypes.c_int32(0)
        py, ldy = _dense(out, self.X.n_rows, d, "out") if out is not None else (None, 0)
        _check(lib().rsc_cache_gather_probe(self._h, *self._b(B, d), inflight, _vec(sink, 0, torch.float32, "sink"),
                                            sink.numel(), py, ldy, ctypes.byref(sl), _stream()))
        return sl.value

    def norms(self, scored: bool = True):
        """(||X||_F^2, ||B||_F^2 of the last scored operand) from the device's
        fixed-order sums (rsc_cache_norms); the second is None with scored=False."""
        fx, fb = ctypes.c_double(), ctypes.c_double()
        _check(lib().rsc_cache_norms(self._h, ctypes.byref(fx), ctypes.byref(fb) if scored else None, _stream()))
        return fx.value, (fb.value if scored else None)

    def staleness(self, order: torch.Tensor):
        """(AUC of the previous selection under the ranking `order` (int32[n],
        best first), |S_prev & S_new|, |S_prev|) from rsc_cache_staleness."""
        auc, both, kp = ctypes.c_double(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().rsc_cache_staleness(self._h, _vec(order, self.X.n_cols, torch.int32, "order"),
                                         ctypes.byref(auc), ctypes.byref(both), ctypes.byref(kp), _stream()))
        return auc.value, both.value, kp.value

    def buffers(self):
        """Device pointers [cn2, colnnz, key, rn2, mask]."""
        p = [ctypes.c_void_p() for _ in range(5)]
        _check(lib().rsc_cache_buffers(self._h, *[ctypes.byref(x) for x in p]))
        return [x.value for x in p]

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            _check(lib().rsc_cache_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def copy_to_host(ptr: int, count: int, np_dtype):
    """Copies `count` elements at device address `ptr` into a new numpy
    array (synchronises the current stream first)."""
    import numpy as np
    out = np.empty(count, dtype=np_dtype)
    if count:
        torch.cuda.current_stream().synchronize()
        r = _hip().hipMemcpy(ctypes.c_void_p(out.ctypes.data), ctypes.c_void_p(ptr),
                             ctypes.c_size_t(out.nbytes), 2)  # hipMemcpyDeviceToHost
        if r != 0:
            raise RuntimeError(f"hipMemcpy failed with code {r}")
    return out


def cache_snapshot(cache: Cache, step: int = 0) -> dict:
    """Host copies of the cached slice and kept indices (for tests)."""
    import numpy as np
    g = cache.get(step)
    s = g["slice"]
    out = dict(g)
    out["nnz"] = s.nnz
    out["rowptr"] = copy_to_host(s.rowptr, s.n_rows + 1, np.int32) if s.rowptr else None
    out["col"] = copy_to_host(s.col, s.nnz, np.int32) if s.col else np.zeros(0, np.int32)
    out["val"] = copy_to_host(s.val, s.nnz, np.float32) if s.val else np.zeros(0, np.float32)
    out["idx"] = copy_to_host(g["idx_ptr"], g["k"], np.int32) if g["idx_ptr"] else np.zeros(0, np.int32)
    return out


_hip_lib = None


def _hip():
    """The HIP runtime already loaded in this process (matched by soname, so
    it is the one torch and librsc.so use)."""
    global _hip_lib
    if _hip_lib is None:
        _hip_lib = ctypes.CDLL("libamdhip64.so.7")
        _hip_lib.hipMemcpy.restype = ctypes.c_int
    return _hip_lib


# ---------------------------------------------------------------- A8
def k_from_fraction(n: int, num: int, den: int) -> int:
    return lib().rsc_k_from_fraction(n, num, den)


def greedy_allocate(keys, colnnz, nnz: int, d, fro_a2: float, fro_b2, C, alpha):
    """Layer-wise k_l (host compute). keys: list of numpy uint64 arrays."""
    import numpy as np
    L = len(keys)
    keys = [np.ascontiguousarray(k, dtype=np.uint64) for k in keys]
    n = len(keys[0])
    ptrs = (ctypes.c_void_p * L)(*[k.ctypes.data for k in keys])
    colnnz = np.ascontiguousarray(colnnz, dtype=np.int32)
    d_arr = np.ascontiguousarray(d, dtype=np.int32)
    fb = np.ascontiguousarray(fro_b2, dtype=np.float64)
    if any(len(k) != n for k in keys) or len(colnnz) != n or len(d_arr) != L or len(fb) != L:
        raise ValueError("keys and colnnz need n entries each; d and fro_b2 one per layer")
    k_out = np.zeros(L, dtype=np.int32)
    bud = ctypes.c_int64()
    _check(lib().rsc_greedy_allocate(L, n, nnz, ctypes.cast(ptrs, ctypes.c_void_p), colnnz.ctypes.data,
                                     d_arr.ctypes.data, float(fro_a2), fb.ctypes.data, C[0], C[1],
                                     alpha[0], alpha[1], k_out.ctypes.data, ctypes.byref(bud)))
    return [int(x) for x in k_out], int(bud.value)


def greedy_profile(key: torch.Tensor, colnnz: torch.Tensor, alpha, with_order: bool = False,
                   ws: torch.Tensor | None = None):
    """Device profile of one layer's ranking for the greedy: (mass float64[nb],
    count int64[nb]) and optionally the ranking int32[n]."""
    n = key.numel()
    nb = lib().rsc_greedy_blocks(n, alpha[0], alpha[1])
    mass = torch.empty(max(nb, 1), dtype=torch.float64, device=key.device)
    count = torch.empty(max(nb, 1), dtype=torch.int64, device=key.device)
    order = torch.empty(max(n, 1), dtype=torch.int32, device=key.device) if with_order else None
    need = lib().rsc_greedy_profile_workspace_bytes(n)
    ws = _workspace(need, key.device) if ws is None else ws
    _check(lib().rsc_greedy_profile(_dp(key), _dp(colnnz), n, alpha[0], alpha[1],
                                    _dp(mass), _dp(count), _ptr(order), _dp(ws),
                                    ws.numel(), _stream()))
    out = (mass[:nb], count[:nb])
    return out + (order[:n],) if with_order else out


def greedy_allocate_profiles(masses, counts, n: int, nnz: int, d, fro_a2: float, fro_b2, C, alpha):
    """Greedy loop on host numpy profiles (one mass/count array per layer)."""
    import numpy as np
    L = len(masses)
    masses = [np.ascontiguousarray(m, dtype=np.float64) for m in masses]
    counts = [np.ascontiguousarray(c, dtype=np.int64) for c in counts]
    mp = (ctypes.c_void_p * L)(*[m.ctypes.data for m in masses])
    cp = (ctypes.c_void_p * L)(*[c.ctypes.data for c in counts])
    d_arr = np.ascontiguousarray(d, dtype=np.int32)
    fb = np.ascontiguousarray(fro_b2, dtype=np.float64)
    nb = lib().rsc_greedy_blocks(n, alpha[0], alpha[1])
    if len(counts) != L or any(len(m) < nb for m in masses) or any(len(c) < nb for c in counts) \
            or len(d_arr) != L or len(fb) != L:
        raise ValueError("one mass and count profile of the greedy's block count per layer; d and fro_b2 per layer")
    k_out = np.zeros(L, dtype=np.int32)
    bud = ctypes.c_int64()
    _check(lib().rsc_greedy_allocate_profiles(L, n, nnz, alpha[0], alpha[1], ctypes.cast(mp, ctypes.c_void_p),
                                              ctypes.cast(cp, ctypes.c_void_p), d_arr.ctypes.data,
                                              float(fro_a2), fb.ctypes.data, C[0], C[1],
                                              k_out.ctypes.data, ctypes.byref(bud)))
    return [int(x) for x in k_out], int(bud.value)
