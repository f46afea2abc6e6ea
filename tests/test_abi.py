"""C-ABI checks that need no GPU: the library loads, exports exactly what
include/rsc.h declares, rejects bad arguments with the documented status
before touching the device, and its host-side budget helpers (the column
budget and the greedy allocation) agree with the oracle."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
import paper_2210_10737_amd as rsc
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rsc.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rsc_[a-z0-9_]+)\s*\(", text)))


def test_header_matches_exports():
    declared = declared_functions()
    assert declared == sorted(rsc.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", rsc.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(set(re.findall(r"\bT (rsc_[a-z0-9_]+)$", out, flags=re.M)))
    assert exported == declared
    L = rsc.lib()
    for name in declared:
        assert getattr(L, name) is not None
    assert L.rsc_abi_version() == 5


def test_status_strings():
    L = rsc.lib()
    for code, name in rsc.STATUS.items():
        assert L.rsc_status_string(code).decode() == name


def _csr(n_rows=4, n_cols=4, nnz=4, rowptr=0x1000, col=0x2000, val=0x3000):
    return rsc.CsrStruct(n_rows, n_cols, nnz, rowptr, col, val)


def _err(status):
    return rsc.STATUS[status]


def test_spmm_argument_validation():
    L = rsc.lib()
    A = _csr()
    ws_need = L.rsc_spmm_workspace_bytes(ctypes.byref(A))
    ws = 0x10000
    good = dict(B=0x4000, d=8, ldb=8, Y=0x8000, ldy=8)

    def call(A=A, B=good["B"], d=good["d"], ldb=good["ldb"], Y=good["Y"], ldy=good["ldy"], ws=ws,
             wsb=ws_need):
        return L.rsc_spmm(ctypes.byref(A) if A is not None else None, B, d, ldb, Y, ldy, ws, wsb, None)

    assert _err(call(A=None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(call(d=0)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(call(ldb=4)) == "RSC_ERR_INVALID_ARGUMENT"          # ld < d
    assert _err(call(ldb=10)) == "RSC_ERR_UNSUPPORTED"              # ld % 4
    assert _err(call(B=0x4004)) == "RSC_ERR_UNSUPPORTED"            # misaligned
    assert _err(call(B=None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(call(A=_csr(nnz=1 << 31))) == "RSC_ERR_UNSUPPORTED"
    assert _err(call(A=_csr(n_rows=-1))) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(call(A=_csr(col=None))) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(call(wsb=ws_need - 1)) == "RSC_ERR_CAPACITY"
    assert _err(call(ws=0x10010)) == "RSC_ERR_UNSUPPORTED"           # ws alignment
    assert "ld" in L.rsc_last_error().decode() or "aligned" in L.rsc_last_error().decode()


def test_topk_and_slice_argument_validation():
    L = rsc.lib()
    n = 100
    need = L.rsc_topk_workspace_bytes(n)
    assert _err(L.rsc_topk_select(0x1000, n, -1, 0x2000, 0x3000, 0x4000, need, None)) == \
        "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_topk_select(0x1000, n, n + 1, 0x2000, 0x3000, 0x4000, need, None)) == \
        "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_topk_select(0x1000, n, 5, None, 0x3000, 0x4000, need, None)) == \
        "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_topk_select(0x1000, n, 5, 0x2000, 0x3000, 0x4000, need - 1, None)) == \
        "RSC_ERR_CAPACITY"
    A = _csr()
    sneed = L.rsc_slice_workspace_bytes(ctypes.byref(A))
    assert _err(L.rsc_slice_csr(ctypes.byref(A), 0x1000, None, 0x2000, 0x3000, 0x4000, -1, 0x5000, 0x10000,
                                sneed, None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_slice_csr(ctypes.byref(A), None, None, 0x2000, 0x3000, 0x4000, 4, 0x5000, 0x10000,
                                sneed, None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_slice_csr(ctypes.byref(A), 0x1000, None, 0x2000, 0x3000, 0x4000, 4, 0x5004, 0x10000,
                                sneed, None)) == "RSC_ERR_UNSUPPORTED"
    assert _err(L.rsc_slice_csr(ctypes.byref(A), 0x1000, 0x1004, 0x2000, 0x3000, 0x4000, 4, 0x5000, 0x10000,
                                sneed, None)) == "RSC_ERR_UNSUPPORTED"
    swn = L.rsc_sample_workspace_bytes(100)
    assert _err(L.rsc_sample_columns(0x1000, 100, -1, 0, 0x2000, 0x3000, 0x4000, 0x10000, swn, None)) == \
        "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_sample_columns(0x1000, 100, 5, 0, 0x2000, 0x3000, 0x4000, 0x10000, swn - 1, None)) == \
        "RSC_ERR_CAPACITY"


def test_cache_argument_validation():
    L = rsc.lib()
    out = ctypes.c_void_p()
    A = _csr()
    bad_t = _csr(n_rows=5)
    assert _err(L.rsc_cache_create(ctypes.byref(A), ctypes.byref(bad_t), 10, None, ctypes.byref(out))) == \
        "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_cache_create(ctypes.byref(A), ctypes.byref(A), 0, None, ctypes.byref(out))) == \
        "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_cache_refresh(None, 0x1000, 4, 4, 1, 0, None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_spmm_sampled(None, 0x1000, 4, 4, 0x2000, 4, None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert _err(L.rsc_cache_staleness(None, 0x1000, None, None, None, None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert L.rsc_cache_destroy(None) == 0
    half = rsc.Allocator(rsc._ALLOC_FN(lambda n, s, c: None), rsc._FREE_FN(), None)  # no free
    assert _err(L.rsc_cache_create_ex(ctypes.byref(A), ctypes.byref(A), 10, ctypes.byref(half), None,
                                      ctypes.byref(out))) == "RSC_ERR_INVALID_ARGUMENT"


def test_csr_validate_argument_checks():
    L = rsc.lib()
    bad = ctypes.c_int64(7)
    assert _err(L.rsc_csr_validate(None, ctypes.byref(bad), None)) == "RSC_ERR_INVALID_ARGUMENT"
    assert bad.value == -1
    big = _csr(nnz=1 << 31)
    assert _err(L.rsc_csr_validate(ctypes.byref(big), None, None)) == "RSC_ERR_UNSUPPORTED"


@pytest.mark.skipif(os.environ.get("HIP_VISIBLE_DEVICES", None) is None and
                    __import__("torch").cuda.is_available(), reason="a GPU is visible")
def test_no_device_status():
    L = rsc.lib()
    A = _csr()
    need = L.rsc_spmm_workspace_bytes(ctypes.byref(A))
    st = L.rsc_spmm(ctypes.byref(A), 0x4000, 8, 8, 0x8000, 8, 0x10000, need, None)
    assert _err(st) == "RSC_ERR_NO_DEVICE"


def test_k_from_fraction_matches_oracle():
    L = rsc.lib()
    for n in (0, 1, 7, 4096, 232_965, 2_449_029, 132_534):
        for num, den in ((0, 100), (10, 100), (30, 100), (50, 100), (1, 3), (100, 100)):
            assert L.rsc_k_from_fraction(n, num, den) == oracle.k_from_fraction(n, num, den)
    assert L.rsc_k_from_fraction(10, 1, 0) == -1
    assert L.rsc_k_from_fraction(10, 3, 2) == -1


def _keys_and_norms(A, ds, seed):
    cn2, colnnz = oracle.col_sqnorms(A.rowptr, A.val)
    keys, fb = [], []
    for l, dl in enumerate(ds):
        o = oracle.pair_keys(cn2, synth.dense_normal(A.n, dl, seed=seed + l))
        keys.append(o["key"]); fb.append(float(o["rn2"].sum()))
    return cn2, colnnz, keys, fb


@pytest.mark.parametrize("C", [(1, 10), (3, 10), (1, 2), (0, 1), (1, 1)])
def test_greedy_matches_oracle(C):
    A = synth.make_graph("tiny", 0)
    ds = [64, 16, 8]
    cn2, colnnz, keys, fb = _keys_and_norms(A, ds, seed=20)
    # ties and NaN keys in the third layer
    keys[2] = keys[2].copy()
    keys[2][::7] = keys[2][3]
    keys[2][5::11] = 0
    k_lib, b_lib = rsc.greedy_allocate(keys, colnnz, A.nnz, ds, cn2.sum(), fb, C, (2, 100))
    k_orc, b_orc = oracle.greedy(keys, colnnz, A.nnz, ds, cn2.sum(), fb, C, (2, 100))
    assert k_lib == k_orc and b_lib == b_orc


def test_greedy_hand_example_through_abi():
    import json
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "greedy_hand_example.json")))
    import struct
    keys = [np.array([struct.unpack("<Q", struct.pack("<d", float(s) ** 2))[0] + 1 for s in row],
                     np.uint64) for row in g["scores"]]
    k, bud = rsc.greedy_allocate(keys, g["colnnz"], g["nnz"], g["d"], g["fro_a2"], g["fro_b2"],
                                 tuple(g["C"]), tuple(g["alpha"]))
    assert k == g["expected_k"] and bud == g["expected_budget"]


def host_profile(key, colnnz, alpha):
    """The greedy's per-block profile from the oracle's ranking: block j
    covers ranks [max(0, n-(j+1)step), n-j*step); sqrt(q) summed in ascending
    rank order one by one (fp64), NaN keys counting 0."""
    import math
    import struct
    n = len(key)
    step = max(1, n * alpha[0] // alpha[1])
    order = oracle.rank_order(key)
    nb = -(-n // step)
    mass, count = np.zeros(nb), np.zeros(nb, np.int64)
    for j in range(nb):
        hi = n - j * step
        lo = max(0, hi - step)
        s = 0.0
        for p in range(lo, hi):
            u = int(key[order[p]])
            if u:
                s += math.sqrt(struct.unpack("<d", struct.pack("<Q", u - 1))[0])
        mass[j] = s
        count[j] = int(colnnz[order[lo:hi]].sum())
    return mass, count


@pytest.mark.parametrize("C", [(1, 10), (3, 10), (1, 2), (0, 1), (1, 1)])
def test_greedy_profiles_match_oracle(C):
    A = synth.make_graph("tiny", 0)
    ds = [64, 16, 8]
    cn2, colnnz, keys, fb = _keys_and_norms(A, ds, seed=30)
    keys[1] = keys[1].copy()
    keys[1][::5] = keys[1][7]
    keys[1][3::13] = 0
    alpha = (3, 100)
    profs = [host_profile(k, colnnz, alpha) for k in keys]
    k_p, b_p = rsc.greedy_allocate_profiles([m for m, _ in profs], [c for _, c in profs], A.n, A.nnz, ds,
                                            cn2.sum(), fb, C, alpha)
    k_o, b_o = oracle.greedy(keys, colnnz, A.nnz, ds, cn2.sum(), fb, C, alpha)
    assert k_p == k_o and b_p == b_o
    assert rsc.lib().rsc_greedy_blocks(A.n, 3, 100) == len(profs[0][0])


def test_greedy_budget_comparison_wide_range():
    """bud * C_den and C_num * total pass 2^63 here (nnz = 2^31 - 1, d = 2^20,
    C = 1 / 2^30); the library must take the same decisions as the oracle's
    exact integer comparison."""
    keys = [np.array([9, 7, 5, 3], np.uint64) << np.uint64(52)]
    colnnz = np.ones(4, np.int32)
    args = (keys, colnnz, 2**31 - 1, [2**20], 1.0, [1.0], (1, 2**30), (1, 4))
    k_lib, b_lib = rsc.greedy_allocate(*args)
    k_orc, b_orc = oracle.greedy(*args)
    assert k_lib == k_orc == [0] and b_lib == b_orc


def test_greedy_rejects_step_above_n_and_budget_overflow():
    """alpha is a fraction of the n columns (section 5.1 uses 2 %): above 1 the
    step n * alpha would not fit int32, so the allocation, the profile's block
    count and the profile itself refuse it; a full budget sum_l nnz d_l past
    int64 is refused too."""
    keys = [np.array([9, 7, 5, 3], np.uint64)]
    with pytest.raises(rsc.RscError, match="alpha"):
        rsc.greedy_allocate(keys, np.ones(4, np.int32), 4, [8], 1.0, [1.0], (1, 2), (5, 4))
    assert rsc.lib().rsc_greedy_blocks(4, 5, 4) == -1
    assert rsc.lib().rsc_greedy_blocks(4, 4, 4) == 1
    assert rsc.lib().rsc_greedy_blocks(2**31 - 1, 3, 1) == -1
    with pytest.raises(rsc.RscError, match="alpha"):
        rsc.greedy_allocate_profiles([np.zeros(1)], [np.zeros(1, np.int64)], 4, 4, [8], 1.0, [1.0], (1, 2), (3, 1))
    with pytest.raises(rsc.RscError, match="int64"):
        rsc.greedy_allocate(keys * 2, np.ones(4, np.int32), 2**40, [2**22, 2**22], 1.0, [1.0, 1.0], (1, 2), (1, 4))
    # one layer at 2^62 still fits
    k, _ = rsc.greedy_allocate(keys, np.ones(4, np.int32), 2**40, [2**22], 1.0, [1.0], (1, 1), (1, 4))
    assert k == [4]


def test_greedy_binding_rejects_short_arrays():
    keys = [np.array([9, 7, 5, 3], np.uint64)]
    with pytest.raises(ValueError):
        rsc.greedy_allocate(keys, np.ones(3, np.int32), 4, [8], 1.0, [1.0], (1, 2), (1, 4))
    with pytest.raises(ValueError):
        rsc.greedy_allocate(keys, np.ones(4, np.int32), 4, [8, 8], 1.0, [1.0], (1, 2), (1, 4))
    with pytest.raises(ValueError):
        rsc.greedy_allocate_profiles([np.zeros(1)], [np.zeros(1, np.int64)], 4, 4, [8], 1.0, [1.0], (1, 2), (1, 4))


def test_plain_c_consumer(tmp_path):
    """include/rsc.h compiles as C11 and a C program linked against
    librsc.so runs its host-only entry points; its greedy result equals the
    oracle's on the same input."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    exe = tmp_path / "c_abi_consumer"
    libdir = os.path.dirname(rsc.LIB_PATH)
    subprocess.run([gcc, "-std=c11", "-Wall", "-Werror", "-Wno-unused-function", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    os.path.join(ROOT, "tests", "c_abi_consumer.c"), "-L", libdir, "-lrsc",
                    f"-Wl,-rpath,{libdir}", "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()
    keys = [np.array([9, 7, 5, 3], np.uint64) << np.uint64(52), np.array([8, 6, 4, 2], np.uint64) << np.uint64(52)]
    k, bud = oracle.greedy(keys, [3, 1, 2, 4], 10, [4, 2], 1.0, [1.0, 1.0], (1, 2), (1, 4))
    assert [int(out[0]), int(out[1])] == k and int(out[2]) == bud


def test_plan_argument_checks():
    L = rsc.lib()
    out = ctypes.c_void_p(7)
    A = rsc.CsrStruct(4, 4, 0, None, None, None)
    assert L.rsc_spmm_plan_create(ctypes.byref(A), None, None) == 1          # out is NULL
    assert L.rsc_spmm_plan_create(ctypes.byref(A), None, ctypes.byref(out)) == 1  # rowptr is NULL
    assert out.value is None
    assert L.rsc_spmm_plan_run(None, None, 4, 4, None, 4, None) == 1
    assert L.rsc_spmm_plan_destroy(None) == 0


def test_binding_refuses_operands_smaller_than_the_call():
    # The library reads and writes rows x d elements through each pointer, so
    # the binding refuses a dense operand with fewer rows or columns, another
    # dtype or a non-unit column stride, and index arrays shorter than the
    # call needs, before any launch (host tensors: the checks come first).
    import torch
    B = torch.zeros((10, 8), dtype=torch.float32)
    with pytest.raises(ValueError, match="holds less"):
        rsc._dense(B, 11, 8, "B")
    with pytest.raises(ValueError, match="holds less"):
        rsc._dense(B, 10, 9, "B")
    with pytest.raises(ValueError, match="float32 expected"):
        rsc._dense(B.double(), 10, 8, "B")
    with pytest.raises(ValueError, match="unit column stride"):
        rsc._dense(B.t(), 8, 10, "B")
    with pytest.raises(ValueError, match="contiguous"):
        rsc._vec(torch.zeros(3, dtype=torch.int32), 4, torch.int32, "mask")
    with pytest.raises(ValueError, match="contiguous"):
        rsc._vec(torch.zeros(4, dtype=torch.int64), 4, torch.int32, "mask")
    with pytest.raises(ValueError, match="contiguous"):
        rsc._vec(torch.zeros(8, dtype=torch.int32)[::2], 4, torch.int32, "mask")
    assert rsc._vec(None, 4, torch.int32, "mask") is None
    A = rsc.DeviceCsr(4, 4, torch.zeros(4, dtype=torch.int32), torch.zeros(0, dtype=torch.int32),
                      torch.zeros(0, dtype=torch.float32))
    with pytest.raises(ValueError, match="rowptr"):
        A.struct()                                   # 4 row pointers for 4 rows
    A = rsc.DeviceCsr(2, 4, torch.zeros(3, dtype=torch.int32), torch.zeros(5, dtype=torch.int32),
                      torch.zeros(4, dtype=torch.float32), nnz=5)
    with pytest.raises(ValueError, match="val"):
        A.struct()                                   # 4 values for 5 entries
