"""Input generators (CPU): the bucketed CSR used for the largest-size cases
is a valid CSR with the requested row lengths, and the row-length plan of
the int32-limit case adds up."""
import numpy as np

import synth


def test_bucket_csr_is_valid_and_seeded():
    lens = [0, 1, 7, 300, 300, 0, 64]
    A = synth.bucket_csr(lens, 300, seed=5)
    assert np.array_equal(np.diff(A.rowptr), lens)
    for i in range(A.n):
        c = A.col[A.rowptr[i]:A.rowptr[i + 1]]
        assert np.all(np.diff(c) > 0) and (len(c) == 0 or (c[0] >= 0 and c[-1] < 300))
    assert np.array_equal(A.col[A.rowptr[3]:A.rowptr[4]], np.arange(300))   # full row
    assert np.all(np.abs(A.val) <= 1.0)
    B = synth.bucket_csr(lens, 300, seed=5)
    assert np.array_equal(A.col, B.col) and np.array_equal(A.val, B.val)


def test_int32_limit_plan():
    import importlib.util, os
    spec = importlib.util.spec_from_file_location(
        "maxsize", os.path.join(os.path.dirname(__file__), "test_gpu_maxsize.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    lens, long_rows = m.max_lens()
    rowptr = np.concatenate([[0], np.cumsum(lens)])
    assert rowptr[-1] == (1 << 31) - 2
    # the last row's second 64-entry run and the long row before it step past 2^31 - 1
    assert rowptr[-2] + 2 * 64 > (1 << 31) - 1 and lens[-1] > 64
    assert lens[m.N - 2] > 1024 and rowptr[m.N - 1] + 512 > (1 << 31) - 1
