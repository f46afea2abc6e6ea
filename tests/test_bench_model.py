"""Byte models and the counter-record digest of bench.py (CPU): the
algorithmic bytes follow their definitions term by term on small cases, and
the digest ignores comments and blank lines but not code."""
import os

import bench


def test_spmm_bytes_terms():
    # rowptr 4(n+1), col+val 8 per entry, each referenced B row once, Y once
    n, nnz, n_src, d = 10, 37, 6, 8
    assert bench.spmm_bytes(n, nnz, n_src, d) == 4 * 11 + 8 * 37 + 4 * 6 * 8 + 4 * 10 * 8
    assert bench.spmm_bytes(2_449_029, 126_197_977, 2_449_029, 256) == 6_034_991_328


def test_refresh_bytes_grow_with_each_term():
    base = bench.refresh_bytes(100, 1000, 200, 30, 16)
    assert bench.refresh_bytes(100, 1001, 200, 30, 16) - base == 12
    assert bench.refresh_bytes(100, 1000, 201, 30, 16) - base == 8
    assert bench.refresh_random_bytes(100, 1000, 201, 30, 16) - bench.refresh_random_bytes(100, 1000, 200, 30, 16) == 16


def test_digest_ignores_comments_only(tmp_path, monkeypatch):
    src = os.path.join(bench.ROOT, "paper_2210_10737_amd", "csrc", "spmm.hip")
    text = open(src).read()
    d0 = bench.kernel_source_digest()
    fake = tmp_path / "paper_2210_10737_amd" / "csrc"
    fake.mkdir(parents=True)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (fake / "spmm.hip").write_text("// a new comment\n\n" + text.replace("namespace rsc {", "namespace rsc {  /* x */"))
    assert bench.kernel_source_digest() == d0
    (fake / "spmm.hip").write_text(text.replace("kUnroll = 8", "kUnroll = 4"))
    assert bench.kernel_source_digest() != d0
