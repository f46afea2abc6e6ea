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
    csrc = os.path.join(bench.ROOT, "paper_2210_10737_amd", "csrc")
    text = open(os.path.join(csrc, "spmm.hip")).read()
    probe = open(os.path.join(csrc, "probe.hip")).read()
    d0 = bench.kernel_source_digest()
    fake = tmp_path / "paper_2210_10737_amd" / "csrc"
    fake.mkdir(parents=True)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    for name in bench.COUNTED_SOURCES:
        (fake / name).write_text(open(os.path.join(csrc, name)).read())
    (fake / "spmm.hip").write_text("// a new comment\n\n" + text.replace("namespace rsc {", "namespace rsc {  /* x */"))
    assert bench.kernel_source_digest() == d0
    (fake / "spmm.hip").write_text(text.replace("kUnroll = 8", "kUnroll = 4"))
    assert bench.kernel_source_digest() != d0
    (fake / "spmm.hip").write_text(text)
    (fake / "probe.hip").write_text(probe.replace("kProbeWaves = 4", "kProbeWaves = 8"))
    assert bench.kernel_source_digest() != d0
    (fake / "probe.hip").write_text(probe)
    slice_src = open(os.path.join(csrc, "slice.hip")).read()
    (fake / "slice.hip").write_text(slice_src.replace("kFusedSub = 3", "kFusedSub = 2"))
    assert bench.kernel_source_digest() != d0


def test_traffic_record_needs_same_source_and_configuration(tmp_path, monkeypatch):
    import json
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    cfg = {"workload": "tiny", "n": 4096, "nnz": 69632, "d": 64, "budget_pct": 50, "aggregator": "gcn",
           "selector": "topk"}
    rec = {"kernel_src_digest": "abc", "config": cfg,
           "ops": {"exact": {"fetch_bytes": 3000.0, "write_bytes": 1000.0, "l2_hit_rate": 0.5}}}
    (prof / "spmm_tiny_counters.json").write_text(json.dumps(rec))
    t = bench.load_traffic(cfg, "abc", {"exact": 2000})
    assert t["ops"]["exact"]["total_bytes"] == 4000 and t["ops"]["exact"]["over_algorithmic"] == 2.0
    assert bench.load_traffic(cfg, "abd", {"exact": 2000}) is None            # other kernel source
    assert bench.load_traffic(dict(cfg, budget_pct=30), "abc", {"exact": 2000}) is None
    assert bench.load_traffic(dict(cfg, workload="social"), "abc", {"exact": 2000}) is None
