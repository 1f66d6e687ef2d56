"""Host-side logic of bench.py (no GPU): the single-GPU guard and the lookup
of measured HBM traffic, which must refuse counter figures taken on other
kernel sources."""
import hashlib
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=60)
    assert res.returncode == 2
    assert "single GPU" in res.stderr
    assert res.stdout == ""          # no JSON line for an unsupported run


def _fake_tree(tmp_path, kernels_src, record_sources):
    csrc = tmp_path / "paper_2010_07565_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "bigcn_kernels.hip").write_bytes(kernels_src)
    (csrc / "bigcn_api.hip").write_bytes(b"// api\n")
    h = hashlib.sha256()
    for part in record_sources:
        h.update(part)
    rec = {"sources_sha256": h.hexdigest(),
           "entries": [{"layer": 0, "entry": "spmm", "fetch_bytes": 1000, "write_bytes": 24},
                       {"layer": 1, "entry": "pack", "fetch_bytes": 7, "write_bytes": 5}]}
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "hbm_traffic_toy.md").write_text(
        "# toy\n\n```json\n" + json.dumps(rec) + "\n```\n")


def test_measured_traffic_matches_entry_and_sources(tmp_path, monkeypatch):
    _fake_tree(tmp_path, b"// kernels\n", [b"// kernels\n", b"// api\n"])
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("toy", 0, "spmm") == 1024
    assert bench.measured_traffic("toy", 1, "pack") == 12
    assert bench.measured_traffic("toy", 1, "spmm") is None      # no such entry
    assert bench.measured_traffic("other", 0, "spmm") is None    # no summary


def test_measured_traffic_is_dropped_when_kernels_changed(tmp_path, monkeypatch):
    _fake_tree(tmp_path, b"// kernels, edited\n", [b"// kernels\n", b"// api\n"])
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("toy", 0, "spmm") is None


def test_committed_traffic_summaries_parse():
    # every committed summary carries a hash and per-entry byte counts
    import re
    prof = os.path.join(ROOT, "profiles")
    names = [f for f in os.listdir(prof) if f.startswith("hbm_traffic_")]
    assert names
    for f in names:
        m = re.search(r"```json\n(.*?)\n```", open(os.path.join(prof, f)).read(), re.S)
        assert m is not None, f
        rec = json.loads(m.group(1))
        assert len(rec["sources_sha256"]) == 64
        assert rec["entries"]
        for e in rec["entries"]:
            assert e["fetch_bytes"] > 0 and e["write_bytes"] > 0
            assert e["entry"] in ("pack", "bgemm", "spmm")


def test_cpu_baseline_times_small_graphs_on_one_thread_too():
    # the oracle's thread count is restored after the one-thread passes
    import oracle
    import workloads
    w = workloads.make_workload(1)
    before = oracle.threads()
    r = bench.cpu_baseline(w, budget_s=0.0)
    assert oracle.threads() == before
    assert r["kind"] == "oracle" and r["cores"] == before and r["value"] > 0
    one = r["single_thread"]
    assert one["cores"] == 1 and one["value"] > 0 and one["unit"] == "nodes/s"
    # above the size limit only the all-threads figure is taken
    r = bench.cpu_baseline(w, budget_s=0.0, single_thread_max_nodes=w.n - 1)
    assert "single_thread" not in r
