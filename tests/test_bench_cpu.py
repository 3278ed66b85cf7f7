"""Host logic of bench.py (no GPU): the counter-reading lookup, the refusal of
more than one GPU, and the oracle baseline's report."""

import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_traffic_lookup_needs_matching_source_and_workload(tmp_path, monkeypatch):
    rec = {"src_hash": "abc", "workload": "w", "kernels": {"residual_add": {"bytes_per_launch": 123.0}}}
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench._traffic_from_profiles("residual_add", "abc", "w") == 123.0
    assert bench._traffic_from_profiles("residual_add", "abd", "w") is None   # the kernel changed since
    assert bench._traffic_from_profiles("residual_add", "abc", "v") is None   # another workload
    assert bench._traffic_from_profiles("merge", "abc", "w") is None


def test_traffic_lookup_without_a_record(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench._traffic_from_profiles("residual_add", "abc", "w") is None


def test_committed_counter_readings_name_a_kernel_source():
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as fh:
        rec = json.load(fh)
    assert len(rec["src_hash"]) == 16 and rec["kernels"]["residual_add"]["bytes_per_launch"] > 0
    # the source hash is a pure function of the add's files
    assert bench._kernel_src_hash() == bench._kernel_src_hash()


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2
    line = json.loads(p.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def test_cpu_baseline_reports_its_sample():
    """The oracle on every block index over a pool of fresh processes, with the
    host's core count and CPU model and the single-thread figure beside it."""
    from paper_2304_00737_amd import workloads as W
    out = bench.cpu_baseline(W.config(1))
    assert out["kind"] == "oracle" and out["unit"] == "elements/s"
    assert out["cores"] == min(os.cpu_count(), bench.CPU_SHARE) and out["nproc"] == os.cpu_count()
    assert out["value"] > 0 and out["single_thread_value"] > 0 and out["cpu_model"]
    assert "block indices" in out["sample"] and "single-thread" in out["sample"]
