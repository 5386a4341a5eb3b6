"""bench.py's command line on a machine without a GPU: more than one GPU is
refused with exit status 2 before anything touches a device, and --help
lists the documented options."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr


def test_help_lists_the_options():
    r = run("--help")
    assert r.returncode == 0
    for opt in ("--gpus", "--steps", "--warmup", "--no-extra", "--no-cpu", "--only-config", "--sweep"):
        assert opt in r.stdout


def test_profiled_traffic_is_found_for_the_timed_kernels(tmp_path, monkeypatch):
    """The profiler byte counts are looked up by kernel, with or without the
    variant suffix the summaries give the assignment, and only while the
    sources they were taken on are unchanged."""
    import json
    sys.path.insert(0, ROOT)
    import bench
    sha = bench.source_sha256()
    t = {"source_sha256": sha, "workloads": {"w": {"kernels": {
        "k_vote_mfma": {"bytes": 11}, "k_assign_mfma (exact search)": {"bytes": 22}}}}}
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps(t))
    monkeypatch.setattr(bench, "TRAFFIC", str(f))
    assert bench.measured_traffic("w", "compact_vote") == 11
    assert bench.measured_traffic("w", "assign_label") == 22
    assert bench.measured_traffic("other", "assign_label") is None
    t["source_sha256"] = "0" * 64
    f.write_text(json.dumps(t))
    assert bench.measured_traffic("w", "assign_label") is None
