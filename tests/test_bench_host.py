"""Host-side pieces of the benchmark driver (no GPU)."""
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_recorded_workloads_skips_cut_lines(tmp_path):
    p = tmp_path / "all.jsonl"
    assert bench.recorded_workloads(str(p)) == set()
    assert bench.recorded_workloads(None) == set()
    lines = [json.dumps({"config": {"workload": w}}) for w in bench.WORKLOADS[:2]]
    p.write_text("\n".join(lines) + "\n" + lines[0][: len(lines[0]) // 2])  # last line cut short
    assert bench.recorded_workloads(str(p)) == set(bench.WORKLOADS[:2])


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
