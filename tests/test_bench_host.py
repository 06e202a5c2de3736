"""bench.py's host-side contract (CPU): one GPU only, one JSON line."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_traffic_figures_belong_to_the_profiled_workload():
    sys.path.insert(0, ROOT)
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    with open(b.TRAFFIC_FILE) as f:
        t = json.load(f)
    # HBM bytes from the counters cover at least the algorithmic bytes, and
    # never apply to another workload
    assert t["bytes_per_launch"] >= t["algorithmic_bytes_per_launch"]
    assert b.measured_traffic("qwen3-32b-decode") is None
