"""bench.py's CPU leg (the oracle timed on a bounded sample of a workload)
and its argument contract, without a GPU."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_cpu_baseline_only_prints_one_json_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--cpu-baseline-only", "--workload", "c1"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    d = json.loads(r.stdout.strip().splitlines()[-1])
    assert d["kind"] == "oracle" and d["unit"] == "tokens/s" and d["value"] > 0
    assert d["cores"] >= 1 and d["host_cpus"] >= 1
    assert "c1 with the first" in d["sample"]


def test_one_thread_child():
    proc = bench.start_one_thread("c1")
    d = bench.finish_one_thread(proc, timeout_s=300)
    assert d is not None and d["cores"] == 1 and d["value"] > 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2 and "not supported" in r.stderr
