"""bench.py's host-side contract (CPU): more than one GPU is refused with a
message, and the counter bytes it reports are tied to the kernel source."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_counter_traffic_follows_the_kernel_source():
    import bench
    path = os.path.join(ROOT, "profiles", "pass1_gpt1p3b_counters.json")
    rec = json.load(open(path))
    assert rec["kernel"] == "k_pass1" and rec["dispatches"] > 0
    want = rec["hbm_bytes_per_launch"] if rec["kernel_sha"] == bench.kernel_source_sha() else None
    assert bench.counter_traffic("gpt1p3b") == want
    assert bench.counter_traffic("no-such-workload") is None
