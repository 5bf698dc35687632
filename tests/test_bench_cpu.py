"""Host-side logic of bench.py that needs no GPU."""
import subprocess
import sys
import os

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_counter_traffic_lookup():
    # no summary covers an unknown kernel or workload
    assert bench.counter_traffic("k_no_such_kernel", "switch_base_8e") == (None, None)
    assert bench.counter_traffic("k_exit_mma", "no_such_workload") == (None, None)
    # a covered kernel gives bytes and the summary's path, or None once the
    # kernel source no longer matches the recorded hash
    val, src = bench.counter_traffic("k_exit_mma", "switch_base_8e")
    assert (val is None and src is None) or (val > 0 and src.startswith("profiles/"))
