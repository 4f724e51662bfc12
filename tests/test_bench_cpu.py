"""CPU checks of bench.py's host logic (no GPU needed)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_is_read_only_for_the_profiled_kernel_source():
    sys.path.insert(0, ROOT)
    import bench
    assert bench.traffic_from_profile("0000000000000000") is None
    h = bench.kernel_source_hash()
    t = bench.traffic_from_profile(h)
    assert t is None or t > 0
