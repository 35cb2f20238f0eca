"""The benchmark's command line on the host (no GPU use): more than one GPU is
refused with a message before anything touches a GPU; the statistics it
reports over timed samples (mean, median, p10, p90)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_stats_of_samples():
    sys.path.insert(0, ROOT)
    import bench
    s = bench.stats_of([4.0, 1.0, 3.0, 2.0, 5.0])
    assert s["mean"] == 3.0 and s["median"] == 3.0 and s["n"] == 5
    assert s["p10"] <= s["median"] <= s["p90"]
