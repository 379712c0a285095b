"""bench.py's command line on a machine without a GPU: more than one GPU is
refused with a message, and the per-set constants describe the kernels."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_set_constants():
    sys.path.insert(0, ROOT)
    import bench
    s12, a15 = bench.SETS["s12"], bench.SETS["a15"]
    assert (s12["r"], s12["products"], s12["plane_bytes"]) == (12, 36, 30)
    assert (a15["r"], a15["products"], a15["plane_bytes"]) == (15, 15, 15)
    assert s12["cres_bytes"] == 12 * 2 and a15["cres_bytes"] == 15
