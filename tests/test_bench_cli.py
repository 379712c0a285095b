"""bench.py's command line on a machine without a GPU: more than one GPU is
refused with a message, the per-set constants describe the kernels, and the
roofline names the kernel the library launches for each workload."""
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


def test_committed_counters_are_plausible():
    """The rocprofv3 counter summaries bench.py reads for roofline.traffic and
    roofline_deconstruct.measured_*: square workload, byte counts at least the
    algorithmic ones (planes read once per GEMM launch; FP64 read, planes
    written and one exponent-scan read per call), and taken on the current
    kernel sources (else skipped: the bench then reports null)."""
    sys.path.insert(0, ROOT)
    import bench
    import workloads
    w = workloads.WORKLOADS["square"]
    stale = []
    for name, cfg in bench.SETS.items():
        path = bench.COUNTER_FILES[name]
        kv = dict(line.split(":", 1) for line in open(path) if ":" in line and not line.startswith("#"))
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        assert kv["workload"] == "square"
        planes = cfg["plane_bytes"] * (w.m * w.k + w.k * w.n)
        assert float(kv["hbm_bytes_per_launch"]) >= planes
        if bench.measured_traffic(w, name) is None:
            stale.append(path)
    kv = dict(line.split(":", 1) for line in open(bench.DEC_COUNTERS) if ":" in line and not line.startswith("#"))
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    for name, cfg in bench.SETS.items():
        alg = (8 + cfg["plane_bytes"] + 8) * (w.m * w.k + w.k * w.n)
        assert 0.95 * alg <= float(kv[f"hbm_bytes_per_call_{name}"]) <= 1.5 * alg
    if bench.measured_deconstruction(w, "s12", 0.2, 1.0)["measured_bytes"] is None:
        stale.append(bench.DEC_COUNTERS)
    if stale:
        import pytest
        pytest.skip(f"counter summaries taken on older kernel sources: {stale}")


def test_gemm_kernel_names(monkeypatch):
    """The kernel named in the roofline object follows the library's rule:
    the persistent forms at an even count of 2-16 K stages with at least two
    tiles per CU (256 CUs here), the grid of one block per tile otherwise."""
    import types

    import torch
    sys.path.insert(0, ROOT)
    import bench
    import workloads
    monkeypatch.setattr(torch.cuda, "get_device_properties",
                        lambda i: types.SimpleNamespace(multi_processor_count=256))
    s12, a15 = bench.SETS["s12"], bench.SETS["a15"]
    W = workloads.WORKLOADS
    assert bench.gemm_kernel_name(W["hpl"], s12) == "residue_gemm_persistent_kernel<int16>"
    assert bench.gemm_kernel_name(W["hpl"], a15) == "residue_gemm_bytes_persistent_kernel<int8>"
    for name in ("square", "ragged", "reach", "tiny"):
        assert bench.gemm_kernel_name(W[name], s12) == "residue_gemm_kernel<int16>", name
        assert bench.gemm_kernel_name(W[name], a15) == "residue_gemm_bytes_kernel<int8>", name
