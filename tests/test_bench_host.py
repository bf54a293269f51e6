"""Host-side logic of bench.py (no GPU): the CPU-baseline leg and the single-GPU guard."""
import dataclasses
import os
import subprocess
import sys

import pytest

from synth import Module, gen_module_inputs, workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_baseline_pool_reports_rate_cores_and_sample():
    """The oracle over spawned worker processes, on a small module: a positive
    rate in candidates/s, the worker count actually used, the CPU model and
    a sample description."""
    import bench

    mods = (Module("t", 64, 256, 0, 0, 0), Module("u", 32, 128, 0, 1, 1))
    wl = dataclasses.replace(workload("block3b", S=8, P=4), modules=mods)
    rows = []
    for m in mods:
        inp = gen_module_inputs(wl, m, "cpu")
        rows.append((inp["W32"][::2].numpy(), inp["d"][::2].numpy()))
    r = bench.cpu_baseline(wl, {"step": 2, "rows": rows}, 0.2)
    assert r["kind"] == "oracle" and r["unit"] == "candidates/s" and r["value"] > 0
    assert 1 <= r["cores"] <= 16 and r["cores"] <= len(os.sched_getaffinity(0))
    assert isinstance(r["cpu"], str) and r["cpu"]
    assert "of the 2 modules" in r["sample"] and "worker processes" in r["sample"]
    assert r["extrapolated_full_encode_s"] > 0


def test_bench_refuses_more_than_one_gpu():
    """--gpus above 1 exits with status 2 and says why, before touching a device."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "single GPU" in r.stderr
