"""Host-side pieces of the benchmark: the one-GPU guard and the step's roofline lower bound."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2 and "one MI355X" in r.stderr and r.stdout == ""


def test_step_lower_bound_takes_the_longer_roof_per_class():
    sys.path.insert(0, ROOT)
    import bench
    classes = {
        # 8 GB at 8 TB/s = 1 ms; 1 TFLOP is shorter: bandwidth-bound
        "a": {"bytes_per_launch": 4e9, "launches_per_step": 2, "flops_per_launch": 0.5e12},
        # 1 MB is negligible; 5.0332 PFLOP at the bf16 peak is 2 s: compute-bound
        "b": {"bytes_per_launch": 1e6, "launches_per_step": 1, "flops_per_launch": 2 * bench.BF16_PEAK_TFLOPS * 1e12},
    }
    lb = bench.step_lower_bound(classes)
    assert lb["bytes_per_step"] == pytest.approx(8e9 + 1e6)
    assert lb["lower_bound_ms"] == pytest.approx(8e9 / (bench.HBM_PEAK_GBS * 1e9) * 1e3 + 2000.0)


def test_host_description_and_class_rooflines():
    sys.path.insert(0, ROOT)
    import bench
    h = bench.host_info()
    assert set(h) == {"cpu", "sockets", "physical_cores", "logical_cpus", "omp_num_threads"}
    assert h["logical_cpus"] >= 1
    gemm = {"bytes_per_launch": 1e8, "flops_per_launch": 1e12, "achieved_GBs": 4000.0, "achieved_TFLOPs": 1258.3}
    assert bench.class_roofline("gemm_tile", gemm, 1237)["bound"] == "mfma"
    assert bench.class_roofline("gemm_tile", gemm, 1237)["frac"] == pytest.approx(0.5)
    assert bench.class_roofline("gemm_ring1", gemm, 171)["bound"] == "hbm"
    assert bench.class_roofline("rows", {"bytes_per_launch": 0, "flops_per_launch": 0}, 171) is None
