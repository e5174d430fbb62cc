"""Host-side logic of bench.py (no GPU): the quasi-DEER pass bound is refused before any GPU
work, and the host description the CPU baseline reports."""
import sys

import numpy as np
import pytest

import bench
from workloads import Workload


def _wl(T, fixed_iters=0):
    return Workload(name=f"plrnn_M64_T{T}_B1", kind="plrnn", B=1, T=T, M=64, n_obs=64, alpha=0.05,
                    params={}, x=np.zeros((1, 2, 64), np.float32), fixed_iters=fixed_iters)


def test_quasi_bound_refuses_long_solves_to_tolerance():
    with pytest.raises(SystemExit, match="quasi-passes"):
        bench.check_quasi_bound(_wl(131072), 0)


def test_quasi_bound_accepts_short_solves_and_fixed_passes():
    bench.check_quasi_bound(_wl(16384), 0)           # the M = 16 workload: T + 2 passes at most
    bench.check_quasi_bound(_wl(131072), 50)         # a fixed number of passes per solve
    bench.check_quasi_bound(_wl(131072, fixed_iters=5), 0)
    with pytest.raises(SystemExit):
        bench.check_quasi_bound(_wl(16384), -1)


def test_host_cpu_description():
    n, model = bench._host_cpu()
    assert n >= 1 and isinstance(model, str) and model


def test_vector_peak_is_the_unpacked_fp32_rate():
    # 256 CUs x 4 SIMDs x 16 lanes x 2 flops per FMA x 2.4 GHz
    assert abs(bench.PEAK_FP32_VALU_TFLOPS - 256 * 4 * 16 * 2 * 2.4e9 / 1e12) < 0.1


@pytest.mark.parametrize("point", ["other,128,32768", "contracting,128,1000", "contracting,128,0"])
def test_fig1a_point_is_checked_before_any_gpu_work(point, monkeypatch):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--fig1a", "--fig1a-point", point])
    with pytest.raises(SystemExit, match="fig1a-point"):
        bench.main()
