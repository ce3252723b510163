"""The performance arithmetic of Section 5.2 against the paper's own
numbers (Table 1 and the Section 5.3 figures, tests/golden/paper_table1.json):
the benchmark reports its step and kernel rates with the same definitions,
Sustained = 3 OPS_conv / t_exec and Peak = 3 OPS_conv / t_comp, t_comp being
the time of the three convolution passes."""
import json
import os

import pytest

import bench

HERE = os.path.dirname(os.path.abspath(__file__))
T1 = json.load(open(os.path.join(HERE, "golden", "paper_table1.json")))
CONV = ("Conv2D_FWD", "Conv2D_BackpropKernel", "Conv2D_BackpropInput")


def test_table1_columns_sum_to_t_exec():
    for col, key in (("tensor_core_ms", "tensor_core"), ("no_tensor_core_ms", "no_tensor_core")):
        assert sum(T1[col].values()) == pytest.approx(T1["t_exec_ms"][key], abs=5e-4)


def test_total_math_ops_is_three_passes():
    assert 3 * T1["ops_conv_per_pass"] == pytest.approx(T1["total_math_ops"], rel=1e-12)


def test_sustained_and_peak_per_gpu():
    t_exec = T1["t_exec_ms"]["tensor_core"] * 1e-3
    t_comp = sum(T1["tensor_core_ms"][k] for k in CONV) * 1e-3
    sus, peak = bench.paper_rates(T1["ops_conv_per_pass"], t_exec, t_comp)
    assert round(sus / 1e12, 2) == T1["sustained_tflops_per_gpu"]          # 59.67
    # 83.927 printed as 83.92: the paper truncates the second decimal
    assert peak / 1e12 == pytest.approx(T1["peak_tflops_per_gpu"], abs=0.01)
    assert int(peak / 1e10) / 100 == T1["peak_tflops_per_gpu"]
    # 49.7% and 70% of the V100's 120 TFLOPS
    assert round(100 * sus / 1e12 / T1["v100_peak_tflops"], 1) == 49.7
    assert round(100 * peak / 1e12 / T1["v100_peak_tflops"]) == 70


def test_t_comp_excludes_the_elementwise_ops():
    """Adding the ReLU column to t_comp would give 71.4 TFLOPS, not the
    printed Peak: t_comp is the convolutions' time alone."""
    with_relu = sum(T1["tensor_core_ms"][k] for k in CONV + ("Relu_ReluGrad",)) * 1e-3
    _, peak = bench.paper_rates(T1["ops_conv_per_pass"], 1.0, with_relu)
    assert abs(peak / 1e12 - T1["peak_tflops_per_gpu"]) > 10


def test_tensor_core_speedup_is_about_six():
    ratios = [T1["no_tensor_core_ms"][k] / T1["tensor_core_ms"][k] for k in CONV]
    assert all(5.5 < r < 6.4 for r in ratios)
    total = sum(T1["no_tensor_core_ms"][k] for k in CONV) / \
        sum(T1["tensor_core_ms"][k] for k in CONV)
    assert round(total) == 6


def test_machine_figures_follow_from_per_gpu_rates():
    """Sustained (peak) EFLOPS = GPUs x per-GPU rate x scaling efficiency,
    within the paper's stated uncertainty."""
    g, eff, u = T1["gpus"], T1["scaling_efficiency"], T1["eflops_uncertainty"]
    sus = g * T1["sustained_tflops_per_gpu"] * eff / 1e6
    peak = g * T1["peak_tflops_per_gpu"] * eff / 1e6
    assert abs(sus - T1["sustained_eflops"]) <= u
    assert abs(peak - T1["peak_eflops"]) <= u
