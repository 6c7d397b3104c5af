"""Host-side logic of bench.py (no GPU): the single-GPU contract, the
algorithmic flop / byte counts behind the roofline fractions, the scaling of
rocprofv3 FETCH_SIZE / WRITE_SIZE readings into HBM bytes, the kernel-name
matching of roofline labels and the automatic one-stream choice."""
import csv
import importlib.util
import os
import subprocess
import sys
import types

import pytest

from fixtures import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stdout + r.stderr


def test_algorithmic_counts(bench):
    heat, sine, deep = configs.ALL["heat-100x100"], configs.ALL["sine-1000x1000"], configs.ALL["deep-sine-1000x1000"]
    # output-layer GEMM: 2 B H D flop
    assert bench.gemm_flops(heat) == 2 * 1024 * 256 * 10_000
    assert bench.gemm_flops(deep) == 2 * 1024 * 2048 * 1_000_000
    # fused Adam: 26 B per output weight (p, m, v read and written, bf16 copy written) + dY + A_{L-1} (bf16)
    assert bench.fused_adam_bytes(sine) == 26 * 1_000_000 * 1024 + 2 * 512 * 1_000_000 + 2 * 512 * 1024
    assert bench.fused_adam_bytes(deep) == 26 * 1_000_000 * 2048 + 2 * 1024 * 1_000_000 + 2 * 1024 * 2048
    # gather: input rows only when the targets are read in place; whole rows otherwise (read + write)
    assert bench.gather_bytes(heat, False) == 2 * 6 * 4 * 1024
    assert bench.gather_bytes(heat, True) == 2 * (10_000 + 6) * 4 * 1024


def write_counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, value in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_pmc_readings_scaled_by_the_calibration_kernel(bench, tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    cal = "void neg_kernel<float>(float const*, float*, long)"
    fwd = "void ot::gemm_f32_kernel<2, 2, 2, 4, (ot::Lay)0, (ot::Lay)0, (ot::Epi)3, 16, 1>(ot::GemmArgs)"
    other = "void ot::gemm_f32_kernel<2, 2, 2, 2, (ot::Lay)1, (ot::Lay)1, (ot::Epi)4, 16, 1>(ot::GemmArgs)"
    # the copy kernel moves 1 GiB each way; FETCH_SIZE reads half of it, WRITE_SIZE all of it
    write_counters(tmp_path / "f", "FETCH_SIZE", [(cal, 524288.0), (fwd, 100.0), (fwd, 110.0), (fwd, 105.0),
                                                  (other, 9999.0)])
    write_counters(tmp_path / "w", "WRITE_SIZE", [(cal, 1048576.0), (fwd, 50.0), (fwd, 60.0), (fwd, 50.0)])
    e = bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), "heat-100x100", "gemm_fp32 (fwd_output)", "cmd")
    assert e["calibration"]["fetch_scale"] == 2.0 and e["calibration"]["write_scale"] == 1.0
    assert e["fetch_kib_per_launch"] == 105.0 and e["write_kib_per_launch"] == 50.0   # medians
    assert e["launches"] == [3, 3]
    assert e["bytes_per_launch"] == 105 * 1024 * 2 + 50 * 1024
    assert bench.traffic_for("heat-100x100", "gemm_fp32 (fwd_output)") == e["bytes_per_launch"]


def test_roofline_labels_match_their_kernels(bench):
    fused = "void ot::gemm_bf16_pipe_kernel<128, 256, 32, 3, 2, (ot::LayB)1, (ot::LayB)1, (ot::EpiB)6, 2>(ot::GemmBArgs)"
    igrad = "void ot::gemm_bf16_pp_kernel<4, (ot::LayB)0, (ot::LayB)1, (ot::EpiB)1>(ot::GemmBArgs)"
    fwd16 = "void ot::gemm_bf16_pp_kernel<4, (ot::LayB)0, (ot::LayB)0, (ot::EpiB)5>(ot::GemmBArgs)"
    fwd32 = "void ot::gemm_f32_kernel<2, 2, 2, 4, (ot::Lay)0, (ot::Lay)0, (ot::Epi)3, 16, 1>(ot::GemmArgs)"
    hidden32 = "void ot::gemm_f32_kernel<2, 2, 2, 4, (ot::Lay)0, (ot::Lay)0, (ot::Epi)2, 16, 0>(ot::GemmArgs)"
    assert bench.kernel_matches("gemm_bf16 (wgrad_output + fused Adam)", fused)
    assert not bench.kernel_matches("gemm_bf16 (wgrad_output + fused Adam)", igrad)
    assert bench.kernel_matches("gemm_bf16 (igrad_output)", igrad)
    assert bench.kernel_matches("gemm_bf16 (fwd_output)", fwd16)
    assert not bench.kernel_matches("gemm_bf16 (fwd_output)", igrad)
    assert bench.kernel_matches("gemm_fp32 (fwd_output)", fwd32)
    assert not bench.kernel_matches("gemm_fp32 (fwd_output)", hidden32)        # hidden layers: ROLE 0
    assert bench.kernel_matches("gather_x_kernel", "ot::gather_x_kernel(int const*, float const*, long)")
    assert not bench.kernel_matches("gather_kernel", "ot::gather_x_kernel(int const*, float const*, long)")


def test_one_stream_for_latency_bound_workloads(bench):
    args = types.SimpleNamespace(one_stream=False)
    assert bench.one_stream(args, configs.ALL["tiny-16x16"])           # 32 x 256 x 4 B of targets
    assert not bench.one_stream(args, configs.ALL["heat-100x100"])     # 41 MB of targets
    assert bench.one_stream(types.SimpleNamespace(one_stream=True), configs.ALL["heat-100x100"])
