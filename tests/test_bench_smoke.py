"""The benchmark's contract: its host logic on the CPU, its JSON line on the GPU.

Thresholds are not asserted (they are reported, not gated); the tests check
that the line carries every field with a consistent value, that the matrix
work per pair follows from the MFMA shapes, and that the per-launch traffic is
reported only for the kernel source it was measured on.
"""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2004_11127_amd import inputs, kred  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_default_run_is_the_headline_with_the_fused_gradient_beside_it():
    old = sys.argv
    try:
        sys.argv = ["bench.py"]
        args = bench.parse()
    finally:
        sys.argv = old
    assert args.workload == "headline" and args.gpus == 1
    gen, gkw, formula, reduction, fpp, bound, desc = bench.WORKLOADS["headline"]
    assert (formula, reduction, fpp, gkw["M"], gkw["N"], gkw["D"]) == ("gauss", "sum", 11, 10**6,
                                                                        10**6, 3)
    assert bench.EXTRA["headline"] == ["c2"]
    assert bench.WORKLOADS["c2"][1] == gkw   # the same inputs


def test_probe_library_exports_its_header():
    import ctypes
    import re
    hdr = open(os.path.join(ROOT, "include", "kred_probe.h")).read()
    names = re.findall(r"^\s*int\s+(kred_[a-z_]+)\s*\(", hdr, flags=re.M)
    assert names == ["kred_probe_peak"]
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2004_11127_amd", "libkred_probe.so"))
    for n in names:
        assert hasattr(lib, n), n


def test_workload_table_is_consistent():
    for name, (gen, gkw, formula, reduction, fpp, bound, desc) in bench.WORKLOADS.items():
        assert callable(getattr(inputs, gen)), name
        assert formula in kred.FORMULAS or formula == "backward", name
        assert reduction is None or reduction in kred.REDUCTIONS, name
        assert (reduction is None) == (formula == "backward"), name
        assert bound in ("alu", "mfma"), name
        assert fpp > 0 and isinstance(desc, str) and desc, name
    for s in bench.SPARSE:
        assert s in bench.WORKLOADS
    for name in bench.REDUCTIONS_PER_STEP:
        assert bench.WORKLOADS[name][2] == "backward"
    for kernel, src in bench.KERNEL_SOURCES.items():
        assert bench.source_sha(kernel) is not None, (kernel, src)


class _W:
    def __init__(self, D, E=1):
        self.D, self.E = D, E


def test_matrix_work_per_pair_follows_the_mfma_shapes():
    # a 16x16x32 product is 2 * 16 * 16 * 32 flops over 16 x 16 pairs and 32 K
    # slots: 64 flops per pair per 32 slots
    per32 = 2 * 16 * 16 * 32 // (16 * 16)
    assert bench.matrix_flops_per_pair("fast_kernel", _W(3), "sum") == {"bf16": per32}
    # exact bf16 k-NN at D = 64: two 32-slot products per 16 x 16 block
    assert bench.matrix_flops_per_pair("knn_bf16_kernel", _W(64), "argkmin") == {"bf16": 2 * per32}
    # split sums at D = 128, E = 16: six partial products per coordinate, and
    # the P.B product as six 16x16x32 bf16 products per 32 columns x 16 rows
    # (2 * 16 * 16 * 32 * 6 / (32 * 16) = 192 flops per pair)
    mx = bench.matrix_flops_per_pair("mfma_split_kernel", _W(128, 16), "sum")
    assert mx == {"bf16": 6 * 4 * per32 + 192}
    # at D = 256 (16-column tiles) P.B stays on the fp32 16x16x4 product
    # (2 * 16 flops per pair per 16 signal columns)
    mx = bench.matrix_flops_per_pair("mfma_split_kernel", _W(256, 16), "sum")
    assert mx == {"bf16": 6 * 8 * per32, "f32": 32}
    # the one-launch sum: one 16x16x4 fp32 product per 16 x 16 pairs
    assert bench.matrix_flops_per_pair("small_kernel", _W(3), "sum") == {"f32": 8}
    # fp32 log-sum-exp at D = 64: the inner product only, no signal product
    assert bench.matrix_flops_per_pair("mfma_kernel", _W(64), "lse") == {"f32": 2 * 64}
    # the split log-sum-exp: six bf16 products per coordinate, no P . B
    assert bench.matrix_flops_per_pair("mfma_split_kernel", _W(64), "lse") == {"bf16": 12 * 64}
    # the fused gradient at D = 128 runs 129 signal columns in two launches of
    # 64 on the matrix cores (the 129th on the vector ALU)
    mx = bench.matrix_flops_per_pair("mfma_split_kernel", _W(128, 1), "sum", "gauss_gradx")
    assert mx == {"bf16": 2 * 6 * 4 * per32 + 192 * (4 + 4)}
    # D = 256 (257 columns, the 16x16x32 kernel): five launches
    mx = bench.matrix_flops_per_pair("mfma_split_kernel", _W(256, 1), "sum", "gauss_gradx")
    assert len(mx) == 2 and mx["f32"] == 32 * (4 + 4 + 4 + 4 + 1)
    assert bench.matrix_flops_per_pair("sum_kernel", _W(3), "sum") == {}


def test_traffic_is_reported_only_for_the_profiled_source(tmp_path):
    sha = bench.source_sha("fast_kernel")
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps({"c2": {"kernel": "fast_kernel", "source_sha": sha,
                                    "hbm_bytes_per_launch": 123.0}}))
    assert bench.traffic_for(str(p), "c2", "fast_kernel") == 123.0
    assert bench.traffic_for(str(p), "c2", "gradx_kernel") is None      # another kernel ran
    assert bench.traffic_for(str(p), "c3", "fast_kernel") is None       # not profiled
    p.write_text(json.dumps({"c2": {"kernel": "fast_kernel", "source_sha": "0" * 12,
                                    "hbm_bytes_per_launch": 123.0}}))
    assert bench.traffic_for(str(p), "c2", "fast_kernel") is None       # source changed since
    assert bench.traffic_for(str(tmp_path / "missing.json"), "c2", "fast_kernel") is None


@pytest.mark.gpu
def test_bench_line_fields_on_the_small_workload():
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "c1",
           "--steps", "3", "--warmup", "1", "--cpu-seconds", "2"]
    print("bench:", " ".join(cmd[2:]), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline", "cpu_baseline"):
        assert k in line, k
    assert line["n_gpus"] == 1 and line["steps"] == 3 and line["warmup"] == 1
    assert line["unit"] == "Gpairs/s" and line["higher_is_better"] is True
    assert line["value"] > 0 and line["ms_per_step"] > 0
    # value is the step's pairs over the step's wall time
    assert line["value"] == pytest.approx(1e8 / (line["ms_per_step"] / 1e3) / 1e9, rel=1e-9)
    assert isinstance(line["config"]["workload"], str)
    rf = line["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in rf, k
    assert rf["bound"] == "alu" and rf["unit"] == "TFLOP/s" and rf["peak"] == 157.3
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-9)
    assert 0 < rf["frac"] < 1.0
    # the kernel time never exceeds the step's wall time
    assert rf["kernel_ms_per_step"] <= line["ms_per_step"] * 1.05
    cb = line["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["unit"] == "Gpairs/s"
    assert cb["value"] > 0 and cb["cores"] >= 1 and isinstance(cb["sample"], str)
    assert cb["max_norm_err_on_sample"] < 1e-4
    assert "-march=native" in cb["build"]
    # per-step events: median and minimum, neither above the slowest step
    st = line["step_ms"]
    assert 0 < st["min"] <= st["median"] <= st["max"]
    # the device's measured sustained rates, and the roofline against them
    dev = line["device"]
    assert 10 < dev["fma_tflops"] < 400 and 100 < dev["exp_gops"] < 1e5
    assert 500 < dev["sclk_mhz"] < 4000 and dev["cus"] > 0
    assert rf["frac_measured"] == pytest.approx(rf["achieved"] / dev["fma_tflops"], rel=1e-9)
    assert 0 < rf["frac_exp_bound"] < 1.0
