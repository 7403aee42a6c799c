"""kred benchmark: Gaussian kernel sum of Eq. (1) with its x-gradient, fused,
at M = N = 1e6, D = 3, E = 1 (one MI355X).

A step is one kred_run over the whole hot path: the packing prologue of y and
b (prescale), the direct-form pair loop with its fused sum and gradient
reduction, and the column-block second pass.  Inputs are seeded synthetic
points (a mixture of 8 isotropic Gaussians, std 0.05, centres in [0,1]^3;
b ~ N(0,1); sigma = 0.05) already resident in HBM when timing starts.

Prints one JSON line.  `value` is pair evaluations per second (Gpairs/s) of
the whole step; `roofline` prices the main kernel's algorithmic flops
(17 per pair) against the FP32 vector peak, timed with HIP events the
library records around that kernel on the launch stream; `cpu_baseline`
times the fp64 oracle on the host over a bounded sample of rows.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FLOPS_PER_PAIR = {"gauss_gradx": 17, "gauss": 11}
PEAK_FP32_VECTOR_TFLOPS = 157.3     # MI355X published FP32 vector peak
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--M", type=int, default=1_000_000)
    ap.add_argument("--N", type=int, default=1_000_000)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-value-only", action="store_true",
                    help="skip the value-only Gaussian sum timed alongside")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="HBM bytes per launch measured with rocprofv3 --pmc (JSON)")
    return ap.parse_args()


def time_steps(ctx, formula, x, y, b, sigma, steps, warmup):
    import torch
    from paper_2004_11127_amd import kred
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        ctx.run(formula, "sum", x, y, b, sigma=sigma, stream=stream)
    torch.cuda.synchronize()
    ctx.profile_collect()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(steps):
        out = ctx.run(formula, "sum", x, y, b, sigma=sigma, flags=kred.FLAG_PROFILE, stream=stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    n, kern_ms, kname = ctx.profile_collect()
    return dict(wall_s=wall, event_ms=ev0.elapsed_time(ev1), kernel_ms=kern_ms / max(n, 1),
                launches=n, kernel=kname, out=out)


def cpu_baseline(w, out_gpu, seconds):
    """Time the fp64 oracle on a bounded sample of rows (all N columns)."""
    import numpy as np

    import oracle
    from paper_2004_11127_amd import inputs

    oracle.build()
    probe = inputs.sample_rows(w.M, 32, seed=777)
    t0 = time.perf_counter()
    oracle.gauss_gradx(w.x, w.y, w.b, w.sigma, rows=probe)
    t_probe = time.perf_counter() - t0
    S = int(min(4096, max(64, 32 * seconds / max(t_probe, 1e-3))))
    rows = inputs.sample_rows(w.M, S, seed=12345)
    t0 = time.perf_counter()
    ref, norm = oracle.gauss_gradx(w.x, w.y, w.b, w.sigma, rows=rows)
    t = time.perf_counter() - t0
    got = out_gpu[rows].astype(np.float64)
    err = float(np.max(np.abs(got - ref) / np.maximum(norm, 1e-30)))
    return dict(value=S * w.N / t / 1e9, unit="Gpairs/s", cores=oracle.num_threads(),
                kind="oracle", sample="%d seeded rows x all %d columns (%.1f s)" % (S, w.N, t),
                seconds=t, max_norm_err_on_sample=err)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2004_11127_amd import inputs, kred

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = inputs.mixture_gauss(M=args.M, N=args.N, D=3, sigma=0.05, seed=0)
    x, y, b = (torch.from_numpy(a).cuda() for a in (w.x, w.y, w.b))
    pairs = float(w.M) * float(w.N)
    with kred.Context(0) as ctx:
        r = time_steps(ctx, "gauss_gradx", x, y, b, w.sigma, args.steps, args.warmup)
        out_gpu = r["out"].cpu().numpy()
        extra = {}
        if not args.no_value_only:
            v = time_steps(ctx, "gauss", x, y, b, w.sigma, args.steps, args.warmup)
            v_ms = v["event_ms"] / args.steps
            extra["gauss_sum_value_only"] = dict(
                gpairs_per_s=pairs / (v_ms / 1e3) / 1e9, ms_per_step=v_ms,
                kernel_ms=v["kernel_ms"],
                tflops=FLOPS_PER_PAIR["gauss"] * pairs / (v["kernel_ms"] / 1e3) / 1e12,
                frac_fp32_vector_peak=FLOPS_PER_PAIR["gauss"] * pairs / (v["kernel_ms"] / 1e3)
                / 1e12 / PEAK_FP32_VECTOR_TFLOPS,
                paper_context="KeOps++ 1.38 s at M=N=1e6, D=3 on an RTX 2080 Ti (Sec. 3 table)")
    ms_per_step = r["wall_s"] * 1e3 / args.steps
    achieved = FLOPS_PER_PAIR["gauss_gradx"] * pairs / (r["kernel_ms"] / 1e3) / 1e12
    traffic = None
    try:
        with open(args.traffic) as f:
            tj = json.load(f)
        traffic = tj.get("gradx_kernel", {}).get("bytes_per_launch")
    except (OSError, ValueError):
        pass
    line = {
        "metric": "kernel pair-evaluations/sec (Gpairs/s) at M=N=1e6 D=3; % of FP32 VALU peak",
        "value": pairs / (ms_per_step / 1e3) / 1e9,
        "unit": "Gpairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "gaussian kernel sum + x-gradient (fused), mixture of 8 Gaussians",
                   "M": w.M, "N": w.N, "D": 3, "E": 1, "sigma": w.sigma,
                   "flops_per_pair": FLOPS_PER_PAIR["gauss_gradx"]},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": PEAK_FP32_VECTOR_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_VECTOR_TFLOPS,
                     "traffic": traffic, "kernel": r["kernel"],
                     "kernel_ms": r["kernel_ms"], "launches_timed": r["launches"]},
        "event_ms_per_step": r["event_ms"] / args.steps,
    }
    line.update(extra)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, out_gpu, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
