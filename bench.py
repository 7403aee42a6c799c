"""kred benchmark on one MI355X.

Default workload: the Gaussian kernel sum of Eq. (1), value only, at
M = N = 1e6, D = 3, E = 1 (the paper's Sec. 3 benchmark problem), on seeded
synthetic points (a mixture of 8 isotropic Gaussians, std 0.05, centres in
[0,1]^3; b ~ N(0,1); sigma = 0.05) already resident in HBM when timing starts.
A step is one kred_run over the whole hot path: the prologue (bounding box,
packing of y and b), the pair loop with its reduction, and the column-block
second pass when there is one.  The same run also times the fused sum +
x-gradient on the same inputs (`extra.c2`), each with its own roofline and
CPU baseline.  `--workload` selects another workload as the main line.

Prints one JSON line.  `value` is pair evaluations per second (Gpairs/s) of
the whole step (each reduction of a step counts its M x N pairs);
`ms_per_step` is wall clock over the timed steps, `step_ms` the median and
minimum of per-step HIP events on the launch stream.  `roofline` prices the
main kernels' algorithmic flops against the FP32 vector peak, or against the
matrix-core peak of the operand type the main kernel multiplies in (fp32 or
bf16), timed with HIP events the library records around each main kernel on
the launch stream; for matrix-core kernels it adds the matrix work they
execute (split operands and padding included) at the published peaks against
the same time, and for vector kernels the measured sustained FMA and exp
rates of the device (`device`, from a microbenchmark run after the timed
steps).  `cpu_baseline` times the fp64 oracle, built for the host's CPU, on
the host's cores over a bounded sample of rows.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_VECTOR_TFLOPS = 157.3     # MI355X published FP32 vector peak
PEAK_FP32_MATRIX_TFLOPS = 157.3     # MI355X published FP32 matrix (MFMA) peak
PEAK_BF16_MATRIX_TFLOPS = 2500.0    # MI355X published dense bf16 matrix peak

# name: (generator kwargs, formula, reduction, flops per pair, bound, description)
WORKLOADS = {
    "c2": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05), "gauss_gradx", "sum",
           17, "alu", "gaussian kernel sum + x-gradient (fused), mixture of 8 Gaussians, 1e6 x 1e6, D=3"),
    "headline": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05), "gauss", "sum",
                 11, "alu", "gaussian kernel sum (value only), mixture of 8 Gaussians, 1e6 x 1e6, D=3"),
    "c1": ("uniform_gauss", dict(M=10_000, N=10_000, D=3, E=1, sigma=0.1), "gauss", "sum",
           11, "alu", "gaussian kernel sum, uniform [0,1]^3, 1e4 x 1e4, D=3"),
    "c3": ("sinkhorn_lse", dict(M=1_000_000, N=1_000_000, D=3, eps=0.01), "sinkhorn", "lse",
           14, "alu", "sinkhorn log-sum-exp, uniform / shifted uniform, 1e6 x 1e6, D=3"),
    "c4": ("highdim_gauss", dict(M=200_000, N=200_000, D=128, E=16, sigma=1.0), "gauss", "sum",
           291, "mfma", "gaussian kernel sum, N(0, I/128), 2e5 x 2e5, D=128, E=16"),
    # the fused value + x-gradient at D = 128: one Gaussian sum with D + 1 = 129
    # signal columns [b, b (y - m)] on the matrix cores (two launches of 64
    # columns, the first also summing the 129th on the vector ALU); 2D + 3
    # flops for the exponent and 2 (D + 1) for the sums
    "gradx_d128": ("highdim_gauss", dict(M=200_000, N=200_000, D=128, E=1, sigma=1.0),
                   "gauss_gradx", "sum", 2 * 128 + 3 + 2 * 129, "mfma",
                   "gaussian kernel sum + x-gradient (fused), N(0, I/128), 2e5 x 2e5, D=128"),
    # Sinkhorn log-sum-exp at D = 64 on the fp32 matrix cores (2D flops for the
    # inner product, 3 for the norms and g, 3 for the running log-sum-exp)
    "lse_d64": ("sinkhorn_lse", dict(M=200_000, N=200_000, D=64, eps=1.0), "sinkhorn", "lse",
                2 * 64 + 6, "mfma", "sinkhorn log-sum-exp, uniform / shifted uniform, 2e5 x 2e5, "
                                    "D=64, eps=1"),
    # the integer coordinates pass the library's exactness guard, so the contraction
    # runs on the bf16 matrix cores
    "c5": ("integer_knn", dict(M=100_000, N=1_000_000, D=64, K=10), "sqdist", "argkmin",
           131, "mfma", "arg-K-min K=10, integer mixture, 1e5 queries x 1e6 points, D=64"),
    # Gaussian backward: the x, y and b gradients of L = sum_i <e_i, a_i>, three
    # reductions over the M x N pairs per step (flops per pair summed over them)
    "backward": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05), "backward",
                 None, 17 + 17 + 11, "alu",
                 "gaussian backward (x, y, b gradients), scalar cotangent, mixture of 8 "
                 "Gaussians, 1e6 x 1e6, D=3"),
    "backward_e16": ("uniform_gauss", dict(M=200_000, N=200_000, D=3, E=16, sigma=0.1), "backward",
                     None, 48 + 48 + 42, "alu",
                     "gaussian backward (x, y, b gradients), E=16 cotangent, uniform [0,1]^3, "
                     "2e5 x 2e5, D=3"),
    # one direction of a Chamfer distance: each query's nearest squared distance
    # (3D - 1 flops for the distance and 1 compare per pair).  The distance runs
    # on the bf16 matrix cores (3-way split) with about half a VALU op per pair
    # left, so the matrix cores bound it.
    "chamfer": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05), "sqdist", "min",
                9, "mfma", "nearest-neighbour squared distance (min reduction, no b), mixture "
                           "of 8 Gaussians, 1e6 x 1e6, D=3"),
    # point-cloud k-NN: the 10 nearest of every query by squared distance, D = 3;
    # the distance runs on the bf16 matrix cores, the lists on the VALU
    "knn3": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05), "sqdist", "argkmin",
             9, "mfma", "arg-K-min K=10 (point-cloud k-NN), mixture of 8 Gaussians, 1e6 x 1e6, D=3"),
    # block-sparse Gaussian sum: grid clusters of side 2 sigma, cluster pairs kept
    # within 6 sigma (+ the cell diagonal); pairs and flops count the kept pairs
    "sparse": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05), "gauss", "sum",
               11, "alu", "block-sparse gaussian kernel sum (grid clusters of side 2 sigma, "
                          "truncation at 6 sigma), mixture of 8 Gaussians, 1e6 x 1e6, D=3"),
    # its backward: the x, y and b gradients of L = sum_i <e_i, a_i> over the kept
    # pairs (x from the row clusters, y and b from the same blocks seen from the
    # column clusters)
    "sparse_backward": ("mixture_gauss", dict(M=1_000_000, N=1_000_000, D=3, sigma=0.05),
                        "backward", None, 17 + 17 + 11, "alu",
                        "block-sparse gaussian backward (x, y, b gradients, scalar cotangent; "
                        "grid clusters of side 2 sigma, truncation at 6 sigma), mixture of 8 "
                        "Gaussians, 1e6 x 1e6, D=3"),
}
SPARSE_CELL, SPARSE_CUTOFF = 2.0, 6.0   # in units of sigma
SPARSE = ("sparse", "sparse_backward")
# the three reductions of a backward step: (rows, columns) = (M, N), (N, M), (N, M)
REDUCTIONS_PER_STEP = {"backward": 3, "backward_e16": 3, "sparse_backward": 3}
LIST_K = {"knn3": 10}   # K of the arg-K-min workloads drawn by a generator without one
KERNEL_SOURCES = {"sum_kernel": "k_direct.hip", "gradx_kernel": "k_direct.hip",
                  "lse_kernel": "k_direct.hip", "knn_kernel": "k_direct.hip",
                  "vjp_kernel": "k_direct.hip", "mfma_kernel": "k_mfma.hip",
                  "mfma_split_kernel": "k_mfma.hip", "knn_bf16_kernel": "k_knn.hip",
                  "fast_kernel": "k_small_mfma.hip", "small_kernel": "k_small.hip"}


def matrix_flops_per_pair(kernel, w, reduction, formula=None):
    """Matrix-core flops a kernel executes per pair (over a step's launches), by operand type.

    The bf16 kernels execute more matrix work than the algorithm needs (split
    operands, padded K slots); this is what their time is measured against in
    `matrix_executed`, beside the algorithmic roofline.
    """
    dp = next((p for p in (32, 64, 128, 256) if w.D <= p), 256)
    sums = reduction == "sum"
    # signal widths of the launches: the fused gradient at D > 16 runs sums of
    # [b, b (y - m)] in chunks of up to 64 columns
    widths = [w.E]
    if formula == "gauss_gradx" and w.D > 16:
        widths = [min(64, w.D + 1 - c) for c in range(0, w.D + 1, 64)]
    ebs = [1 if e <= 16 else (2 if e <= 32 else 4) for e in widths]
    if kernel == "mfma_split_kernel":     # 6 split products per coordinate
        if reduction == "lse":            # the log-sum-exp has no P . B
            return {"bf16": 12 * dp}
        if dp <= 128:                     # P . B: 6 bf16 16x16x32 products per 32 x 16 pairs
            if len(widths) > 1 and widths[-1] == 1:
                # a last single column is summed on the vector ALU by the first
                # launch (its own launch returns at once)
                ebs = ebs[:-1]
            return {"bf16": 12 * dp * len(ebs) + sum(192 * eb for eb in ebs)}
        return {"bf16": 12 * dp * len(ebs), "f32": sum(32 * eb for eb in ebs)}
    if kernel == "mfma_kernel":
        return {"f32": sum(2 * dp + (32 * eb if sums else 0) for eb in ebs)}
    if kernel == "knn_bf16_kernel":       # one exact bf16 product per coordinate
        return {"bf16": 2 * dp}
    if kernel == "fast_kernel":           # one 16x16x32 product per 16x16 pairs (32 K slots)
        return {"bf16": 64}
    if kernel == "small_kernel":          # one fp32 16x16x4 product per 16x16 pairs
        return {"f32": 8}
    return {}


def call_latency(ctx, w, formula, reduction, reps=200):
    """Per-call latency: HIP events around each call, the stream drained before
    the next one (so each call starts on an idle GPU and the span includes its
    host-side enqueue); median and minimum over `reps` calls, in microseconds."""
    import torch
    x, y = torch.from_numpy(w.x).cuda(), torch.from_numpy(w.y).cuda()
    b = torch.from_numpy(w.b).cuda()
    out = torch.empty((w.M, w.E), device="cuda")
    stream = torch.cuda.current_stream()
    kw = dict(sigma=w.sigma, eps=w.eps, K=w.K)
    for _ in range(10):
        ctx.run(formula, reduction, x, y, b, out=out, stream=stream, **kw)
    torch.cuda.synchronize()
    each = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        ctx.run(formula, reduction, x, y, b, out=out, stream=stream, **kw)
        e1.record(stream)
        e1.synchronize()
        each.append(e0.elapsed_time(e1) * 1e3)
    each.sort()
    return {"us_median": each[reps // 2], "us_min": each[0], "reps": reps,
            "mode": "HIP events around each call, stream drained between calls"}


# workloads the default run times beside the main line (same inputs, more work per pair)
EXTRA = {"headline": ["c2"]}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="headline", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of each oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="time the main workload only (not the workloads in EXTRA)")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the sustained-rate microbenchmark of the device")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run one 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="HBM bytes per launch measured with rocprofv3 --pmc")
    return ap.parse_args()


def source_sha(kernel):
    path = os.path.join(ROOT, "paper_2004_11127_amd", "csrc", KERNEL_SOURCES.get(kernel, ""))
    try:
        with open(path, "rb") as f:
            return hashlib.sha1(f.read()).hexdigest()[:12]
    except OSError:
        return None


def traffic_for(path, workload, kernel):
    """Bytes per launch from the committed counter summary, if it matches the current source."""
    try:
        with open(path) as f:
            tj = json.load(f)
    except (OSError, ValueError):
        return None
    ent = tj.get(workload)
    if not ent or ent.get("kernel") != kernel or ent.get("source_sha") != source_sha(kernel):
        return None
    return ent.get("hbm_bytes_per_launch")


def cotangent(w):
    """Seeded N(0, 1) cotangent e (M x E) of the Gaussian sum, for the backward workloads."""
    import numpy as np
    return np.random.default_rng(1).standard_normal((w.M, w.E)).astype(np.float32)


def sparse_pattern(ctx, w, name):
    """Sorted copy of the workload and its block-sparse pattern (setup, not in the steps).

    The forward workload builds the pattern on the GPU (kred_cluster_pattern:
    grid labels, stable sort, ranges and truncation) and permutes x, y and b
    there (kred_gather_rows); only the pattern's four counts come back to the
    host, to size the call, and `prologue_ms` times the build and the gathers
    (HIP events).  The host copies below serve the CPU baseline only.  The
    backward workload also needs the column-side view (transpose_pattern) and
    builds its pattern on the host."""
    import numpy as np
    cell, cut = SPARSE_CELL * w.sigma, SPARSE_CUTOFF * w.sigma
    if name == "sparse":
        import torch
        x, y, b = (torch.from_numpy(a).cuda() for a in (w.x, w.y, w.b))
        t = ctx.cluster_pattern(x, y, cell, cut)          # sizing pass, then the pattern
        cap = int(t["col_ranges"].shape[0])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        t = ctx.cluster_pattern(x, y, cell, cut, col_cap=cap)
        xs, ys, bs = (ctx.gather_rows(v, t[o]) for v, o in ((x, "order_x"), (y, "order_y"),
                                                           (b, "order_y")))
        e1.record()
        torch.cuda.synchronize()
        counts = t["counts"].cpu().numpy()
        nr, nnz = int(counts[0]), int(counts[1])
        dev = dict(x=xs, y=ys, b=bs, row_ranges=t["row_ranges"][:nr], col_ptr=t["col_ptr"][:nr + 1],
                   col_ranges=t["col_ranges"][:nnz])
        w.x, w.y, w.b = (v.cpu().numpy() for v in (xs, ys, bs))
        return dict(device=dev, pairs=int(counts[2]), prologue_ms=e0.elapsed_time(e1),
                    row_ranges=dev["row_ranges"].cpu().numpy(), col_ptr=dev["col_ptr"].cpu().numpy(),
                    col_ranges=dev["col_ranges"].cpu().numpy())
    from paper_2004_11127_amd import clusters
    pat = clusters.truncation_pattern(w.x, w.y, cell, cut)
    w.x = w.x[pat["order_x"]].copy(); w.y = w.y[pat["order_y"]].copy()
    w.b = w.b[pat["order_y"]].copy()
    pat["transposed"] = clusters.transpose_pattern(pat["row_ranges"], pat["col_ptr"],
                                                   pat["col_ranges"], w.M, w.N)
    return pat


def time_steps(ctx, w, formula, reduction, steps, warmup, pattern=None):
    """Time `steps` calls; kernel_ms is the main kernels' time per step (HIP events)."""
    import torch
    from paper_2004_11127_amd import kred
    x, y = torch.from_numpy(w.x).cuda(), torch.from_numpy(w.y).cuda()
    b = torch.from_numpy(w.b).cuda() if w.b is not None else None
    if formula == "sqdist" and reduction in ("min", "argkmin"):
        b = None   # reductions of the bare squared distance
    stream = torch.cuda.current_stream()
    if pattern is not None and formula == "backward":
        e = torch.from_numpy(cotangent(w)).cuda()
        fwd = tuple(torch.from_numpy(pattern[k]).cuda() for k in ("row_ranges", "col_ptr",
                                                                  "col_ranges"))
        tr = tuple(torch.from_numpy(a).cuda() for a in pattern["transposed"])

        def call(flags):
            return ctx.gauss_backward_ranges(x, y, b, e, fwd, tr, sigma=w.sigma, flags=flags,
                                             stream=stream)
    elif pattern is not None:
        if "device" in pattern:      # built and permuted on the GPU
            d = pattern["device"]
            x, y, b = d["x"], d["y"], d["b"]
            rr, cp, cr = d["row_ranges"], d["col_ptr"], d["col_ranges"]
        else:
            rr, cp, cr = (torch.from_numpy(pattern[k]).cuda() for k in ("row_ranges", "col_ptr",
                                                                         "col_ranges"))
        kw = dict(sigma=w.sigma, eps=w.eps, K=w.K)

        def call(flags):
            return ctx.run_ranges(formula, reduction, x, y, b, rr, cp, cr, flags=flags,
                                  stream=stream, **kw)
    elif formula == "backward":
        e = torch.from_numpy(cotangent(w)).cuda()

        def call(flags):
            return ctx.gauss_backward(x, y, b, e, sigma=w.sigma, flags=flags, stream=stream)
    else:
        kw = dict(sigma=w.sigma, eps=w.eps, K=w.K)

        def call(flags):
            return ctx.run(formula, reduction, x, y, b, flags=flags, stream=stream, **kw)
    for _ in range(warmup):
        call(0)
    torch.cuda.synchronize()
    ctx.profile_collect()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record(stream)
        out = call(kred.FLAG_PROFILE)
        e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    n, kern_ms, kname = ctx.profile_collect()
    if formula == "backward":
        out = out[0]   # the x-gradient, for the CPU baseline's check
    each = sorted(e0.elapsed_time(e1) for e0, e1 in ev)
    return dict(wall_s=wall, event_ms=ev[0][0].elapsed_time(ev[-1][1]), kernel_ms=kern_ms / steps,
                step_ms=dict(median=each[len(each) // 2] if len(each) % 2 else
                             0.5 * (each[len(each) // 2 - 1] + each[len(each) // 2]),
                             min=each[0], max=each[-1]),
                launches=n, kernel=kname, out=out.cpu().numpy())


NATIVE_BUILD = {}


def cpu_baseline(w, formula, reduction, out_gpu, seconds, pattern=None):
    """Time the fp64 oracle on a bounded sample of rows (all N columns, or the
    pattern's columns of the sampled rows' clusters)."""
    import numpy as np

    import oracle
    from paper_2004_11127_amd import inputs

    if "cmd" not in NATIVE_BUILD:
        NATIVE_BUILD["cmd"] = oracle.use_native()   # gcc -O3 -march=native, built on this host

    def clustered(rows, rr, cp, cr, ncols, reduce, width):
        # the sampled rows' clusters, each reduced over its pattern columns;
        # rows in no cluster hold zero
        cl = np.searchsorted(rr[:, 1], rows, side="right")
        inside = cl < len(rr)
        inside[inside] &= rows[inside] >= rr[cl[inside], 0]
        val = np.zeros((len(rows), width)); nrm = np.zeros_like(val)
        for I in np.unique(cl[inside]):
            sel = inside & (cl == I)
            cols = oracle._cluster_columns(cp, cr, I, ncols)
            if cols.size:
                v, n = reduce(rows[sel], cols)
                val[sel] = v; nrm[sel] = n
        return val, nrm

    def run(rows):
        if pattern is not None and formula == "backward":
            # gx of the sampled rows over their clusters' columns; gy and gb of
            # the same indices as columns, over their column clusters' rows
            e = cotangent(w)
            gx = clustered(rows, pattern["row_ranges"], pattern["col_ptr"], pattern["col_ranges"],
                           w.N, lambda r, c: oracle.gauss_vjp(w.x[r], w.y[c], w.b[c], e[r],
                                                              w.sigma), w.D)
            cc, rp, rt = pattern["transposed"]
            clustered(rows, cc, rp, rt, w.M,
                      lambda r, c: oracle.gauss_vjp(w.y[r], w.x[c], e[c], w.b[r], w.sigma), w.D)
            clustered(rows, cc, rp, rt, w.M,
                      lambda r, c: oracle.kernel_sum("gauss", w.y[r], w.x[c], e[c], sigma=w.sigma),
                      w.E)
            return gx
        if pattern is not None:
            return clustered(rows, pattern["row_ranges"], pattern["col_ptr"],
                             pattern["col_ranges"], w.N,
                             lambda r, c: oracle.kernel_sum("gauss", w.x[r], w.y[c], w.b[c],
                                                            sigma=w.sigma), w.E)
        if formula == "backward":
            # the three reductions of a step on the same sampled row indices
            e = cotangent(w)
            gx, nx = oracle.gauss_vjp(w.x, w.y, w.b, e, w.sigma, rows=rows)
            oracle.gauss_vjp(w.y, w.x, e, w.b, w.sigma, rows=rows)
            oracle.kernel_sum("gauss", w.y, w.x, e, sigma=w.sigma, rows=rows)
            return gx, nx
        if formula == "gauss_gradx":
            return oracle.gauss_gradx(w.x, w.y, w.b, w.sigma, rows=rows)
        if reduction == "lse":
            return oracle.sinkhorn_lse(w.x, w.y, w.b, w.eps, rows=rows)
        if reduction == "argkmin":
            return oracle.argkmin(w.x, w.y, w.K, rows=rows)
        if reduction == "min":
            val, _, scale = oracle.extreme("sqdist", "min", w.x, w.y, rows=rows)
            return val, scale
        return oracle.kernel_sum(formula, w.x, w.y, w.b, sigma=w.sigma, rows=rows)

    # a probe large enough that thread start-up does not dominate its time
    probe = inputs.sample_rows(w.M, min(w.M, 256), seed=777)
    t0 = time.perf_counter()
    run(probe)
    t_probe = time.perf_counter() - t0
    S = int(min(w.M, 65536, max(64, len(probe) * seconds / max(t_probe, 1e-3))))
    rows = inputs.sample_rows(w.M, S, seed=12345)
    t0 = time.perf_counter()
    ref, aux = run(rows)
    t = time.perf_counter() - t0
    got = out_gpu[rows]
    if reduction == "argkmin":
        # indices may differ where fp32 and fp64 order near-equal distances
        # differently; the distances of the returned points must still be the
        # K smallest (relative to each row's K-th distance)
        dist = ((w.x[rows, None, :].astype(np.float64) - w.y[got].astype(np.float64)) ** 2).sum(-1)
        kth = np.maximum(aux[:, -1:], 1e-30)
        check = {"index_mismatches_on_sample": int((got != ref).sum()),
                 "max_rel_dist_err_on_sample": float(np.max(np.abs(dist - aux) / kth))}
    elif reduction == "min":
        check = {"max_rel_err_on_sample": float(np.max(np.abs(got - ref) / np.maximum(aux, 1e-30)))}
    elif reduction == "lse":
        check = {"max_abs_err_on_sample": float(np.max(np.abs(got[:, 0] - ref)))}
    else:
        check = {"max_norm_err_on_sample": float(np.max(np.abs(got - ref) / np.maximum(aux, 1e-30)))}
    red = 3 if formula == "backward" else 1
    cols = w.N if pattern is None else pattern["pairs"] / w.M   # columns per row (mean)
    res = dict(value=red * S * cols / t / 1e9, unit="Gpairs/s", cores=oracle.num_threads(),
               kind="oracle", build=NATIVE_BUILD.get("cmd"),
               sample="%d seeded rows x %s%s (%.1f s)"
                      % (S, "all %d columns" % w.N if pattern is None else "their pattern columns",
                         " for each of the 3 gradients" if red > 1 else "", t),
               seconds=t)
    res.update(check)
    if pattern is not None and formula != "backward":
        # what the truncation drops: the block-sparse result against the dense sum
        few = rows[:: max(1, len(rows) // 64)]
        dense, dn = oracle.kernel_sum("gauss", w.x[few], w.y, w.b, sigma=w.sigma)
        res["truncation_err_vs_dense"] = float(np.max(np.abs(out_gpu[few] - dense) /
                                                      np.maximum(dn, 1e-30)))
    return res


def probe_device():
    """Sustained fp32 FMA and v_exp_f32 rates and the shader clock (libkred_probe.so)."""
    import ctypes

    class Peak(ctypes.Structure):
        _fields_ = [("fma_tflops", ctypes.c_double), ("exp_gops", ctypes.c_double),
                    ("sclk_mhz", ctypes.c_double), ("fma_ms", ctypes.c_double),
                    ("exp_ms", ctypes.c_double), ("cus", ctypes.c_int)]

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2004_11127_amd", "libkred_probe.so"))
    lib.kred_probe_peak.argtypes = [ctypes.c_int, ctypes.POINTER(Peak)]
    lib.kred_probe_peak.restype = ctypes.c_int
    pk = Peak()
    rc = lib.kred_probe_peak(0, ctypes.byref(pk))
    if rc != 0:
        return {"error": "kred_probe_peak returned %d" % rc}
    return {"fma_tflops": pk.fma_tflops, "exp_gops": pk.exp_gops, "sclk_mhz": pk.sclk_mhz,
            "cus": pk.cus, "probe": "libkred_probe.so kred_probe_peak (peak_probe.hip)"}


def measure(ctx, name, args):
    """Time one workload; the fields of its JSON object (without the device figures)."""
    from paper_2004_11127_amd import inputs

    gen, gkw, formula, reduction, fpp, bound, desc = WORKLOADS[name]
    w = getattr(inputs, gen)(seed=0, **gkw)
    if name in LIST_K:
        w.K = LIST_K[name]
    pattern = sparse_pattern(ctx, w, name) if name in SPARSE else None
    pairs = (float(pattern["pairs"]) if pattern is not None else float(w.M) * float(w.N)) \
        * REDUCTIONS_PER_STEP.get(name, 1)
    r = time_steps(ctx, w, formula, reduction, args.steps, args.warmup, pattern)
    ms_per_step = r["wall_s"] * 1e3 / args.steps
    # fpp counts the flops of one (i, j) over all reductions of a step
    step_pairs = pairs / REDUCTIONS_PER_STEP.get(name, 1)   # pairs of one reduction
    achieved = fpp * step_pairs / (r["kernel_ms"] / 1e3) / 1e12
    mx = matrix_flops_per_pair(r["kernel"], w, reduction, formula)
    mdtype = ("bf16" if "bf16" in mx else "f32") if bound == "mfma" else None
    peak = {None: PEAK_FP32_VECTOR_TFLOPS, "f32": PEAK_FP32_MATRIX_TFLOPS,
            "bf16": PEAK_BF16_MATRIX_TFLOPS}[mdtype]
    # the executed matrix work at the published peaks, against the kernel time
    ms_at_peak = pairs * (mx.get("bf16", 0) / (PEAK_BF16_MATRIX_TFLOPS * 1e12) +
                          mx.get("f32", 0) / (PEAK_FP32_MATRIX_TFLOPS * 1e12)) * 1e3
    sub = {
        "value": pairs / (ms_per_step / 1e3) / 1e9,
        "unit": "Gpairs/s",
        "ms_per_step": ms_per_step,
        "step_ms": r["step_ms"],
        "config": {"workload": desc, "M": w.M, "N": w.N, "D": w.D, "E": w.E, "K": w.K,
                   "sigma": w.sigma, "eps": w.eps, "flops_per_pair": fpp},
        "roofline": {"bound": bound, "matrix_dtype": mdtype,
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak,
                     "traffic": traffic_for(args.traffic, name, r["kernel"]),
                     "kernel": r["kernel"], "kernel_ms_per_step": r["kernel_ms"],
                     "launches_timed": r["launches"],
                     "launches_per_step": r["launches"] / args.steps},
        "event_ms_per_step": r["event_ms"] / args.steps,
    }
    if mx:
        sub["roofline"]["matrix_executed"] = {
            "flops_per_pair": mx, "ms_at_peak_per_step": ms_at_peak,
            "frac": ms_at_peak / r["kernel_ms"]}
    if name in ("c1", "headline"):
        sub["paper_context"] = ("KeOps++ on an RTX 2080 Ti (Sec. 3 table): 0.4 ms at 1e4 and "
                                "1.38 s at 1e6 points, D=3, fp32")
    if name == "c1":
        sub["latency"] = call_latency(ctx, w, formula, reduction)
    if pattern is not None:
        sub["config"]["pattern_pairs_fraction"] = pattern["pairs"] / (float(w.M) * w.N)
        sub["config"]["clusters"] = int(len(pattern["row_ranges"]))
        if "prologue_ms" in pattern:
            sub["config"]["pattern"] = "built on the GPU (kred_cluster_pattern)"
            sub["prologue_ms"] = pattern["prologue_ms"]
    if not args.no_cpu_baseline:
        sub["cpu_baseline"] = cpu_baseline(w, formula, reduction, r["out"], args.cpu_seconds,
                                           pattern)
    # exp-bearing vector kernels: one v_exp_f32 per pair bounds the pair rate too
    sub["_exp_per_pair"] = 1 if (bound == "alu" and formula in ("gauss", "gauss_gradx", "sinkhorn",
                                                                   "backward", "laplace")) else 0
    sub["_pairs_per_s_kernel"] = step_pairs / (r["kernel_ms"] / 1e3)
    return sub


def with_device(sub, dev):
    """Add the measured sustained rates to a workload's roofline."""
    rl = sub["roofline"]
    if "fma_tflops" in dev and rl["bound"] == "alu":
        rl["peak_measured"] = dev["fma_tflops"]
        rl["frac_measured"] = rl["achieved"] / dev["fma_tflops"]
    if "exp_gops" in dev and sub["_exp_per_pair"]:
        exp_bound = dev["exp_gops"] * 1e9 / sub["_exp_per_pair"]   # pairs/s if exp alone bound
        rl["exp_bound_gpairs"] = exp_bound / 1e9
        rl["frac_exp_bound"] = sub["_pairs_per_s_kernel"] / exp_bound
    del sub["_exp_per_pair"], sub["_pairs_per_s_kernel"]
    return sub


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2004_11127_amd import kred

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    extras = [] if args.no_extra else EXTRA.get(args.workload, [])
    with kred.Context(0) as ctx:
        main_sub = measure(ctx, args.workload, args)
        extra = {name: measure(ctx, name, args) for name in extras}
    if args.copy_probe:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
    dev = {} if args.no_probe else probe_device()
    main_sub = with_device(main_sub, dev)
    extra = {k: with_device(v, dev) for k, v in extra.items()}
    line = {
        "metric": "kernel pair-evaluations/sec (Gpairs/s) at M=N=1e6 D=3; % of FP32 VALU peak",
        "value": main_sub["value"],
        "unit": "Gpairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_sub["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
    }
    for k, v in main_sub.items():
        if k not in ("value", "unit", "ms_per_step"):
            line[k] = v
    if extra:
        line["extra"] = extra
    if dev:
        line["device"] = dev
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
