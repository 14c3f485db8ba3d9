#!/usr/bin/env python3
"""Benchmark of the IVF routing and construction hot path on one MI355X.

Every workload is measured at its stated size, with its inputs resident in
HBM before timing, and next to the CPU oracle on this host:

  1. routing, tiny: 1,024 centroids, D = 128, 1,000 integer-valued queries,
     nprobe 16 (oracle in full);
  2. routing, uint8-valued: 65,536 centroids, D = 128, 10,000 queries,
     nprobe 64;
  3. routing, normalised floats: 262,144 unit-norm centroids, D = 96, 10,000
     queries, nprobe 128;
  4. k-means: 10 Lloyd iterations on 10M uint8 rows (65,536-component
     mixture, std 20), 65,536 centroids from a seeded row sample;
  5. assign-build: 1e9 uint8 rows of the same generator (128 GB resident,
     produced on the device in 64M-row chunks) assigned to the 65,536
     mixture means by top-1 L2, then the inverted-list build.

The timed step (`--steps`, after `--warmup` untimed ones) is workload 5, the
largest: one ivf_assign_build call over all 1e9 rows. `value` = rows / step
time. `roofline` is that step's dominant kernel (the single-plane int8
screen); `cpu_baseline` is the oracle on a bounded sample of the same
assignment. The other workloads are in `configs`, each with its own rate,
roofline fraction and oracle timing. NEXT-row kernels (list-major layout,
residual PQ, ADC scan, candidate-restricted assignment) run on the k-means
output and are reported under `extra`.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3  # MI355X dense fp32 matrix peak
PEAK_INT8_MFMA_TOPS = 5000.0   # MI355X dense int8 matrix peak
PEAK_HBM_GBS = 8000.0
PEAK_FP64_VECTOR_TFLOPS = 78.6

C_BIG, D_U8 = 65536, 128


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3, help="timed assign-build calls over the 1e9 rows")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--rows", type=int, default=10**9, help="rows of the assign-build workload")
    ap.add_argument("--kmeans-rows", type=int, default=10_000_000)
    ap.add_argument("--kmeans-iters", type=int, default=10)
    ap.add_argument("--only", default="", help="comma-separated subset of 1,2,3,4,5 and b (the list build "
                                               "alone on 1e9 labels; profiling runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the NEXT-row kernels")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target oracle time for the headline CPU baseline")
    ap.add_argument("--copy-calibration-gib", type=float, default=0.0,
                    help="also run one device copy of this size (HBM counter calibration for rocprofv3)")
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def dev(a):
    import numpy as np
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def call_times(ctx, fn, reps, warm=3):
    """Whole-call times (ms) of `fn` from HIP events on the stream the
    library runs on (torch's current stream, which the context binds to),
    after `warm` untimed calls; plus the per-kernel timeline of the last call."""
    import torch

    import paper_2608_08751_amd as ivf

    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    fn()
    tl = ctx.kernel_times()
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    return ts, tl


def oracle_rate(fn, n_probe, n_max, target_s):
    """Runs fn(n) on a probe of n_probe units, then on as many units as fit
    about target_s seconds (at most n_max); returns (units, seconds)."""
    t = time.perf_counter()
    fn(n_probe)
    dt = time.perf_counter() - t
    n = int(min(n_max, max(n_probe, n_probe * target_s / max(dt, 1e-6))))
    t = time.perf_counter()
    fn(n)
    return n, time.perf_counter() - t


# ------------------------------------------------------------------ routing

def bench_route(ctx, name, d, k, oracle_s, full_oracle=False):
    """Routing of d["queries"] against d["centroids"], nprobe k: median of 10
    whole calls; the oracle's queries/s on all its queries (full_oracle) or
    a bounded sample of them."""
    import numpy as np
    import torch

    import paper_2608_08751_amd as ivf

    q, c = dev(d["queries"]), dev(d["centroids"])
    Q, D = q.shape
    C = c.shape[0]
    ids = torch.empty((Q, k), dtype=torch.int32, device="cuda")
    dist = torch.empty((Q, k), dtype=torch.float32, device="cuda")
    fn = lambda: ivf.ivf_route(ctx, q, c, k, out_ids=ids, out_dist=dist)
    ts, tl = call_times(ctx, fn, 10)
    st = ctx.last_stats()
    t = float(np.median(ts))
    flops = 2.0 * Q * C * D
    tf = flops / (t * 1e-3) / 1e12
    out = {"queries": Q, "centroids": C, "dim": D, "nprobe": k, "ms_per_call": t,
           "queries_per_s": Q / (t * 1e-3), "kernels_ms": {n.split("/", 1)[1]: ms for n, ms in tl}, "stats": st}
    if st["screen_i8"]:
        # uint8-valued queries: keys and filter on the two int8 planes (each
        # plane executes the algorithmic 2QCD operations once)
        out["screen"] = "int8 MFMA, two planes"
        out["algorithmic_tops"] = tf
        out["int8_mfma_frac"] = tf / PEAK_INT8_MFMA_TOPS
        out["int8_mfma_executed_frac"] = 2.0 * tf / PEAK_INT8_MFMA_TOPS
        out["vs_fp32_mfma_peak_ratio"] = tf / PEAK_FP32_MFMA_TFLOPS
    else:
        out["screen"] = "fp32 MFMA"
        out["tflops"] = tf
        out["fp32_mfma_frac"] = tf / PEAK_FP32_MFMA_TFLOPS
    if oracle_s is not None:
        import oracle

        qh, ch = d["queries"], d["centroids"]
        if full_oracle:
            t0 = time.perf_counter()
            oids, _ = oracle.route(qh, ch, k)
            n, dt = Q, time.perf_counter() - t0
            same = bool((oids == ids.cpu().numpy()).all())
        else:
            n, dt = oracle_rate(lambda m: oracle.route(qh[:m], ch, k), 16, Q, oracle_s)
            same = None
        out["oracle"] = {"queries_per_s": n / dt, "queries": n, "seconds": dt, "cores": oracle.num_threads(0),
                         "sample": "all queries" if full_oracle else "the first %d queries" % n}
        if same is not None:
            out["oracle"]["ids_equal"] = same
    log("%s: %.3f ms per call, %.1f T(FL)OP/s algorithmic on %s" % (name, t, tf, out["screen"]))
    return out


# ------------------------------------------------------------------ k-means

def bench_kmeans(ctx, N, iters, oracle_s, hints=True):
    """Lloyd's algorithm from the seeded row sample: `iters` iterations, each
    one ivf_kmeans_step timed with HIP events (from the second on with the
    previous iteration's labels as hints); per iteration its time, objective
    and screening statistics."""
    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    C, D = C_BIG, D_U8
    means = dev(synth.uniform_means(C, D, seed=0))
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(means, 0, N, x, seed=0)
    c0 = x[dev(synth.kmeans_init(N, C, seed=0))].float().contiguous()
    labs = [torch.empty(N, dtype=torch.int32, device="cuda") for _ in range(2)]
    lab = labs[0]
    cnt = torch.empty(C, dtype=torch.int64, device="cuda")
    obj = torch.empty(1, dtype=torch.float64, device="cuda")
    cbuf = [torch.empty((C, D), dtype=torch.float32, device="cuda") for _ in range(2)]
    # one untimed iteration loads the kernels and sizes the workspace
    ivf.ivf_kmeans_step(ctx, x, c0, seed=0, it=0, out_labels=lab, out_centroids=cbuf[0], out_counts=cnt,
                        out_objective=obj)
    torch.cuda.synchronize()
    rows = []
    c = c0
    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    for it in range(iters):
        out = cbuf[it % 2]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        lab = labs[it % 2]
        hint = labs[(it + 1) % 2] if hints and it > 0 else None
        e0.record()
        ivf.ivf_kmeans_step(ctx, x, c, seed=0, it=it, out_labels=lab, out_centroids=out, out_counts=cnt,
                            out_objective=obj, hint_labels=hint)
        e1.record()
        e1.synchronize()
        tl = ctx.kernel_times()
        rows.append({"iteration": it, "ms": e0.elapsed_time(e1), "objective": float(obj.item()),
                     "screen_single_plane_ms": sum(ms for n, ms in tl if n.endswith("/screen_top1_i8s")),
                     "screen_two_planes_ms": sum(ms for n, ms in tl if n.endswith("/screen_top1_i8")),
                     "update_ms": sum(ms for n, ms in tl if n.endswith("/kmeans_update")),
                     "build_ms": sum(ms for n, ms in tl if "/build_" in n),
                     "stats": ctx.last_stats()})
        c = out
        log("k-means iteration %d: %.1f ms, objective %.6e" % (it, rows[-1]["ms"], rows[-1]["objective"]))
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    total = sum(r["ms"] for r in rows)
    ops = 2.0 * N * C * D * iters
    tops = ops / (total * 1e-3) / 1e12
    res = {"rows": N, "centroids": C, "dim": D, "iterations": iters, "label_hints": bool(hints),
           "total_s": total * 1e-3,
           "ms_per_iteration": total / iters, "vectors_per_s": N * iters / (total * 1e-3),
           "algorithmic_tops": tops, "int8_mfma_frac": tops / PEAK_INT8_MFMA_TOPS,
           "vs_fp32_mfma_peak_ratio": tops / PEAK_FP32_MFMA_TFLOPS,
           "objective_non_increasing": all(b["objective"] <= a["objective"] * (1 + 1e-9)
                                           for a, b in zip(rows, rows[1:])),
           "per_iteration": rows}
    if oracle_s is not None:
        import oracle

        ch = c0.cpu().numpy()
        rng = np.random.default_rng(98)
        idx = np.sort(rng.choice(N, 200000, replace=False))
        xs = x[dev(idx)].cpu().numpy()
        n, dt = oracle_rate(lambda m: oracle.assign(xs[:m], ch), 16, len(idx), oracle_s)
        res["oracle"] = {"vectors_per_s": n / dt, "rows": n, "seconds": dt, "cores": oracle.num_threads(0),
                         "sample": "nearest-centroid search of %d sampled training rows against the initial "
                                   "65,536 centroids (the assignment of one iteration)" % n}
    return res, x, c, lab


# ------------------------------------------------------------- assign-build

def gen_rows(N, means_dev):
    import torch

    import synth

    chunk = 64 * 2**20
    x = torch.empty((N, D_U8), dtype=torch.uint8, device="cuda")
    for r0 in range(0, N, chunk):
        synth.device_mixture_rows_u8(means_dev, r0, min(chunk, N - r0), x[r0:r0 + chunk], seed=0)
    torch.cuda.synchronize()
    return x


def measured_traffic(rows_per_launch, record):
    """HBM bytes per launch of the dominant kernel from a committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (calibrated against a device copy), if it
    was taken on the current kernel sources (the record's `sources`, hashed
    in order) and launch size; otherwise None."""
    import hashlib

    path = os.path.join(ROOT, "profiles", record)
    try:
        with open(path) as f:
            rec = json.load(f)
        h = hashlib.sha256()
        for src in rec["sources"]:
            with open(os.path.join(ROOT, src), "rb") as f:
                h.update(f.read())
        sha = h.hexdigest()
    except (OSError, ValueError, KeyError, TypeError):
        return None, None
    if not sha.startswith(rec["sources_sha256_prefix"]) or rec["rows_per_launch"] != rows_per_launch:
        return None, None
    return rec["traffic_bytes"], "profiles/" + record


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (queries, rows "
              "or centroids would be sharded with one exchange each); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    only = set(args.only.split(",")) if args.only else {"1", "2", "3", "4", "5"}
    osec = None if args.no_cpu_baseline else 3.0
    ctx = ivf.Context(0)
    configs = {}
    extra = {}

    if "1" in only:
        configs["1_route_tiny"] = bench_route(ctx, "route tiny", synth.uniform_mixture_route(1024, 1000, 128, seed=0, plants=0),
                                              16, osec, full_oracle=True)
    if "2" in only:
        configs["2_route_uint8"] = bench_route(ctx, "route uint8-valued",
                                               synth.uniform_mixture_route(C_BIG, 10000, 128, seed=0, plants=0), 64, osec)
    if "3" in only:
        configs["3_route_normalised"] = bench_route(ctx, "route normalised",
                                                    synth.normalised_route(262144, 10000, 96, seed=0), 128, osec)
    if "4" in only:
        km, x_train, c_km, lab_km = bench_kmeans(ctx, args.kmeans_rows, args.kmeans_iters,
                                                 None if osec is None else 6.0)
        configs["4_kmeans"] = km
        if not args.no_extra:
            extra = bench_next_rows(ctx, x_train, c_km, lab_km, configs["4_kmeans"])
        del x_train, c_km, lab_km
        torch.cuda.empty_cache()

    result = {
        "metric": "routed queries/s and assigned vectors/s at 1 GPU; % of fp32 MFMA peak",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8",
        "data": "synthetic: seeded uint8 Gaussian mixture (65,536 components uniform in [0,255]^128, std 20, "
                "rounded and clipped), generated on the device; stands in for SIFT-1B",
    }

    if "5" in only:
        N, C, D = args.rows, C_BIG, D_U8
        t0 = time.time()
        means_h = synth.uniform_means(C, D, seed=0)
        means = dev(means_h)
        x = gen_rows(N, means)
        log("generated %d rows in %.1f s" % (N, time.time() - t0))
        lab = torch.empty(N, dtype=torch.int32, device="cuda")
        cnt = torch.empty(C, dtype=torch.int64, device="cuda")
        off = torch.empty(C + 1, dtype=torch.int64, device="cuda")
        perm = torch.empty(N, dtype=torch.int32, device="cuda")

        def step():
            ivf.ivf_assign_build(ctx, x, means, out_labels=lab, out_counts=cnt, out_offsets=off, out_perm=perm)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        stats = ctx.last_stats()
        log("warmup done; stats:", stats)
        ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
        ctx.kernel_times()
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for i in range(args.steps):
            step()
            torch.cuda.synchronize()
            log("step %d done" % i)
        t_total = time.perf_counter() - t_start
        timeline = ctx.kernel_times()
        ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
        ms_per_step = 1e3 * t_total / args.steps
        stats = ctx.last_stats()  # of the last timed step

        agg = {}
        for name, ms in timeline:
            a = agg.setdefault(name.split("/", 1)[1], [0, 0.0])
            a[0] += 1
            a[1] += ms
        kernels = {n: {"launches": c_, "avg_ms": t / c_, "ms_per_step": t / args.steps} for n, (c_, t) in agg.items()}
        # dominant kernel: the single-plane int8 screen, one launch per slice
        # of at most 2^28 rows; algorithmic work = 2 * rows * C * D multiply
        # and add operations (the -2 x.c contraction), which it executes
        # exactly (one int8 plane per centroid)
        scr = [ms for n, ms in timeline if n.endswith("/screen_top1_i8s")]
        ops_step = 2.0 * N * C * D
        achieved = ops_step * args.steps / (sum(scr) * 1e-3) / 1e12
        launches_per_step = len(scr) // args.steps
        traffic, traffic_src = measured_traffic(min(N, 2**28), "screen_top1_i8s_traffic.json")
        _, probe = ctx.mfma_probe_i8(200000)
        roofline = {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_INT8_MFMA_TOPS,
            "unit": "TOP/s",
            "frac": achieved / PEAK_INT8_MFMA_TOPS,
            "traffic": traffic,
            "traffic_source": traffic_src or "not measured on the current kernel sources",
            "kernel": "screen1_kernel<128, 8> (single-plane int8 MFMA, fused top-1)",
            "ops_per_step": ops_step,
            "launches_per_step": launches_per_step,
            "rows_per_launch": min(N, 2**28),
            "avg_launch_ms": sum(scr) / len(scr),
            "measured_peak": probe,
            "frac_of_measured_peak": achieved / probe,
            "vs_fp32_mfma_peak_ratio": achieved / PEAK_FP32_MFMA_TFLOPS,
        }
        build = [ms for n, ms in timeline if "/build_" in n]
        build_ms = sum(build) / args.steps
        gbs = 12.0 * N / (build_ms * 1e-3) / 1e9
        cfg5 = {
            "rows": N, "centroids": C, "dim": D, "ms_per_call": ms_per_step,
            "vectors_per_s": N / (ms_per_step * 1e-3),
            "assign_ms": sum(ms for n, ms in timeline if "/build_" not in n) / args.steps,
            "algorithmic_tops": ops_step / (ms_per_step * 1e-3) / 1e12,
            "build_lists": {"ms": build_ms, "bytes_per_row": 12, "GBps": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
                            "kernels_ms": {n: k["ms_per_step"] for n, k in kernels.items() if n.startswith("build_")}},
            "stats": stats,
        }
        result.update({
            "value": N / (ms_per_step * 1e-3),
            "unit": "vectors/s",
            "ms_per_step": ms_per_step,
            "config": {
                "workload": "assign-build: 1e9 uint8 rows (D = 128, 128 GB resident, generated on the device in "
                            "64M-row chunks) assigned to 65,536 fp32 centroids (the mixture means) by top-1 "
                            "squared L2, then counts, offsets and the stable list permutation",
                "rows": N, "centroids": C, "dim": D,
                "screen": "int8 MFMA (one plane per centroid; two planes for the rows it leaves); exact fp64 "
                          "re-evaluation of near-ties",
            },
            "roofline": roofline,
            "kernels": kernels,
        })
        if osec is not None:
            import oracle

            oracle.build()
            rng = np.random.default_rng(99)
            idx = np.sort(rng.choice(N, 262144, replace=False))
            xs = x[dev(idx)].cpu().numpy()
            n, dt = oracle_rate(lambda m: oracle.assign(xs[:m], means_h), 16, len(idx), args.cpu_seconds)
            result["cpu_baseline"] = {
                "value": n / dt, "unit": "vectors/s", "cores": oracle.num_threads(0), "kind": "oracle",
                "cpu": cpu_model(),
                "sample": "nearest-centroid search of %d rows sampled from the 1e9 (copied back from the "
                          "device) against the 65,536 centroids, %.1f s" % (n, dt),
            }
            # the list build on a 1e8-label prefix of the GPU labels
            nb = min(N, 10**8)
            labh = lab[:nb].cpu().numpy()
            t = time.perf_counter()
            oracle.build_lists(labh, C)
            dt = time.perf_counter() - t
            cfg5["oracle"] = {"assign_vectors_per_s": result["cpu_baseline"]["value"],
                              "build_vectors_per_s": nb / dt,
                              "sample": "assignment as cpu_baseline; counting-sort list build of the first "
                                        "%d GPU labels (one thread), %.1f s" % (nb, dt)}
        configs["5_assign_build"] = cfg5
        del x, lab, perm
        torch.cuda.empty_cache()

    if "b" in only:
        configs["list_build"] = bench_build(ctx, args.rows)
    if args.copy_calibration_gib > 0:
        # one device copy of known size, for scaling rocprofv3 byte counters
        n = int(args.copy_calibration_gib * 2**30)
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
        del src, dst
    result["configs"] = configs
    if extra:
        result["extra"] = extra
    print(json.dumps(result), flush=True)


def bench_build(ctx, N):
    """ivf_build_lists alone on N uniform labels over 65,536 lists (device
    generator): median of 3 calls, per-kernel times; 12 algorithmic bytes per
    row against the HBM peak."""
    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    C = C_BIG
    lab = torch.empty(N, dtype=torch.int32, device="cuda")
    synth.device_labels(N, C, lab, seed=3)
    cnt = torch.empty(C, dtype=torch.int64, device="cuda")
    off = torch.empty(C + 1, dtype=torch.int64, device="cuda")
    perm = torch.empty(N, dtype=torch.int32, device="cuda")
    fn = lambda: ivf.ivf_build_lists(ctx, lab, C, out_counts=cnt, out_offsets=off, out_perm=perm)
    ts, tl = call_times(ctx, fn, 3, warm=1)
    t = float(np.median(ts))
    gbs = 12.0 * N / (t * 1e-3) / 1e9
    log("list build of %d labels: %.3f ms" % (N, t))
    del lab, perm
    torch.cuda.empty_cache()
    return {"labels": N, "lists": C, "ms_per_call": t, "bytes_per_row": 12, "GBps": gbs,
            "hbm_frac": gbs / PEAK_HBM_GBS, "kernels_ms": {n.split("/", 1)[1]: ms for n, ms in tl}}


# ---------------------------------------------------------------- NEXT rows

def bench_next_rows(ctx, x, cent, prev, km):
    """The NEXT-row kernels on the k-means workload's 10M rows and trained
    centroids: assign-build, list-major layout with residuals, residual PQ
    (one training step, encoding), the ADC scan of 10,000 routed queries,
    and the candidate-restricted assignment."""
    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    N, D = x.shape
    C = cent.shape[0]
    lab, cnt, off, perm = ivf.ivf_assign_build(ctx, x, cent)
    torch.cuda.synchronize()
    out = {}
    lm, res = bench_list_major(ctx, x, cent, off, perm)
    out["list_major"] = lm
    pq, codes, cb = bench_pq(ctx, res)
    out["pq"] = pq
    del res
    q = dev(synth.uniform_mixture_route(C, 10000, D, seed=0)["queries"])
    probes, _ = ivf.ivf_route(ctx, q, cent, 64, want_dist=False)
    out["adc_scan"] = bench_adc(ctx, q, cent, probes, off, perm, codes, cb)
    out["adc_scan_zipf"] = bench_adc_zipf(ctx, q, cent, codes, cb)
    full_ms = km["per_iteration"][-1]["screen_single_plane_ms"] + km["per_iteration"][-1]["screen_two_planes_ms"]
    out["assign_graph"] = bench_assign_graph(ctx, x, cent, prev, full_ms)
    out["assign_cells"] = bench_assign_cells(ctx)
    return out


def _timed(ctx, fn, reps=3):
    import numpy as np

    import paper_2608_08751_amd as ivf

    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    ts = []
    for _ in range(reps):
        fn()
        ts.append(sum(ms for _, ms in ctx.kernel_times()))
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    return float(np.median(ts))


def bench_list_major(ctx, x, cent, offsets, perm):
    """ivf_list_major (uint8 rows, 65,536 lists): list-major copy plus fp32
    residuals, median of 3 calls. Algorithmic bytes per row: read the row and
    its id, write the row and its residual (D + 4 + D + 4 D)."""
    import torch

    import paper_2608_08751_amd as ivf

    N, D = x.shape
    rows = torch.empty_like(x)
    res = torch.empty((N, D), dtype=torch.float32, device=x.device)
    fn = lambda: ivf.ivf_list_major(ctx, x, cent, offsets, perm, out_rows=rows, out_residuals=res)
    fn()
    torch.cuda.synchronize()
    t = _timed(ctx, fn)
    per_row = D + 4 + D + 4 * D
    gbs = per_row * N / (t * 1e-3) / 1e9
    del rows
    return ({"rows": N, "dim": D, "ms": t, "bytes_per_row": per_row, "GBps": gbs,
             "hbm_frac": gbs / PEAK_HBM_GBS}, res)


def bench_pq(ctx, res, M=16, train_rows=1 << 20):
    """Residual PQ on the list-major residuals (M = 16 subspaces of 8 dims,
    256 codewords): one codebook training step on the first 1M residuals and
    the encoding of all of them, median of 3 calls each. The encoding's
    algorithmic work is 3 flops (subtract, multiply, add) per codeword and
    dim, in fp64: 3 * 256 * D per row, against the fp64 vector peak."""
    import numpy as np
    import torch

    import paper_2608_08751_amd as ivf

    N, D = res.shape
    train = res[:train_rows]
    rng = np.random.default_rng(0)
    pick = torch.from_numpy(rng.choice(train_rows, 256, replace=False)).to(res.device)
    cb0 = train[pick].reshape(256, M, D // M).permute(1, 0, 2).contiguous()
    cb, cnt, obj = ivf.ivf_pq_train_step(ctx, train, cb0, seed=0, it=0)
    codes = ivf.ivf_pq_encode(ctx, res, cb)
    torch.cuda.synchronize()
    t_train = _timed(ctx, lambda: ivf.ivf_pq_train_step(ctx, train, cb0, seed=0, it=0, out_codebooks=cb,
                                                        out_counts=cnt, out_objective=obj))
    t_enc = _timed(ctx, lambda: ivf.ivf_pq_encode(ctx, res, cb, out_codes=codes))
    flops = 3.0 * 256 * D * N
    tf = flops / (t_enc * 1e-3) / 1e12
    return ({"rows": N, "dim": D, "subspaces": M, "train_rows": train_rows, "train_step_ms": t_train,
             "train_members_per_codeword_max": int(cnt.max()),
             "encode_ms": t_enc, "encode_rows_per_s": N / (t_enc * 1e-3), "encode_fp64_tflops": tf,
             "encode_fp64_frac": tf / PEAK_FP64_VECTOR_TFLOPS}, codes, cb)


def bench_adc(ctx, queries, cent, probes, offsets, perm, codes, cb, k=512):
    """Residual-PQ ADC scan of 10,000 routed queries (nprobe 64) over the PQ
    codes of the list-major rows, handoff k = 512 per query (the paper's
    N_rerank): median of 3 calls."""
    import torch

    import paper_2608_08751_amd as ivf

    Q, P = probes.shape
    out_ids = torch.empty((Q, k), dtype=torch.int32, device=queries.device)
    out_d = torch.empty((Q, k), dtype=torch.float32, device=queries.device)
    fn = lambda: ivf.ivf_adc_scan(ctx, queries, cent, probes, offsets, perm, codes, cb, k, out_ids=out_ids,
                                  out_dist=out_d)
    fn()
    torch.cuda.synchronize()
    lens = (offsets[1:] - offsets[:-1])[probes.long()].sum().item()
    t = _timed(ctx, fn)
    return {"queries": Q, "nprobe": P, "k": k, "subspaces": codes.shape[1], "codes_scanned": int(lens),
            "ms": t, "queries_per_s": Q / (t * 1e-3), "codes_per_s": lens / (t * 1e-3)}


def bench_adc_zipf(ctx, queries, cent, codes, cb, k=512, P=64, skew=1.0):
    """The same scan over a Zipf-skewed list layout (list sizes ~ 1/rank over
    the 65,536 lists, so the largest holds about 8 % of the codes): the
    codes are reassigned to seeded Zipf labels, and every query probes 64
    distinct random lists. Median of 3 calls."""
    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    N = codes.shape[0]
    C = cent.shape[0]
    lab = synth.random_labels(N, C, seed=7, skew=skew)
    perm = dev(np.argsort(lab, kind="stable").astype(np.int32))
    cnt = np.bincount(lab, minlength=C)
    off = dev(np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64))
    rng = np.random.default_rng(8)
    Q = queries.shape[0]
    probes = dev(np.stack([rng.choice(C, P, replace=False) for _ in range(Q)]).astype(np.int32))
    out_ids = torch.empty((Q, k), dtype=torch.int32, device=queries.device)
    out_d = torch.empty((Q, k), dtype=torch.float32, device=queries.device)
    fn = lambda: ivf.ivf_adc_scan(ctx, queries, cent, probes, off, perm, codes, cb, k, out_ids=out_ids,
                                  out_dist=out_d)
    fn()
    torch.cuda.synchronize()
    lens = (off[1:] - off[:-1])[probes.long()].sum().item()
    t = _timed(ctx, fn)
    return {"queries": Q, "nprobe": P, "k": k, "lists": C, "zipf_exponent": skew,
            "largest_list": int(cnt.max()), "codes_scanned": int(lens), "ms": t,
            "queries_per_s": Q / (t * 1e-3), "codes_per_s": lens / (t * 1e-3)}


def bench_assign_graph(ctx, x, cent, prev, full_ms, S=8):
    """Candidate-restricted assignment (fast construction mode): the
    8-nearest-centroid graph from ivf_route of the centroids against
    themselves, then each row scored against the 8 neighbours of its previous
    centroid, rows taken grouped by previous label (and, for comparison, in
    row order). Median of 3 calls. HBM bytes per row: the row, its previous
    label, its label and distance (centroid rows come from the cache)."""
    import torch

    import paper_2608_08751_amd as ivf

    N, D = x.shape
    C = cent.shape[0]
    graph, _ = ivf.ivf_route(ctx, cent, cent, S, want_dist=False)
    lab = torch.empty(N, dtype=torch.int32, device=x.device)
    dist = torch.empty(N, dtype=torch.float32, device=x.device)
    # rows grouped by previous label (that label's list permutation): rows
    # next to each other share their candidates
    _, _, order = ivf.ivf_build_lists(ctx, prev, C)
    ivf.ivf_assign_graph(ctx, x, cent, graph, prev, order=order, out_labels=lab, out_dist=dist)
    torch.cuda.synchronize()
    t_graph = _timed(ctx, lambda: ivf.ivf_route(ctx, cent, cent, S, out_ids=graph, want_dist=False))
    t_rows = _timed(ctx, lambda: ivf.ivf_assign_graph(ctx, x, cent, graph, prev, out_labels=lab, out_dist=dist))
    t = _timed(ctx, lambda: ivf.ivf_assign_graph(ctx, x, cent, graph, prev, order=order, out_labels=lab,
                                                 out_dist=dist))
    per_row = D + 12
    gbs = per_row * N / (t * 1e-3) / 1e9
    return {"rows": N, "centroids": C, "degree": S, "graph_ms": t_graph, "assign_ms": t,
            "assign_ms_row_order": t_rows,
            "rows_per_s": N / (t * 1e-3), "GBps": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
            "speedup_vs_full_assignment": full_ms / t}



def bench_assign_cells(ctx, N=10_000_000, G=1024, S=8, hops=8):
    """Candidates for rows without a previous label (graph-assisted assignment
    of the base set) on the assign-build workload's generator: 10M base rows,
    the 65,536 mixture means as centroids. A coarse table of 1,024 centroids
    (three Lloyd steps over the centroid table), the cells of the centroids
    and of the rows against it (ivf_assign_build), the 8-nearest-centroid
    graph, then the nearest member of each row's cell and up to 8 greedy
    graph moves, rows taken in cell order (and the nearest member alone,
    first_choice_ms). Median of 3 calls of each timed part; agreement
    with, and time against, the exact assignment of the same rows."""
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    C, D = C_BIG, D_U8
    cent = dev(synth.uniform_means(C, D, seed=0))
    x = torch.empty((N, D), dtype=torch.uint8, device="cuda")
    synth.device_mixture_rows_u8(cent, 0, N, x, seed=0)
    exact, _, _, _ = ivf.ivf_assign_build(ctx, x, cent)
    t_full = _timed(ctx, lambda: ivf.ivf_assign_build(ctx, x, cent, out_labels=exact))
    coarse = cent[dev(synth.kmeans_init(C, G, seed=1))].contiguous()
    t_coarse = 0.0
    for it in range(3):
        t_coarse += _timed(ctx, lambda: ivf.ivf_kmeans_step(ctx, cent, coarse, seed=1, it=it), reps=1)
        _, coarse, _, _ = ivf.ivf_kmeans_step(ctx, cent, coarse, seed=1, it=it)
    _, c_cnt, c_off, c_mem = ivf.ivf_assign_build(ctx, cent, coarse)
    t_members = _timed(ctx, lambda: ivf.ivf_assign_build(ctx, cent, coarse))
    graph, _ = ivf.ivf_route(ctx, cent, cent, S, want_dist=False)
    t_graph = _timed(ctx, lambda: ivf.ivf_route(ctx, cent, cent, S, out_ids=graph, want_dist=False))
    cell, _, _, by_cell = ivf.ivf_assign_build(ctx, x, coarse)
    t_cell = _timed(ctx, lambda: ivf.ivf_assign_build(ctx, x, coarse, out_labels=cell, out_perm=by_cell))
    lab = torch.empty(N, dtype=torch.int32, device=x.device)
    dist = torch.empty(N, dtype=torch.float32, device=x.device)
    fn = lambda: ivf.ivf_assign_cells(ctx, x, cent, cell, c_off, c_mem, graph, hops, order=by_cell,
                                      out_labels=lab, out_dist=dist)
    fn()
    torch.cuda.synchronize()
    t = _timed(ctx, fn)
    agree = float((lab == exact).float().mean())
    fn0 = lambda: ivf.ivf_assign_cells(ctx, x, cent, cell, c_off, c_mem, None, 0, order=by_cell, out_labels=lab,
                                       out_dist=dist)
    t0 = _timed(ctx, fn0)
    agree0 = float((lab == exact).float().mean())
    members_per_row = float(c_cnt[cell.long()].double().mean())
    per_row = t + t_cell
    out = {"rows": N, "centroids": C, "cells": G, "degree": S, "hops": hops, "coarse_train_ms": t_coarse,
           "members_ms": t_members, "graph_ms": t_graph, "row_cells_ms": t_cell, "assign_ms": t,
           "first_choice_ms": t0,
           "members_per_cell_max": int(c_cnt.max()), "members_per_row_mean": members_per_row,
           "rows_per_s": N / (per_row * 1e-3), "agreement_with_exact": agree,
           "agreement_first_choice_only": agree0, "exact_assignment_ms": t_full,
           "speedup_vs_exact_assignment": t_full / per_row}
    del x
    torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    main()
