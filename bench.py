#!/usr/bin/env python3
"""Benchmark of the IVF routing / construction hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input,
on the 65,536-centroid, D = 128 index of the uint8-valued workloads:
  1. ivf_kmeans_step  on 10M uint8 training rows (centroid quantisation,
                      fused single-plane int8-MFMA screening with register
                      top-1, certified fp64 refine, two-plane int8 screen of
                      the rows the single plane leaves, list build, Lloyd
                      update with reseeding, objective);
  2. ivf_assign_build on a batch of 10M uint8 base rows with the new
                      centroids (full assignment + histogram / scan / stable
                      scatter into cluster-major lists);
  3. ivf_route        of 10,000 integer-valued fp32 queries, nprobe 64
                      (threshold sample, fused filter, certified selection).
Every routed query and every assigned row is one vector scored against all
65,536 centroids with top-k selection, so `value` = (train rows + base rows +
queries) / step time, in vectors/s. Inputs are resident in HBM before timing.

The JSON line also carries, per call, the rates; the dominant kernel's
roofline measured live with HIP events on the library's stream; and the CPU
oracle timed on a bounded sample on this host (`cpu_baseline`). The
normalised-float routing workload (262,144 centroids, D = 96, nprobe 128) is
timed separately as an extra.
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


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--train-rows", type=int, default=10_000_000)
    ap.add_argument("--base-rows", type=int, default=10_000_000)
    ap.add_argument("--queries", type=int, default=10_000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="skip the normalised routing extra")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target oracle time for the CPU baseline")
    ap.add_argument("--build-rows", type=int, default=1_000_000_000,
                    help="rows for the separately timed list build at scale (0 = skip)")
    ap.add_argument("--copy-calibration-gib", type=float, default=0.0,
                    help="also run one device copy of this size (HBM counter calibration for rocprofv3)")
    ap.add_argument("--fp32-screen", action="store_true",
                    help="screen the uint8 rows on fp32 MFMA (IVF_OPT_FP32_SCREEN) instead of int8")
    ap.add_argument("--two-plane", action="store_true",
                    help="screen the uint8 rows on two int8 planes only (IVF_OPT_I8_TWO_PLANE_ONLY)")
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
    dev = torch.device("cuda:0")
    C, D, K = 65536, 128, 64
    Nt, Nb, Q = args.train_rows, args.base_rows, args.queries

    t0 = time.time()
    means = torch.from_numpy(synth.uniform_means(C, D, seed=0)).to(dev)
    x_train = torch.empty((Nt, D), dtype=torch.uint8, device=dev)
    x_base = torch.empty((Nb, D), dtype=torch.uint8, device=dev)
    qrows = torch.empty((Q, D), dtype=torch.uint8, device=dev)
    synth.device_mixture_rows_u8(means, 0, Nt, x_train, seed=0)
    synth.device_mixture_rows_u8(means, Nt, Nb, x_base, seed=0)
    synth.device_mixture_rows_u8(means, Nt + Nb, Q, qrows, seed=0)
    queries = qrows.float().contiguous()
    init = torch.from_numpy(synth.kmeans_init(Nt, C, seed=0)).to(dev)
    c0 = x_train[init].float().contiguous()
    torch.cuda.synchronize()
    log("inputs generated on the device in %.1f s" % (time.time() - t0))

    ctx = ivf.Context(0)
    if args.fp32_screen:
        ctx.set_option(ivf.IVF_OPT_FP32_SCREEN, 1)
        top1_name = "screen_top1"
    elif args.two_plane:
        ctx.set_option(ivf.IVF_OPT_I8_TWO_PLANE_ONLY, 1)
        top1_name = "screen_top1_i8"
    else:
        top1_name = "screen_top1_i8s"
    lab_t = torch.empty(Nt, dtype=torch.int32, device=dev)
    c1 = torch.empty((C, D), dtype=torch.float32, device=dev)
    cnt_t = torch.empty(C, dtype=torch.int64, device=dev)
    obj = torch.empty(2, dtype=torch.float64, device=dev)
    lab_b = torch.empty(Nb, dtype=torch.int32, device=dev)
    cnt_b = torch.empty(C, dtype=torch.int64, device=dev)
    off_b = torch.empty(C + 1, dtype=torch.int64, device=dev)
    perm_b = torch.empty(Nb, dtype=torch.int32, device=dev)
    ids = torch.empty((Q, K), dtype=torch.int32, device=dev)
    dist = torch.empty((Q, K), dtype=torch.float32, device=dev)

    stats = {}

    def step(record=False):
        ivf.ivf_kmeans_step(ctx, x_train, c0, seed=0, it=0, out_labels=lab_t, out_centroids=c1,
                            out_counts=cnt_t, out_objective=obj)
        if record:
            stats["kmeans"] = ctx.last_stats()
        ivf.ivf_assign_build(ctx, x_base, c1, out_labels=lab_b, out_counts=cnt_b, out_offsets=off_b,
                             out_perm=perm_b)
        if record:
            stats["assign_build"] = ctx.last_stats()
        ivf.ivf_route(ctx, queries, c1, K, out_ids=ids, out_dist=dist)
        if record:
            stats["route"] = ctx.last_stats()

    for _ in range(args.warmup):
        step(record=True)
    torch.cuda.synchronize()
    log("warmup done; fallback/refine stats:", stats)

    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()  # clear
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step()
        log("step %d enqueued" % i)
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    timeline = ctx.kernel_times()
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)

    ms_per_step = 1e3 * t_total / args.steps
    vectors = Nt + Nb + Q
    value = vectors / (t_total / args.steps)

    # per-kernel aggregation over the timed steps
    agg = {}
    for name, ms in timeline:
        a = agg.setdefault(name, [0, 0.0])
        a[0] += 1
        a[1] += ms
    kernels = {n: {"launches": c, "avg_ms": t / c, "ms_per_step": t / args.steps} for n, (c, t) in agg.items()}
    # the dominant kernel: fused screening with top-1 (one launch on Nt rows,
    # one on Nb rows per step); algorithmic work = 2 * rows * C * D multiply
    # and add operations (the -2 x.c contraction)
    top1 = [ms for n, ms in timeline if n.endswith("/" + top1_name)]
    ops_top1 = 2.0 * C * D * (Nt + Nb) * args.steps
    achieved = ops_top1 / (sum(top1) * 1e-3) / 1e12
    if args.fp32_screen:
        roofline = {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_FP32_MFMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_MFMA_TFLOPS,
            "traffic": measured_traffic(Nt, "screen_top1_fp32_traffic.json"),
            "kernel": "screen_kernel<128, uint8, top1> (fp32 MFMA)",
            "ops_per_launch": 2.0 * C * D * Nt,
            "avg_launch_ms": sum(top1) / len(top1),
        }
        _, probe = ctx.mfma_probe()
    elif args.two_plane:
        # the two-plane int8 screen runs two int8 MFMA planes per centroid: it
        # executes twice the algorithmic operations on the int8 pipe
        roofline = {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_INT8_MFMA_TOPS,
            "unit": "TOP/s",
            "frac": achieved / PEAK_INT8_MFMA_TOPS,
            "traffic": measured_traffic(Nt, "screen_top1_traffic.json"),
            "kernel": "screen_i8_kernel<128, 8> (two-plane int8 MFMA)",
            "ops_per_launch": 2.0 * C * D * Nt,
            "executed_int8_ops_per_launch": 2 * 2.0 * C * D * Nt,
            "executed_frac": 2 * achieved / PEAK_INT8_MFMA_TOPS,
            "fp32_mfma_equivalent_frac": achieved / PEAK_FP32_MFMA_TFLOPS,
            "avg_launch_ms": sum(top1) / len(top1),
        }
        _, probe = ctx.mfma_probe_i8(200000)
    else:
        # the single-plane int8 screen executes exactly the algorithmic
        # operations (one int8 plane per centroid)
        roofline = {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_INT8_MFMA_TOPS,
            "unit": "TOP/s",
            "frac": achieved / PEAK_INT8_MFMA_TOPS,
            "traffic": measured_traffic(Nt, "screen_top1_i8s_traffic.json"),
            "kernel": "screen1_kernel<128, 8> (single-plane int8 MFMA)",
            "ops_per_launch": 2.0 * C * D * Nt,
            "fp32_mfma_equivalent_frac": achieved / PEAK_FP32_MFMA_TFLOPS,
            "avg_launch_ms": sum(top1) / len(top1),
        }
        _, probe = ctx.mfma_probe_i8(200000)
    # the MFMA pipe as the library's probe kernel measures it on this GPU
    # (register operands only; for int8, pseudo-random operands over about
    # 0.1 s, which the part runs at its power-limited clock), after the timed
    # region
    roofline["measured_peak"] = probe
    roofline["frac_of_measured_peak"] = achieved / probe
    if args.two_plane:
        roofline["executed_frac_of_measured_peak"] = 2 * achieved / probe

    def call_ms(call):
        return sum(ms for n, ms in timeline if n.startswith(call + "/")) / args.steps

    per_call = {
        "kmeans_step_vectors_per_s": Nt / (call_ms("kmeans_step") * 1e-3),
        "assign_build_vectors_per_s": Nb / (call_ms("assign_build") * 1e-3),
        "route_queries_per_s": Q / (call_ms("route") * 1e-3),
        "route_tflops": 2.0 * Q * C * D / (call_ms("route") * 1e-3) / 1e12,
    }
    build_ms = [ms for n, ms in timeline if "/build_" in n]
    # two builds per step: Nt rows (inside the k-means step) and Nb rows
    per_call["build_lists_gbs"] = 12.0 * (Nt + Nb) * args.steps / (sum(build_ms) * 1e-3) / 1e9
    per_call["build_lists_hbm_frac"] = per_call["build_lists_gbs"] / PEAK_HBM_GBS
    # the whole step's algorithmic rate against the fp32 MFMA peak (the uint8
    # rows run on int8 MFMA, so this exceeds 1)
    per_call["step_fp32_mfma_equivalent_frac"] = (2.0 * C * D * vectors / (ms_per_step * 1e-3) / 1e12
                                                  / PEAK_FP32_MFMA_TFLOPS)

    result = {
        "metric": "routed queries/s and assigned vectors/s at 1 GPU; % of fp32 MFMA peak",
        "value": value,
        "unit": "vectors/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.fp32_screen else "i8",
        "data": "synthetic (seeded uint8 Gaussian mixture, 65,536 components, std 20, generated on the device)",
        "config": {
            "workload": "ivf_pipeline: kmeans_step(10M u8 rows) + assign_build(10M u8 rows) + route(10,000 queries, nprobe 64); C=65536, D=128",
            "train_rows": Nt, "base_rows": Nb, "queries": Q, "centroids": C, "dim": D, "nprobe": K,
            "screen": ("fp32 MFMA" if args.fp32_screen else "int8 MFMA (two planes per centroid)" if args.two_plane
                       else "int8 MFMA (one plane per centroid; two planes for the rows it leaves)")
            + " for the uint8 rows, fp32 MFMA for the fp32 queries; exact fp64 re-evaluation of near-ties",
        },
        "roofline": roofline,
        "per_call": per_call,
        "kernels": kernels,
        "stats": stats,
    }

    if args.copy_calibration_gib > 0:
        n = int(args.copy_calibration_gib * 2**30)
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(x_train, c0, args.cpu_seconds)

    if not args.no_extra:
        lm, res = bench_list_major(ctx, x_base, c1, off_b, perm_b)
        pq, codes, cb = bench_pq(ctx, res)
        del res
        result["extra"] = {"route_normalised": bench_route_normalised(ctx), "list_major": lm, "pq": pq,
                           "adc_scan": bench_adc(ctx, queries, c1, ids, off_b, perm_b, codes, cb),
                           "assign_graph": bench_assign_graph(ctx, x_train, c1, lab_t,
                                                              kernels["kmeans_step/" + top1_name]["avg_ms"])}
        del codes
        if args.build_rows > 0:
            # free the pipeline's buffers first: the 1e9-row build needs ~8 GB
            del x_train, x_base, lab_t, lab_b, perm_b
            torch.cuda.empty_cache()
            result["extra"]["build_lists_at_scale"] = bench_build(ctx, args.build_rows, C)

    print(json.dumps(result), flush=True)


def measured_traffic(rows_per_launch, record):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary (calibrated against a device
    copy), if it was taken on the current kernel sources (the record's
    `sources`, hashed in order) and launch size; otherwise None."""
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
        return None
    if not sha.startswith(rec["sources_sha256_prefix"]) or rec["rows_per_launch"] != rows_per_launch:
        return None
    return rec["traffic_bytes"]


def bench_route_normalised(ctx):
    """Routing of 10,000 normalised queries against 262,144 unit-norm centroids
    (D = 96), nprobe 128: median of 5 calls, whole-call event time."""
    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    d = synth.normalised_route(262144, 10000, 96, seed=0)
    q = torch.from_numpy(d["queries"]).cuda()
    c = torch.from_numpy(d["centroids"]).cuda()
    ids = torch.empty((10000, 128), dtype=torch.int32, device="cuda")
    dist = torch.empty((10000, 128), dtype=torch.float32, device="cuda")
    ivf.ivf_route(ctx, q, c, 128, out_ids=ids, out_dist=dist)
    torch.cuda.synchronize()
    st = ctx.last_stats()
    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    times = []
    for _ in range(5):
        ivf.ivf_route(ctx, q, c, 128, out_ids=ids, out_dist=dist)
        tl = ctx.kernel_times()
        times.append(sum(ms for _, ms in tl))
        filt = sum(ms for n, ms in tl if n.endswith(("/screen_filter", "/screen_keys")))
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    t = float(np.median(times))
    flops = 2.0 * 10000 * 262144 * 96
    return {
        "queries_per_s": 10000 / (t * 1e-3),
        "ms_per_call": t,
        "tflops": flops / (t * 1e-3) / 1e12,
        "mfma_frac": flops / (t * 1e-3) / 1e12 / PEAK_FP32_MFMA_TFLOPS,
        "screen_ms": filt,
        "stats": st,
    }


def bench_list_major(ctx, x, cent, offsets, perm):
    """ivf_list_major on the step's assign-build output (10M uint8 base rows,
    65,536 lists): list-major copy plus fp32 residuals, median of 3 calls.
    Algorithmic bytes per row: read the row and its id, write the row and
    its residual (D + 4 + D + 4 D)."""
    import numpy as np
    import torch

    import paper_2608_08751_amd as ivf

    N, D = x.shape
    rows = torch.empty_like(x)
    res = torch.empty((N, D), dtype=torch.float32, device=x.device)
    ivf.ivf_list_major(ctx, x, cent, offsets, perm, out_rows=rows, out_residuals=res)
    torch.cuda.synchronize()
    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    times = []
    for _ in range(3):
        ivf.ivf_list_major(ctx, x, cent, offsets, perm, out_rows=rows, out_residuals=res)
        times.append(sum(ms for _, ms in ctx.kernel_times()))
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    t = float(np.median(times))
    per_row = D + 4 + D + 4 * D
    gbs = per_row * N / (t * 1e-3) / 1e9
    del rows
    return ({"rows": N, "dim": D, "ms": t, "bytes_per_row": per_row, "GBps": gbs,
             "hbm_frac": gbs / PEAK_HBM_GBS}, res)


def bench_pq(ctx, res, M=16, train_rows=1 << 20):
    """Residual PQ on the list-major residuals (10M x 128, M = 16 subspaces of
    8 dims, 256 codewords): one codebook training step on the first 1M
    residuals and the encoding of all of them, median of 3 calls each. The
    encoding's algorithmic work is 3 flops (subtract, multiply, add) per
    codeword and dim, in fp64: 3 * 256 * D per row, against the 78.6 TFLOP/s
    fp64 vector peak."""
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

    def timed(fn):
        ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
        ctx.kernel_times()
        ts = []
        for _ in range(3):
            fn()
            ts.append(sum(ms for _, ms in ctx.kernel_times()))
        ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
        return float(np.median(ts))

    t_train = timed(lambda: ivf.ivf_pq_train_step(ctx, train, cb0, seed=0, it=0, out_codebooks=cb,
                                                  out_counts=cnt, out_objective=obj))
    t_enc = timed(lambda: ivf.ivf_pq_encode(ctx, res, cb, out_codes=codes))
    flops = 3.0 * 256 * D * N
    tf = flops / (t_enc * 1e-3) / 1e12
    return ({"rows": N, "dim": D, "subspaces": M, "train_rows": train_rows, "train_step_ms": t_train,
             "encode_ms": t_enc, "encode_rows_per_s": N / (t_enc * 1e-3), "encode_fp64_tflops": tf,
             "encode_fp64_frac": tf / PEAK_FP64_VECTOR_TFLOPS}, codes, cb)


def bench_adc(ctx, queries, cent, probes, offsets, perm, codes, cb, k=512):
    """Residual-PQ ADC scan of the step's 10,000 routed queries (nprobe 64)
    over the PQ codes of the 10M list-major base rows, handoff k = 512 per
    query (the paper's N_rerank): median of 3 calls. Work per query: one
    M x 256 LUT per probed list and M lookups per code of the probed lists."""
    import numpy as np
    import torch

    import paper_2608_08751_amd as ivf

    Q, P = probes.shape
    out_ids = torch.empty((Q, k), dtype=torch.int32, device=queries.device)
    out_d = torch.empty((Q, k), dtype=torch.float32, device=queries.device)
    ivf.ivf_adc_scan(ctx, queries, cent, probes, offsets, perm, codes, cb, k, out_ids=out_ids, out_dist=out_d)
    torch.cuda.synchronize()
    lens = (offsets[1:] - offsets[:-1])[probes.long()].sum().item()
    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    ts = []
    for _ in range(3):
        ivf.ivf_adc_scan(ctx, queries, cent, probes, offsets, perm, codes, cb, k, out_ids=out_ids, out_dist=out_d)
        ts.append(sum(ms for _, ms in ctx.kernel_times()))
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    t = float(np.median(ts))
    return {"queries": Q, "nprobe": P, "k": k, "subspaces": codes.shape[1], "codes_scanned": int(lens),
            "ms": t, "queries_per_s": Q / (t * 1e-3), "codes_per_s": lens / (t * 1e-3)}


def bench_assign_graph(ctx, x, cent, prev, full_top1_ms, S=8):
    """Candidate-restricted assignment (fast construction mode) of the step's
    10M training rows to the new centroids: the 8-nearest-centroid graph from
    ivf_route of the centroids against themselves, then each row scored
    against the 8 neighbours of its previous centroid. Median of 3 calls.
    HBM bytes per row: the row, its previous label, its label and distance
    (centroid rows come from the cache)."""
    import numpy as np
    import torch

    import paper_2608_08751_amd as ivf

    N, D = x.shape
    C = cent.shape[0]
    graph, _ = ivf.ivf_route(ctx, cent, cent, S, want_dist=False)
    lab = torch.empty(N, dtype=torch.int32, device=x.device)
    dist = torch.empty(N, dtype=torch.float32, device=x.device)
    ivf.ivf_assign_graph(ctx, x, cent, graph, prev, out_labels=lab, out_dist=dist)
    torch.cuda.synchronize()

    def timed(fn):
        ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
        ctx.kernel_times()
        ts = []
        for _ in range(3):
            fn()
            ts.append(sum(ms for _, ms in ctx.kernel_times()))
        ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
        return float(np.median(ts))

    t_graph = timed(lambda: ivf.ivf_route(ctx, cent, cent, S, out_ids=graph, want_dist=False))
    t = timed(lambda: ivf.ivf_assign_graph(ctx, x, cent, graph, prev, out_labels=lab, out_dist=dist))
    per_row = D + 12
    gbs = per_row * N / (t * 1e-3) / 1e9
    return {"rows": N, "centroids": C, "degree": S, "graph_ms": t_graph, "assign_ms": t,
            "rows_per_s": N / (t * 1e-3), "GBps": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
            "speedup_vs_full_assignment": full_top1_ms / t}


def bench_build(ctx, N, C):
    """ivf_build_lists on N uniform device-generated labels over C lists:
    median of 3 calls; algorithmic bytes = 12 per row (histogram reads a 4-byte
    label; the scatter reads it again and writes a 4-byte id)."""
    import numpy as np
    import torch

    import synth
    import paper_2608_08751_amd as ivf

    lab = torch.empty(N, dtype=torch.int32, device="cuda")
    synth.device_labels(N, C, lab, seed=0)
    cnt = torch.empty(C, dtype=torch.int64, device="cuda")
    off = torch.empty(C + 1, dtype=torch.int64, device="cuda")
    perm = torch.empty(N, dtype=torch.int32, device="cuda")
    ivf.ivf_build_lists(ctx, lab, C, cnt, off, perm)
    torch.cuda.synchronize()
    ctx.set_option(ivf.IVF_OPT_PROFILE, 1)
    ctx.kernel_times()
    runs = []
    for _ in range(3):
        ivf.ivf_build_lists(ctx, lab, C, cnt, off, perm)
        runs.append(ctx.kernel_times())
    ctx.set_option(ivf.IVF_OPT_PROFILE, 0)
    totals = [sum(ms for _, ms in r) for r in runs]
    i = int(np.argsort(totals)[len(totals) // 2])
    t = totals[i]
    gbs = 12.0 * N / (t * 1e-3) / 1e9
    return {
        "rows": N, "lists": C, "ms": t, "GBps": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
        "kernels_ms": {n.split("/", 1)[1]: ms for n, ms in runs[i]},
    }


def cpu_baseline(x_train, c0, target_s):
    """The oracle (plain C, fp64, all host threads) on a bounded sample of the
    same work: nearest-centroid search of sampled training rows against the
    65,536 centroids. Each routed query / assigned row costs the same C*D
    distance work, so its rate is the oracle's vectors/s for the step."""
    import numpy as np

    import oracle

    oracle.build()
    cent = c0.cpu().numpy()
    threads = oracle.num_threads(0)
    rng = np.random.default_rng(99)
    probe = max(8, threads)
    rows = x_train[:probe].cpu().numpy()
    t = time.perf_counter()
    oracle.assign(rows, cent)
    dt = time.perf_counter() - t
    n = int(min(max(probe, probe * target_s / max(dt, 1e-6)), 200000))
    idx = np.sort(rng.choice(x_train.shape[0], n, replace=False))
    import torch

    rows = x_train[torch.from_numpy(idx).cuda()].cpu().numpy()
    t = time.perf_counter()
    oracle.assign(rows, cent)
    dt = time.perf_counter() - t
    return {
        "value": n / dt,
        "unit": "vectors/s",
        "cores": threads,
        "kind": "oracle",
        "cpu": cpu_model(),
        "sample": "nearest-centroid search of %d sampled training rows against the 65,536 centroids (%.1f s)" % (n, dt),
    }


if __name__ == "__main__":
    main()
