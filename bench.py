#!/usr/bin/env python3
"""Benchmark of the low-bit substitute-layer qlinear on one MI355X.

Default workload: Qwen2.5-7B-shaped MLP projections (gate|up fused K=3584 N=37888,
down K=18944 N=3584), 4-bit codes, groups of 128, fp16 scale/zero, bf16
activations, at draft-tree batches M in {1, 8, 32, 64}.  One step = both launches
at every M (8 launches).  Weights are rotated over enough distinct packed copies
(>= 1 GB) that no launch finds its weights in the 256 MB last-level cache.

Prints one JSON line: effective weight GB/s (codes + scales + zeros bytes / time)
of the whole step, the dominant kernel's roofline and the CPU oracle's rate on a
bounded sample.  ``--workload`` selects another workload for exploration.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen7b_mlp")
    ap.add_argument("--ms", default=None, help="comma-separated M values (default: the workload's)")
    ap.add_argument("--rotate-gb", type=float, default=1.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-cols", type=int, default=1 << 30)
    ap.add_argument("--path", type=int, default=0, help="0 auto, 1 GEMV, 2 MFMA")
    ap.add_argument("--json-out", default=None)
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (reference "
                         "for the HBM traffic counters) and exit")
    return ap.parse_args()


def build_launches(wl, ms, rotate_gb, torch, ss, synth, helpers_quant):
    """Distinct packed weight copies and per-M activations/outputs."""
    from paper_2509_18344_amd.workloads import fused_layer, weight_bytes
    projs = fused_layer(wl.projs) if wl.fused else wl.projs
    if wl.key == "qwen7b_mlp":  # gate|up share x: one fused launch, like the layer plan
        projs = (type(projs[0])("gate_up", 3584, 2 * 18944), projs[2])
    per_copy = sum(weight_bytes(p.N, p.K, wl.bits, wl.group) for p in projs)
    copies = max(1, int(np.ceil(rotate_gb * 1e9 / per_copy)))
    weights = []
    for c in range(copies):
        wc = []
        for pi, p in enumerate(projs):
            w = synth.weights_torch(p.N, p.K, 11, c, pi, device="cuda")
            wc.append(helpers_quant(w, wl.bits, wl.group))
            del w
        weights.append(wc)
    torch.cuda.synchronize()
    acts = {}
    for M in ms:
        for pi, p in enumerate(projs):
            x = synth.activations(M, p.K, 12, M, pi, outlier_frac=wl.outlier_frac).to("cuda")
            y = torch.empty((M, p.N), dtype=torch.bfloat16, device="cuda")
            acts[(M, pi)] = (x, y)
    return projs, weights, acts, per_copy


def device_quantize(torch, ss):
    def q(w, bits, group):
        N, K = w.shape
        codes = torch.empty((N, K), dtype=torch.uint8, device=w.device)
        sc = torch.empty((K // group, N), dtype=torch.float16, device=w.device)
        zr = torch.empty((K // group, N), dtype=torch.float16, device=w.device)
        ss.subspec_quantize(w, bits, group, N, K, codes, sc, zr)
        qw = torch.empty(ss.subspec_qpack_bytes(bits, N, K), dtype=torch.uint8, device=w.device)
        ss.subspec_qpack(codes, bits, N, K, qw)
        del codes
        return {"qweight": qw, "scales": sc, "zeros": zr, "N": N, "K": K}
    return q


def cpu_baseline(wl, sample_cols):
    """Time the fp64 oracle (unpack + exact dequant + float64 matmul) on one whole
    projection of the workload at each of its M values; report weight GB/s."""
    import oracle
    import paper_2509_18344_amd as ss
    from paper_2509_18344_amd import synth
    from paper_2509_18344_amd.workloads import weight_bytes
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl missing
        blas_threads = len(os.sched_getaffinity(0))
    p = max(wl.projs, key=lambda q: (q.K, q.N))
    N = min(p.N, sample_cols)
    K = p.K
    w = synth.weights_np(N, K, 13)
    q, s16, z16 = oracle.quantize_minmax(w, wl.bits, wl.group)
    del w
    packed = np.zeros(ss.subspec_qpack_bytes(wl.bits, N, K), np.uint8)
    ss.subspec_qpack_host(q, wl.bits, N, K, packed)
    xs = {M: synth.bf16_bits(synth.activations(M, K, 14, M)) for M in wl.ms}
    np.ones((64, 64)) @ np.ones((64, 64))  # start the BLAS thread pool outside the timing
    t0 = time.perf_counter()
    for M in wl.ms:
        codes = oracle.unpack(packed, wl.bits, N, K)
        y = oracle.qlinear_ref(xs[M], codes, s16, z16, wl.group)
        assert y.shape == (M, N)
    dt = time.perf_counter() - t0
    wb = weight_bytes(N, K, wl.bits, wl.group) * len(wl.ms)
    return {"value": round(wb / dt / 1e9, 4), "unit": "GB/s", "cores": int(blas_threads),
            "kind": "oracle", "seconds": round(dt, 3),
            "sample": f"{p.name} projection K={K} N={N} (of {p.N}) at M in {list(wl.ms)}: "
                      f"unpack + fp64 dequant (one thread) + fp64 BLAS matmul "
                      f"({blas_threads} threads); {wb / 1e6:.1f} MB of weights"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2509_18344_amd as ss
    from paper_2509_18344_amd import synth
    from paper_2509_18344_amd.workloads import WORKLOADS, weight_bytes

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration_mb:
        n = args.copy_calibration_mb << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n}))
        return
    ss.load_library()
    wl = WORKLOADS[args.workload]
    ms = tuple(int(m) for m in args.ms.split(",")) if args.ms else wl.ms
    t_setup = time.perf_counter()
    projs, weights, acts, per_copy = build_launches(wl, ms, args.rotate_gb, torch, ss, synth,
                                                    device_quantize(torch, ss))
    # Reserve the split-K workspace up front so no launch allocates.
    need = 0
    for M in ms:
        for p in projs:
            need = max(need, ss.subspec_qlinear_plan(M, p.N, p.K, wl.bits, wl.group,
                                                     args.path)["workspace_bytes"])
    ss.subspec_reserve(need)
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup

    launches = [(M, pi) for M in ms for pi in range(len(projs))]
    copies = len(weights)
    stream = torch.cuda.current_stream()
    counter = [0]

    def step(events=None):
        for li, (M, pi) in enumerate(launches):
            wc = weights[counter[0] % copies][pi]
            counter[0] += 1
            x, y = acts[(M, pi)]
            p = projs[pi]
            if events is not None:
                events[li][0].record(stream)
            ss.subspec_qlinear_path(x, wc["qweight"], wc["scales"], wc["zeros"], wl.bits,
                                    wl.group, M, p.N, p.K, y, args.path, stream.cuda_stream)
            if events is not None:
                events[li][1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    per_launch = {li: [] for li in range(len(launches))}
    ev = [[[torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
           for _ in launches] for _ in range(args.steps)]
    t_all0 = torch.cuda.Event(enable_timing=True)
    t_all1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_all0.record(stream)
    for s in range(args.steps):
        step(ev[s])
    t_all1.record(stream)
    torch.cuda.synchronize()
    total_ms = t_all0.elapsed_time(t_all1)
    for s in range(args.steps):
        for li in range(len(launches)):
            per_launch[li].append(ev[s][li][0].elapsed_time(ev[s][li][1]))

    step_weight_bytes = sum(weight_bytes(projs[pi].N, projs[pi].K, wl.bits, wl.group)
                            for (_, pi) in launches)
    ms_per_step = total_ms / args.steps
    value = step_weight_bytes / (ms_per_step * 1e-3) / 1e9

    detail = []
    best = None
    for li, (M, pi) in enumerate(launches):
        p = projs[pi]
        t = np.array(per_launch[li])
        avg_us = float(t.mean() * 1e3)
        wb = weight_bytes(p.N, p.K, wl.bits, wl.group)
        ab = wb + 2 * M * p.K + 2 * M * p.N
        flops = 2.0 * M * p.N * p.K
        plan = ss.subspec_qlinear_plan(M, p.N, p.K, wl.bits, wl.group, args.path)
        d = {"proj": p.name, "M": M, "N": p.N, "K": p.K, "path": plan["path"],
             "grid": plan["grid"], "splits": plan["splits"], "avg_us": round(avg_us, 2),
             "p10_us": round(float(np.percentile(t, 10) * 1e3), 2),
             "p90_us": round(float(np.percentile(t, 90) * 1e3), 2),
             "weight_GBs": round(wb / (avg_us * 1e-6) / 1e9, 1),
             "alg_GBs": round(ab / (avg_us * 1e-6) / 1e9, 1),
             "TFLOPs": round(flops / (avg_us * 1e-6) / 1e12, 2),
             "total_ms": float(t.sum())}
        detail.append(d)
        if best is None or d["total_ms"] > best["total_ms"]:
            best = d | {"alg_bytes": ab, "flops": flops}
    peak_frac_hbm = best["alg_GBs"] / HBM_PEAK_GBS
    roofline = {"bound": "hbm", "achieved": best["alg_GBs"], "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(peak_frac_hbm, 4), "traffic": None,
                "kernel": f"{'k_qgemv' if best['path'] == 1 else 'k_qgemm_mfma'} "
                          f"{best['proj']} M={best['M']} N={best['N']} K={best['K']}",
                "alg_bytes_per_launch": best["alg_bytes"], "avg_us": best["avg_us"]}

    out = {
        "metric": "effective weight GB/s and % HBM roofline of low-bit qlinear at draft-tree M",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: N(0,0.02) fp32 weights min/max-quantized on the GPU, N(0,1) bf16 "
                "activations, seeded",
        "config": {"workload": wl.description, "bits": wl.bits, "group": wl.group,
                   "ms": list(ms), "launches_per_step": len(launches),
                   "weight_bytes_per_step": step_weight_bytes,
                   "distinct_weight_copies": copies,
                   "rotation_GB": round(copies * per_copy / 1e9, 2),
                   "hbm_fraction_of_8TBs": round(value / HBM_PEAK_GBS, 4)},
        "roofline": roofline,
        "per_launch": [{k: v for k, v in d.items() if k != "total_ms"} for d in detail],
        "setup_s": round(setup_s, 2),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_cols)
    line = json.dumps(out)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)


if __name__ == "__main__":
    main()
