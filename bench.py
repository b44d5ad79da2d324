#!/usr/bin/env python3
"""Benchmark of the low-bit substitute-layer qlinear on one MI355X.

Default (``--workload suite``): the headline is the Qwen2.5-32B-shaped 64-layer
substitute stack (q|k|v, o, gate|up, down per layer; 3-bit codes, groups of 128,
fp16 scale/zero) at draft-tree batches M in {1, 16, 64, 128}: one step = one pass
of all 64 layers at every M, each M's pass captured as one HIP graph.  The same
JSON line carries, under "configs", the tiny layer (K=256 N=512 4-bit g64 at M = 1
and 4: per-call latency, weights cache-resident), the Qwen2.5-7B-shaped MLP
projections (gate|up fused K=3584 N=37888, down K=18944 N=3584, 4-bit g128, M in
{1, 8, 32, 64}, weights rotated over >= 1 GB of distinct copies), the same at the
small draft batches M in {2, 4, 6, 8}, the 28-layer
Qwen2.5-7B-shaped stack at M = 64, and the 64-layer 2-bit g64 32B-shaped stack
with 1% outlier input channels at M = 128, each with its own roofline entry.

Timing: untimed steps of the same work for half a second (the shader clock ramps up
from idle over a few hundred ms), W untimed warm-up steps, then K steps back to back
between HIP events on the launch stream (ms_per_step = their total / K; step_ms = median, p10 and p90 of the
per-step times).  Per launch: a HIP graph of that projection's launches over all
layers (or weight copies) is replayed several times, one event pair per replay,
so no host work sits between the timed calls; the dominant launch's roofline
comes from that figure.  host_us_per_call is the host time of one eager
subspec_qlinear call.  The GPU's clock levels are sampled (sysfs DPM tables) while
the timed steps run, and a plain device copy's rate is given as context for the
fraction of 8 TB/s.

Prints one JSON line: effective weight GB/s (codes + scales + zeros bytes / time)
of the whole step, the dominant kernel's roofline and the CPU oracle's rate on a
bounded sample (one layer of the headline workload, host CPU model and BLAS named).
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
# Per kernel family: where its measured traffic is kept, which sources it depends on
# and which kernel names belong to it.
FAMILIES = {
    "qlinear": {"json": os.path.join(ROOT, "profiles", "traffic.json"),
                "sources": ("kernels_qlinear.hip", "kernels_qmma.hip", "qmma_kernel.h", "qlinear_device.h",
                            "device_common.h", "kernels.h"),
                "kernels": ("k_qgemv", "k_qgemm_mfma", "k_qmma")},
    "tree": {"json": os.path.join(ROOT, "profiles", "traffic_tree.json"),
             "sources": ("kernels_tree.hip", "kernels_tree.h", "device_common.h", "kernels.h"),
             "kernels": ("k_tree_expand",)},
    "attn": {"json": os.path.join(ROOT, "profiles", "traffic_attn.json"),
             "sources": ("kernels_attn.hip", "kernels_attn.h", "device_common.h", "kernels.h"),
             "kernels": ("k_attn_partial", "k_attn_combine")},
}
WORKLOAD_FAMILY = {"tree_expand": "tree", "tree_attn": "attn"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="suite",
                    help="suite (default: qwen32b_stack as the headline, then tiny, qwen7b_mlp, "
                         "qwen7b_mlp_draft, qwen7b_stack and qwen32b_2bit as extra entries), or one "
                         "of those, "
                         "or tree_expand (the draft-tree expansion step; --ms gives its rows) "
                         "or tree_attn (one layer's tree attention over the shared KV cache) "
                         "or prefetch (verification pass over offloaded layers with cross-layer "
                         "weight prefetch) or hqq (HQQ-style quantization of one Qwen2.5-7B layer)")
    ap.add_argument("--ms", default=None, help="comma-separated M values (default: the workload's)")
    ap.add_argument("--rotate-gb", type=float, default=1.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-clocks", action="store_true",
                    help="do not sample the GPU clock levels (sysfs) during the timed steps")
    ap.add_argument("--path", type=int, default=0, help="0 auto, 1 GEMV, 2 MFMA")
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches of the projection workloads instead of HIP-graph "
                         "replays (always eager with --path other than 0)")
    ap.add_argument("--per-launch-reps", type=int, default=20,
                    help="launches per timed burst of the tree and attention workloads")
    ap.add_argument("--json-out", default=None)
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (reference "
                         "for the HBM traffic counters) and exit")
    ap.add_argument("--summarize-trace", default=None, metavar="TRACE_DIR",
                    help="print a markdown table of a rocprofv3 --kernel-trace run's "
                         "library kernels per (kernel, grid) and exit")
    ap.add_argument("--summarize-sq", nargs=3, default=None, metavar=("PASS_A_DIR", "PASS_B_DIR", "TRACE_DIR"),
                    help="print a markdown table of the SQ counters (two --pmc passes of SQ_PASS_A "
                         "and SQ_PASS_B) and kernel-trace durations of --workload's launches at "
                         "--ms, and exit")
    ap.add_argument("--summarize-pmc", nargs=4, default=None,
                    metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"))
    return ap.parse_args()


# --- kernel identity and measured traffic ----------------------------------------

_COMMENT = re.compile(r"//[^\n]*|/\*.*?\*/", re.S)


def kernel_source_hash(family: str = "qlinear") -> str:
    """Hash of the family's kernel sources with comments and whitespace removed (what
    the compiler sees), so that measured counters stay attached to unchanged code."""
    h = hashlib.sha256()
    for f in FAMILIES[family]["sources"]:
        with open(os.path.join(ROOT, "paper_2509_18344_amd", "csrc", f), encoding="utf-8") as fh:
            code = _COMMENT.sub(" ", fh.read())
        h.update(" ".join(code.split()).encode())
    return h.hexdigest()[:16]


def dispatch_key(family: str, targs, grid_items: int, wg_items: int) -> str:
    """Kernel identity: template name with its first six arguments (bits, group,
    rows or row tiles, tiles per wavefront, chunk, wavefronts) and the grid."""
    return f"{family}<{', '.join(str(a) for a in targs[:6])}> grid={grid_items} wg={wg_items}"


def plan_key(plan, bits, group) -> str:
    wg = plan["waves"] * 64
    if plan["path"] == 1:
        family = "k_qgemv"
        targs = (bits, group, plan["rows"], plan["tiles_per_wave"], plan["chunk_blocks"], plan["waves"])
    elif plan["mfma_rows"] == 32:
        family = "k_qmma"
        targs = (bits, group, plan["rows"] // 32, plan["tiles_per_wave"] // 2, plan["ring_chunks"],
                 plan["waves"])
    else:
        family = "k_qgemm_mfma"
        targs = (bits, group, plan["rows"] // 16, plan["tiles_per_wave"], plan["chunk_blocks"], plan["waves"])
    # the whole launch: row blocks are its grid's y dimension
    return dispatch_key(family, targs, plan["grid"] * plan["row_blocks"] * wg, wg)


def _counter_rows(d, counter):
    files = [os.path.join(dp, f) for dp, _, fs in os.walk(d) for f in fs
             if f.endswith("counter_collection.csv")]
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    per = collections.defaultdict(float)
    meta = {}
    for fn in files:
        with open(fn) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                k = (fn, r["Dispatch_Id"])
                per[k] += float(r["Counter_Value"])
                meta[k] = (r["Kernel_Name"], int(r["Grid_Size"]), int(r["Workgroup_Size"]))
    return [(meta[k][0], meta[k][1], meta[k][2], v) for k, v in per.items()]


def summarize_pmc(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, family="qlinear",
                  calib_bytes=1 << 30):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of one kernel family, scaled by what
    the same counters read for a plain copy of known size."""
    fam = FAMILIES[family]
    pat = re.compile(r"(" + "|".join(fam["kernels"]) + r")(<([^>]*)>)?")
    cf = max(v for (_, _, _, v) in _counter_rows(copy_fetch_dir, "FETCH_SIZE"))
    cw = max(v for (_, _, _, v) in _counter_rows(copy_write_dir, "WRITE_SIZE"))
    f_scale = calib_bytes / (cf * 1024.0)
    w_scale = calib_bytes / (cw * 1024.0)
    acc = collections.defaultdict(lambda: {"fetch": [], "write": [], "names": set()})
    for d, which, counter in ((fetch_dir, "fetch", "FETCH_SIZE"), (write_dir, "write", "WRITE_SIZE")):
        for name, grid, wg, v in _counter_rows(d, counter):
            m = pat.search(name)
            if not m:
                continue
            targs = [int(a) for a in m.group(3).split(",")] if m.group(3) else []
            if family == "qlinear":
                e = acc[dispatch_key(m.group(1), targs, grid, wg)]
            else:
                e = acc[f"{m.group(0)} grid={grid} wg={wg}"]
            e[which].append(v)
            e["names"].add(m.group(0))
    kernels = {}
    for key, e in sorted(acc.items()):
        if not e["fetch"] or not e["write"]:
            continue
        if len(e["names"]) != 1:  # two template instances share a grid: ambiguous
            continue
        fk = float(np.mean(e["fetch"]))
        wk = float(np.mean(e["write"]))
        kernels[key] = {"kernel": e["names"].pop(), "dispatches": len(e["fetch"]),
                        "fetch_kib_raw": round(fk, 1), "write_kib_raw": round(wk, 1),
                        "hbm_bytes_per_launch": int(round(fk * 1024 * f_scale + wk * 1024 * w_scale))}
    out = {"kernel_source_sha256_16": kernel_source_hash(family),
           "calibration": {"copy_bytes": calib_bytes, "fetch_kib_raw": cf, "write_kib_raw": cw,
                           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)},
           "kernels": kernels}
    os.makedirs(os.path.dirname(fam["json"]), exist_ok=True)
    with open(fam["json"], "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps({"wrote": fam["json"], "kernels": len(kernels),
                      "fetch_scale": out["calibration"]["fetch_scale"],
                      "write_scale": out["calibration"]["write_scale"]}))


def library_key(name, grid, wg):
    """Dispatch key of a library kernel from its full name, grid and workgroup size
    (work-items), the same key plan_key gives the qlinear kernels; None otherwise."""
    m = re.search(r"(k_\w+)(<[^>]*>)?", name)
    if not m or "subspec::" not in name:
        return None
    targs = [int(a) for a in m.group(2)[1:-1].split(",")] if m.group(2) else []
    if m.group(1) in ("k_qgemv", "k_qgemm_mfma", "k_qmma"):
        return dispatch_key(m.group(1), targs, grid, wg)
    return f"{m.group(0)} grid={grid} wg={wg}"


def trace_durations(d):
    """Per dispatch key, the durations (us) of the library's kernels in a rocprofv3
    kernel trace."""
    files = [os.path.join(dp, f) for dp, _, fs in os.walk(d) for f in fs
             if f.endswith("kernel_trace.csv")]
    if not files:
        raise SystemExit(f"no kernel_trace.csv under {d}")
    durs = collections.defaultdict(list)
    for fn in files:
        with open(fn) as f:
            for r in csv.DictReader(f):
                grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
                key = library_key(r["Kernel_Name"], grid, int(r["Workgroup_Size_X"]))
                if key:
                    durs[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return durs


def summarize_trace(d):
    """Per (kernel, grid) dispatch durations of the library's kernels in a rocprofv3
    kernel trace, as a markdown table (microseconds)."""
    durs = trace_durations(d)
    print("| kernel (template args, grid and workgroup in work-items) | dispatches | avg us | median us | min us | max us |")
    print("|---|---|---|---|---|---|")
    for key, v in sorted(durs.items()):
        a = np.array(v)
        print(f"| `{key}` | {len(a)} | {a.mean():.2f} | {np.median(a):.2f} | {a.min():.2f} | {a.max():.2f} |")


SQ_PASS_A = ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY",
             "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU")
SQ_PASS_B = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_MFMA",
             "SQ_INSTS_LDS", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS")
SIMDS = 1024
SCLK_GHZ = 2.4


def summarize_sq(dir_a, dir_b, trace_dir, wl_key, ms):
    """Markdown table of the SQ counters of every launch of a qlinear workload: two
    rocprofv3 --pmc passes (SQ_PASS_A, SQ_PASS_B) and a kernel trace of the same
    command.  Run where the counters were taken (the launch plans, hence the dispatch
    keys, depend on the device)."""
    import paper_2509_18344_amd as ss
    from paper_2509_18344_amd.workloads import WORKLOADS, Proj, fused_layer
    wl = WORKLOADS[wl_key]
    if wl.key.startswith("qwen7b_mlp"):
        projs = (Proj("gate_up", 3584, 2 * 18944), Proj("down", 18944, 3584))
    else:
        projs = fused_layer(wl.projs) if wl.layers > 1 else wl.projs
    labels = {}
    for M in ms:
        for p in projs:
            plan = ss.subspec_qlinear_plan(M, p.N, p.K, wl.bits, wl.group)
            key = plan_key(plan, wl.bits, wl.group)
            name, msk = labels.get(key, (p.name, []))
            labels[key] = (name, msk + [M])
    labels = {k: f"{n} M={','.join(str(m) for m in msk)}" for k, (n, msk) in labels.items()}
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for d, names in ((dir_a, SQ_PASS_A), (dir_b, SQ_PASS_B)):
        for c in names:
            for name, grid, wg, v in _counter_rows(d, c):
                key = library_key(name, grid, wg)
                if key in labels:
                    vals[key][c].append(v)
    durs = trace_durations(trace_dir)
    print("| launch | kernel | dispatches | waves | issuing % | waiting for issue % | of which LDS % | "
          "waitcnt/barrier % | VALU / wave | MFMA / wave | LDS / wave | trace avg us | MFMA busy % |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|---|")
    for key, label in labels.items():
        v = {c: float(np.mean(x)) for c, x in vals[key].items()}
        if not all(c in v for c in SQ_PASS_A + SQ_PASS_B) or key not in durs:
            continue
        waves = v["SQ_WAVES"]
        wc = v["SQ_WAVE_CYCLES"]
        avg = float(np.mean(durs[key]))
        busy = v["SQ_VALU_MFMA_BUSY_CYCLES"] / (avg * 1e-6 * SCLK_GHZ * 1e9 * SIMDS)
        print(f"| {label} | `{key.split(' grid')[0]}` | {len(vals[key]['SQ_WAVES'])} | {int(waves)} | "
              f"{100 * v['SQ_ACTIVE_INST_ANY'] / wc:.0f} | {100 * v['SQ_WAIT_INST_ANY'] / wc:.0f} | "
              f"{100 * v['SQ_WAIT_INST_LDS'] / wc:.0f} | {100 * v['SQ_WAIT_ANY'] / wc:.0f} | "
              f"{v['SQ_INSTS_VALU'] / waves:.0f} | {v['SQ_INSTS_MFMA'] / waves:.0f} | "
              f"{v['SQ_INSTS_LDS'] / waves:.0f} | {avg:.1f} | {100 * busy:.1f} |")


def measured_traffic(key: str, family: str = "qlinear"):
    """HBM bytes per launch for `key` from the family's traffic file, if those
    counters were taken on the current kernel sources; else None."""
    try:
        with open(FAMILIES[family]["json"]) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("kernel_source_sha256_16") != kernel_source_hash(family):
        return None
    entry = data.get("kernels", {}).get(key)
    return None if entry is None else entry.get("hbm_bytes_per_launch")


# --- host and device context ------------------------------------------------------

def host_info():
    """The host CPU model (from /proc/cpuinfo) and the BLAS numpy uses (threadpoolctl)."""
    info = {"cpu_model": None, "blas": None, "blas_threads": None,
            "affinity_cpus": len(os.sched_getaffinity(0))}
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    info["cpu_model"] = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if blas:
            info["blas"] = f"{blas[0].get('internal_api')} {blas[0].get('version')}".strip()
            info["blas_threads"] = max(int(i.get("num_threads", 1)) for i in blas)
    except Exception:  # pragma: no cover - threadpoolctl missing
        pass
    return info


def _dpm_level(path):
    """The current level of a sysfs DPM table (the line marked '*'), e.g. '2400Mhz'."""
    try:
        with open(path) as f:
            for ln in f:
                if ln.rstrip().endswith("*"):
                    return ln.split(":", 1)[1].replace("*", "").strip()
    except OSError:
        pass
    return None


class ClockSampler:
    """Samples the GPU's shader and memory clock levels from sysfs (pp_dpm_sclk /
    pp_dpm_mclk of the first card that has them) every `period` seconds on a thread
    while a timed region runs; no child process, no GPU call."""

    def __init__(self, period=0.05, enabled=True):
        import glob
        import threading
        cards = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")) if enabled else []
        self.dev = os.path.dirname(cards[0]) if cards else None
        self.period = period
        self.samples = []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            self.samples.append((_dpm_level(os.path.join(self.dev, "pp_dpm_sclk")),
                                 _dpm_level(os.path.join(self.dev, "pp_dpm_mclk"))))
            self._stop.wait(self.period)

    def __enter__(self):
        if self.dev:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        if self.dev:
            self._stop.set()
            self._thread.join()

    def summary(self):
        if not self.samples:
            return None
        sclk = collections.Counter(a for a, _ in self.samples)
        mclk = collections.Counter(b for _, b in self.samples)
        return {"samples": len(self.samples), "sclk": dict(sclk.most_common()),
                "mclk": dict(mclk.most_common()), "source": self.dev + "/pp_dpm_{sclk,mclk}"}


def copy_rate(torch, stream, mib=2048, replays=5):
    """Device-to-device copy rate of torch's copy kernel over `mib` MiB, counting
    the bytes read plus the bytes written: context for the fraction of 8 TB/s."""
    n = mib << 20
    with torch.cuda.stream(stream):
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        src.fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(replays):
            dst.copy_(src)
        e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / replays
    del src, dst
    return {"torch_copy_GBs_read_plus_write": round(2 * n / (ms * 1e-3) / 1e9, 1), "MiB": mib}


# --- CPU oracle baseline --------------------------------------------------------

def cpu_baseline(wl, ms, min_seconds=10.0):
    """Time the fp64 oracle (unpack + exact dequant + float64 matmul) on the bench
    step's own launches (every projection at every M), repeating the step until
    `min_seconds` have passed; report weight GB/s.  Stacks use one layer."""
    import oracle
    import paper_2509_18344_amd as ss
    from paper_2509_18344_amd import synth
    from paper_2509_18344_amd.workloads import Proj, fused_layer, weight_bytes
    host = host_info()
    threads = host["blas_threads"] or host["affinity_cpus"]
    if wl.key.startswith("qwen7b_mlp"):
        projs = (Proj("gate_up", 3584, 2 * 18944), Proj("down", 18944, 3584))
    elif wl.layers > 1:
        projs = fused_layer(wl.projs)
    else:
        projs = wl.projs
    prepared = []
    for pi, p in enumerate(projs):
        w = synth.weights_np(p.N, p.K, 13, pi)
        q, s16, z16 = oracle.quantize_minmax(w, wl.bits, wl.group)
        del w
        packed = np.zeros(ss.subspec_qpack_bytes(wl.bits, p.N, p.K), np.uint8)
        ss.subspec_qpack_host(q, wl.bits, p.N, p.K, packed)
        del q
        xs = {M: synth.bf16_bits(synth.activations(M, p.K, 14, M, pi, outlier_frac=wl.outlier_frac))
              for M in ms}
        prepared.append((p, packed, s16, z16, xs))
    np.ones((64, 64)) @ np.ones((64, 64))  # start the BLAS thread pool outside the timing
    steps = 0
    t0 = time.perf_counter()
    while True:
        for M in ms:
            for (p, packed, s16, z16, xs) in prepared:
                codes = oracle.unpack(packed, wl.bits, p.N, p.K)
                y = oracle.qlinear_ref(xs[M], codes, s16, z16, wl.group)
                assert y.shape == (M, p.N)
                del codes, y
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    wb = steps * len(ms) * sum(weight_bytes(p.N, p.K, wl.bits, wl.group) for p in projs)
    names = "+".join(f"{p.name}(K={p.K},N={p.N})" for p in projs)
    return {"value": round(wb / dt / 1e9, 4), "unit": "GB/s", "cores": int(threads),
            "kind": "oracle", "seconds": round(dt, 3),
            "cpu_model": host["cpu_model"], "blas": host["blas"],
            "sample": f"{steps} pass(es) of {names} at M in {list(ms)}"
                      f"{' (one layer of the stack)' if wl.layers > 1 else ''}: unpack + fp64 "
                      f"dequant (one thread) + fp64 BLAS matmul ({threads} threads); "
                      f"{wb / 1e6:.1f} MB of weights"}


# --- GPU timing -------------------------------------------------------------------

def timed(torch, stream, fn, warmup, steps):
    for s in range(warmup):
        fn(s)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for s in range(steps):
        fn(warmup + s)
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1)


SPIN_UP_S = 0.5  # the shader clock takes a few hundred ms to ramp from idle


def timed_steps(torch, stream, fn, warmup, steps, clocks=True):
    """Spin-up (untimed steps of the same work for SPIN_UP_S seconds, so the clock is
    at its working level), `warmup` untimed steps, then `steps` steps back to back
    between events on `stream` (one event after each step, nothing waits between
    them).  Returns the total milliseconds, the per-step milliseconds and the clock
    levels sampled while the timed steps ran."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < SPIN_UP_S:
        fn(0)
        torch.cuda.synchronize()
    for s in range(warmup):
        fn(s)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    with ClockSampler(enabled=clocks) as cs:
        ev[0].record(stream)
        for s in range(steps):
            fn(warmup + s)
            ev[s + 1].record(stream)
        torch.cuda.synchronize()
    per = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)])
    return ev[0].elapsed_time(ev[-1]), per, cs.summary()


def pct(a, q):
    return round(float(np.percentile(a, q)), 4)


def per_launch_graph(torch, ss, wl, M, p, argsets, stream, replays=7, min_launches=32):
    """Per-call time of one projection without host work between calls: a HIP graph
    of n back-to-back launches of it (cycling through `argsets`, i.e. distinct weight
    copies or layers) is replayed `replays` times, each replay between two events on
    the launch stream; a call's time is the replay's time / n (for the 32x32 kernel
    this includes its x-sum pre-pass)."""
    from paper_2509_18344_amd.workloads import weight_bytes
    n = max(min_launches, len(argsets))
    lst = [dict(argsets[i % len(argsets)], N=p.N, K=p.K) for i in range(n)]
    g = ss.subspec_stack_capture(lst, wl.bits, wl.group, M, stream)
    try:
        ss.subspec_graph_launch(g, stream)  # untimed first replay
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(replays + 1)]
        ev[0].record(stream)
        for r in range(replays):
            ss.subspec_graph_launch(g, stream)
            ev[r + 1].record(stream)
        torch.cuda.synchronize()
        t = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(replays)]) * 1e3 / n  # us
    finally:
        ss.subspec_graph_destroy(g)
    plan = ss.subspec_qlinear_plan(M, p.N, p.K, wl.bits, wl.group)
    wb = weight_bytes(p.N, p.K, wl.bits, wl.group)
    ab = wb + 2 * M * p.K + 2 * M * p.N
    flops = 2.0 * M * p.N * p.K
    med = float(np.median(t))
    return {"proj": p.name, "M": M, "N": p.N, "K": p.K, "path": plan["path"],
            "key": plan_key(plan, wl.bits, wl.group), "grid": plan["grid"], "splits": plan["splits"],
            "median_us": round(med, 2), "p10_us": pct(t, 10), "p90_us": pct(t, 90),
            "calls_per_replay": n, "replays": replays,
            "weight_GBs": round(wb / (med * 1e-6) / 1e9, 1),
            "alg_GBs": round(ab / (med * 1e-6) / 1e9, 1),
            "TFLOPs": round(flops / (med * 1e-6) / 1e12, 2),
            "alg_bytes": ab, "flops": flops}


def host_us_per_call(ss, wl, M, p, a, stream, calls=200):
    """Host time of one eager subspec_qlinear call (argument marshalling, the plan,
    the launch), averaged over `calls` calls issued without waiting."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(calls):
        ss.subspec_qlinear(a["x"], a["qweight"], a["scales"], a["zeros"], wl.bits, wl.group, M, p.N, p.K,
                           a["y"], stream)
    t1 = time.perf_counter()
    torch.cuda.synchronize()
    return {"us": round((t1 - t0) * 1e6 / calls, 2), "call": f"{p.name} M={M} N={p.N} K={p.K}"}


def roofline_of(dom, family="qlinear"):
    """Roofline entry of the dominant launch (bound by HBM or by bf16 MFMA,
    whichever its arithmetic intensity puts it under)."""
    ridge = (MFMA_BF16_PEAK_TFLOPS * 1e12) / (HBM_PEAK_GBS * 1e9)
    if dom["flops"] / dom["alg_bytes"] > ridge:
        r = {"bound": "mfma", "achieved": dom["TFLOPs"], "peak": MFMA_BF16_PEAK_TFLOPS,
             "unit": "TFLOP/s", "frac": round(dom["TFLOPs"] / MFMA_BF16_PEAK_TFLOPS, 4)}
    else:
        r = {"bound": "hbm", "achieved": dom["alg_GBs"], "peak": HBM_PEAK_GBS,
             "unit": "GB/s", "frac": round(dom["alg_GBs"] / HBM_PEAK_GBS, 4)}
    r.update({"traffic": measured_traffic(dom["key"], family),
              "kernel": f"{dom['key']} ({dom['proj']} M={dom['M']} N={dom['N']} K={dom['K']})",
              "avg_us": dom["median_us"], "alg_bytes_per_launch": dom["alg_bytes"],
              "flops_per_launch": dom["flops"],
              "kernel_source_sha256_16": kernel_source_hash(family)})
    return r


def run_projections(args, torch, ss, wl, ms, stream):
    """Independent projections at several M; weights rotate over distinct copies so
    that no launch finds its weights in the last-level cache (the tiny workload,
    a latency measurement, keeps one copy)."""
    from paper_2509_18344_amd import prepare, synth
    from paper_2509_18344_amd.workloads import Proj, weight_bytes
    projs = wl.projs
    if wl.key.startswith("qwen7b_mlp"):  # gate|up share x: one fused launch, as in the layer plan
        projs = (Proj("gate_up", 3584, 2 * 18944), Proj("down", 18944, 3584))
    per_copy = sum(weight_bytes(p.N, p.K, wl.bits, wl.group) for p in projs)
    copies = 1 if wl.key == "tiny" else max(1, int(math.ceil(args.rotate_gb * 1e9 / per_copy)))
    weights = []
    for c in range(copies):
        wc = []
        for pi, p in enumerate(projs):
            w = synth.weights_torch(p.N, p.K, 11, c, pi, device="cuda")
            wc.append(prepare.quantize_pack(w, wl.bits, wl.group))
            del w
        weights.append(wc)
    acts = {}
    for M in ms:
        for pi, p in enumerate(projs):
            x = synth.activations(M, p.K, 12, M, pi, outlier_frac=wl.outlier_frac).to("cuda")
            acts[(M, pi)] = (x, torch.empty((M, p.N), dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    launches = [(M, pi) for M in ms for pi in range(len(projs))]
    nl = len(launches)
    need = max(ss.subspec_qlinear_plan(M, projs[pi].N, projs[pi].K, wl.bits, wl.group,
                                       args.path)["workspace_bytes"] for (M, pi) in launches)
    ss.subspec_reserve(need)

    def proj_dict(s, li):
        M, pi = launches[li]
        wc = weights[(s * nl + li) % copies][pi]
        x, y = acts[(M, pi)]
        return {"x": x, "y": y, "qweight": wc["qweight"], "scales": wc["scales"],
                "zeros": wc["zeros"], "N": projs[pi].N, "K": projs[pi].K}

    graphs = []
    period = copies // math.gcd(copies, nl)
    use_graph = not args.eager and args.path == 0
    if use_graph:
        for s in range(period):  # one graph per M (the API captures one M at a time)
            gs = []
            for M in ms:
                lst = [proj_dict(s, li) for li in range(nl) if launches[li][0] == M]
                gs.append(ss.subspec_stack_capture(lst, wl.bits, wl.group, M, stream))
            graphs.append(gs)

    def step(s):
        if use_graph:
            for g in graphs[s % period]:
                ss.subspec_graph_launch(g, stream)
            return
        for li in range(nl):
            d = proj_dict(s, li)
            ss.subspec_qlinear_path(d["x"], d["qweight"], d["scales"], d["zeros"], wl.bits,
                                    wl.group, launches[li][0], d["N"], d["K"], d["y"],
                                    args.path, stream)

    total_ms, per_step, clocks = timed_steps(torch, stream, step, args.warmup, args.steps, not args.no_clocks)
    for gs in graphs:
        for g in gs:
            ss.subspec_graph_destroy(g)
    per = []
    for (M, pi) in launches:
        x, y = acts[(M, pi)]
        argsets = [{"x": x, "y": y, **{k: weights[c][pi][k] for k in ("qweight", "scales", "zeros")}}
                   for c in range(copies)]
        per.append(per_launch_graph(torch, ss, wl, M, projs[pi], argsets, stream))
    M0, p0 = launches[0][0], projs[launches[0][1]]
    host = host_us_per_call(ss, wl, M0, p0, dict(proj_dict(0, 0)), stream)
    return {"total_ms": total_ms, "per_step": per_step, "per_launch": per, "launches_per_step": nl,
            "copies": copies, "rotation_GB": round(copies * per_copy / 1e9, 2),
            "step_bytes": sum(weight_bytes(projs[pi].N, projs[pi].K, wl.bits, wl.group)
                              for (_, pi) in launches),
            "step_flops": sum(2.0 * M * projs[pi].N * projs[pi].K for (M, pi) in launches),
            "timing": "HIP graph replays" if use_graph else "eager launches",
            "host_us_per_call": host, "clocks": clocks}


def run_stack(args, torch, ss, wl, ms, stream):
    """All layers of a substitute stack, 4 launches per layer, one HIP graph per M;
    one step = one pass of the stack at every M."""
    from paper_2509_18344_amd import prepare, synth
    from paper_2509_18344_amd.workloads import fused_layer, weight_bytes
    plan = fused_layer(wl.projs)
    packed = []
    for l in range(wl.layers):
        w = synth.layer_weights(wl.projs, 20, l)
        parts = [[w["q"], w["k"], w["v"]], [w["o"]], [w["gate"], w["up"]], [w["down"]]]
        packed.append([prepare.fused(ps, wl.bits, wl.group) if len(ps) > 1 else
                       prepare.quantize_pack(ps[0], wl.bits, wl.group) for ps in parts])
        del w
    torch.cuda.synchronize()
    # every plan's workspace up front: no growth between the captures below
    ss.subspec_reserve(max(ss.subspec_qlinear_plan(M, p.N, p.K, wl.bits, wl.group)["workspace_bytes"]
                           for M in ms for p in plan))
    xs, ys, graphs = {}, {}, []
    for M in ms:
        xs[M] = [[synth.activations(M, p.K, 21, l, li, outlier_frac=wl.outlier_frac).to("cuda")
                  for li, p in enumerate(plan)] for l in range(wl.layers)]
        ys[M] = [[torch.empty((M, p.N), dtype=torch.bfloat16, device="cuda") for p in plan]
                 for _ in range(wl.layers)]
        launches = []
        for l in range(wl.layers):
            launches += prepare.layer_launches(packed[l], xs[M][l], ys[M][l])
        graphs.append(ss.subspec_stack_capture(launches, wl.bits, wl.group, M, stream))

    def step(s):
        for g in graphs:
            ss.subspec_graph_launch(g, stream)

    total_ms, per_step, clocks = timed_steps(torch, stream, step, args.warmup, args.steps, not args.no_clocks)
    for g in graphs:
        ss.subspec_graph_destroy(g)
    per = []
    for M in ms:
        for li, p in enumerate(plan):
            argsets = [{"x": xs[M][l][li], "y": ys[M][l][li],
                        **{k: packed[l][li][k] for k in ("qweight", "scales", "zeros")}}
                       for l in range(wl.layers)]
            per.append(per_launch_graph(torch, ss, wl, M, p, argsets, stream))
    # host cost of an eager call: the shortest launch of the stack (o at the smallest M)
    M0 = min(ms)
    a = {"x": xs[M0][0][1], "y": ys[M0][0][1], **{k: packed[0][1][k] for k in ("qweight", "scales", "zeros")}}
    host = host_us_per_call(ss, wl, M0, plan[1], a, stream)
    layer_bytes = sum(weight_bytes(p.N, p.K, wl.bits, wl.group) for p in plan)
    del packed, xs, ys
    return {"total_ms": total_ms, "per_step": per_step, "per_launch": per,
            "launches_per_step": 4 * wl.layers * len(ms),
            "copies": 1, "rotation_GB": round(layer_bytes * wl.layers / 1e9, 2),
            "step_bytes": layer_bytes * wl.layers * len(ms),
            "step_flops": sum(wl.layers * 2.0 * M * p.N * p.K for M in ms for p in plan),
            "timing": "HIP graph replays", "host_us_per_call": host, "clocks": clocks}


def run_qlinear(args, torch, ss, key, ms=None):
    """One qlinear workload: the step's rate, its spread, the per-launch table and
    the dominant launch's roofline."""
    from paper_2509_18344_amd.workloads import WORKLOADS
    wl = WORKLOADS[key]
    ms = ms or wl.ms
    stream = torch.cuda.Stream()
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        r = run_stack(args, torch, ss, wl, ms, stream) if wl.layers > 1 else \
            run_projections(args, torch, ss, wl, ms, stream)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    ms_per_step = r["total_ms"] / args.steps
    value = r["step_bytes"] / (ms_per_step * 1e-3) / 1e9
    per = r["per_launch"]
    # dominant launch: the largest share of the step's kernel time
    dom = max(per, key=lambda d: d["median_us"])
    return {
        "value": round(value, 1), "unit": "GB/s", "ms_per_step": round(ms_per_step, 4),
        "step_ms": {"median": pct(r["per_step"], 50), "p10": pct(r["per_step"], 10),
                    "p90": pct(r["per_step"], 90)},
        "config": {"workload": f"{key}: {wl.description}", "bits": wl.bits, "group": wl.group,
                   "ms": list(ms), "layers": wl.layers, "launches_per_step": r["launches_per_step"],
                   "weight_bytes_per_step": r["step_bytes"], "distinct_weight_copies": r["copies"],
                   "rotation_GB": r["rotation_GB"], "timing": r["timing"],
                   "hbm_fraction_of_8TBs": round(value / HBM_PEAK_GBS, 4),
                   "TFLOPs": round(r["step_flops"] / (ms_per_step * 1e-3) / 1e12, 2)},
        "roofline": roofline_of(dom),
        "gpu_clocks_during_steps": r["clocks"],
        "host_us_per_call": r["host_us_per_call"],
        "per_launch": [{k: v for k, v in d.items() if k not in ("alg_bytes", "flops")} for d in per],
        "wall_s": round(time.perf_counter() - t0, 2),
    }


HEADLINE = "qwen32b_stack"
EXTRA_CONFIGS = ("tiny", "qwen7b_mlp", "qwen7b_mlp_draft", "qwen7b_stack", "qwen32b_2bit")


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, family=WORKLOAD_FAMILY.get(args.workload, "qlinear"))
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_sq:
        from paper_2509_18344_amd.workloads import WORKLOADS
        key = HEADLINE if args.workload == "suite" else args.workload
        ms = tuple(int(m) for m in args.ms.split(",")) if args.ms else WORKLOADS[key].ms
        summarize_sq(*args.summarize_sq, key, ms)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2509_18344_amd as ss

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
    if args.workload == "tree_expand":
        run_tree(args, torch, ss)
        return
    if args.workload == "tree_attn":
        run_attn(args, torch, ss)
        return
    if args.workload == "prefetch":
        run_prefetch(args, torch, ss)
        return
    if args.workload == "hqq":
        run_hqq(args, torch, ss)
        return
    suite = args.workload == "suite"
    key = HEADLINE if suite else args.workload
    ms = tuple(int(m) for m in args.ms.split(",")) if args.ms else None
    t_all = time.perf_counter()
    head = run_qlinear(args, torch, ss, key, ms)
    extras = {}
    if suite:
        for k in EXTRA_CONFIGS:
            extras[k] = run_qlinear(args, torch, ss, k)
    out = {
        "metric": "effective weight GB/s and % HBM roofline of low-bit qlinear at draft-tree M",
        "value": head["value"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: N(0,0.02) fp32 weights min/max-quantized on the GPU, N(0,1) bf16 "
                "activations, seeded",
        "config": head["config"],
        "roofline": head["roofline"],
        "step_ms": head["step_ms"],
        "gpu_clocks_during_steps": head["gpu_clocks_during_steps"],
        "host_us_per_call": head["host_us_per_call"],
        "per_launch": head["per_launch"],
    }
    if suite:
        out["configs"] = extras
    out["hbm_context"] = copy_rate(torch, torch.cuda.Stream())
    if not args.no_cpu_baseline:
        from paper_2509_18344_amd.workloads import WORKLOADS
        wl = WORKLOADS[key]
        out["cpu_baseline"] = cpu_baseline(wl, ms or wl.ms)
    out["wall_s"] = round(time.perf_counter() - t_all, 2)
    line = json.dumps(out)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)


# --- draft-tree expansion (Sec. 4.2, App. D) --------------------------------------

TREE_V = 152064      # Qwen2.5 vocabulary
TREE_K = 6           # leaves kept per draft pass (Sec. 5.1)
TREE_T = 0.2         # draft temperature for greedy decoding (Sec. 4.2, App. D)


def tree_cpu_baseline(rs, min_seconds=10.0):
    """Time the fp64 oracle on the same expansion inputs until `min_seconds` pass."""
    import oracle
    rng = np.random.default_rng(3)
    cases = [(oracle.bf16_round_bits(rng.normal(0, 3, (R, TREE_V)).astype(np.float32)),
              rng.uniform(-12, 0, R)) for R in rs]
    steps = 0
    t0 = time.perf_counter()
    while True:
        for bits, parent in cases:
            oracle.tree_expand(bits, parent, TREE_T, TREE_K)
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    nbytes = steps * sum(2 * R * TREE_V for R in rs)
    return {"value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "seconds": round(dt, 3),
            "sample": f"{steps} pass(es) of the expansion at R in {list(rs)}, V={TREE_V}, "
                      f"k={TREE_K}, T={TREE_T} (NumPy fp64, one thread)"}


def run_tree(args, torch, ss):
    """One step = one expansion per R (leaves of the tree) over V = 152064 bf16 logits,
    logits rotating over >= --rotate-gb of distinct copies (they sit in HBM, not in the
    last-level cache, when a call starts)."""
    rs = tuple(int(m) for m in args.ms.split(",")) if args.ms else (TREE_K,)
    stream = torch.cuda.Stream()
    rng = np.random.default_rng(3)
    sets = []
    for R in rs:
        per = 2 * R * TREE_V
        copies = max(2, int(math.ceil(args.rotate_gb * 1e9 / per)))
        base = torch.from_numpy(rng.normal(0, 3, (R, TREE_V)).astype(np.float32)).to("cuda").bfloat16()
        lg = [base.roll(c, dims=1).contiguous() for c in range(copies)]
        parent = torch.from_numpy(rng.uniform(-12, 0, R).astype(np.float32)).to("cuda")
        out = (torch.empty(TREE_K, dtype=torch.int32, device="cuda"),
               torch.empty(TREE_K, dtype=torch.int32, device="cuda"),
               torch.empty(TREE_K, dtype=torch.float32, device="cuda"))
        sets.append((R, lg, parent, out))
    ss.subspec_reserve(max(ss.subspec_tree_workspace_bytes(R, TREE_V, TREE_K) for R in rs))
    torch.cuda.synchronize()

    def call(R, lg, parent, out, s):
        ss.subspec_tree_expand(lg[s % len(lg)], parent, R, TREE_V, TREE_T, TREE_K, out[0], out[1],
                               out[2], stream)

    def step(s):
        for (R, lg, parent, out) in sets:
            call(R, lg, parent, out, s)

    with torch.cuda.stream(stream):
        total_ms = timed(torch, stream, step, args.warmup, args.steps)
        # Per R: a burst of back-to-back launches between two events on the launch
        # stream (one event pair per launch would add the events' own cost).
        per_launch = []
        for (R, lg, parent, out) in sets:
            reps = max(args.per_launch_reps, len(lg))
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for r in range(reps):
                call(R, lg, parent, out, r)
            e1.record(stream)
            torch.cuda.synchronize()
            avg_us = e0.elapsed_time(e1) * 1e3 / reps
            nbytes = 2 * R * TREE_V + 4 * R + 12 * TREE_K
            chunks, _, list_len = ss.subspec_tree_plan(R, TREE_V, TREE_K)
            key = f"k_tree_expand<{list_len}> grid={R * chunks * 256} wg=256"
            per_launch.append({"R": R, "V": TREE_V, "k": TREE_K, "key": key,
                               "avg_us": round(avg_us, 2), "launches_timed": reps,
                               "alg_bytes": nbytes,
                               "alg_GBs": round(nbytes / (avg_us * 1e-6) / 1e9, 1)})
    ms_per_step = total_ms / args.steps
    step_bytes = sum(2 * R * TREE_V for R in rs)
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    dom = max(per_launch, key=lambda d: d["avg_us"])
    out = {
        "metric": "logits GB/s of the draft-tree expansion step (sharpened log-softmax, parent "
                  "scores, global top-k)",
        "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic: N(0,3) bf16 logits, U(-12,0) parent scores, seeded",
        "config": {"workload": f"draft-tree expansion, V={TREE_V}, k={TREE_K}, T={TREE_T}",
                   "rows": list(rs), "launches_per_step": len(rs), "timing": "eager launches"},
        "roofline": {"bound": "hbm", "achieved": dom["alg_GBs"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(dom["alg_GBs"] / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(dom["key"], "tree"), "kernel": dom["key"],
                     "avg_us": dom["avg_us"], "alg_bytes_per_launch": dom["alg_bytes"],
                     "kernel_source_sha256_16": kernel_source_hash("tree")},
        "per_launch": per_launch,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = tree_cpu_baseline(rs)
    line = json.dumps(out)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)




# One draft layer's tree attention, Qwen2.5-7B heads, at the last pass of a depth-48
# tree with k = 6 (Sec. 5.1): 47 earlier passes x 6 tokens = 282 tree tokens.
ATTN_CFG = {"M": 6, "Hq": 28, "Hkv": 4, "P": 2048, "T": 282}


def attn_bytes(M, Hq, Hkv, P, T):
    """Algorithmic bytes of one call: every visible-or-not key and value row of the
    head's range read once (bf16), q and the output, the appended rows, the mask."""
    L = P + T + M
    W = (T + M + 31) // 32
    return 2 * Hkv * L * 128 * 2 + 2 * M * Hq * 128 * 2 + 2 * M * Hkv * 128 * 2 + 4 * M * W


def attn_cpu_baseline(min_seconds=10.0):
    """Time the fp64 oracle on the bench configuration until `min_seconds` pass."""
    import oracle
    from paper_2509_18344_amd import synth
    c = ATTN_CFG
    S = c["P"] + c["T"] + c["M"]
    x = synth.tree_attn_inputs(c["M"], c["Hq"], c["Hkv"], 128, S, 5)
    mask = synth.tree_levels_mask(c["T"], 6, c["M"], 5)
    steps = 0
    t0 = time.perf_counter()
    while True:
        oracle.tree_attention(x["q"], x["k_cache"], x["v_cache"], c["P"], c["T"], x["k_new"], x["v_new"],
                              mask, 1.0 / math.sqrt(128))
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    nbytes = steps * attn_bytes(**c)
    return {"value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "seconds": round(dt, 3),
            "sample": f"{steps} call(s) of the tree attention at {c} (NumPy fp64, one thread)"}


def run_attn(args, torch, ss):
    """One step = one call (two kernels) on one layer's cache; the caches rotate over
    >= --rotate-gb of distinct copies so that they come from HBM."""
    from paper_2509_18344_amd import synth
    c = ATTN_CFG
    M, Hq, Hkv, P, T = c["M"], c["Hq"], c["Hkv"], c["P"], c["T"]
    S = P + T + M
    x = synth.tree_attn_inputs(M, Hq, Hkv, 128, S, 5)
    mask = synth.tree_levels_mask(T, 6, M, 5)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda")
    per = 2 * Hkv * S * 128 * 2
    copies = max(2, int(math.ceil(args.rotate_gb * 1e9 / per)))
    kc0, vc0 = dev(x["k_cache"]), dev(x["v_cache"])
    caches = [(kc0.clone(), vc0.clone()) for _ in range(copies)]
    q, kn, vn = dev(x["q"]), dev(x["k_new"]), dev(x["v_new"])
    mk = torch.from_numpy(mask.view(np.int32)).to("cuda")
    out = torch.empty((M, Hq, 128), dtype=torch.int16, device="cuda")
    scale = 1.0 / math.sqrt(128)
    ss.subspec_reserve(ss.subspec_tree_attention_workspace_bytes(M, Hq, Hkv, P, T))
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()

    def step(s):
        kc, vc = caches[s % copies]
        ss.subspec_tree_attention(q, kc, vc, kn, vn, mk, M, Hq, Hkv, S, P, T, scale, out, stream)

    with torch.cuda.stream(stream):
        total_ms = timed(torch, stream, step, args.warmup, args.steps)
        reps = max(args.per_launch_reps, copies)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for r in range(reps):
            step(r)
        e1.record(stream)
        torch.cuda.synchronize()
        avg_us = e0.elapsed_time(e1) * 1e3 / reps
    ms_per_step = total_ms / args.steps
    nbytes = attn_bytes(**c)
    splits, tps = ss.subspec_tree_attention_plan(M, Hq, Hkv, P, T)
    qt = -(-(Hq // Hkv * M) // 16)
    # keys name the whole grid (k_attn_partial: splits x Hkv workgroups)
    keys = [f"k_attn_partial<{qt}> grid={splits * 256 * Hkv} wg=256", f"k_attn_combine grid={M * Hq * 128} wg=128"]
    tr = [measured_traffic(k, "attn") for k in keys]
    achieved = nbytes / (avg_us * 1e-6) / 1e9
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    out_line = {
        "metric": "KV-cache GB/s of the draft model's tree attention (one layer, one draft pass)",
        "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: N(0,1) bf16 q, keys, values; random depth-48 tree mask; seeded",
        "config": {"workload": f"tree attention, Qwen2.5-7B heads (Hq=28, Hkv=4, D=128), M={M} new tree "
                               f"tokens, P={P} committed, T={T} earlier tree tokens",
                   "splits": splits, "tiles_per_split": tps, "cache_copies": copies,
                   "timing": "eager calls (two kernels each)"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None if None in tr else sum(tr),
                     "kernel": " + ".join(keys) + " (one call)", "avg_us": round(avg_us, 2),
                     "calls_timed": reps, "alg_bytes_per_launch": nbytes,
                     "kernel_source_sha256_16": kernel_source_hash("attn")},
    }
    if not args.no_cpu_baseline:
        out_line["cpu_baseline"] = attn_cpu_baseline()
    line = json.dumps(out_line)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)



# Verification pass over offloaded target layers (Sec. 4.3, App. E): Qwen2.5-7B
# projections in bf16, 289 tokens (a depth-48 tree of k = 6 plus the root).
PF_PROJS = (("q", 3584, 3584), ("k", 512, 3584), ("v", 512, 3584), ("o", 3584, 3584),
            ("gate", 18944, 3584), ("up", 18944, 3584), ("down", 3584, 18944))
PF_TOKENS = 289
PF_LAYERS = 6          # offloaded layers per timed pass
PF_DISTINCT = 2        # distinct pinned host copies of a layer, cycled
PCIE5_X16_GBS = 64.0   # host link of the MI355X platform, one direction (PCIe 5.0 x16)
PF_SLOTS = 3           # device slots of the largest projection
PF_SLOT_CHOICES = (2, 3, 4)


def run_prefetch(args, torch, ss):
    """One step = one verification pass over PF_LAYERS offloaded layers: every
    projection's bf16 weights copied from pinned host memory into a reused device slot
    (2 slots) while the previous projection's GEMM runs."""

    class DevView:
        def __init__(self, ptr, n, k):
            self.__cuda_array_interface__ = {"shape": (n, k), "typestr": "<f2", "data": (ptr, False),
                                             "version": 2}

    def as_bf16(ptr, n, k):
        return torch.as_tensor(DevView(ptr, n, k), device="cuda").view(torch.bfloat16)

    g = torch.Generator().manual_seed(11)
    host = [[(torch.randn(n, k, generator=g) * 0.02).to(torch.bfloat16).pin_memory() for _, n, k in PF_PROJS]
            for _ in range(PF_DISTINCT)]
    dev_w = [(torch.randn(n, k, device="cuda") * 0.02).to(torch.bfloat16) for _, n, k in PF_PROJS]
    xs = {k: torch.randn(PF_TOKENS, k, device="cuda").to(torch.bfloat16) for k in {k for _, _, k in PF_PROJS}}
    order = [(layer, j) for layer in range(PF_LAYERS) for j in range(len(PF_PROJS))]
    nbytes = sum(2 * n * k for _, n, k in PF_PROJS) * PF_LAYERS
    flops = sum(2 * PF_TOKENS * n * k for _, n, k in PF_PROJS) * PF_LAYERS
    slot = max(2 * n * k for _, n, k in PF_PROJS)
    pfs = {n: ss.Prefetcher(slot, n) for n in PF_SLOT_CHOICES}
    comp = torch.cuda.Stream()
    copy_s = torch.cuda.Stream()
    ybuf = {n: torch.empty(PF_TOKENS, n, device="cuda", dtype=torch.bfloat16) for _, n, _ in PF_PROJS}
    staging = torch.empty(slot // 2, device="cuda", dtype=torch.bfloat16)

    def gemm(j, w):
        torch.matmul(xs[PF_PROJS[j][2]], w.t(), out=ybuf[PF_PROJS[j][1]])

    def pass_pipelined(nslots=PF_SLOTS):
        # up to nslots - 1 tensors ahead of the one being computed; the copy into a
        # slot waits for the GEMM that used it nslots tensors earlier
        pf = pfs[nslots]
        ahead = nslots - 1
        tickets = [pf.begin(host[order[i][0] % PF_DISTINCT][order[i][1]]) for i in range(min(ahead, len(order)))]
        with torch.cuda.stream(comp):
            for i, (layer, j) in enumerate(order):
                _, n, k = PF_PROJS[j]
                ptr = pf.acquire(tickets[i], comp)
                gemm(j, as_bf16(ptr, n, k))
                pf.release(tickets[i], comp)
                if i + ahead < len(order):
                    nl, nj = order[i + ahead]
                    tickets.append(pf.begin(host[nl % PF_DISTINCT][nj]))

    def pass_copies():
        with torch.cuda.stream(copy_s):
            for layer, j in order:
                h = host[layer % PF_DISTINCT][j]
                staging[:h.numel()].view(h.shape).copy_(h, non_blocking=True)

    def pass_gemms():
        with torch.cuda.stream(comp):
            for layer, j in order:
                gemm(j, dev_w[j])

    def pass_serial():
        with torch.cuda.stream(comp):
            for layer, j in order:
                h = host[layer % PF_DISTINCT][j]
                w = staging[:h.numel()].view(h.shape)
                w.copy_(h, non_blocking=True)
                gemm(j, w)

    def timed_pass(fn, reps):
        fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            fn()
            torch.cuda.synchronize()
        return (time.perf_counter() - t0) / reps

    for _ in range(max(1, args.warmup)):
        pass_pipelined()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        # a verification pass ends on the host: the accepted tokens decide the next
        # speculation, so each step synchronises
        pass_pipelined()
        torch.cuda.synchronize()
    t_pipe = (time.perf_counter() - t0) / args.steps
    # the comparison passes, interleaved over three rounds (the host link's rate drifts
    # by a few per cent from one second to the next); medians
    variants = {"copies_only": pass_copies, "gemms_only": pass_gemms, "copy_then_gemm": pass_serial}
    variants.update({f"slots_{n}": (lambda n=n: pass_pipelined(n)) for n in PF_SLOT_CHOICES})
    samples = collections.defaultdict(list)
    for _ in range(3):
        for name, fn in variants.items():
            samples[name].append(timed_pass(fn, 2))
    med = {name: float(np.median(v)) for name, v in samples.items()}
    t_copy, t_gemm, t_serial = med["copies_only"], med["gemms_only"], med["copy_then_gemm"]
    t_slots = {n: med[f"slots_{n}"] for n in PF_SLOT_CHOICES}
    for p_ in pfs.values():
        p_.close()
    value = nbytes / t_pipe / 1e9
    copy_gbs = nbytes / t_copy / 1e9
    out = {
        "metric": "weight GB/s delivered to and consumed by the verification pass over offloaded layers "
                  "(cross-layer asynchronous prefetch)",
        "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(t_pipe * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: N(0,0.02) bf16 weights in pinned host memory, N(0,1) bf16 activations, seeded",
        "config": {"workload": f"verification pass, Qwen2.5-7B projections, {PF_LAYERS} offloaded layers "
                               f"({PF_DISTINCT} distinct host copies), {PF_TOKENS} tokens, {PF_SLOTS} device slots",
                   "bytes_per_pass": nbytes, "gflop_per_pass": round(flops / 1e9, 1),
                   "slot_bytes": slot, "timing": "host clock around whole passes, each ending in a synchronisation"},
        "roofline": {"bound": "host link (PCIe 5.0 x16, one direction)", "achieved": round(value, 2),
                     "peak": PCIE5_X16_GBS, "unit": "GB/s", "frac": round(value / PCIE5_X16_GBS, 4),
                     "traffic": None, "kernel": "host-to-device copies on the prefetcher's copy stream"},
        "parts_ms": {"pipelined_timed_steps": round(t_pipe * 1e3, 3), "copies_only": round(t_copy * 1e3, 3),
                     "gemms_only": round(t_gemm * 1e3, 3), "copy_then_gemm": round(t_serial * 1e3, 3),
                     "pipelined_by_slots": {str(n): round(t * 1e3, 3) for n, t in t_slots.items()}},
        "copy_only_GBs": round(copy_gbs, 2),
        "gemm_hidden_frac": round((t_serial - t_slots[PF_SLOTS]) / t_gemm, 3) if t_gemm > 0 else None,
    }
    line = json.dumps(out)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)



def hqq_cpu_baseline(min_seconds=10.0):
    """The fp64 oracle's HQQ quantizer on 1024 x 3584 weights, repeated for min_seconds."""
    import oracle
    from paper_2509_18344_amd import synth
    w = synth.weights_np(1024, 3584, 51)
    steps = 0
    t0 = time.perf_counter()
    while True:
        oracle.quantize_hqq(w, 4, 64)
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    n = steps * w.size
    return {"value": round(n / dt / 1e6, 3), "unit": "M weights/s", "cores": 1, "kind": "oracle",
            "seconds": round(dt, 3),
            "sample": f"{steps} x 1024 x 3584 fp32 weights, 4-bit g64 (NumPy fp64, one thread)"}


def run_hqq(args, torch, ss):
    """One step = quantizing the 7 projections of one Qwen2.5-7B layer (233 M fp32
    weights, on the device) to 4 bits, groups of 64, with the optimised zero."""
    from paper_2509_18344_amd import synth
    bits, group = 4, 64
    ws, outs = [], []
    for i, (_, n, k) in enumerate(PF_PROJS):
        w = synth.weights_torch(n, k, 61, i)
        ws.append(w)
        outs.append((torch.empty((n, k), dtype=torch.uint8, device="cuda"),
                     torch.empty((k // group, n), dtype=torch.float16, device="cuda"),
                     torch.empty((k // group, n), dtype=torch.float16, device="cuda")))
    stream = torch.cuda.Stream()
    n_weights = sum(n * k for _, n, k in PF_PROJS)

    def step_with(fn):
        def step(_s):
            for (name, n, k), w, (c, sc, zr) in zip(PF_PROJS, ws, outs):
                fn(w, bits, group, n, k, c, sc, zr, stream)
        return step

    with torch.cuda.stream(stream):
        total_ms = timed(torch, stream, step_with(ss.subspec_quantize_hqq), args.warmup, args.steps)
        mm_ms = timed(torch, stream, step_with(ss.subspec_quantize), 1, max(3, args.steps))
    ms = total_ms / args.steps
    mm = mm_ms / max(3, args.steps)
    nbytes = n_weights * (4 + 1) + 2 * 2 * n_weights // group  # fp32 in, codes, fp16 scale and zero out
    gbs = nbytes / (ms * 1e-3) / 1e9
    out = {
        "metric": "weights quantized per second with the HQQ-style optimised zero-point (one Qwen2.5-7B layer, "
                  "4-bit, groups of 64)",
        "value": round(n_weights / (ms * 1e-3) / 1e9, 3), "unit": "G weights/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic: N(0,0.02) fp32 weights generated on the device, seeded",
        "config": {"workload": "HQQ-style quantization of the 7 projections of one Qwen2.5-7B layer, 4-bit g64",
                   "weights": n_weights, "minmax_ms_per_step": round(mm, 3), "timing": "eager launches"},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "k_quantize_hqq<64> (7 launches per step)", "alg_bytes_per_step": nbytes,
                     "note": "float64 arithmetic (a power per weight and round) bounds it, not HBM"},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = hqq_cpu_baseline()
    line = json.dumps(out)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(line + "\n")
    print(line, flush=True)


if __name__ == "__main__":
    main()
