"""Benchmark: ResNet-50-shaped CNN inference (bf16, batch 32) on one MI355X
through the routine-selection library, plus batch 1, the fixed-routine paths,
per-layer roofline fractions and the CPU oracle baseline.

A step is one inference of the whole net over one batch of synthetic input
with the DPRS-selected routine path (the tuning -- profiling and selection --
runs once before the timed region and is reported as tuning_s).  Prints one
JSON line.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "img/s ResNet-50-shape bs1/32 bf16; conv MFMA util %; DP-path vs best fixed"
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0
LAYOUTS = ("NCHW", "NHWC", "NC8HW8")
ALGOS = ("direct", "igemm", "winograd")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def layer_kind(spec, i):
    """Layer type of layer i (1-based), convolutions by filter size and grouping."""
    layer = spec["layers"][i - 1]
    if layer["type"] == "conv":
        if layer["groups"] > 1:
            return "dwconv"
        return "conv%dx%d" % (layer["r"], layer["s"])
    return layer["type"]


def layer_work(spec, g, i, routine):
    """(category, flops, algorithmic bytes) of layer i (1-based) for a routine.
    The bytes follow the formula input + filters + output (+ residual); see
    bytes_needed for the bytes a strided 1x1 convolution actually reads."""
    layer = spec["layers"][i - 1]
    es = 4 if spec["dtype"] == "f32" else 2
    n, k, p, q = g.layer_shape(i)
    ins = [g.layer_shape(j) for j in layer["in"]]
    _, c, h, w = ins[0]
    t = layer["type"]
    if t == "conv":
        r, s, grp = layer["r"], layer["s"], layer["groups"]
        wbytes = k * (c // grp) * r * s * es
        byt = es * (n * c * h * w + n * k * p * q) + wbytes + 4 * k
        flops = 2 * n * k * c * r * s * p * q
        if layer.get("proj"):  # the shortcut (whole, by the formula) and its 1x1 weights
            _, c2, h2, w2 = ins[1]
            byt += es * (n * c2 * h2 * w2 + k * c2)
            flops += 2 * n * k * c2 * p * q
        elif len(layer["in"]) > 1:  # residual read in the epilogue
            byt += es * n * k * p * q
        if grp > 1:
            return "dwconv", 2 * n * k * r * s * p * q, byt
        if routine["algo"] == 2:  # Winograd: the MFMA work is the 16 tile GEMMs
            tiles = n * ((h + 1) // 2) * ((w + 1) // 2)
            flops = 2 * 16 * k * c * tiles
        cat = "conv_stem" if c <= 4 else "conv%dx%d" % (r, s)
        return cat, flops, byt
    if t == "add":
        return "add", n * k * p * q, 3 * es * n * k * p * q
    if t == "maxpool":
        return "maxpool", 0, es * (n * c * h * w + n * k * p * q)
    if t == "gap":
        return "gap", n * c * h * w, es * (n * c * h * w + n * k)
    if t == "fc":
        return "fc", 2 * n * c * k, es * (n * c + c * k + n * k)
    return t, 0, 0


def bytes_needed(spec, g, i, routine):
    """Algorithmic bytes with the input counted as the pixels the layer
    reads: a 1x1 convolution without padding at stride s reads one input
    pixel in s x s (the formula of layer_work counts the whole input)."""
    _, _, byt = layer_work(spec, g, i, routine)
    layer = spec["layers"][i - 1]
    es = 4 if spec["dtype"] == "f32" else 2
    if layer["type"] == "conv" and layer["r"] == 1 and layer["s"] == 1 and layer["pad"] == 0 and layer["stride"] > 1:
        n, k, p, q = g.layer_shape(i)
        _, c, h, w = g.layer_shape(layer["in"][0])
        byt -= es * n * c * (h * w - p * q)
    if layer.get("proj") and layer["proj"]["stride"] > 1:  # a strided shortcut: the pixels read
        n, k, p, q = g.layer_shape(i)
        _, c2, h2, w2 = g.layer_shape(layer["in"][1])
        byt -= es * n * c2 * (h2 * w2 - p * q)
    return byt


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_resnet50_bs32_bf16.json")
KDIR = os.path.join(ROOT, "paper_2110_06037_amd", "csrc", "kernels")
# sources each dominant kernel is built from (its traffic summary goes stale
# when any of them changes)
KERNEL_SOURCES = {
    "add_kernel": ("misc.hip", "kcommon.hpp"),
    "igemm_dma_kernel": ("igemm.hpp", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
    "igemm_kernel": ("igemm.hpp", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
    "conv3x3_patch_kernel": ("conv_patch.hip", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
    "conv1x1_stream_kernel": ("conv1x1_stream.hip", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
    "conv_smallc_kernel": ("conv_smallc.hip", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
    "dw3x3_kernel": ("dwconv.hip", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
    "wino_fused_kernel": ("wino_fused.hip", "wino.hpp", "gemm_common.hpp", "kcommon.hpp", "launch.hpp"),
}
ALL_KERNEL_SOURCES = ("conv.hip", "conv_igemm_bf16.hip", "conv_igemm_f16.hip", "conv1x1_stream.hip", "conv_patch.hip",
                      "conv_smallc.hip", "convert.hip", "dwconv.hip", "fc.hip", "igemm.hpp", "misc.hip",
                      "wino.hpp", "wino_fused.hip",
                      "gemm_common.hpp",
                      "kcommon.hpp", "launch.hpp")


def kernel_source_hash(ksub=None):
    """Hash of the sources a kernel (by a part of its symbol) is built from."""
    import hashlib
    h = hashlib.sha256()
    files = next((v for k, v in KERNEL_SOURCES.items() if ksub and k in ksub), ALL_KERNEL_SOURCES)
    for f in files:
        with open(os.path.join(KDIR, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _traffic_summary(path=TRAFFIC_FILE):
    try:
        with open(path) as f:
            return json.load(f)
    except (OSError, ValueError):
        return {}


def traffic_for_layers(layers, routine, summary=None, workload=None):
    """HBM bytes per launch of `routine` averaged over `layers` from the
    committed per-layer PMC summary: only when the summary was taken on this
    workload and holds every one of those layers run by this same routine,
    with kernel sources unchanged since the counters were taken; else
    (None, reason)."""
    summary = _traffic_summary() if summary is None else summary
    if workload is not None and summary.get("workload") != workload:
        return None, f"no counter summary for workload {workload}"
    by_layer = {e["layer"]: e for e in summary.get("layers", [])}
    tot = 0
    for i in layers:
        e = by_layer.get(i)
        if e is None or e.get("routine") != routine:
            return None, f"layer {i} was profiled with another routine (or not at all)"
        if e.get("source_hash") != kernel_source_hash(e.get("kernels", [""])[0]):
            return None, f"the kernel sources of layer {i} changed since its counters were taken"
        if e.get("bytes") is None:
            return None, "no calibration"
        tot += e["bytes"]
    return tot // max(1, len(layers)), None


def _pmc_rows(d):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows += list(csv.DictReader(open(f)))
    return rows


def summarize_pmc(fetch_dir, write_dir, pass_file, out, calib_mib):
    """Per-layer HBM traffic of a pinned path from two rocprofv3 --pmc runs of
    `bench.py --pmc-pass` (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch):
    the library's kernels (namespace sn::k) of the run are the warm-up and
    timed steps in order, each step's launches attributed to layers by the
    plan's launch list; counters of the timed steps are averaged per launch,
    summed per layer and scaled by what each counter reads for a device copy
    of known size."""
    with open(pass_file) as f:
        info = json.load(f)
    launch_layer = info["launch_layers"]
    L = len(launch_layer)
    per_counter = {}
    calib = {}
    kernels = None
    for name, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = [r for r in _pmc_rows(d) if r["Counter_Name"] == name]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        ours = [r for r in rows if r["Kernel_Name"].startswith("_ZN2sn1k") or "sn::k::" in r["Kernel_Name"]]
        steps = len(ours) // L
        if steps * L != len(ours) or steps < info["warmup"] + info["steps"]:
            raise SystemExit(f"{name}: {len(ours)} library dispatches, not a whole number of {L}-launch steps")
        copy = [float(r["Counter_Value"]) for r in rows if "copy" in r["Kernel_Name"].lower()]
        calib[name] = calib_mib * 1024.0 / max(copy) if copy and calib_mib else None
        timed = ours[(steps - info["steps"]) * L:]
        per_launch = [0.0] * L
        for k, r in enumerate(timed):
            per_launch[k % L] += float(r["Counter_Value"]) / info["steps"]
        per_counter[name] = per_launch
        kernels = [timed[k]["Kernel_Name"] for k in range(L)]
    layers = []
    for i, rname in enumerate(info["routines"]):
        idx = [k for k in range(L) if launch_layer[k] == i]
        if not idx:
            continue
        kib_f = sum(per_counter["FETCH_SIZE"][k] for k in idx)
        kib_w = sum(per_counter["WRITE_SIZE"][k] for k in idx)
        ks = [kernels[k] for k in idx]
        ok = calib["FETCH_SIZE"] and calib["WRITE_SIZE"]
        layers.append({"layer": i, "routine": rname, "launches": len(idx), "kernels": ks,
                       "fetch_kib": round(kib_f, 1), "write_kib": round(kib_w, 1),
                       "bytes": int((kib_f * calib["FETCH_SIZE"] + kib_w * calib["WRITE_SIZE"]) * 1024) if ok else None,
                       "source_hash": kernel_source_hash(ks[0])})
    res = {"workload": info["workload"], "steps": info["steps"], "calibration":
           {"copy_mib": calib_mib, "fetch_scale": calib["FETCH_SIZE"], "write_scale": calib["WRITE_SIZE"]},
           "layers": layers}
    with open(out, "w") as fh:
        json.dump(res, fh, indent=1)
    print(json.dumps({"layers": len(layers), "calibration": res["calibration"]}))


def summarize_trace(trace_dir, pass_file, out):
    """Per-layer kernel time of a pinned path from a rocprofv3 --kernel-trace
    run of `bench.py --pmc-pass`: the library's dispatches are the warm-up and
    timed steps in order, attributed to layers by the plan's launch list;
    each launch's duration (end - start timestamp) is averaged over the timed
    steps and summed per layer.  Adds the layer's minimum bytes (input +
    filters + output, + residual; strided 1x1 layers count the pixels they
    read) and the GB/s they give over that time."""
    import csv
    import glob
    with open(pass_file) as f:
        info = json.load(f)
    launch_layer = info["launch_layers"]
    L = len(launch_layer)
    rows = []
    for fn in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        rows += list(csv.DictReader(open(fn)))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    ours = [r for r in rows if r["Kernel_Name"].startswith("_ZN2sn1k") or "sn::k::" in r["Kernel_Name"]]
    steps = len(ours) // L
    if steps * L != len(ours) or steps < info["warmup"] + info["steps"]:
        raise SystemExit(f"trace: {len(ours)} library dispatches, not a whole number of {L}-launch steps")
    timed = ours[(steps - info["steps"]) * L:]
    dur = [0.0] * L
    for k, r in enumerate(timed):
        dur[k % L] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / info["steps"]
    need = info.get("bytes_needed", {})
    layers = []
    for i, rname in enumerate(info["routines"]):
        idx = [k for k in range(L) if launch_layer[k] == i]
        if not idx:
            continue
        ns = sum(dur[k] for k in idx)
        b = need.get(str(i))
        layers.append({"layer": i, "routine": rname, "launches": len(idx),
                       "kernels": [timed[k]["Kernel_Name"] for k in idx],
                       "kernel_ns": [round(dur[k], 1) for k in idx], "us": round(ns / 1e3, 3),
                       "bytes_needed": b, "gbs": round(b / ns, 1) if b and ns else None})
    res = {"workload": info["workload"], "steps": info["steps"], "layers": layers,
           "step_kernel_us": round(sum(dur) / 1e3, 2)}
    with open(out, "w") as fh:
        json.dump(res, fh, indent=1)
    print(json.dumps({"layers": len(layers), "step_kernel_us": res["step_kernel_us"]}))


def _mask_name(m):
    return "+".join(n for i, n in enumerate(("NCHW", "NHWC", "NC8HW8")) if m >> i & 1)


def _nets():
    from workloads import mobilenet_v2, resnet18, resnet50, vgg16
    return {"resnet50": resnet50, "resnet18": resnet18, "mobilenetv2": mobilenet_v2, "vgg16": vgg16}


NETS = {"resnet50": None, "resnet18": None, "mobilenetv2": None, "vgg16": None}


def sweep(args):
    """Cost table of the 3x3 stride-1 sweep (C = K in 64..512 at 56..7 pixels, batch 32):
    every routine of the conv layer and every converter of its input, as profiled."""
    from paper_2110_06037_amd import build_from_spec
    from workloads import CONV_SWEEP_SHAPES, conv_sweep, generate
    dt = args.dtype
    out = []
    for c, hw in CONV_SWEEP_SHAPES:
        spec = conv_sweep(c, hw, args.batch, dt)
        g = build_from_spec(spec, generate(spec), device=0)
        g.profile(warmup=5, reps=args.profile_reps)
        costs = g.costs()
        flops = 2 * args.batch * c * c * 9 * hw * hw
        tiles = args.batch * ((hw + 1) // 2) ** 2
        es = 4 if dt == "f32" else 2
        mbytes = es * 2 * args.batch * c * hw * hw + es * c * c * 9 + 4 * c
        rows = []
        for r in costs["layers"][1]["routines"]:
            if r["ns"] is None or r["ns"] < 0:
                continue
            if "f4x4" in r["name"]:   # F(4x4,3x3): 36 tile GEMMs over 4x4-pixel tiles
                f = 2 * 36 * c * c * args.batch * ((hw + 3) // 4) ** 2
            elif "winograd" in r["name"]:
                f = 2 * 16 * c * c * tiles
            else:
                f = flops
            tfl = f / (r["ns"] * 1e-9) / 1e12
            rows.append({"routine": r["name"], "us": round(r["ns"] / 1e3, 2),
                         "tflops": round(tfl, 1),
                         "mfma_frac": round(tfl / PEAK_MFMA_TFLOPS[dt], 4) if "direct" not in r["name"] else None,
                         "gbs": round(mbytes / (r["ns"] * 1e-9) / 1e9, 1)})
        cvt = {}
        e = next(e for e in costs["edges"] if e["from"] == 0)   # the conv's input tensor
        for a, row in enumerate(e["ns"]):
            for b, v in enumerate(row):
                if a != b and v > 0:
                    cvt[f"{LAYOUTS[a]}>{LAYOUTS[b]}"] = {
                        "us": round(v / 1e3, 2),
                        "gbs": round(2 * es * args.batch * c * hw * hw / (v * 1e-9) / 1e9, 1)}
        best = min(rows, key=lambda r: r["us"])
        out.append({"shape": f"C=K={c} HxW={hw}x{hw} bs{args.batch} {dt}", "gflop": round(flops / 1e9, 2),
                    "best": best["routine"], "routines": rows, "converters": cvt})
        log(f"[sweep] {out[-1]['shape']}: best {best['routine']} {best['us']} us "
            f"({best['tflops']} TFLOP/s)")
        g.close()
    print(json.dumps({"sweep": out}), flush=True)


def time_steps(g, x, out, steps, warmup):
    import torch
    for _ in range(warmup):
        g.run(x, out)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.run(x, out)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def step_stats(g, x, out, n):
    """Per-step latency distribution of the selected path: n steps, each between
    its own pair of HIP events on the stream the path runs on (the pair adds a
    few microseconds of dispatch gap that the block-timed value does not have)."""
    import statistics
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in ev:
        a.record()
        g.run(x, out)
        b.record()
    torch.cuda.synchronize()
    ms = [a.elapsed_time(b) for a, b in ev]
    return {"median": round(statistics.median(ms), 4), "mean": round(statistics.fmean(ms), 4),
            "std": round(statistics.pstdev(ms), 4), "min": round(min(ms), 4), "runs": n}


def cpu_baseline(spec, t, budget_s, storage="dtype"):
    """The oracle (naive float64, OpenMP) on the first images of the batch,
    with every layer output rounded to the run dtype (storage "dtype", the
    parity mode) or exact (storage "f64")."""
    import numpy as np
    from oracle import numeric as O
    from workloads import decode, with_batch
    d = decode(t, spec["dtype"])
    done = 0
    t0 = time.perf_counter()
    while done < spec["batch"]:
        one = dict(d)
        one["x"] = d["x"][done:done + 1]
        O.forward(with_batch(spec, 1), one, storage=storage)
        done += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": round(done / el, 4), "unit": "img/s", "cores": O.num_threads(),
            "kind": "oracle",
            "sample": f"{done} image(s) of the batch-{spec['batch']} {spec['name'].split('_')[0]} input, "
                      f"naive float64 direct convolution, "
                      + (f"{spec['dtype']} storage rounding" if storage == "dtype" else "exact float64 storage")
                      + f", {el:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batch", type=int, default=32)
    ap.add_argument("--dtype", default="bf16")
    ap.add_argument("--profile-reps", type=int, default=20)
    ap.add_argument("--profile-flush-mib", type=int, default=0,
                    help="cache-cold unit profiling: MiB written before each timed run (0 = warm)")
    ap.add_argument("--timing-reps", type=int, default=50,
                    help="back-to-back repetitions per layer in the per-layer timing pass")
    ap.add_argument("--net", default="resnet50", choices=sorted(NETS),
                    help="workload (the headline line is resnet50 at batch 32)")
    ap.add_argument("--sweep", action="store_true",
                    help="print the measured cost table of the four 3x3 sweep shapes and exit")
    ap.add_argument("--no-fixed", action="store_true", help="skip the fixed-path sweep")
    ap.add_argument("--no-bs1", action="store_true", help="skip the batch-1 measurement")
    ap.add_argument("--no-fuse", action="store_true",
                    help="keep residual adds as their own layers (default: fold each into the 1x1 "
                         "convolution that produces its operand)")
    ap.add_argument("--no-proj", action="store_true",
                    help="keep projection shortcuts as their own 1x1 convolutions (default: fold each, "
                         "with its residual add, into the convolution the add follows)")
    ap.add_argument("--refine-reps", type=int, default=15,
                    help="in-path refinement after integrated profiling: timed runs per trial "
                         "(0 = off; near-tied routines of each layer timed inside the whole path)")
    ap.add_argument("--refine-tol", type=int, default=150,
                    help="in-path refinement: alternatives within this many per mille of the "
                         "selected routine's unit-profiled time")
    ap.add_argument("--refine-alts", type=int, default=3,
                    help="in-path refinement: alternatives tried per layer (the fastest by unit cost)")
    ap.add_argument("--integrated-reps", type=int, default=20,
                    help="runs per candidate in integrated profiling (0 = keep the DPRS path)")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--costs-out", default=None, help="write the measured cost table here")
    ap.add_argument("--costs-in", default=None,
                    help="select from this cost table instead of profiling (same workload)")
    ap.add_argument("--tune-only", action="store_true",
                    help="profile and select, write --costs-out, and exit")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed region, run one device copy of this size "
                         "(a known-size kernel for scaling PMC byte counters)")
    ap.add_argument("--path-out", default=None, help="write the selected routine path here")
    ap.add_argument("--path-in", default=None,
                    help="run this routine path (from --path-out) instead of selecting one")
    ap.add_argument("--pmc-pass", default=None, metavar="PASS_JSON",
                    help="run only warmup + steps of the path (then the calibration copy) for "
                         "counter collection, write the launch list to PASS_JSON, and exit")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "PASS_JSON", "OUT"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of --pmc-pass into "
                         "the per-layer traffic summary OUT, and exit")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("TRACE_DIR", "PASS_JSON", "OUT"),
                    help="per-layer kernel durations of a --pmc-pass run under rocprofv3 --kernel-trace")
    ap.add_argument("--rotate-layouts", action="store_true",
                    help="with --tune-only: a path whose layer i takes layout i mod 3 (converters on every "
                         "edge), for profiling the adapt routines")
    ap.add_argument("--compare-rounds", type=int, default=4,
                    help="alternating rounds timing the DPRS path against the best fixed paths")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, calib_mib=args.calib_copy_mib)
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the path would shard over "
              "the batch (one graph per GPU, tuned at its share of the batch, no exchange)",
              file=sys.stderr)
        sys.exit(2)

    if args.sweep:
        sweep(args)
        return

    import numpy as np
    import torch
    from paper_2110_06037_amd import build_from_spec, native as N, to_device as to_dev
    from workloads import fuse_projection, fuse_residual, generate, resnet50

    spec = _nets()[args.net](args.batch, args.dtype)
    if not args.no_fuse:
        spec = fuse_residual(spec)
        if not args.no_proj:
            spec = fuse_projection(spec)
    t = generate(spec)
    log(f"[bench] {spec['name']}: building graph")
    g = build_from_spec(spec, t, device=0)
    t0 = time.perf_counter()
    if args.costs_in:
        with open(args.costs_in) as f:
            g.set_costs(f.read())
    else:
        # cache-cold unit profiling when asked: the library evicts the caches
        # before every timed run and takes the median
        g.set_option(N.OPT_FLUSH, args.profile_flush_mib << 20)
        g.profile(warmup=5, reps=args.profile_reps)
        g.set_option(N.OPT_FLUSH, 0)
    t_prof = time.perf_counter() - t0
    t1 = time.perf_counter()
    g.select("dprs")
    t_sel = time.perf_counter() - t1
    log(f"[bench] {'loaded costs' if args.costs_in else 'profiled'} in {t_prof:.1f} s, "
        f"selected in {t_sel * 1e3:.2f} ms")
    if args.costs_out:
        with open(args.costs_out, "w") as f:
            json.dump(g.costs(), f)
    if args.rotate_layouts:
        # a path for profiling the adapt routines: layer i runs the fastest
        # routine in layout i mod 3, so every edge between layers converts
        table = g.costs()["layers"]
        rot = [0]
        for i in range(1, g.num_layers()):
            ns = {r["id"]: (c["ns"] if c["ns"] is not None and c["ns"] >= 0 else float("inf"))
                  for r, c in zip(g.routines(i), table[i]["routines"])}
            want = [r for r in g.routines(i) if r["layout"] == i % 3 and ns[r["id"]] < float("inf")]
            rot.append(min(want or g.routines(i), key=lambda r: ns[r["id"]])["id"])
        g.set_path(rot)
    dp_ids, dp_model_ns = g.path()
    pinned = None
    if args.path_in:
        with open(args.path_in) as f:
            pinned = json.load(f)["path"]
        args.integrated_reps = 0
    if args.tune_only:
        if args.integrated_reps > 0:
            g.profile_integrated(warmup=2, reps=args.integrated_reps)
        if args.refine_reps > 0 and not args.rotate_layouts:
            n_ref = g.refine_in_path(tol_permille=args.refine_tol, max_alts=args.refine_alts, reps=args.refine_reps)
            log(f"[bench] in-path refinement: {n_ref} layer(s) changed")
        if args.path_out:
            with open(args.path_out, "w") as f:
                json.dump({"path": g.path()[0], "routines": [g.routines(i)[r]["name"] for i, r in
                                                              enumerate(g.path()[0])]}, f)
        g.close()
        return
    x = to_dev(t["x"], args.dtype)
    out = g.empty_output()
    if args.pmc_pass:
        # counter collection: the pinned path's steps and nothing else (the
        # library's dispatches are then whole steps in order), then one copy
        # of known size for scaling the byte counters
        if pinned:
            g.set_path(pinned)
        for _ in range(args.warmup + args.steps):
            g.run(x, out)
        torch.cuda.synchronize()
        if args.calib_copy_mib:
            src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
            dst = torch.zeros_like(src)
            dst.copy_(src)
            torch.cuda.synchronize()
        ids = g.path()[0]
        need = {str(i): bytes_needed(spec, g, i, g.routines(i)[ids[i]]) for i in range(1, g.num_layers())}
        with open(args.pmc_pass, "w") as f:
            json.dump({"workload": spec["name"], "warmup": args.warmup, "steps": args.steps,
                       "routines": [g.routines(i)[r]["name"] for i, r in enumerate(ids)],
                       "launch_layers": g.plan_launches(), "bytes_needed": need}, f)
        g.close()
        return

    sec_dp = time_steps(g, x, out, args.steps, args.warmup)
    log(f"[bench] DPRS path: {sec_dp * 1e3:.3f} ms/step, {args.batch / sec_dp:.1f} img/s")
    if pinned:
        g.set_path(pinned)
    # integrated profiling (Sec. III-C): the DPRS candidates and the fixed
    # paths timed end to end; the library keeps the fastest
    integ = None
    t_int = 0.0
    sec = sec_dp
    if args.integrated_reps > 0:
        t2 = time.perf_counter()
        cands = g.profile_integrated(warmup=2, reps=args.integrated_reps)
        t_int = time.perf_counter() - t2
        ids, _ = g.path()
        pick = next(c for c in cands if c["path"] == ids)
        label = (f"dprs/{_mask_name(pick['a'])}" if pick["kind"] == "dprs"
                 else f"fixed/{N.LAYOUT_NAME[pick['a']]}/{N.ALGO_NAME[pick['b']]}")
        if ids != dp_ids:
            sec = time_steps(g, x, out, args.steps, args.warmup)
        integ = {"candidates": len(cands), "selected": label, "seconds": round(t_int, 2),
                 "measured_ms": {(f"dprs/{_mask_name(c['a'])}" if c["kind"] == "dprs" else
                                  f"fixed/{N.LAYOUT_NAME[c['a']]}/{N.ALGO_NAME[c['b']]}"):
                                 round(c["measured_ns"] / 1e6, 4) for c in cands}}
        log(f"[bench] integrated profiling: {len(cands)} candidates in {t_int:.1f} s, "
            f"selected {label}: {sec * 1e3:.3f} ms/step")
    # in-path refinement: near-tied routines of each layer's schema timed
    # inside the whole path; the library keeps the refined path only if it
    # also wins end to end
    refine = None
    t_ref = 0.0
    if args.refine_reps > 0 and not pinned:
        before = g.path()[0]
        t3 = time.perf_counter()
        n_ref = g.refine_in_path(tol_permille=args.refine_tol, max_alts=args.refine_alts, reps=args.refine_reps)
        t_ref = time.perf_counter() - t3
        after = g.path()[0]
        refine = {"layers_changed": n_ref, "seconds": round(t_ref, 2), "tol_permille": args.refine_tol,
                  "changes": {str(i): [g.routines(i)[before[i]]["name"], g.routines(i)[after[i]]["name"]]
                              for i in range(len(after)) if after[i] != before[i]}}
        if n_ref:
            sec = time_steps(g, x, out, args.steps, args.warmup)
        log(f"[bench] in-path refinement: {n_ref} layer(s) changed in {t_ref:.1f} s: {sec * 1e3:.3f} ms/step")
    if pinned:
        sec = time_steps(g, x, out, args.steps, args.warmup)
        log(f"[bench] pinned path: {sec * 1e3:.3f} ms/step")
    ids, model_ns = g.path()
    if args.path_out:
        with open(args.path_out, "w") as f:
            json.dump({"path": ids, "routines": [g.routines(i)[r]["name"] for i, r in enumerate(ids)]}, f)
    value = args.batch / sec
    steps_dist = step_stats(g, x, out, min(max(args.steps, 10), 100))
    log(f"[bench] per-step latency (ms): {steps_dist}")

    # per-layer times over K instrumented steps: each layer's launches are
    # repeated back to back with HIP events tied to the first and last dispatch
    nl = g.num_layers()
    acc = np.zeros(nl)
    passes = min(args.steps, 20)
    for _ in range(passes):
        _, ms = g.run_timed(x, out, reps=args.timing_reps)
        acc += np.array(ms)
    layer_ms = acc / passes
    # cache-cold per-layer times: the library writes a 512 MiB buffer (more
    # than L2 and the Infinity Cache hold) before each layer; one repetition
    # per layer, median over 5 passes
    g.set_option(N.OPT_FLUSH, 512 << 20)
    cold = np.median(np.array([g.run_timed(x, out, reps=1)[1] for _ in range(5)]), axis=0)
    g.set_option(N.OPT_FLUSH, 0)
    groups = {}      # (routine, layer type) -> its launches in one step: one kernel symbol each
                     # (the direct routine of an add and of a pool are different kernels)
    cats = {}        # layer category -> totals (for the 3x3 MFMA utilisation)
    per_layer = []
    for i in range(1, nl):
        rt = g.routines(i)[ids[i]]
        cat, flops, byt = layer_work(spec, g, i, rt)
        need = bytes_needed(spec, g, i, rt)
        for key, d in ((f"{rt['name']} on {layer_kind(spec, i)}", groups), (cat, cats)):
            gr = d.setdefault(key, {"ms": 0.0, "flops": 0, "bytes": 0, "needed": 0, "launches": 0, "cats": set(),
                                    "layers": [], "routine": rt["name"]})
            gr["ms"] += layer_ms[i]
            gr["flops"] += flops
            gr["bytes"] += byt
            gr["needed"] += need
            gr["launches"] += 1
            gr["cats"].add(cat)
            gr["layers"].append(i)
        per_layer.append({"layer": i, "type": cat, "routine": rt["name"],
                          "us": round(layer_ms[i] * 1e3, 2), "us_cold": round(float(cold[i]) * 1e3, 2),
                          "tflops": round(flops / (layer_ms[i] * 1e-3) / 1e12, 2) if flops and layer_ms[i] else 0,
                          "gbs": round(byt / (layer_ms[i] * 1e-3) / 1e9, 1) if layer_ms[i] else 0,
                          "gbs_needed": round(need / (layer_ms[i] * 1e-3) / 1e9, 1) if layer_ms[i] else 0})
    dom_key = max(groups, key=lambda k: groups[k]["ms"])
    dom = groups[dom_key]
    avg_s = dom["ms"] / dom["launches"] * 1e-3
    # the roof that binds: MFMA when the routine's arithmetic intensity is above
    # the ridge point (peak flops / peak bandwidth), HBM otherwise
    ridge = PEAK_MFMA_TFLOPS[args.dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    if (any(c.startswith("conv") for c in dom["cats"]) and "direct" not in dom_key
            and dom["flops"] > ridge * dom["bytes"]):
        ach = dom["flops"] / dom["launches"] / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_MFMA_TFLOPS[args.dtype],
                "unit": "TFLOP/s"}
    else:
        ach = dom["bytes"] / dom["launches"] / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    # HBM traffic from the committed per-layer counter summary, only where it
    # covers these very layers run by this routine (else null, with the reason)
    traffic, why = traffic_for_layers(dom["layers"], dom["routine"], workload=spec["name"])
    roof["traffic"] = traffic
    if traffic:
        roof["traffic_ratio"] = round(traffic / (dom["bytes"] / dom["launches"]), 3)
    else:
        roof["traffic_null_reason"] = why
    roof["kernel"] = (f"routine {dom_key} ({dom['launches']} launches/step on "
                      f"{'/'.join(sorted(dom['cats']))} layers {dom['layers']})")
    roof["avg_launch_us"] = round(avg_s * 1e6, 2)
    roof["algorithmic"] = {"flops_per_launch": dom["flops"] // dom["launches"],
                           "bytes_per_launch": dom["bytes"] // dom["launches"],
                           "bytes_needed_per_launch": dom["needed"] // dom["launches"]}
    if roof["bound"] == "hbm":
        # the same with a strided 1x1 layer's input counted as the pixels it reads
        roof["achieved_needed"] = round(dom["needed"] / dom["launches"] / avg_s / 1e9, 1)
    # headline: MFMA utilisation over the 3x3 convolutions
    c3 = cats.get("conv3x3")
    conv3_util = (c3["flops"] / (c3["ms"] * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS[args.dtype]) if c3 else None
    # every layer category against both roofs (per-layer block means): the
    # dominant routine above is one tile configuration, this is the whole
    # category (all routines and tiles of that layer kind)
    step_layer_ms = float(layer_ms[1:].sum())
    cat_roof = {}
    for cname, cv in sorted(cats.items(), key=lambda kv: -kv[1]["ms"]):
        sec_c = cv["ms"] * 1e-3
        cat_roof[cname] = {
            "layers": cv["launches"], "ms": round(cv["ms"], 4), "share": round(cv["ms"] / step_layer_ms, 4),
            "mfma_frac": round(cv["flops"] / sec_c / 1e12 / PEAK_MFMA_TFLOPS[args.dtype], 4) if cv["flops"] else 0.0,
            "hbm_frac": round(cv["bytes"] / sec_c / 1e9 / PEAK_HBM_GBS, 4),
            "hbm_frac_needed": round(cv["needed"] / sec_c / 1e9 / PEAK_HBM_GBS, 4)}

    if args.calib_copy_mib:
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.zeros_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    fixed = {}
    fixed_model = {}   # the additive model's T(S) of each fixed path, from the same cost table
    best_fixed = None
    if not args.no_fixed:
        for lay in LAYOUTS:
            for algo in ALGOS:
                g.select("fixed", lay, algo)
                fixed_model[f"{lay}/{algo}"] = round(g.path()[1] / 1e6, 4)
                s = time_steps(g, x, out, args.steps, args.warmup)
                fixed[f"{lay}/{algo}"] = round(args.batch / s, 2)
                log(f"[bench] fixed {lay}/{algo}: {args.batch / s:.1f} img/s")
        best_fixed = max(fixed, key=fixed.get)
        g.set_path(ids)
    dp_vs_fixed = round(args.batch / sec_dp / fixed[best_fixed], 4) if best_fixed else None
    sel_vs_fixed = round(value / fixed[best_fixed], 4) if best_fixed else None
    # the DPRS path, the selected path and the two best fixed paths timed in
    # alternating rounds (order reversed every other round), so drift and
    # warm-up favour none of them; medians and per-round ratios reported
    comparison = None
    if best_fixed and args.compare_rounds > 0:
        top = sorted(fixed, key=fixed.get, reverse=True)[:2]
        cands = [("dprs", dp_ids)] + ([("selected", ids)] if ids != dp_ids else [])
        for name in top:
            lay, algo = name.split("/")
            g.select("fixed", lay, algo)
            cands.append((f"fixed/{name}", g.path()[0]))
        if refine:
            # the fastest fixed path given the same in-path refinement (it
            # stays within its one layout), so the selected path is also
            # compared with a fixed path tuned as far as the DPRS one
            lay, algo = top[0].split("/")
            g.select("fixed", lay, algo)
            g.refine_in_path(tol_permille=args.refine_tol, max_alts=args.refine_alts, reps=args.refine_reps)
            cands.append((f"fixed_refined/{top[0]}", g.path()[0]))
        times = {nm: [] for nm, _ in cands}
        for r in range(args.compare_rounds):
            for nm, path in (cands if r % 2 == 0 else cands[::-1]):
                g.set_path(path)
                times[nm].append(time_steps(g, x, out, args.steps, min(args.warmup, 5)) * 1e3)
        g.set_path(ids)
        med = {nm: float(np.median(v)) for nm, v in times.items()}
        bf = min((nm for nm in med if nm.startswith("fixed/")), key=med.get)
        ratios = [f / d for f, d in zip(times[bf], times["dprs"])]
        comparison = {"rounds": args.compare_rounds, "steps_per_round": args.steps,
                      "ms": {nm: {"median": round(med[nm], 4), "min": round(min(v), 4), "max": round(max(v), 4)}
                             for nm, v in times.items()},
                      "best_fixed": bf, "dp_vs_best_fixed": round(med[bf] / med["dprs"], 4),
                      "dp_vs_best_fixed_per_round": [round(q, 4) for q in ratios]}
        if "selected" in med:
            comparison["selected_vs_best_fixed"] = round(med[bf] / med["selected"], 4)
            fr = next((nm for nm in med if nm.startswith("fixed_refined/")), None)
            if fr:
                comparison["selected_vs_refined_best_fixed"] = round(med[fr] / med["selected"], 4)
        log(f"[bench] alternating comparison: {comparison}")

    bs1 = bs1_detail = None
    if not args.no_bs1 and args.net == "resnet50":
        spec1 = resnet50(1, args.dtype)
        if not args.no_fuse:
            spec1 = fuse_residual(spec1)
            if not args.no_proj:
                spec1 = fuse_projection(spec1)
        t1_ = generate(spec1)
        g1 = build_from_spec(spec1, t1_, device=0)
        g1.profile(warmup=5, reps=args.profile_reps)
        g1.select("dprs")
        if args.integrated_reps > 0:
            g1.profile_integrated(warmup=2, reps=max(args.integrated_reps, 20))
        if args.refine_reps > 0:
            g1.refine_in_path(tol_permille=args.refine_tol, max_alts=args.refine_alts, reps=args.refine_reps)
        x1 = to_dev(t1_["x"], args.dtype)
        o1 = g1.empty_output()
        # eager launches and the same plan replayed as a HIP graph; the
        # faster is reported (on this stack graph replay has been the slower)
        s1 = time_steps(g1, x1, o1, max(args.steps, 50), args.warmup)
        g1.set_option(N.OPT_HIPGRAPH, 1)
        s1g = time_steps(g1, x1, o1, max(args.steps, 50), args.warmup)
        bs1 = round(1.0 / min(s1, s1g), 1)
        bs1_detail = {"eager_ms": round(s1 * 1e3, 4), "hip_graph_ms": round(s1g * 1e3, 4)}
        log(f"[bench] bs1 DP path: eager {s1 * 1e3:.3f} ms, HIP graph {s1g * 1e3:.3f} ms, {bs1} img/s")
        g1.close()

    cpu = cpu_baseline(spec, t, args.cpu_budget)
    if args.cpu_budget > 0:
        cpu64 = cpu_baseline(spec, t, args.cpu_budget / 2, storage="f64")
        cpu["value_f64_storage"] = cpu64["value"]
        cpu["sample_f64_storage"] = cpu64["sample"]
    log(f"[bench] cpu oracle: {cpu}")

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "img/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": args.dtype,
        "data": "synthetic (seeded random input and He-normal weights)",
        "config": {"workload": f"{args.net}-shaped CNN, batch {args.batch}, {args.dtype}, 224x224"
                               + ("" if not any(l["type"] == "conv" and len(l["in"]) > 1 for l in spec["layers"])
                                  else ", residual adds folded into the 1x1 convolutions that produce them")
                               + (", projection shortcuts folded into the convolution their add follows"
                                  if any(l.get("proj") for l in spec["layers"]) else ""),
                   "batch": args.batch,
                   "path": ("DPRS candidates + fixed paths, integrated profiling keeps the fastest"
                            if integ else "DPRS-selected routines")
                           + (", in-path refinement" if refine else "")},
        "roofline": roof,
        "cpu_baseline": cpu,
        "step_ms": steps_dist,
        "layer_sum_ms": {"warm": round(float(layer_ms[1:].sum()), 4), "cold": round(float(cold[1:].sum()), 4)},
        "img_s_bs1": bs1, "bs1_ms": bs1_detail,
        "conv3x3_mfma_util": round(conv3_util, 4) if conv3_util else None,
        "category_roofline": cat_roof,
        "dprs_img_s": round(args.batch / sec_dp, 2),
        "dp_vs_best_fixed": comparison["dp_vs_best_fixed"] if comparison else dp_vs_fixed,
        "selected_vs_best_fixed": (comparison.get("selected_vs_best_fixed", comparison["dp_vs_best_fixed"])
                                   if comparison else sel_vs_fixed),
        "selected_vs_refined_best_fixed": comparison.get("selected_vs_refined_best_fixed") if comparison else None,
        "comparison": comparison, "single_pass_dp_vs_best_fixed": dp_vs_fixed,
        "best_fixed": best_fixed, "fixed_img_s": fixed, "fixed_model_time_ms": fixed_model, "integrated": integ,
        "in_path_refinement": refine,
        "model_time_ms": round(model_ns / 1e6, 4), "dprs_model_time_ms": round(dp_model_ns / 1e6, 4),
        "tuning_s": round(t_prof + t_sel + t_int + t_ref, 2),
        "unit_profiling": ("loaded" if args.costs_in else
                           f"cold/{args.profile_flush_mib}MiB/median" if args.profile_flush_mib else "warm/mean"),
    }
    sel = {}
    for i in range(1, nl):
        nm = g.routines(i)[ids[i]]["name"]
        sel[nm] = sel.get(nm, 0) + 1
    line["selected"] = sel
    if os.environ.get("SN_BENCH_LAYERS"):
        with open(os.environ["SN_BENCH_LAYERS"], "w") as f:
            json.dump(per_layer, f, indent=1)
    print(json.dumps(line), flush=True)
    g.close()


if __name__ == "__main__":
    main()
