#!/usr/bin/env python3
"""Benchmark of the block-pruned ResNet-50 layer forward on one MI355X.

Workload: every conv layer of ResNet-50 v1.5 at ImageNet shape (224x224) plus
the fc layer, batch 64, bf16 activations and weights, fp32 accumulation.
1x1 convs: 32x32 blocks, 2x row pruning; 3x3 convs: 16x32 blocks, 4x column
pruning; conv1 (7x7/2) and fc dense.  Weights are seeded He-normal draws,
pruned and packed on the GPU once (reported as prep time); each layer reads
its own seeded N(0,1) input, resident in HBM before timing starts.

One step = the forward of all 54 layers (gather + MFMA contraction + fused
epilogue), launched as one captured HIP graph.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5]
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms/layer + kept-FLOP TFLOP/s (% MFMA roofline), ResNet-50 layers at 4× pruning"
PEAK_BF16 = 2516.6e12     # dense MFMA bf16, FLOP/s
PEAK_HBM = 8.0e12         # bytes/s
KERNEL_TAGS = ("bsp::fwd::k_fwd<", "bsp::pw::k_pw<")   # the forward kernels (general, pointwise)
CALIB_BYTES = 256 << 20   # plain copy kernel (torch.neg on bf16) that calibrates the HBM counters
COUNTERS_FILE = os.path.join(ROOT, "profiles", "forward_resnet50_b64_hbm_counters.txt")


def is_forward(name: str) -> bool:
    return any(t in name for t in KERNEL_TAGS)


def source_hash() -> str:
    """Hash of the kernel sources; counter figures taken on other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2111_11581_amd", "csrc")
    for d, names in ((csrc, sorted(os.listdir(csrc))), (os.path.join(ROOT, "include"), ["bsp.h"])):
        for n in names:
            if n.endswith((".hip", ".cpp", ".h")):
                with open(os.path.join(d, n), "rb") as f:
                    h.update(n.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def read_counters():
    """Per-launch HBM bytes of the forward kernels from the committed counter summary,
    or None when it is missing or was taken on different kernel sources."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    kv = {}
    with open(COUNTERS_FILE) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_hash") != source_hash():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def layer_cost(layer, nnz: int, n_values: int, n_indices: int, n_rowptr: int):
    """Kept FLOPs, dense FLOPs and algorithmic bytes (input once + output once +
    packed values + index metadata) of one layer forward."""
    P = layer.pixels
    f_kept = 2.0 * nnz * P
    f_dense = 2.0 * layer.scheme.rows * layer.scheme.cols * P
    x_el = 1
    for v in layer.x_shape:
        x_el *= v
    y_el = 1
    for v in layer.y_shape:
        y_el *= v
    b_alg = 2.0 * (x_el + y_el + n_values) + 4.0 * (n_indices + n_rowptr)
    t_roof = max(f_kept / PEAK_BF16, b_alg / PEAK_HBM)
    return f_kept, f_dense, b_alg, t_roof


def cpu_baseline(layers, images: int, threads: int):
    """Time the fp64 oracle (direct conv / matmul on masked weights) on the
    first `images` images of every layer; inputs from the host generator."""
    import numpy as np
    from oracle import direct
    from oracle import prune as OP
    from synthetic import draw, seed_for, SEED_X, SEED_W
    direct.build(force=False)
    t_total, kept_flops = 0.0, 0.0
    for i, l in enumerate(layers):
        w = draw(seed_for(3, i, SEED_W), l.w_shape, l.w_dist, "bf16")
        wg = OP.as_f64(w, "bf16").reshape(l.scheme.rows, -1)
        m = OP.prune_mask(wg, l.scheme.bh, l.scheme.bw, l.scheme.regularity, l.scheme.rate)
        wm = (wg * m).reshape(l.w_shape)
        if l.kind == "conv":
            xs = (images,) + tuple(l.x_shape[1:])
            x = OP.as_f64(draw(seed_for(3, i, SEED_X), xs, l.x_dist, "bf16"), "bf16")
            t0 = time.perf_counter()
            direct.conv2d(x, wm, None, (l.sh, l.sw), (l.ph, l.pw), threads=threads)
            t_total += time.perf_counter() - t0
            kept_flops += 2.0 * int(m.sum()) * images * l.ho * l.wo
        else:
            x = OP.as_f64(draw(seed_for(3, i, SEED_X), (l.in_f, images), l.x_dist, "bf16"), "bf16")
            t0 = time.perf_counter()
            direct.linear(x, wm, threads=threads)
            t_total += time.perf_counter() - t0
            kept_flops += 2.0 * int(m.sum()) * images
    return t_total, kept_flops


def _csv_rows(d: str, suffix: str):
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not files:
        raise SystemExit("no *%s under %s" % (suffix, d))
    rows = []
    for fn in files:
        with open(fn, newline="") as f:
            rows += list(csv.DictReader(f))
    return rows


def _pmc_per_launch(d: str, counter: str, n_layers: int):
    """Mean counter value (KiB) per forward dispatch of the timed steps (the first,
    eager step is skipped) and the value of the calibration copy kernel."""
    rows = [r for r in _csv_rows(d, "counter_collection.csv") if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    conv = [float(r["Counter_Value"]) for r in rows if is_forward(r["Kernel_Name"])]
    calib = [float(r["Counter_Value"]) for r in rows if "neg" in r["Kernel_Name"]]
    if len(conv) <= n_layers or not calib:
        raise SystemExit("%s: %d forward dispatches, %d copy dispatches" % (d, len(conv), len(calib)))
    steady = conv[n_layers:]
    return sum(steady) / len(steady), len(steady), max(calib)


def summarize(args):
    """Write the forward-kernel summary (kernel trace statistics and, when given, the
    HBM counters scaled by the calibration copy) to the profiles folder."""
    from synthetic import workload
    n_layers = len(workload(3, batch=args.batch))
    stats = _csv_rows(args.summarize, "kernel_stats.csv")
    conv = [r for r in stats if is_forward(r["Name"])]
    calls = sum(int(r["Calls"]) for r in conv)
    total_ns = sum(float(r["TotalDurationNs"]) for r in conv)
    lines = ["# Forward kernels (k_fwd: conv1 and the 3x3 layers; k_pw: the 1x1 layers and fc) on the "
             "ResNet-50 v1.5 layer pass (batch 64, bf16, 54 launches per step)", "",
             "Kernel trace statistics (rocprofv3 --kernel-trace --stats), command:", "",
             "    " + args.trace_cmd, "",
             "| kernel | calls | total us | average us | min us | max us |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        nm = r["Name"]
        short = nm.replace("void ", "").replace("bsp::fwd::", "").replace("bsp::pw::", "").split("(")[0] \
            if is_forward(nm) else nm[:60]
        lines.append("| %s | %s | %.1f | %.3f | %.3f | %.3f |" % (
            short, r["Calls"], float(r["TotalDurationNs"]) / 1e3, float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3))
    lines += ["", "Forward kernels, all instantiations: %d calls, average %.3f us per launch, %.1f us per step of %d launches"
              % (calls, total_ns / calls / 1e3, total_ns / calls * n_layers / 1e3, n_layers), ""]
    kv = {"source_hash": source_hash(), "kernel_avg_us_trace": "%.3f" % (total_ns / calls / 1e3)}
    if args.pmc_fetch and args.pmc_write:
        f_kib, nf, f_cal = _pmc_per_launch(args.pmc_fetch, "FETCH_SIZE", n_layers)
        w_kib, nw, w_cal = _pmc_per_launch(args.pmc_write, "WRITE_SIZE", n_layers)
        f_scale = CALIB_BYTES / (f_cal * 1024.0)
        w_scale = CALIB_BYTES / (w_cal * 1024.0)
        fetch = f_kib * 1024.0 * f_scale
        write = w_kib * 1024.0 * w_scale
        lines += ["HBM counters (one rocprofv3 --pmc pass each), commands:", "",
                  "    " + args.fetch_cmd, "    " + args.write_cmd, "",
                  "Calibration: a plain copy kernel (torch.neg, %d MiB in, %d MiB out) reads FETCH_SIZE %.0f KiB and "
                  "WRITE_SIZE %.0f KiB, so the scale factors are %.4f (fetch) and %.4f (write)."
                  % (CALIB_BYTES >> 20, CALIB_BYTES >> 20, f_cal, w_cal, f_scale, w_scale), "",
                  "Forward kernels per launch (mean over %d / %d dispatches of the timed steps): fetch %.3f MB, write %.3f MB, "
                  "traffic %.3f MB" % (nf, nw, fetch / 1e6, write / 1e6, (fetch + write) / 1e6), ""]
        kv.update({"fetch_bytes_per_launch": "%.0f" % fetch, "write_bytes_per_launch": "%.0f" % write,
                   "traffic_bytes_per_launch": "%.0f" % (fetch + write),
                   "fetch_scale": "%.5f" % f_scale, "write_scale": "%.5f" % w_scale})
    os.makedirs(os.path.dirname(os.path.abspath(args.out)), exist_ok=True)
    with open(args.out, "w") as f:
        f.write("\n".join(lines))
    if args.pmc_fetch and args.pmc_write:
        with open(COUNTERS_FILE, "w") as f:
            f.write("# forward-kernel HBM bytes per launch on the ResNet-50 layer pass; written by bench.py --summarize\n")
            f.write("# from the passes listed in %s\n" % os.path.basename(args.out))
            for k, v in kv.items():
                f.write("%s: %s\n" % (k, v))
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-images", type=int, default=40, help="images per layer in the CPU oracle sample")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--layers-out", default=None, help="write the per-layer table (JSON) here")
    ap.add_argument("--no-layers", action="store_true", help="skip the per-layer timing (profiling passes)")
    ap.add_argument("--summarize", default=None, metavar="TRACE_DIR",
                    help="no GPU: summarize a rocprofv3 --stats output folder (and --pmc-fetch/--pmc-write)")
    ap.add_argument("--pmc-fetch", default=None)
    ap.add_argument("--pmc-write", default=None)
    ap.add_argument("--trace-cmd", default="")
    ap.add_argument("--fetch-cmd", default="")
    ap.add_argument("--write-cmd", default="")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "forward_resnet50_b64.md"))
    args = ap.parse_args()
    if args.summarize:
        summarize(args)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each GPU would run its "
              "own batch shard with no exchange); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2111_11581_amd as B
    from paper_2111_11581_amd.layers import PackedLayer
    from synthetic import workload, draw, draw_device, seed_for, SEED_X, SEED_W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.lib()   # raises if the HIP library is not built
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layers = workload(3, batch=args.batch)

    # ---- weights: seeded host draws -> device; prune + pack on the GPU (prep) ----
    wdev = []
    for i, l in enumerate(layers):
        w = draw(seed_for(3, i, SEED_W), l.w_shape, l.w_dist, "bf16")
        wdev.append(torch.from_numpy(w.reshape(l.scheme.rows, -1).view(np.int16)).view(torch.bfloat16).to(dev))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    packed = []
    for l, w in zip(layers, wdev):
        conv = None if l.kind != "conv" else B.ConvShape(l.n, l.cin, l.h, l.w, l.kh, l.kw, l.sh, l.sw, l.ph, l.pw)
        packed.append(PackedLayer(l.scheme, B.BF16, w, conv=conv))
    torch.cuda.synchronize()
    prep_ms = (time.perf_counter() - t0) * 1e3

    # ---- activations (seeded, on device) and outputs ----
    xs, ys = [], []
    for i, l in enumerate(layers):
        xs.append(draw_device(seed_for(3, i, SEED_X), l.x_shape, l.x_dist, "bf16", dev))
        ys.append(torch.empty(l.y_shape, dtype=torch.bfloat16, device=dev))
    torch.cuda.synchronize()

    costs = []
    for l, p in zip(layers, packed):
        nnz = int(p.mask.sum().item())
        costs.append(layer_cost(l, nnz, p.n_values, p.n_indices, p.n_rowptr))

    def run_layer(i):
        l, p = layers[i], packed[i]
        if l.kind == "conv":
            p.conv2d(xs[i], ys[i], l.n, B.BF16)
        else:
            p.linear(xs[i], ys[i], l.batch, B.BF16)

    def step():
        for i in range(len(layers)):
            run_layer(i)

    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        step()            # eager once (also loads the code objects)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()

    # one graph for the whole step; one graph per layer (REPS launches) for per-layer times
    g_step = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_step):
        step()
    REPS = 10
    g_layer = []
    for i in range(len(layers)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(REPS):
                run_layer(i)
        g_layer.append(g)
    torch.cuda.synchronize()

    # plain copy kernel of known size: its HBM counters calibrate the forward kernels
    cal_src = torch.zeros(CALIB_BYTES // 2, dtype=torch.bfloat16, device=dev)
    cal_dst = torch.empty_like(cal_src)
    torch.neg(cal_src, out=cal_dst)
    torch.cuda.synchronize()
    del cal_src, cal_dst

    for _ in range(args.warmup):
        g_step.replay()
    torch.cuda.synchronize()

    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        g_step.replay()
    ev1.record()
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - w0
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    # per-layer kernel durations (graph of REPS back-to-back launches, same stream)
    layer_us = []
    for i in range(0 if args.no_layers else len(layers)):
        g_layer[i].replay()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            g_layer[i].replay()
        e1.record()
        torch.cuda.synchronize()
        layer_us.append(e0.elapsed_time(e1) * 1e3 / (3 * REPS))

    f_kept = sum(c[0] for c in costs)
    f_dense = sum(c[1] for c in costs)
    b_alg = sum(c[2] for c in costs)
    t_roof = sum(c[3] for c in costs)
    t_step = ms_per_step * 1e-3
    n = len(layers)
    achieved_gbs = b_alg / t_step / 1e9

    traffic = read_counters()
    table = []
    for l, c, us in zip(layers, costs, layer_us):
        table.append({"layer": l.name, "scheme": l.scheme.label(), "us": round(us, 3),
                      "roof_us": round(c[3] * 1e6, 3), "roof_frac": round(c[3] * 1e6 / us, 4),
                      "kept_tflops": round(c[0] / (us * 1e-6) / 1e12, 2),
                      "hbm_gbs": round(c[2] / (us * 1e-6) / 1e9, 1)})
    print("%-36s %-22s %9s %9s %7s %9s %9s" % ("layer", "scheme", "us", "roof_us", "frac", "kTFLOP/s", "GB/s"),
          file=sys.stderr)
    for r in table:
        print("%-36s %-22s %9.2f %9.2f %7.3f %9.1f %9.0f" % (r["layer"], r["scheme"], r["us"], r["roof_us"],
                                                            r["roof_frac"], r["kept_tflops"], r["hbm_gbs"]),
              file=sys.stderr)
    if args.layers_out:
        with open(args.layers_out, "w") as f:
            json.dump(table, f, indent=1)

    out = {
        "metric": METRIC,
        "value": round(f_kept / t_step / 1e12, 3),
        "unit": "TFLOP/s (kept FLOPs, whole ResNet-50 layer pass)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_layer": round(ms_per_step / n, 5),
        "effective_tflops": round(f_dense / t_step / 1e12, 3),
        "roof_frac_step": round(t_roof / t_step, 4),
        "roof_ms_step": round(t_roof * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations, He-normal weights; no dataset)",
        "config": {"workload": "ResNet-50 v1.5 conv layers + fc at 224x224, batch %d: 1x1 row 32x32 2x, "
                               "3x3 col 16x32 4x, conv1 and fc dense" % args.batch,
                   "batch": args.batch, "layers": n},
        "roofline": {"bound": "hbm",
                     "kernel": "forward kernels k_fwd + k_pw (all instantiations, %d launches per step)" % n,
                     "achieved": round(achieved_gbs, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": round(achieved_gbs * 1e9 / PEAK_HBM, 4),
                     "traffic": None if traffic is None else round(traffic),
                     "algorithmic_bytes_per_launch": round(b_alg / n),
                     "algorithmic_bytes_per_step": int(b_alg),
                     "avg_launch_us": round(ms_per_step * 1e3 / n, 3)},
        "prep_ms": round(prep_ms, 1),
        "wall_s_timed": round(wall_s, 4),
    }
    if not args.no_cpu:
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        t_cpu, kf = cpu_baseline(layers, args.cpu_images, threads)
        out["cpu_baseline"] = {"value": round(kf / t_cpu / 1e12, 6),
                               "unit": "TFLOP/s (kept FLOPs; oracle does every dense MAC in fp64)",
                               "cores": threads, "kind": "oracle",
                               "sample": "all %d layers, first %d of %d images, %.1f s" % (
                                   n, args.cpu_images, args.batch, t_cpu),
                               "cpu": platform.processor() or platform.machine()}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
