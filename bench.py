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


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-images", type=int, default=40, help="images per layer in the CPU oracle sample")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--layers-out", default=None, help="write the per-layer table (JSON) here")
    args = ap.parse_args()

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
    for i in range(len(layers)):
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
        "roofline": {"bound": "hbm", "kernel": "k_conv (all tile instantiations, %d launches per step)" % n,
                     "achieved": round(achieved_gbs, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": round(achieved_gbs * 1e9 / PEAK_HBM, 4), "traffic": None,
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
