#!/usr/bin/env python3
"""Benchmark of the block-pruned layer forward on one MI355X.

Default workload (--workload 3): every conv layer of ResNet-50 v1.5 at ImageNet
shape (224x224) plus the fc layer, batch 64, bf16 activations and weights, fp32
accumulation.  1x1 convs: 32x32 blocks, 2x row pruning; 3x3 convs: 16x32
blocks, 4x column pruning; conv1 (7x7/2) and fc dense.  Weights are seeded
He-normal draws, pruned and packed on the GPU once (reported as prep time);
each layer reads its own seeded N(0,1) input, resident in HBM before timing
starts.  The other workloads (same measurement):
  --workload 1  one fp32 3x3 conv, 64 -> 64 at 32x32, 16x16 column blocks 4x
  --workload 2  the VGG-16 CIFAR stack at batch 32 (13 convs with ReLU, 2x2
                max-pool after convs 2, 4, 7 and 10; chained), 8x16 column 8x
  --workload 4  the FC stack: 4 x 4096 -> 4096 at batch 512 (chained), 32x32
                column blocks at rate 10
(the block-size sweep layer is measured by paper_2111_11581_amd.latency).

One step = the forward of all layers (gather + MFMA contraction + fused
epilogue, and the max-pool glue of the VGG stack), launched as one captured HIP
graph.  Prints one JSON line; a per-layer table (hot-cache and cold-cache
kernel times against each layer's roofline) goes to stderr.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload 3]
"""

from __future__ import annotations

import argparse
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms/layer + kept-FLOP TFLOP/s (% MFMA roofline), ResNet-50 layers at 4× pruning"
PEAK = {"bf16": 2516.6e12, "f32": 157.3e12}   # dense MFMA, FLOP/s
PEAK_HBM = 8.0e12         # bytes/s
N_SIMD = 1024             # 256 CUs x 4 SIMDs
N_XCD = 8                 # GRBM_GUI_ACTIVE reads as the sum over the 8 XCDs
# forward kernels: general, pointwise, pipelined pointwise, stride-2 stem
KERNEL_TAGS = ("bsp::fwd::k_fwd<", "bsp::pw::k_pw<", "bsp::pl::k_pl<", "bsp::stem::k_stem(")
AUX_TAGS = ("k_im2col", "k_splitk_sum")   # expansion and partial-sum kernels some layers add to a step
CALIB_BYTES = 256 << 20   # plain copy kernel (torch.neg on bf16) that calibrates the HBM counters
COLD_BYTES = 512 << 20    # buffer sets rotated through for cold-cache layer times (2x the last-level cache)
COUNTERS_FILE = os.path.join(ROOT, "profiles", "forward_resnet50_b64_hbm_counters.txt")
MFMA_FILE = os.path.join(ROOT, "profiles", "forward_resnet50_b64_mfma_counters.txt")
MFMA_COUNTERS = ["SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES",
                 "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_ANY", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE"]
WORKLOAD_NAMES = {
    1: "single 3x3 conv 64->64 @32x32, batch 1, fp32: col 16x16 4x",
    2: "VGG-16 CIFAR stack, batch 32, bf16: conv1 dense, convs 2-13 col 8x16 8x, ReLU + 2x2 max-pool glue",
    3: "ResNet-50 v1.5 conv layers + fc at 224x224, batch 64: 1x1 row 32x32 2x, 3x3 col 16x32 4x, "
       "conv1 and fc dense",
    4: "FC stack 4 x 4096->4096, batch 512, bf16: col 32x32 rate 10 (8x effective)",
}


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


def _read_kv(path):
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    return kv if kv.get("source_hash") == source_hash() else None


def read_counters():
    """Per-launch HBM bytes of the forward kernels from the committed counter summary,
    or None when it is missing or was taken on different kernel sources."""
    kv = _read_kv(COUNTERS_FILE)
    try:
        return float(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def read_mfma_counters():
    """Executed MFMA FLOPs per step (bf16 MOPs x 512) and the counter MFMA busy
    fraction from the committed counter summary, or None (missing / stale)."""
    kv = _read_kv(MFMA_FILE)
    try:
        return (float(kv["executed_mfma_flops_per_step"]), float(kv["mfma_busy_frac_step"])) if kv else None
    except (KeyError, ValueError):
        return None


def layer_cost(layer, nnz: int, n_values: int, n_indices: int, n_rowptr: int, esize: int, dt: str):
    """Kept FLOPs, dense FLOPs and algorithmic bytes (input once + output once +
    packed values + index metadata) of one layer forward, and its roofline time."""
    P = layer.pixels
    f_kept = 2.0 * nnz * P
    f_dense = 2.0 * layer.scheme.rows * layer.scheme.cols * P
    x_el = math.prod(layer.x_shape)
    y_el = math.prod(layer.y_shape)
    b_alg = esize * (x_el + y_el + n_values) + 4.0 * (n_indices + n_rowptr)
    t_roof = max(f_kept / PEAK[dt], b_alg / PEAK_HBM)
    return f_kept, f_dense, b_alg, t_roof


def cpu_info():
    """CPU model name and physical core count of this host (Linux /proc/cpuinfo)."""
    model, cores = platform.processor() or platform.machine(), set()
    try:
        phys, core = None, None
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k, v = k.strip(), v.strip()
                if k == "model name":
                    model = v
                elif k == "physical id":
                    phys = v
                elif k == "core id":
                    core = v
                elif not k and phys is not None:
                    cores.add((phys, core))
                    phys, core = None, None
        if phys is not None:
            cores.add((phys, core))
    except OSError:
        pass
    return model, (len(cores) or None)


def cpu_baseline(layers, config: int, images: int, threads: int, dt: str):
    """Time the fp64 oracle (direct conv / matmul on masked weights) on the first
    `images` images (batch vectors) of every layer; inputs from the host generator."""
    from oracle import direct
    from oracle import prune as OP
    from synthetic import draw, seed_for, SEED_X, SEED_W
    direct.build(force=False)
    t_total, kept_flops = 0.0, 0.0
    for i, l in enumerate(layers):
        w = draw(seed_for(config, i, SEED_W), l.w_shape, l.w_dist, dt)
        wg = OP.as_f64(w, dt).reshape(l.scheme.rows, -1)
        m = OP.prune_mask(wg, l.scheme.bh, l.scheme.bw, l.scheme.regularity, l.scheme.rate)
        wm = (wg * m).reshape(l.w_shape)
        if l.kind == "conv":
            n = min(images, l.n)
            xs = (n,) + tuple(l.x_shape[1:])
            x = OP.as_f64(draw(seed_for(config, i, SEED_X), xs, l.x_dist, dt), dt)
            t0 = time.perf_counter()
            direct.conv2d(x, wm, None, (l.sh, l.sw), (l.ph, l.pw), relu=l.relu, threads=threads)
            t_total += time.perf_counter() - t0
            kept_flops += 2.0 * int(m.sum()) * n * (l.y_shape[2] * l.y_shape[3])
        else:
            n = min(images, l.batch)
            x = OP.as_f64(draw(seed_for(config, i, SEED_X), (l.in_f, n), l.x_dist, dt), dt)
            t0 = time.perf_counter()
            direct.linear(x, wm, threads=threads)
            t_total += time.perf_counter() - t0
            kept_flops += 2.0 * int(m.sum()) * n
    return t_total, kept_flops


# ------------------------------------------------------------ profile summaries ---
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


def _short(nm: str) -> str:
    return nm.replace("void ", "").replace("bsp::fwd::", "").replace("bsp::pw::", "").replace("bsp::pl::", "").replace("bsp::stem::", "").split("(")[0]


def _layer_counters(d: str, n_layers: int):
    """Per layer (dispatch order inside a step, the eager first step skipped): the
    kernel name and the mean of every counter over the timed steps."""
    rows = [r for r in _csv_rows(d, "counter_collection.csv") if is_forward(r["Kernel_Name"])]
    by_id = {}
    for r in rows:
        e = by_id.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"], "c": {}})
        e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    ids = sorted(by_id)
    if len(ids) < 2 * n_layers or len(ids) % n_layers:
        raise SystemExit("%s: %d forward dispatches, not whole steps of %d" % (d, len(ids), n_layers))
    steps = len(ids) // n_layers - 1
    out = []
    for li in range(n_layers):
        sel = [by_id[ids[(s + 1) * n_layers + li]] for s in range(steps)]
        names = {e["name"] for e in sel}
        keys = set().union(*(e["c"].keys() for e in sel))
        out.append({"kernel": _short(sorted(names)[0]),
                    "c": {k: sum(e["c"].get(k, 0.0) for e in sel) / steps for k in keys}})
    return out, steps


def summarize(args):
    """Write the forward-kernel summaries (kernel trace statistics; the HBM counters
    scaled by the calibration copy; the per-layer MFMA / VALU / LDS counters) to
    the profiles folder."""
    from synthetic import workload
    layers = workload(3, batch=args.batch)
    n_layers = len(layers)
    lines = []
    kv = {"source_hash": source_hash()}
    if args.summarize:
        stats = _csv_rows(args.summarize, "kernel_stats.csv")
        conv = [r for r in stats if is_forward(r["Name"])]
        calls = sum(int(r["Calls"]) for r in conv)
        total_ns = sum(float(r["TotalDurationNs"]) for r in conv)
        lines += ["# Forward kernels (k_stem: conv1; k_fwd: the 3x3 layers; k_pl: 1x1 layers with more than 64 input channels; "
                  "k_pw: the other 1x1 layers and fc) on the "
                  "ResNet-50 v1.5 layer pass (batch 64, bf16, %d launches per step)" % n_layers, "",
                  "Kernel trace statistics (rocprofv3 --kernel-trace --stats), command:", "",
                  "    " + args.trace_cmd, "",
                  "| kernel | calls | total us | average us | min us | max us |", "|---|---|---|---|---|---|"]
        for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
            nm = r["Name"]
            short = _short(nm) if is_forward(nm) else nm[:60]
            lines.append("| %s | %s | %.1f | %.3f | %.3f | %.3f |" % (
                short, r["Calls"], float(r["TotalDurationNs"]) / 1e3, float(r["AverageNs"]) / 1e3,
                float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3))
        aux_ns = sum(float(r["TotalDurationNs"]) for r in stats if any(t in r["Name"] for t in AUX_TAGS))
        n_steps = calls / n_layers
        lines += ["", "Forward kernels, all instantiations: %d calls, average %.3f us per launch, %.1f us per step "
                  "of %d launches" % (calls, total_ns / calls / 1e3, total_ns / calls * n_layers / 1e3, n_layers),
                  "", "Expansion (im2col) and split-K sum kernels of the layers that take them: %.1f us per step; "
                  "all kernels of a step: %.1f us" % (aux_ns / n_steps / 1e3, (total_ns + aux_ns) / n_steps / 1e3), ""]
        kv["kernel_avg_us_trace"] = "%.3f" % (total_ns / calls / 1e3)
        if args.pmc_fetch and args.pmc_write:
            f_kib, nf, f_cal = _pmc_per_launch(args.pmc_fetch, "FETCH_SIZE", n_layers)
            w_kib, nw, w_cal = _pmc_per_launch(args.pmc_write, "WRITE_SIZE", n_layers)
            f_scale = CALIB_BYTES / (f_cal * 1024.0)
            w_scale = CALIB_BYTES / (w_cal * 1024.0)
            fetch = f_kib * 1024.0 * f_scale
            write = w_kib * 1024.0 * w_scale
            lines += ["HBM counters (one rocprofv3 --pmc pass each), commands:", "",
                      "    " + args.fetch_cmd, "    " + args.write_cmd, "",
                      "Calibration: a plain copy kernel (torch.neg, %d MiB in, %d MiB out) reads FETCH_SIZE %.0f KiB "
                      "and WRITE_SIZE %.0f KiB, so the scale factors are %.4f (fetch) and %.4f (write)."
                      % (CALIB_BYTES >> 20, CALIB_BYTES >> 20, f_cal, w_cal, f_scale, w_scale), "",
                      "Forward kernels per launch (mean over %d / %d dispatches of the timed steps): fetch %.3f MB, "
                      "write %.3f MB, traffic %.3f MB" % (nf, nw, fetch / 1e6, write / 1e6, (fetch + write) / 1e6), ""]
            kv.update({"fetch_bytes_per_launch": "%.0f" % fetch, "write_bytes_per_launch": "%.0f" % write,
                       "traffic_bytes_per_launch": "%.0f" % (fetch + write),
                       "fetch_scale": "%.5f" % f_scale, "write_scale": "%.5f" % w_scale})
        os.makedirs(os.path.dirname(os.path.abspath(args.out)), exist_ok=True)
        with open(args.out, "w") as f:
            f.write("\n".join(lines))
        if args.pmc_fetch and args.pmc_write:
            with open(COUNTERS_FILE, "w") as f:
                f.write("# forward-kernel HBM bytes per launch on the ResNet-50 layer pass; written by "
                        "bench.py --summarize\n")
                f.write("# from the passes listed in %s\n" % os.path.basename(args.out))
                for k, v in kv.items():
                    f.write("%s: %s\n" % (k, v))
        print("\n".join(lines))
    if args.pmc_mfma:
        summarize_mfma(args, layers)


def summarize_mfma(args, layers):
    """Per-layer MFMA / VALU / LDS counters of the ResNet-50 pass: executed MFMA
    FLOPs (bf16 MOPs x 512: dense-expanded zeros and K padding included) against the
    kept FLOPs of the method, the counters' MFMA busy fraction, VALU and LDS
    instructions per MFMA, LDS bank-conflict cycles."""
    import numpy as np
    from synthetic import draw, seed_for, SEED_W
    from oracle import prune as OP
    n_layers = len(layers)
    per, steps = None, None
    for d in args.pmc_mfma.split(","):      # one or more passes; counters merged per layer
        p2, s2 = _layer_counters(d, n_layers)
        if per is None:
            per, steps = p2, s2
        else:
            for a, b in zip(per, p2):
                assert a["kernel"] == b["kernel"], (a["kernel"], b["kernel"])
                for k, v in b["c"].items():
                    a["c"].setdefault(k, v)
            steps = min(steps, s2)
    rows = []
    tot = {"exec": 0.0, "kept": 0.0, "busy": 0.0, "active": 0.0}
    by_kernel = {}
    for i, (l, e) in enumerate(zip(layers, per)):
        c = e["c"]
        w = draw(seed_for(3, i, SEED_W), l.w_shape, l.w_dist, "bf16")
        m = OP.prune_mask(OP.as_f64(w, "bf16").reshape(l.scheme.rows, -1), l.scheme.bh, l.scheme.bw,
                          l.scheme.regularity, l.scheme.rate)
        kept = 2.0 * float(m.sum()) * l.pixels
        exe = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512.0
        mfma = max(c.get("SQ_INSTS_MFMA", 0.0), 1.0)
        busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        active = max(c.get("GRBM_GUI_ACTIVE", 0.0) / N_XCD, 1.0)   # GPU cycles the kernel was active
        valu_other = c.get("SQ_INSTS_VALU", 0.0) - c.get("SQ_INSTS_MFMA", 0.0)
        rows.append((l.name, e["kernel"], kept / 1e9, exe / 1e9, exe / max(kept, 1.0), busy / (active * N_SIMD),
                     valu_other / mfma, c.get("SQ_INSTS_LDS", 0.0) / mfma,
                     c.get("SQ_LDS_BANK_CONFLICT", 0.0) / active / 256.0))
        tot["exec"] += exe
        tot["kept"] += kept
        tot["busy"] += busy
        tot["active"] += active
        k = by_kernel.setdefault(e["kernel"], [0, 0.0, 0.0, 0.0, 0.0, 0.0])
        k[0] += 1
        k[1] += kept
        k[2] += exe
        k[3] += valu_other
        k[4] += mfma
        k[5] += c.get("SQ_INSTS_LDS", 0.0)
    lines = ["# MFMA, VALU and LDS counters of the forward kernels on the ResNet-50 v1.5 layer pass "
             "(batch 64, bf16)", "",
             "rocprofv3 --pmc passes (%s), commands:" % ", ".join(MFMA_COUNTERS), "",
             *["    " + c.strip() for c in args.mfma_cmd.split(";")], "",
             "Per layer, mean over %d timed steps.  executed GF = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 (what the "
             "MFMA units ran, zero-expanded rows and K padding included); kept GF = 2 x kept weights x output "
             "pixels (the method's work); MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / %d XCDs x %d SIMDs); "
             "VALU/MFMA and LDS/MFMA are instructions issued per MFMA instruction; bank conflicts are LDS "
             "bank-conflict cycles per CU per active cycle." % (steps, N_XCD, N_SIMD), "",
             "| layer | kernel | kept GF | executed GF | exec/kept | MFMA busy | VALU/MFMA | LDS/MFMA | bank confl. |",
             "|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| %s | %s | %.2f | %.2f | %.2f | %.3f | %.1f | %.2f | %.3f |" % r)
    lines += ["", "Per kernel instantiation (sums over its layers):", "",
              "| kernel | layers | kept GF | executed GF | exec/kept | VALU/MFMA | LDS/MFMA |", "|---|---|---|---|---|---|---|"]
    for k, v in sorted(by_kernel.items(), key=lambda kv: -kv[1][2]):
        lines.append("| %s | %d | %.2f | %.2f | %.2f | %.1f | %.2f |" % (k, v[0], v[1] / 1e9, v[2] / 1e9,
                                                                        v[2] / max(v[1], 1.0), v[3] / max(v[4], 1.0),
                                                                        v[5] / max(v[4], 1.0)))
    busy_frac = tot["busy"] / (tot["active"] * N_SIMD)
    lines += ["", "Pass: kept %.1f GF, executed %.1f GF (%.2fx), MFMA busy %.3f of the active time." % (
        tot["kept"] / 1e9, tot["exec"] / 1e9, tot["exec"] / tot["kept"], busy_frac), ""]
    with open(args.mfma_out, "w") as f:
        f.write("\n".join(lines))
    with open(MFMA_FILE, "w") as f:
        f.write("# forward-kernel MFMA counters of the ResNet-50 layer pass; written by bench.py --pmc-mfma\n")
        f.write("# from the pass listed in %s\n" % os.path.basename(args.mfma_out))
        f.write("source_hash: %s\n" % source_hash())
        f.write("executed_mfma_flops_per_step: %.0f\n" % tot["exec"])
        f.write("kept_flops_per_step: %.0f\n" % tot["kept"])
        f.write("mfma_busy_frac_step: %.5f\n" % busy_frac)
    print("\n".join(lines))


# ------------------------------------------------------------------- the run ---
def build_ops(args, dev):
    """Layers of the workload, packed on the GPU, with their inputs and outputs.
    Returns (ops, prep_ms, dt): ops are dicts with a run(x, y) closure, the layer's
    input / output tensors and its cost (None for the max-pool glue)."""
    import numpy as np
    import torch
    import paper_2111_11581_amd as B
    from paper_2111_11581_amd.layers import PackedLayer
    from synthetic import workload, draw, draw_device, seed_for, SEED_X, SEED_W

    cfg = args.workload
    layers = workload(cfg, batch=args.batch) if cfg == 3 else workload(cfg)
    dt = layers[0].dtype
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    bdt = B.F32 if dt == "f32" else B.BF16
    esize = 4 if dt == "f32" else 2
    wdev = []
    for i, l in enumerate(layers):
        w = draw(seed_for(cfg, i, SEED_W), l.w_shape, l.w_dist, dt)
        t = torch.from_numpy(w.reshape(l.scheme.rows, -1)) if dt == "f32" else \
            torch.from_numpy(w.reshape(l.scheme.rows, -1).view(np.int16)).view(torch.bfloat16)
        wdev.append(t.to(dev))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    packed = []
    for l, w in zip(layers, wdev):
        conv = None if l.kind != "conv" else B.ConvShape(l.n, l.cin, l.h, l.w, l.kh, l.kw, l.sh, l.sw, l.ph, l.pw)
        packed.append(PackedLayer(l.scheme, bdt, w, conv=conv))
    torch.cuda.synchronize()
    prep_ms = (time.perf_counter() - t0) * 1e3

    ops = []
    chained = cfg in (2, 4)
    cur = None
    for i, (l, p) in enumerate(zip(layers, packed)):
        x = cur if (chained and cur is not None) else draw_device(seed_for(cfg, i, SEED_X), l.x_shape, l.x_dist, dt,
                                                                  dev)
        y = torch.empty(l.y_shape, dtype=tdt, device=dev)
        nnz = int(p.mask.sum().item())
        cost = layer_cost(l, nnz, p.n_values, p.n_indices, p.n_rowptr, esize, dt)

        def run(xx, yy, l=l, p=p):
            if l.kind == "conv":
                p.conv2d(xx, yy, l.n, bdt, None, l.relu)
            else:
                p.linear(xx, yy, l.batch, bdt, None, l.relu)
        ops.append({"name": l.name, "scheme": l.scheme.label(), "x": x, "y": y, "run": run, "cost": cost})
        cur = y
        if getattr(l, "pool_after", False):
            h, w_ = l.y_shape[2], l.y_shape[3]
            yp = torch.empty((l.n, l.cout, h // 2, w_ // 2), dtype=tdt, device=dev)

            def pool(xx, yy, l=l, h=h, w_=w_):
                B.bsp_maxpool2x2(bdt, l.n, l.cout, h, w_, xx, yy)
            b_pool = esize * (y.numel() + yp.numel())
            ops.append({"name": "  max-pool 2x2 (glue)", "scheme": "-", "x": y, "y": yp, "run": pool,
                        "cost": (0.0, 0.0, float(b_pool), b_pool / PEAK_HBM)})
            cur = yp
    return ops, prep_ms, dt, len(layers)


def time_graph(g, reps: int) -> float:
    """Seconds per replay of a captured graph (events on the current stream)."""
    import torch
    g.replay()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / reps


def per_layer_times(ops, reps: int = 10):
    """Hot-cache and cold-cache kernel time of each op, seconds.  Hot: a graph of
    `reps` back-to-back launches on the same buffers (inputs stay in the caches).
    Cold: a graph of launches that rotate through buffer sets of at least 512 MiB in
    total (twice the last-level cache), each set used once per replay."""
    import torch
    out = []
    for op in ops:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                op["run"](op["x"], op["y"])
        hot = time_graph(g, 3)
        del g
        set_bytes = op["x"].numel() * op["x"].element_size() + op["y"].numel() * op["y"].element_size()
        nset = max(reps, min(4096, math.ceil(COLD_BYTES / max(set_bytes, 1))))
        xs = [op["x"]] + [op["x"].clone() for _ in range(min(nset, 64) - 1)]
        ys = [torch.empty_like(op["y"]) for _ in range(len(xs))]
        # beyond 64 distinct sets, reuse inputs with distinct outputs still cycling through >= 512 MiB
        while len(ys) < nset:
            ys.append(torch.empty_like(op["y"]))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for k in range(nset):
                op["run"](xs[k % len(xs)], ys[k])
        cold = time_graph(g, 2) / nset
        del g, xs, ys
        torch.cuda.synchronize()
        out.append((hot / reps, cold))
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, choices=(1, 2, 3, 4))
    ap.add_argument("--cpu-images", type=int, default=40, help="images (vectors) per layer in the CPU oracle sample")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--batch", type=int, default=64, help="batch of the ResNet-50 workload")
    ap.add_argument("--layers-out", default=None, help="write the per-layer table (JSON) here")
    ap.add_argument("--no-layers", action="store_true", help="skip the per-layer timing (profiling passes)")
    ap.add_argument("--summarize", default=None, metavar="TRACE_DIR",
                    help="no GPU: summarize a rocprofv3 --stats output folder (and --pmc-fetch/--pmc-write)")
    ap.add_argument("--pmc-fetch", default=None)
    ap.add_argument("--pmc-write", default=None)
    ap.add_argument("--pmc-mfma", default=None, metavar="PMC_DIR[,PMC_DIR...]",
                    help="no GPU: summarize rocprofv3 --pmc passes of the MFMA / VALU / LDS counters per layer")
    ap.add_argument("--trace-cmd", default="")
    ap.add_argument("--fetch-cmd", default="")
    ap.add_argument("--write-cmd", default="")
    ap.add_argument("--mfma-cmd", default="", help="the commands of the --pmc-mfma passes, separated by ';'")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "forward_resnet50_b64.md"))
    ap.add_argument("--mfma-out", default=os.path.join(ROOT, "profiles", "forward_resnet50_b64_mfma_counters.md"))
    args = ap.parse_args()
    if args.summarize or args.pmc_mfma:
        summarize(args)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each GPU would run its "
              "own batch shard with no exchange); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2111_11581_amd as B

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.lib()   # raises if the HIP library is not built
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ops, prep_ms, dt, n_layers = build_ops(args, dev)
    torch.cuda.synchronize()

    def step():
        for op in ops:
            op["run"](op["x"], op["y"])

    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        step()            # eager once (also loads the code objects)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()

    g_step = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_step):
        step()
    torch.cuda.synchronize()

    # plain copy kernel of known size: its HBM counters calibrate the forward kernels, and
    # its rate (bytes read + written per second) is what a plain streaming kernel reaches
    # on this GPU, beside the nominal 8 TB/s
    cal_src = torch.zeros(CALIB_BYTES // 2, dtype=torch.bfloat16, device=dev)
    cal_dst = torch.empty_like(cal_src)
    torch.neg(cal_src, out=cal_dst)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(5):
        torch.neg(cal_src, out=cal_dst)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * CALIB_BYTES / (c0.elapsed_time(c1) * 1e-3) / 1e9
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

    times = [] if args.no_layers else per_layer_times(ops)

    costs = [op["cost"] for op in ops]
    f_kept = sum(c[0] for c in costs)
    f_dense = sum(c[1] for c in costs)
    b_alg = sum(c[2] for c in costs)
    t_roof = sum(c[3] for c in costs)
    t_step = ms_per_step * 1e-3
    achieved_gbs = b_alg / t_step / 1e9
    peak = PEAK[dt]

    table = []
    for op, tt in zip(ops, times):
        c = op["cost"]
        hot, cold = tt
        table.append({"layer": op["name"], "scheme": op["scheme"], "us_hot": round(hot * 1e6, 3),
                      "us_cold": round(cold * 1e6, 3), "roof_us": round(c[3] * 1e6, 3),
                      "frac_hot": round(c[3] / hot, 4), "frac_cold": round(c[3] / cold, 4),
                      "kept_tflops_cold": round(c[0] / cold / 1e12, 2), "gbs_cold": round(c[2] / cold / 1e9, 1)})
    if table:
        print("per-layer kernel time: hot = back-to-back launches on one buffer set (inputs in the caches); "
              "cold = launches rotating through >= 512 MiB of buffer sets", file=sys.stderr)
        print("%-36s %-20s %9s %9s %9s %7s %7s %9s %8s" % ("layer", "scheme", "us_hot", "us_cold", "roof_us",
                                                          "f_hot", "f_cold", "kTF/s", "GB/s"), file=sys.stderr)
        for r in table:
            print("%-36s %-20s %9.2f %9.2f %9.2f %7.3f %7.3f %9.1f %8.0f" % (
                r["layer"], r["scheme"], r["us_hot"], r["us_cold"], r["roof_us"], r["frac_hot"], r["frac_cold"],
                r["kept_tflops_cold"], r["gbs_cold"]), file=sys.stderr)
    if args.layers_out:
        with open(args.layers_out, "w") as f:
            json.dump({"workload": WORKLOAD_NAMES[args.workload], "ms_per_step": ms_per_step, "layers": table}, f,
                      indent=1)

    roof = {"bound": "hbm",
            "kernel": "forward kernels k_stem + k_fwd + k_pl + k_pw (all instantiations, %d launches per step; the step time also holds the im2col expansion and split-K sums of the layers that take them)" % len(ops),
            "achieved": round(achieved_gbs, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": round(achieved_gbs * 1e9 / PEAK_HBM, 4), "traffic": None,
            "algorithmic_bytes_per_launch": round(b_alg / len(ops)),
            "algorithmic_bytes_per_step": int(b_alg),
            "avg_launch_us": round(ms_per_step * 1e3 / len(ops), 3),
            "copy_gbs": round(copy_gbs, 1), "frac_of_copy": round(achieved_gbs / copy_gbs, 4)}
    kept_util = f_kept / t_step / peak
    roof["mfma"] = {"peak_tflops": peak / 1e12, "kept_tflops": round(f_kept / t_step / 1e12, 3),
                    "kept_frac": round(kept_util, 4), "executed_tflops": None, "executed_frac": None,
                    "counter_busy_frac": None}
    if args.workload == 3:
        traffic = read_counters()
        roof["traffic"] = None if traffic is None else round(traffic)
        mf = read_mfma_counters()
        if mf is not None:
            roof["mfma"]["executed_tflops"] = round(mf[0] / t_step / 1e12, 3)
            roof["mfma"]["executed_frac"] = round(mf[0] / t_step / peak, 4)
            roof["mfma"]["counter_busy_frac"] = round(mf[1], 4)

    out = {
        "metric": METRIC,
        "value": round(f_kept / t_step / 1e12, 3),
        "unit": "TFLOP/s (kept FLOPs, whole %s)" % ("ResNet-50 layer pass" if args.workload == 3 else "workload pass"),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_layer": round(ms_per_step / n_layers, 5),
        "effective_tflops": round(f_dense / t_step / 1e12, 3),
        "roof_frac_step": round(t_roof / t_step, 4),
        "roof_ms_step": round(t_roof * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded %s; no dataset)" % (
            "N(0,1) activations, He-normal weights" if args.workload in (2, 3) else
            "U[-1,1] activations, N(0,0.05) weights" if args.workload == 1 else "U[-1,1] activations, N(0,0.02) weights"),
        "config": {"workload": WORKLOAD_NAMES[args.workload], "layers": n_layers,
                   "batch": args.batch if args.workload == 3 else {1: 1, 2: 32, 4: 512}[args.workload]},
        "roofline": roof,
        "prep_ms": round(prep_ms, 1),
        "wall_s_timed": round(wall_s, 4),
    }
    if not args.no_cpu:
        from synthetic import workload
        layers = workload(3, batch=args.batch) if args.workload == 3 else workload(args.workload)
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        t_cpu, kf = cpu_baseline(layers, args.workload, args.cpu_images, threads, dt)
        model, phys = cpu_info()
        out["cpu_baseline"] = {"value": round(kf / t_cpu / 1e12, 6),
                               "unit": "TFLOP/s (kept FLOPs; oracle does every dense MAC in fp64)",
                               "cores": threads, "kind": "oracle",
                               "sample": "all %d layers, first %d images (vectors) of each, %.1f s" % (
                                   n_layers, args.cpu_images, t_cpu),
                               "cpu": model, "physical_cores": phys, "threads": threads}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
