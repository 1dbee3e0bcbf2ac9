"""Latency model and rule-based block-size selection (Sec. 5.2.1 and 5.2.2).

The latency model is a table of forward latencies measured on this GPU for layer
settings: layer shape, regularity (row or column), block size (``0`` = the whole
matrix, i.e. coarse structured pruning) and pruning rate.  It is built once per
device by timing the library's own forward call (``measure``) and saved as JSON.

The selection rule is host logic over the table (``select_block_size``): the
latency of each candidate block size is normalised by the layer's dense MACs; a
candidate is valid when that latency is at most (1 + beta) times the latency of
structured pruning (whole-matrix blocks) at the same rate and regularity; of the
valid candidates the smallest block (finest granularity) is selected.  When none
is valid, structured pruning is returned.

Usage (GPU):
    python -m paper_2111_11581_amd.latency build --out model.json
    python -m paper_2111_11581_amd.latency select --model model.json --beta 0.2
"""

from __future__ import annotations

import argparse
import json
import math
import sys
from dataclasses import asdict, dataclass

REG_NAMES = {0: "row", 1: "col", 2: "unstructured", 3: "dense", 4: "punched", 6: "pattern"}
BLOCK_REGS = (0, 1, 4)   # regularities with a block size (the rule selects among them)


@dataclass(frozen=True)
class Setting:
    """One layer setting of the latency model (a conv; a linear layer is a 1x1 conv
    over a 1 x batch image with cin = input features)."""
    cin: int
    cout: int
    h: int
    w: int
    kh: int
    kw: int
    stride: int
    pad: int
    batch: int
    regularity: int   # 0 row, 1 column, 2 unstructured, 3 dense, 4 block-punched (package constants)
    bh: int           # block height (0: whole matrix; 1 for unstructured; punched: filters)
    bw: int           # block width (0: whole matrix; 1 for unstructured; punched: input channels)
    rate: int

    def key(self) -> str:
        if self.regularity == 3:
            b = "-"
        elif self.regularity == 2:
            b = "1x1"
        elif self.regularity == 6:
            b = f"{self.bh}p"
        else:
            b = "whole" if self.bh == 0 and self.bw == 0 else f"{self.bh}x{self.bw}"
        return (f"{self.kh}x{self.kw}/{self.stride} {self.cin}->{self.cout} {self.h}x{self.w} b{self.batch} "
                f"{REG_NAMES[self.regularity]} {b} r{self.rate}")

    def layer_key(self) -> str:
        """The setting without regularity, block and rate: the layer the rule selects for."""
        return f"{self.kh}x{self.kw}/{self.stride} {self.cin}->{self.cout} {self.h}x{self.w} b{self.batch}"

    @property
    def ho(self) -> int:
        return (self.h + 2 * self.pad - self.kh) // self.stride + 1

    @property
    def wo(self) -> int:
        return (self.w + 2 * self.pad - self.kw) // self.stride + 1

    def macs(self) -> int:
        """Dense multiply-accumulates of the layer (the normaliser of Sec. 5.2.2)."""
        return self.batch * self.cout * self.ho * self.wo * self.cin * self.kh * self.kw

    def area(self) -> int:
        """Block area in weight elements (whole matrix: rows x cols; a block-punched
        block of bh filters x bw channels holds bh * bw kernels)."""
        if self.regularity == 4:
            return (self.bh or self.cout) * (self.bw or self.cin) * self.kh * self.kw
        rows, cols = self.cout, self.cin * self.kh * self.kw
        return (self.bh or rows) * (self.bw or cols)


# MI355X peaks the roofline fractions are taken against (dense bf16 MFMA, HBM3E)
PEAK_BF16_FLOPS = 2.5166e15
PEAK_HBM_BYTES = 8.0e12


def _kept_of(extent: int, block: int, rate: int) -> int:
    """Kept groups of an extent cut into blocks (0: one block), each keeping
    ceil(block / rate) (Sec. 4.1.1; the last block may be ragged)."""
    b = block or extent
    full, last = divmod(extent, b)
    return full * -(-b // rate) + (-(-last // rate) if last else 0)


def kept_fraction(s: Setting) -> float:
    """Fraction of the GEMM-form weights a setting keeps, from its scheme alone."""
    khw = s.kh * s.kw
    rows, cols = s.cout, s.cin * khw
    if s.regularity == 3:
        return 1.0
    if s.regularity == 1:
        return _kept_of(cols, s.bw, s.rate) / cols
    if s.regularity == 0:
        return _kept_of(rows, s.bh, s.rate) / rows
    if s.regularity == 4:
        return -(-khw // s.rate) / khw
    if s.regularity == 6:      # 4 of 9 weights of each kept kernel; connectivity keeps ceil(9 n / 4 r) of n
        n = rows * s.cin
        return 4.0 * min(n, -(-9 * n // (4 * s.rate))) / (9 * n)
    n = rows * cols
    return -(-n // s.rate) / n


def roofline(s: Setting, ms: float):
    """(roofline fraction, bound) of one measured setting: the larger of the kept-FLOP
    time at the bf16 MFMA peak and the algorithmic HBM time (input, output, kept
    weights, bf16) at the HBM peak, over the measured time."""
    kept = kept_fraction(s)
    t_mfma = 2.0 * s.macs() * kept / PEAK_BF16_FLOPS
    nbytes = 2.0 * (s.batch * s.cin * s.h * s.w + s.batch * s.cout * s.ho * s.wo +
                    kept * s.cout * s.cin * s.kh * s.kw)
    t_hbm = nbytes / PEAK_HBM_BYTES
    return max(t_mfma, t_hbm) / (ms * 1e-3), ("mfma" if t_mfma > t_hbm else "hbm")


class LatencyModel:
    """Measured forward latency (milliseconds) per setting."""

    def __init__(self, entries=None, meta=None):
        self.ms = {}          # key -> ms
        self.settings = {}    # key -> Setting
        self.meta = dict(meta or {})
        for s, ms in (entries or []):
            self.add(s, ms)

    def add(self, s: Setting, ms: float):
        if not (ms > 0 and math.isfinite(ms)):
            raise ValueError(f"latency of {s.key()} must be a positive number, got {ms}")
        self.ms[s.key()] = float(ms)
        self.settings[s.key()] = s

    def latency(self, s: Setting) -> float:
        return self.ms[s.key()]

    def normalized(self, s: Setting) -> float:
        """Latency per dense MAC (Sec. 5.2.2)."""
        return self.ms[s.key()] / s.macs()

    def save(self, path: str):
        with open(path, "w") as f:
            json.dump({"meta": self.meta,
                       "entries": [dict(asdict(self.settings[k]), ms=self.ms[k]) for k in sorted(self.ms)]},
                      f, indent=1)

    @classmethod
    def load(cls, path: str) -> "LatencyModel":
        with open(path) as f:
            d = json.load(f)
        m = cls(meta=d.get("meta"))
        for e in d["entries"]:
            ms = e.pop("ms")
            m.add(Setting(**e), ms)
        return m


def select_block_size(model: LatencyModel, layer: Setting, regularity: int, rate: int, beta: float = 0.2):
    """The smallest block whose normalised latency is within (1 + beta) of structured
    pruning (whole-matrix blocks) at the same regularity and rate (Sec. 5.2.2).

    ``layer`` gives the layer shape (its regularity, block and rate fields are
    ignored).  Returns (bh, bw); (0, 0) is structured pruning, also returned when no
    block size qualifies.  Raises KeyError when the model holds no structured entry
    for the layer, regularity and rate.
    """
    if beta < 0:
        raise ValueError("beta must be >= 0")
    lk = layer.layer_key()
    cands = [s for s in model.settings.values()
             if s.layer_key() == lk and s.regularity == regularity and s.rate == rate]
    ref = [s for s in cands if s.bh == 0 and s.bw == 0]
    if not ref:
        raise KeyError(f"no structured (whole-matrix) entry for {lk} {REG_NAMES[regularity]} r{rate}")
    limit = (1.0 + beta) * model.normalized(ref[0])
    valid = [s for s in cands if not (s.bh == 0 and s.bw == 0) and model.normalized(s) <= limit]
    if not valid:
        return (0, 0)
    best = min(valid, key=lambda s: (s.area(), s.bh, s.bw))
    return (best.bh, best.bw)


# ---- building the model on the GPU ----

def sweep_settings(cin=256, cout=256, h=56, w=56, k=3, batch=64, blocks=(4, 8, 16, 32, 64, 0),
                   rates=(2, 4, 8, 16), regularities=BLOCK_REGS, references=False):
    """The block-size sweep of one conv layer: square blocks (0 = whole matrix) x
    regularity x rate (defaults: 3x3 256->256 at 56x56, batch 64; row, column and
    block-punched, whose blocks are filters x input channels).  With
    ``references``, also unstructured magnitude pruning at each rate and the dense
    layer (reference points; the selection rule does not use them)."""
    st = [Setting(cin, cout, h, w, k, k, 1, k // 2, batch, reg, b, b, r)
          for b in blocks for reg in regularities for r in rates]
    if references:
        st += [Setting(cin, cout, h, w, k, k, 1, k // 2, batch, 2, 1, 1, r) for r in rates]
        if k == 3:   # pattern-based pruning (8 patterns), the 3x3 comparison point of Sec. 5.2.3
            st += [Setting(cin, cout, h, w, k, k, 1, k // 2, batch, 6, 8, 0, r) for r in rates]
        st.append(Setting(cin, cout, h, w, k, k, 1, k // 2, batch, 3, 0, 0, 1))
    return st


def network_settings(layers, blocks=(4, 8, 16, 32, 64, 0), rates=(4,)):
    """Settings of a network's conv layers (distinct shapes): every block size at each
    rate, column and row blocks for every layer and block-punched blocks for K x K
    kernels (K > 1), plus the whole-matrix reference of each regularity.  ``layers``
    holds (cin, cout, h, w, k, stride, batch) tuples."""
    seen, st = set(), []
    for cin, cout, h, w, k, stride, batch in layers:
        key = (cin, cout, h, w, k, stride, batch)
        if key in seen:
            continue
        seen.add(key)
        regs = (0, 1, 4) if k > 1 else (0, 1)
        for reg in regs:
            for b in blocks:
                for r in rates:
                    st.append(Setting(cin, cout, h, w, k, k, stride, k // 2, batch, reg, b, b, r))
    return st


def measure(settings, reps: int = 10, rounds: int = 10, seed: int = 1234, device=None) -> LatencyModel:
    """Times the library's forward call for each setting (bf16): a graph of ``reps``
    back-to-back launches of the layer (the test model of ten layers of one setting,
    Sec. 5.2.1), replayed ``rounds`` times (100 runs by default); mean per launch.
    Weights and activations are seeded normal draws made on the device (He-normal
    weights): the latency depends on the shapes and the kept structure only."""
    import torch
    from . import BF16, BspError, ConvShape, Scheme, bsp_version
    from .layers import PackedLayer

    dev = torch.device(device or "cuda:0")
    gen = torch.Generator(device=dev)
    model = LatencyModel(meta={"device": torch.cuda.get_device_name(dev), "library_version": bsp_version(),
                               "dtype": "bf16", "reps": reps, "rounds": rounds})
    for s in settings:
        gen.manual_seed(seed)
        rows, cols = s.cout, s.cin * s.kh * s.kw
        wd = (torch.randn(rows, cols, generator=gen, device=dev) * math.sqrt(2.0 / cols)).to(torch.bfloat16)
        x = torch.randn(s.batch, s.cin, s.h, s.w, generator=gen, device=dev).to(torch.bfloat16)
        y = torch.empty(s.batch, s.cout, s.ho, s.wo, dtype=torch.bfloat16, device=dev)
        scheme = Scheme(rows, cols, s.bh, s.bw, s.regularity, s.rate, s.kh * s.kw)
        conv = ConvShape(s.batch, s.cin, s.h, s.w, s.kh, s.kw, s.stride, s.stride, s.pad, s.pad)
        try:
            p = PackedLayer(scheme, BF16, wd, conv=conv)
        except BspError as e:   # a setting the library does not run is left out of the model
            print(f"skipped {s.key()}: {e}", flush=True)
            continue
        p.conv2d(x, y, s.batch, BF16)
        torch.cuda.synchronize(dev)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                p.conv2d(x, y, s.batch, BF16)
        g.replay()
        torch.cuda.synchronize(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(rounds):
            g.replay()
        e1.record()
        torch.cuda.synchronize(dev)
        model.add(s, e0.elapsed_time(e1) / (reps * rounds))
        del g, p
    return model


def summary(model: LatencyModel, beta: float = 0.2) -> str:
    """Markdown table of the rule's block size per layer, regularity and rate at one
    beta, with the chosen setting's latency beside the whole-matrix one (us)."""
    layers = {}
    for s in model.settings.values():
        layers.setdefault(s.layer_key(), []).append(s)
    out = []
    for r in sorted({s.rate for s in model.settings.values() if s.regularity in BLOCK_REGS}):
        regs = [g for g in BLOCK_REGS if any(s.regularity == g and s.rate == r for s in model.settings.values())]
        out.append(f"## Block size per layer at beta = {beta:g} (rate {r}): choice (its latency / whole-matrix "
                   f"latency, us)\n")
        out.append("| layer | " + " | ".join(REG_NAMES[g] for g in regs) + " |")
        out.append("|---|" + "---|" * len(regs))
        for lk in sorted(layers):
            st = layers[lk]
            cells = []
            for g in regs:
                try:
                    bh, bw = select_block_size(model, st[0], g, r, beta)
                except KeyError:
                    cells.append("-")
                    continue
                pick = [s for s in st if s.regularity == g and s.rate == r and (s.bh, s.bw) == (bh, bw)]
                whole = [s for s in st if s.regularity == g and s.rate == r and (s.bh, s.bw) == (0, 0)]
                name = "whole" if (bh, bw) == (0, 0) else f"{bh}x{bw}"
                cells.append(f"{name} ({model.latency(pick[0]) * 1e3:.0f} / {model.latency(whole[0]) * 1e3:.0f})")
            out.append(f"| {lk} | " + " | ".join(cells) + " |")
        out.append("")
    return "\n".join(out)


def report(model: LatencyModel, betas=(0.0, 0.1, 0.2, 0.5)) -> str:
    """Markdown summary of a model: per layer, the latency of every block size and
    rate (and its ratio to whole-matrix pruning at the same regularity and rate), the
    reference points, and the rule's choice for each beta.  A model of several layers
    starts with the per-layer choice at beta 0.2 (or the middle beta given)."""
    out = []
    layers = {}
    for s in model.settings.values():
        layers.setdefault(s.layer_key(), []).append(s)
    if len(layers) > 1:
        out.append(summary(model, 0.2 if 0.2 in betas else betas[len(betas) // 2]))
    for lk in sorted(layers):
        st = layers[lk]
        rates = sorted({s.rate for s in st if s.regularity in BLOCK_REGS})
        out.append(f"### {lk}\n")
        for reg in BLOCK_REGS:
            rs = [s for s in st if s.regularity == reg]
            if not rs:
                continue
            out.append(f"{REG_NAMES[reg]} pruning: latency in us (ratio to whole-matrix blocks at the same rate)\n")
            out.append("| block | " + " | ".join(f"{r}x" for r in rates) + " |")
            out.append("|---|" + "---|" * len(rates))
            blocks = sorted({(s.bh, s.bw) for s in rs}, key=lambda b: (b == (0, 0), b))
            for b in blocks:
                cells = []
                for r in rates:
                    x = [s for s in rs if (s.bh, s.bw) == b and s.rate == r]
                    w = [s for s in rs if (s.bh, s.bw) == (0, 0) and s.rate == r]
                    if not x:
                        cells.append("-")
                        continue
                    us = model.latency(x[0]) * 1e3
                    cells.append(f"{us:.1f} ({model.latency(x[0]) / model.latency(w[0]):.2f})" if w else f"{us:.1f}")
                name = "whole" if b == (0, 0) else f"{b[0]}x{b[1]}"
                out.append(f"| {name} | " + " | ".join(cells) + " |")
            out.append("")
        out.append("roofline fraction of each setting (the larger of the kept-FLOP time at the bf16 MFMA peak and the "
                   "algorithmic HBM time at 8 TB/s, over the measured time; m: MFMA-bound, h: HBM-bound)\n")
        out.append("| regularity | block | " + " | ".join(f"{r}x" for r in rates) + " |")
        out.append("|---|---|" + "---|" * len(rates))
        for reg in BLOCK_REGS:
            rs = [s for s in st if s.regularity == reg]
            for b in sorted({(s.bh, s.bw) for s in rs}, key=lambda b: (b == (0, 0), b)):
                cells = []
                for r in rates:
                    x = [s for s in rs if (s.bh, s.bw) == b and s.rate == r]
                    if not x:
                        cells.append("-")
                        continue
                    f, bound = roofline(x[0], model.latency(x[0]))
                    cells.append(f"{f:.3f} {bound[0]}")
                name = "whole" if b == (0, 0) else f"{b[0]}x{b[1]}"
                out.append(f"| {REG_NAMES[reg]} | {name} | " + " | ".join(cells) + " |")
        out.append("")
        refs = [s for s in st if s.regularity in (2, 3, 6)]
        if refs:
            names = {2: "unstructured", 3: "dense", 6: "pattern (8 patterns)"}
            out.append("reference points: " + ", ".join(
                f"{names[s.regularity]}{'' if s.regularity == 3 else f' {s.rate}x'} {model.latency(s) * 1e3:.1f} us "
                f"(roofline {roofline(s, model.latency(s))[0]:.3f})"
                for s in sorted(refs, key=lambda s: (s.regularity, s.rate))) + "\n")
        out.append("rule choice (smallest block within (1 + beta) of whole-matrix blocks, latency per dense MAC):\n")
        out.append("| regularity | rate | " + " | ".join(f"beta {b:g}" for b in betas) + " |")
        out.append("|---|---|" + "---|" * len(betas))
        for reg in BLOCK_REGS:
            for r in rates:
                cells = []
                for b in betas:
                    try:
                        bh, bw = select_block_size(model, st[0], reg, r, b)
                    except KeyError:
                        cells.append("-")
                        continue
                    cells.append("whole" if (bh, bw) == (0, 0) else f"{bh}x{bw}")
                out.append(f"| {REG_NAMES[reg]} | {r}x | " + " | ".join(cells) + " |")
        out.append("")
    return "\n".join(out)


def _main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    b = sub.add_parser("build", help="measure the block-size sweep of one 3x3 conv on the GPU")
    b.add_argument("--out", required=True)
    b.add_argument("--cin", type=int, default=256)
    b.add_argument("--hw", type=int, default=56)
    b.add_argument("--batch", type=int, default=64)
    b.add_argument("--resnet50", action="store_true",
                   help="the distinct ResNet-50 v1.5 conv shapes at 224x224 (rate 4) instead of the sweep layer")
    s = sub.add_parser("select", help="block size per regularity and rate from a saved model")
    s.add_argument("--model", required=True)
    s.add_argument("--beta", type=float, default=0.2)
    r = sub.add_parser("report", help="markdown summary of a saved model and the rule's choices")
    r.add_argument("--model", required=True)
    r.add_argument("--betas", type=float, nargs="+", default=[0.0, 0.1, 0.2, 0.5])
    a = ap.parse_args(argv)
    if a.cmd == "report":
        print(report(LatencyModel.load(a.model), tuple(a.betas)))
        return 0
    if a.cmd == "build":
        if a.resnet50:
            from synthetic import workload   # layer shapes only
            st = network_settings([(l.cin, l.cout, l.h, l.w, l.kh, l.sh, a.batch) for l in workload(3)
                                   if l.kind == "conv" and not (l.kh == 7)])
        else:
            st = sweep_settings(cin=a.cin, cout=a.cin, h=a.hw, w=a.hw, batch=a.batch, references=True)
        m = measure(st)
        m.save(a.out)
        for k in sorted(m.ms):
            print(f"{k:56s} {m.ms[k] * 1e3:9.1f} us", flush=True)
        return 0
    m = LatencyModel.load(a.model)
    layers = {x.layer_key(): x for x in m.settings.values()}
    for lk, layer in sorted(layers.items()):
        for reg in BLOCK_REGS:
            for rate in sorted({x.rate for x in m.settings.values() if x.layer_key() == lk}):
                try:
                    bh, bw = select_block_size(m, layer, reg, rate, a.beta)
                except KeyError:
                    continue
                print(f"{lk} {REG_NAMES[reg]} r{rate}: beta {a.beta:.2f} -> "
                      f"{'whole matrix' if bh == 0 else f'{bh}x{bw}'}")
    return 0


if __name__ == "__main__":
    sys.exit(_main())
