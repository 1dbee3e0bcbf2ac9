"""Layer shapes and pruning schemes of the five synthetic workloads.

Each workload stands in for a layer mix the paper evaluates (CIFAR- and
ImageNet-shaped VGG-16 / ResNet-50 layers, large FC layers, and a block-size
sweep on one 3x3 layer, Sec. 6.2); no dataset items are used, only seeded
tensors of those shapes.

The GEMM form of a conv weight (Cout, Cin, kh, kw) has rows = Cout and
columns = Cin*kh*kw with column q = (c*kh + r)*kw + s.  A block size of 0
means the whole extent of that dimension.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

ROW, COL, UNSTRUCTURED, DENSE, PUNCHED, ROWCOL, PATTERN = 0, 1, 2, 3, 4, 5, 6
REG_NAMES = {ROW: "row", COL: "col", UNSTRUCTURED: "unstructured", DENSE: "dense", PUNCHED: "punched",
             ROWCOL: "row+col", PATTERN: "pattern"}


@dataclass(frozen=True)
class Scheme:
    rows: int
    cols: int
    bh: int            # 0 => whole extent
    bw: int            # 0 => whole extent
    regularity: int    # ROW / COL / UNSTRUCTURED / DENSE / PUNCHED
    rate: int          # integer >= 1
    khw: int = 1       # kernel locations per input channel (block-punched: blocks are
                       # bh filters x bw input channels)

    def label(self) -> str:
        if self.regularity in (UNSTRUCTURED, DENSE):
            return f"{REG_NAMES[self.regularity]} r{self.rate}"
        b = "whole" if (self.bh == 0 and self.bw == 0) else f"{self.bh}x{self.bw}"
        return f"{REG_NAMES[self.regularity]} {b} r{self.rate}"


@dataclass(frozen=True)
class ConvLayer:
    name: str
    n: int
    cin: int
    h: int
    w: int
    cout: int
    kh: int
    kw: int
    sh: int
    sw: int
    ph: int
    pw: int
    bh: int
    bw: int
    regularity: int
    rate: int
    dtype: str                      # 'f32' or 'bf16'
    x_dist: tuple
    w_dist: tuple
    relu: bool = False
    pool_after: bool = False
    count: int = 1                  # how many times the shape occurs in the net
    kind: str = field(default="conv")

    @property
    def ho(self) -> int:
        return (self.h + 2 * self.ph - self.kh) // self.sh + 1

    @property
    def wo(self) -> int:
        return (self.w + 2 * self.pw - self.kw) // self.sw + 1

    @property
    def x_shape(self):
        return (self.n, self.cin, self.h, self.w)

    @property
    def w_shape(self):
        return (self.cout, self.cin, self.kh, self.kw)

    @property
    def y_shape(self):
        return (self.n, self.cout, self.ho, self.wo)

    @property
    def pixels(self) -> int:
        return self.n * self.ho * self.wo

    @property
    def scheme(self) -> Scheme:
        return Scheme(self.cout, self.cin * self.kh * self.kw, self.bh, self.bw,
                      self.regularity, self.rate, self.kh * self.kw)


@dataclass(frozen=True)
class LinearLayer:
    name: str
    batch: int
    in_f: int
    out_f: int
    bh: int
    bw: int
    regularity: int
    rate: int
    dtype: str
    x_dist: tuple
    w_dist: tuple
    relu: bool = False
    count: int = 1
    kind: str = field(default="linear")

    @property
    def cout(self) -> int:
        return self.out_f

    @property
    def x_shape(self):           # feature-major [in_features][batch]
        return (self.in_f, self.batch)

    @property
    def w_shape(self):
        return (self.out_f, self.in_f)

    @property
    def y_shape(self):
        return (self.out_f, self.batch)

    @property
    def pixels(self) -> int:
        return self.batch

    @property
    def scheme(self) -> Scheme:
        return Scheme(self.out_f, self.in_f, self.bh, self.bw, self.regularity, self.rate)


def he_normal(fan_in: int) -> tuple:
    return ("normal", 0.0, math.sqrt(2.0 / fan_in))


def _conv(name, n, cin, h, w, cout, k, s, p, bh, bw, reg, rate, dtype, xd, wd=None, **kw):
    wd = wd or he_normal(cin * k * k)
    return ConvLayer(name, n, cin, h, w, cout, k, k, s, s, p, p, bh, bw, reg, rate, dtype, xd, wd, **kw)


def c1_single_conv():
    """One 3x3 conv, 64->64 at 32x32, batch 1, fp32; 16x16 blocks, 4x column pruning."""
    return [_conv("c1 conv3x3 64", 1, 64, 32, 32, 64, 3, 1, 1, 16, 16, COL, 4, "f32",
                  ("uniform", -1.0, 1.0), ("normal", 0.0, 0.05))]


def c2_vgg16_cifar():
    """VGG-16 on 32x32 inputs, batch 32, bf16: 13 3x3 convs, ReLU after each,
    2x2 max-pool after convs 2, 4, 7 and 10.  The first conv is dense; every
    other one has 8x16 blocks with 8x column pruning."""
    chans = [64, 64, 128, 128, 256, 256, 256, 512, 512, 512, 512, 512, 512]
    pool_after = {1, 3, 6, 9}
    layers, cin, hw = [], 3, 32
    for i, c in enumerate(chans):
        dense = i == 0
        layers.append(_conv(f"c2 conv{i + 1} {cin}->{c} @{hw}", 32, cin, hw, hw, c, 3, 1, 1,
                            0 if dense else 8, 0 if dense else 16, DENSE if dense else COL,
                            1 if dense else 8, "bf16", ("normal", 0.0, 1.0),
                            relu=True, pool_after=i in pool_after))
        cin = c
        if i in pool_after:
            hw //= 2
    return layers


def c3_resnet50_layers(batch: int = 64):
    """All conv layers of ResNet-50 v1.5 at ImageNet shape (224x224), bf16.

    conv1 (7x7/2) and fc stay dense; 1x1 convs use 32x32 blocks with 2x row
    pruning, 3x3 convs use 16x32 blocks with 4x column pruning.  The stride-2
    of each downsampling stage sits on the 3x3 conv and on the 1x1 shortcut.
    Each layer gets its own seeded N(0,1) input of its shape.
    """
    xd = ("normal", 0.0, 1.0)
    L = [_conv("conv1 7x7/2 3->64", batch, 3, 224, 224, 64, 7, 2, 3, 0, 0, DENSE, 1, "bf16", xd)]

    def c1x1(name, cin, hw, cout, s=1):
        return _conv(name, batch, cin, hw, hw, cout, 1, s, 0, 32, 32, ROW, 2, "bf16", xd)

    def c3x3(name, c, hw, s=1):
        return _conv(name, batch, c, hw, hw, c, 3, s, 1, 16, 32, COL, 4, "bf16", xd)

    cin, hw = 64, 56
    for si, (nb, mid, out) in enumerate([(3, 64, 256), (4, 128, 512), (6, 256, 1024), (3, 512, 2048)]):
        st = 1 if si == 0 else 2
        for b in range(nb):
            s = st if b == 0 else 1
            tag = f"s{si + 1}b{b + 1}"
            L.append(c1x1(f"{tag} 1x1 {cin}->{mid} @{hw}", cin, hw, mid))
            L.append(c3x3(f"{tag} 3x3 {mid} s{s} @{hw}", mid, hw, s))
            hwo = hw // s
            L.append(c1x1(f"{tag} 1x1 {mid}->{out} @{hwo}", mid, hwo, out))
            if b == 0:
                L.append(c1x1(f"{tag} ds 1x1 {cin}->{out} s{s} @{hw}", cin, hw, out, s))
            cin, hw = out, hwo
    L.append(LinearLayer("fc 2048->1000", batch, 2048, 1000, 0, 0, DENSE, 1, "bf16",
                         xd, he_normal(2048)))
    return L


def c4_fc_stack():
    """Four 4096->4096 linear layers, 512 feature-major input vectors, bf16;
    32x32 blocks with rate 10 column pruning (keeps 4 of 32, i.e. 8x)."""
    return [LinearLayer(f"c4 fc{i + 1} 4096->4096", 512, 4096, 4096, 32, 32, COL, 10, "bf16",
                        ("uniform", -1.0, 1.0), ("normal", 0.0, 0.02)) for i in range(4)]


def c5_sweep(batch: int = 64):
    """One 3x3 conv 256->256 at 56x56: block sizes x {row, col} x rates, plus
    unstructured magnitude pruning at the same rates and the dense layer."""
    xd = ("normal", 0.0, 1.0)
    L = []
    for b in (4, 8, 16, 32, 64, 0):
        for reg in (ROW, COL):
            for r in (2, 4, 8, 16):
                bs = "whole" if b == 0 else f"{b}x{b}"
                L.append(_conv(f"c5 {REG_NAMES[reg]} {bs} r{r}", batch, 256, 56, 56, 256, 3, 1, 1,
                               b, b, reg, r, "bf16", xd))
    for r in (2, 4, 8, 16):
        L.append(_conv(f"c5 unstructured r{r}", batch, 256, 56, 56, 256, 3, 1, 1, 1, 1,
                       UNSTRUCTURED, r, "bf16", xd))
    L.append(_conv("c5 dense", batch, 256, 56, 56, 256, 3, 1, 1, 0, 0, DENSE, 1, "bf16", xd))
    return L


WORKLOADS = {
    1: ("single 3x3 conv 64ch 32x32 fp32", c1_single_conv),
    2: ("VGG-16 CIFAR stack b32 bf16", c2_vgg16_cifar),
    3: ("ResNet-50 ImageNet conv layers b64 bf16", c3_resnet50_layers),
    4: ("FC 4096x4096 x4 b512 bf16", c4_fc_stack),
    5: ("3x3 conv 256ch 56x56 scheme sweep b64 bf16", c5_sweep),
}


def workload(config: int, **kw):
    return WORKLOADS[config][1](**kw)
