"""GPU parity: the HIP path through the C ABI against the CPU oracle on the same
seeded inputs.  Masks, indices, rowptr and packed values are compared bit-exact.
Every forward output is gated three ways (tests/helpers.check_output): relative L2
error over the whole output (<= 1e-5 for fp32, <= 5e-3 for bf16 inputs with fp32
accumulation and bf16 output), the same per (image, output channel) plane, and an
element-wise rounding bound, so that a localised mistake cannot hide in the norm."""

import numpy as np
import pytest

from oracle import prune as OP
from synthetic import (workload, draw, draw_layer, seed_for, ConvLayer, LinearLayer, ROW, COL, UNSTRUCTURED, DENSE,
                       PUNCHED, ROWCOL, PATTERN)
from tests.helpers import (DT, TOL, to_dev, from_dev, as_f64, rel_l2, oracle_mask, oracle_conv, oracle_linear,
                           out_to_f64, gate_conv, gate_linear)

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module")
def B():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2111_11581_amd as B
    B.lib()
    return B


def _layers():
    from paper_2111_11581_amd import layers
    return layers


# ------------------------------------------------------------------ masks/pack ---
MATS = [  # name, R, C, bh, bw, reg, rate, dtype, dist
    ("c1 64x576 col16x16 r4 f32", 64, 576, 16, 16, COL, 4, "f32", ("normal", 0, 0.05)),
    ("c2 256x1152 col8x16 r8", 256, 1152, 8, 16, COL, 8, "bf16", ("normal", 0, 0.04)),
    ("c3 512x4608 col16x32 r4", 512, 4608, 16, 32, COL, 4, "bf16", ("normal", 0, 0.02)),
    ("c3 2048x512 row32x32 r2", 2048, 512, 32, 32, ROW, 2, "bf16", ("normal", 0, 0.06)),
    ("c4 4096x4096 col32x32 r10", 4096, 4096, 32, 32, COL, 10, "bf16", ("normal", 0, 0.02)),
    ("c5 4x4 row r16", 256, 2304, 4, 4, ROW, 16, "bf16", ("normal", 0, 0.03)),
    ("c5 64x64 col r2", 256, 2304, 64, 64, COL, 2, "bf16", ("normal", 0, 0.03)),
    ("c5 whole col r8", 256, 2304, 0, 0, COL, 8, "bf16", ("normal", 0, 0.03)),
    ("c5 whole row r4", 256, 2304, 0, 0, ROW, 4, "bf16", ("normal", 0, 0.03)),
    ("c5 unstructured r4", 256, 2304, 1, 1, UNSTRUCTURED, 4, "bf16", ("normal", 0, 0.03)),
    ("unstructured r3 f32", 100, 77, 1, 1, UNSTRUCTURED, 3, "f32", ("normal", 0, 1.0)),
    ("dense", 64, 147, 0, 0, DENSE, 1, "bf16", ("normal", 0, 0.1)),
    ("ragged col", 37, 53, 8, 16, COL, 3, "bf16", ("normal", 0, 1.0)),
    ("ragged row", 37, 53, 8, 16, ROW, 3, "f32", ("normal", 0, 1.0)),
    ("ties col", 48, 96, 16, 32, COL, 4, "bf16", ("ties",)),
    ("ties row", 96, 48, 32, 16, ROW, 4, "f32", ("ties",)),
    ("ties unstructured", 64, 64, 1, 1, UNSTRUCTURED, 5, "bf16", ("ties",)),
    ("rowcol 16x32 r2", 64, 576, 16, 32, ROWCOL, 2, "bf16", ("normal", 0, 0.05)),
    ("rowcol ragged 8x16 r3 f32", 37, 53, 8, 16, ROWCOL, 3, "f32", ("normal", 0, 1.0)),
    ("rowcol whole r4", 96, 300, 0, 0, ROWCOL, 4, "bf16", ("normal", 0, 0.05)),
    ("ties rowcol", 48, 96, 16, 32, ROWCOL, 4, "bf16", ("ties",)),
]


def _mat(i, R, C, dtype, dist):
    if dist[0] == "ties":   # small integers: many exactly equal scores
        a = np.random.default_rng(900 + i).integers(-2, 3, size=(R, C)).astype(np.float32)
        return a if dtype == "f32" else (a.view(np.uint32) >> 16).astype(np.uint16)
    return draw(seed_for(9, i, 1), (R, C), dist, dtype)


@pytest.mark.parametrize("i", range(len(MATS)), ids=[m[0] for m in MATS])
def test_prune_and_pack_bit_exact(B, i):
    import torch
    name, R, C, bh, bw, reg, rate, dtype, dist = MATS[i]
    w = _mat(i, R, C, dtype, dist)
    scheme = B.Scheme(R, C, bh, bw, reg, rate)
    wd = to_dev(w, dtype)
    layer = _layers().PackedLayer(scheme, DT[dtype], wd)
    torch.cuda.synchronize()
    m_ref = oracle_mask(w, dtype, scheme)
    m_gpu = layer.mask.cpu().numpy().reshape(R, C)
    assert np.array_equal(m_gpu, m_ref), f"{name}: {int((m_gpu != m_ref).sum())} mask entries differ"
    pk = OP.pack(w, m_ref, bh, bw, reg, rate)
    vals = from_dev(layer.values[:layer.n_values], dtype)
    assert np.array_equal(vals.view(np.uint8), np.ascontiguousarray(pk["values"]).view(np.uint8))
    if reg in (ROW, COL, ROWCOL):
        assert np.array_equal(layer.indices[:layer.n_indices].cpu().numpy(), pk["indices"])
        assert np.array_equal(layer.rowptr[:layer.n_rowptr].cpu().numpy(), pk["rowptr"])
    back = from_dev(layer.unpack(), dtype).reshape(R, C)
    expect = np.where(m_ref == 1, w, np.zeros_like(w))
    assert np.array_equal(back.view(np.uint8), expect.view(np.uint8))


PUNCHED_MATS = [  # name, R, cin, khw, bh (filters), bw (channels), rate, dtype, dist
    ("3x3 16x8 r2", 64, 64, 9, 16, 8, 2, "bf16", ("normal", 0, 0.05)),
    ("3x3 ragged 8xwhole r3 f32", 37, 20, 9, 8, 0, 3, "f32", ("normal", 0, 1.0)),
    ("c5 3x3 whole r4", 256, 256, 9, 0, 0, 4, "bf16", ("normal", 0, 0.03)),
    ("5x5 whole x5 r4", 48, 12, 25, 0, 5, 4, "bf16", ("normal", 0, 0.1)),
    ("7x7 4x1 r16", 16, 3, 49, 4, 1, 16, "bf16", ("normal", 0, 0.1)),
    ("ties 3x3 16x4 r3", 48, 16, 9, 16, 4, 3, "bf16", ("ties",)),
]


@pytest.mark.parametrize("i", range(len(PUNCHED_MATS)), ids=[m[0] for m in PUNCHED_MATS])
def test_punched_prune_and_pack_bit_exact(B, i):
    name, R, cin, khw, bh, bw, rate, dtype, dist = PUNCHED_MATS[i]
    C = cin * khw
    w = _mat(60 + i, R, C, dtype, dist)
    scheme = B.Scheme(R, C, bh, bw, PUNCHED, rate, khw)
    layer = _layers().PackedLayer(scheme, DT[dtype], to_dev(w, dtype))
    m_ref = oracle_mask(w, dtype, scheme)
    m_gpu = layer.mask.cpu().numpy().reshape(R, C)
    assert np.array_equal(m_gpu, m_ref), f"{name}: {int((m_gpu != m_ref).sum())} mask entries differ"
    pk = OP.pack(w, m_ref, bh, bw, PUNCHED, rate)
    vals = from_dev(layer.values[:layer.n_values], dtype)
    assert np.array_equal(vals.view(np.uint8), np.ascontiguousarray(pk["values"]).view(np.uint8))
    assert np.array_equal(layer.indices[:layer.n_indices].cpu().numpy(), pk["indices"])
    assert np.array_equal(layer.rowptr[:layer.n_rowptr].cpu().numpy(), pk["rowptr"])
    back = from_dev(layer.unpack(), dtype).reshape(R, C)
    expect = np.where(m_ref == 1, w, np.zeros_like(w))
    assert np.array_equal(back.view(np.uint8), expect.view(np.uint8))


def test_pack_rejects_a_block_punched_mask_off_its_pattern(B):
    import torch
    R, cin, khw = 32, 16, 9
    w = draw(seed_for(9, 51, 1), (R, cin * khw), ("normal", 0, 1), "bf16")
    scheme = B.Scheme(R, cin * khw, 8, 4, PUNCHED, 3, khw)
    m = oracle_mask(w, "bf16", scheme).reshape(R, cin, khw)
    m[3, 5] = np.roll(m[3, 5], 1)            # one kernel with other locations
    with pytest.raises(B.BspError) as e:
        _layers().PackedLayer(scheme, B.BF16, to_dev(w, "bf16"), mask=torch.from_numpy(m.reshape(-1)).cuda())
    assert e.value.status == -4


def test_pack_rejects_a_mask_without_block_structure(B):
    import torch
    R, C = 64, 256
    w = draw(seed_for(9, 50, 1), (R, C), ("normal", 0, 1), "bf16")
    m = oracle_mask(w, "bf16", B.Scheme(R, C, 16, 32, COL, 4))
    m[5, np.nonzero(m[5])[0][0]] = 0         # one hole in a kept column
    with pytest.raises(B.BspError) as e:
        _layers().PackedLayer(B.Scheme(R, C, 16, 32, COL, 4), B.BF16, to_dev(w, "bf16"),
                              mask=torch.from_numpy(m.reshape(-1)).cuda())
    assert e.value.status == -4


# ----------------------------------------------------------------------- conv ---
def _conv_case(name, n, cin, h, w, cout, k, s, p, bh, bw, reg, rate, dtype="bf16", relu=False,
               bias=False, out="same"):
    return dict(name=name, layer=ConvLayer(name, n, cin, h, w, cout, k, k, s, s, p, p, bh, bw, reg, rate,
                                           dtype, ("normal", 0, 1.0), ("normal", 0, (2.0 / (cin * k * k)) ** 0.5),
                                           relu=relu), bias=bias, out=out)


CONV_CASES = [
    _conv_case("3x3 col16x32 r4 ragged-wo", 2, 64, 13, 11, 64, 3, 1, 1, 16, 32, COL, 4),
    _conv_case("3x3 col16x32 r4 s2", 2, 64, 15, 15, 64, 3, 2, 1, 16, 32, COL, 4),
    _conv_case("3x3 col8x16 r8 relu bias", 3, 64, 8, 8, 128, 3, 1, 1, 8, 16, COL, 8, relu=True, bias=True),
    _conv_case("1x1 row32x32 r2", 2, 96, 14, 14, 160, 1, 1, 0, 32, 32, ROW, 2),
    _conv_case("1x1 row32x32 r2 s2", 2, 64, 14, 14, 96, 1, 2, 0, 32, 32, ROW, 2),
    _conv_case("7x7/2 dense", 1, 3, 40, 40, 64, 7, 2, 3, 0, 0, DENSE, 1),
    _conv_case("5x5 pad2 col whole r4", 2, 20, 9, 9, 24, 5, 1, 2, 0, 0, COL, 4),
    _conv_case("3x3 pad0 col4x4 r2 fp32out", 2, 8, 10, 12, 20, 3, 1, 0, 4, 4, COL, 2, out="f32"),
    _conv_case("3x3 row whole r4 bias", 1, 16, 12, 12, 40, 3, 1, 1, 0, 0, ROW, 4, bias=True),
    _conv_case("3x3 unstructured r4", 2, 32, 12, 12, 48, 3, 1, 1, 1, 1, UNSTRUCTURED, 4),
    _conv_case("3x3 col r4 7x7 spans images", 5, 128, 7, 7, 96, 3, 1, 1, 16, 32, COL, 4),
    _conv_case("3x3 s3 general stride", 2, 16, 17, 17, 32, 3, 3, 1, 16, 16, COL, 2),
    _conv_case("f32 3x3 col16x16 r4", 1, 64, 32, 32, 64, 3, 1, 1, 16, 16, COL, 4, dtype="f32", out="f32"),
    _conv_case("f32 3x3 s2 row", 2, 16, 11, 11, 48, 3, 2, 1, 16, 16, ROW, 2, dtype="f32", out="f32"),
    _conv_case("3x3 col r16 many chunks", 1, 512, 6, 6, 64, 3, 1, 1, 16, 64, COL, 16),
    _conv_case("1x1 col whole r2 4x4 image", 3, 256, 4, 4, 64, 1, 1, 0, 0, 0, COL, 2),
    # whole-width row blocks: only the kept filters are computed (row map + pruned-row fill)
    _conv_case("1x1 row whole r4 relu bias", 2, 64, 14, 14, 100, 1, 1, 0, 0, 0, ROW, 4, relu=True, bias=True),
    _conv_case("1x1 row 32xwhole r2 s2", 2, 64, 14, 14, 96, 1, 2, 0, 32, 0, ROW, 2),
    _conv_case("3x3 row 16xwhole r3 ragged", 2, 24, 9, 11, 70, 3, 1, 1, 16, 0, ROW, 3, bias=True),
    _conv_case("3x3 row whole r16 relu", 1, 32, 10, 10, 64, 3, 1, 1, 0, 0, ROW, 16, relu=True),
    _conv_case("f32 3x3 row whole r4 bias", 1, 16, 12, 12, 40, 3, 1, 1, 0, 0, ROW, 4, dtype="f32", out="f32",
               bias=True),
    # block-punched (Sec. 4.1.2): bh filters x bw input channels, kernel locations removed per block
    _conv_case("3x3 punched 16x8 r3", 2, 64, 12, 12, 64, 3, 1, 1, 16, 8, PUNCHED, 3),
    _conv_case("3x3 punched whole r4 s2", 2, 32, 15, 15, 48, 3, 2, 1, 0, 0, PUNCHED, 4),
    _conv_case("5x5 punched 8x4 r5 relu bias", 1, 20, 11, 11, 24, 5, 1, 2, 8, 4, PUNCHED, 5, relu=True, bias=True),
    _conv_case("3x3 punched 16x1 r9 ragged", 3, 24, 9, 13, 40, 3, 1, 1, 16, 1, PUNCHED, 9),
    _conv_case("f32 3x3 punched 4x4 r2", 1, 16, 10, 10, 32, 3, 1, 1, 4, 4, PUNCHED, 2, dtype="f32", out="f32"),
    _conv_case("1x1 punched 32x16 r2 keeps all", 2, 64, 14, 14, 96, 1, 1, 0, 32, 16, PUNCHED, 2),
    # rows and columns removed in the same block (Eqs. 2-3 together)
    _conv_case("3x3 rowcol 16x32 r2 bias relu", 2, 64, 12, 12, 64, 3, 1, 1, 16, 32, ROWCOL, 2, relu=True, bias=True),
    _conv_case("1x1 rowcol 32x32 r2 s2", 2, 64, 14, 14, 96, 1, 2, 0, 32, 32, ROWCOL, 2),
    _conv_case("f32 3x3 rowcol 8x8 r2", 1, 16, 10, 10, 32, 3, 1, 1, 8, 8, ROWCOL, 2, dtype="f32", out="f32"),
    # output planes of at most 16 pixels run as a 1x1 layer over the im2col input
    _conv_case("im2col 3x3 col8x16 r8 2x2", 5, 64, 2, 2, 64, 3, 1, 1, 8, 16, COL, 8),
    _conv_case("im2col 3x3 col16x32 r4 4x4 relu bias", 3, 96, 4, 4, 80, 3, 1, 1, 16, 32, COL, 4, relu=True,
               bias=True),
    _conv_case("im2col 3x3 s2 8x8 row whole r4 bias", 2, 32, 8, 8, 40, 3, 2, 1, 0, 0, ROW, 4, bias=True),
    _conv_case("im2col 3x3 punched 16x8 r3 4x4", 2, 32, 4, 4, 48, 3, 1, 1, 16, 8, PUNCHED, 3),
    _conv_case("im2col f32 3x3 col16x16 r2 4x4", 2, 16, 4, 4, 32, 3, 1, 1, 16, 16, COL, 2, dtype="f32", out="f32"),
    _conv_case("im2col 5x5 pad0 dense 6x6", 3, 12, 6, 6, 24, 5, 1, 0, 0, 0, DENSE, 1),
    _conv_case("im2col 3x3 pad0 unstructured 4x5", 4, 24, 4, 5, 40, 3, 1, 0, 1, 1, UNSTRUCTURED, 4),
    _conv_case("im2col 3x3 row32x32 r2 3x3 ragged", 7, 40, 3, 3, 72, 3, 1, 1, 32, 32, ROW, 2),
    # planes of at most 64 pixels with per-block-row lists: im2col planes padded to whole
    # granules, the pipelined kernel with gathered lists (1, 2 or 4 list groups per m-block)
    _conv_case("im2col lists 3x3 col16x32 r4 7x7", 3, 256, 7, 7, 64, 3, 1, 1, 16, 32, COL, 4),
    _conv_case("im2col lists 3x3 col32x32 r4 8x8 ragged rows bias", 2, 40, 8, 8, 72, 3, 1, 1, 32, 32, COL, 4,
               bias=True),
    _conv_case("im2col lists 3x3 col64x16 r2 6x6 relu", 3, 16, 6, 6, 128, 3, 1, 1, 64, 16, COL, 2, relu=True),
    _conv_case("im2col lists 5x5 punched 16x8 r5 7x7 bias relu", 2, 24, 7, 7, 40, 5, 1, 2, 16, 8, PUNCHED, 5,
               relu=True, bias=True),
    _conv_case("im2col lists 3x3 s2 col8x16 r8 13x13", 3, 48, 13, 13, 64, 3, 2, 1, 8, 16, COL, 8),
    _conv_case("im2col lists 3x3 rowcol 16x32 r2 5x7", 2, 64, 5, 7, 48, 3, 1, 1, 16, 32, ROWCOL, 2),
    # 1x1 stride-2 layers over one identity list: planes of at most 196 pixels run over the
    # subsampled input (stride-1 pointwise kernel), larger ones on the strided kernel
    _conv_case("subsample 1x1/2 dense odd 15x13 relu bias f32out", 3, 48, 15, 13, 40, 1, 2, 0, 0, 0, DENSE, 1,
               relu=True, bias=True, out="f32"),
    _conv_case("subsample 1x1/2 row16x16 r2 28x28 (196-pixel plane)", 2, 64, 28, 28, 96, 1, 2, 0, 16, 16, ROW, 2),
    _conv_case("strided 1x1/2 row16x16 r2 30x30 (225-pixel plane)", 2, 64, 30, 30, 96, 1, 2, 0, 16, 16, ROW, 2),
    # stride-2 stems with an identity list: the stem kernel (output channels as MFMA rows)
    _conv_case("stem 7x7/2 dense relu bias f32out", 2, 3, 32, 48, 40, 7, 2, 3, 0, 0, DENSE, 1, relu=True,
               bias=True, out="f32"),
    _conv_case("stem 7x7/2 dense ragged row groups", 1, 3, 26, 64, 64, 7, 2, 3, 0, 0, DENSE, 1),
    _conv_case("stem 3x3/2 row16x16 r2 zero-expanded 9 rows bias", 2, 8, 18, 16, 48, 3, 2, 1, 16, 16, ROW, 2,
               bias=True),
]


def run_conv(B, layer, x, w, dtype, out_dt, bias=None, relu=False, mask=None):
    import torch
    scheme = layer.scheme
    conv = B.ConvShape(layer.n, layer.cin, layer.h, layer.w, layer.kh, layer.kw, layer.sh, layer.sw,
                       layer.ph, layer.pw)
    L = _layers().PackedLayer(scheme, DT[dtype], to_dev(w.reshape(layer.cout, -1), dtype), conv=conv,
                              mask=mask)
    xd = to_dev(x, dtype)
    tdt = torch.float32 if out_dt == "f32" else torch.bfloat16
    y = torch.full(layer.y_shape, float("nan"), dtype=tdt, device="cuda")
    bd = None if bias is None else torch.from_numpy(bias.astype(np.float32)).cuda()
    L.conv2d(xd, y, layer.n, DT[out_dt], bd, relu)
    torch.cuda.synchronize()
    return L, y


@pytest.mark.parametrize("case", CONV_CASES, ids=[c["name"] for c in CONV_CASES])
def test_conv_matches_oracle(B, case):
    layer = case["layer"]
    dtype = layer.dtype
    out_dt = dtype if case["out"] == "same" else case["out"]
    d = draw_layer(layer, 8, CONV_CASES.index(case), with_bias=case["bias"])
    bias = d.get("bias")
    L, y = run_conv(B, layer, d["x"], d["w"], dtype, out_dt, bias, layer.relu)
    m = L.mask.cpu().numpy().reshape(layer.cout, -1)
    assert np.array_equal(m, oracle_mask(d["w"], dtype, layer.scheme))
    got = out_to_f64(from_dev(y, out_dt), out_dt)
    gate_conv(got, d["x"], d["w"], m, dtype, out_dt, layer, bias=bias, relu=layer.relu, name=case["name"])


def test_filter_pruning_writes_the_bias_of_pruned_filters_exactly(B):
    """Whole-matrix row pruning removes whole filters (Sec. 4.4): their outputs are
    exactly ReLU(b[o]) in the output precision, the kept filters match the oracle."""
    import torch
    for relu in (False, True):
        layer = ConvLayer("fp", 2, 32, 9, 9, 48, 3, 3, 1, 1, 1, 1, 0, 0, ROW, 4, "bf16", ("normal", 0, 1.0),
                          ("normal", 0, 0.08), relu=relu)
        d = draw_layer(layer, 8, 77, with_bias=True)
        bias = d["bias"]
        L, y = run_conv(B, layer, d["x"], d["w"], "bf16", "bf16", bias, relu)
        m = L.mask.cpu().numpy().reshape(layer.cout, -1)
        pruned = np.nonzero(m.sum(axis=1) == 0)[0]
        assert len(pruned) == 36
        got = out_to_f64(from_dev(y, "bf16"), "bf16")
        b32 = bias.astype(np.float32)
        expect = np.maximum(b32, 0) if relu else b32
        expect_bf16 = out_to_f64(from_dev(torch.from_numpy(expect).to(torch.bfloat16).cuda(), "bf16"), "bf16")
        for o in pruned:
            assert np.all(got[:, o] == expect_bf16[o]), o
        gate_conv(got, d["x"], d["w"], m, "bf16", "bf16", layer, bias=bias, relu=relu)


def test_conv_is_deterministic_and_empty_batch_is_a_noop(B):
    import torch
    case = CONV_CASES[0]
    layer = case["layer"]
    d = draw_layer(layer, 8, 0)
    L, y1 = run_conv(B, layer, d["x"], d["w"], "bf16", "bf16")
    y2 = torch.empty_like(y1)
    L.conv2d(to_dev(d["x"], "bf16"), y2, layer.n, B.BF16)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    y3 = torch.zeros(4, dtype=torch.bfloat16, device="cuda")
    L.conv2d(to_dev(d["x"], "bf16"), y3, 0, B.BF16)
    torch.cuda.synchronize()
    assert torch.count_nonzero(y3.float()) == 0


MISMATCH_CASES = [  # name, layer, bias: tiles packed for stride 2 used at stride 1
    ("3x3 col16x32", ConvLayer("mm col", 2, 64, 13, 11, 64, 3, 3, 1, 1, 1, 1, 16, 32, COL, 4, "bf16",
                               ("normal", 0, 1.0), ("normal", 0, 0.06)), False),
    ("1x1 row whole (row map, pointwise kernel)", ConvLayer("mm rowmap pw", 2, 64, 14, 14, 100, 1, 1, 1, 1, 0, 0,
                                                            0, 0, ROW, 4, "bf16", ("normal", 0, 1.0),
                                                            ("normal", 0, 0.1)), True),
    ("3x3 row 16xwhole (row map, general kernel)", ConvLayer("mm rowmap fwd", 2, 24, 9, 11, 70, 3, 3, 1, 1, 1, 1,
                                                             16, 0, ROW, 3, "bf16", ("normal", 0, 1.0),
                                                             ("normal", 0, 0.1)), True),
]


@pytest.mark.parametrize("name,layer,with_bias", MISMATCH_CASES, ids=[c[0] for c in MISMATCH_CASES])
def test_tiles_packed_for_another_geometry_give_nan(B, name, layer, with_bias):
    """dev_tiles of another plan (here: packed for stride 2, used at stride 1) give NaN
    in every output element, never numbers, and never a row outside the output
    (row-mapped layers read no row map from such tiles)."""
    import torch
    d = draw_layer(layer, 8, 0, with_bias=with_bias)
    k, p = layer.kh, layer.ph
    other = B.ConvShape(1, layer.cin, layer.h, layer.w, k, k, 2, 2, p, p)
    shape = B.ConvShape(layer.n, layer.cin, layer.h, layer.w, k, k, 1, 1, p, p)
    scheme = layer.scheme
    nv, ni, nr, nb_other = B.bsp_packed_sizes(scheme, other, B.BF16)
    nb = B.bsp_packed_sizes(scheme, shape, B.BF16)[3]
    w = to_dev(d["w"].reshape(layer.cout, -1), "bf16")
    mask = torch.empty(layer.cout * w.shape[1], dtype=torch.uint8, device="cuda")
    B.bsp_prune(scheme, B.BF16, w, mask)
    vals = torch.empty(max(nv, 1), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty(max(ni, 1), dtype=torch.int32, device="cuda")
    rp = torch.empty(max(nr, 1), dtype=torch.int32, device="cuda")
    tiles = torch.zeros(max(nb, nb_other), dtype=torch.uint8, device="cuda")
    B.bsp_pack(scheme, B.BF16, w, mask, vals, idx, rp, tiles, other)
    y = torch.zeros(layer.y_shape, dtype=torch.bfloat16, device="cuda")
    bd = torch.from_numpy(d["bias"].astype(np.float32)).cuda() if with_bias else None
    B.bsp_conv2d(scheme, shape, B.BF16, B.BF16, to_dev(d["x"], "bf16"), tiles, bd, True, y)
    torch.cuda.synchronize()
    assert torch.isnan(y.float()).all()


def test_stem_tiles_of_another_geometry_give_nan(B):
    """The stem kernel checks the tile header too: tiles packed for stride 1 used at
    stride 2 give NaN everywhere."""
    import torch
    layer = ConvLayer("mm stem", 2, 3, 40, 40, 64, 7, 7, 2, 2, 3, 3, 0, 0, DENSE, 1, "bf16", ("normal", 0, 1.0),
                      ("normal", 0, 0.1))
    d = draw_layer(layer, 8, 1)
    other = B.ConvShape(1, layer.cin, layer.h, layer.w, 7, 7, 1, 1, 3, 3)
    shape = B.ConvShape(layer.n, layer.cin, layer.h, layer.w, 7, 7, 2, 2, 3, 3)
    scheme = layer.scheme
    nv, ni, nr, nb_other = B.bsp_packed_sizes(scheme, other, B.BF16)
    nb = B.bsp_packed_sizes(scheme, shape, B.BF16)[3]
    w = to_dev(d["w"].reshape(layer.cout, -1), "bf16")
    mask = torch.empty(layer.cout * w.shape[1], dtype=torch.uint8, device="cuda")
    B.bsp_prune(scheme, B.BF16, w, mask)
    vals = torch.empty(max(nv, 1), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty(max(ni, 1), dtype=torch.int32, device="cuda")
    rp = torch.empty(max(nr, 1), dtype=torch.int32, device="cuda")
    tiles = torch.zeros(max(nb, nb_other), dtype=torch.uint8, device="cuda")
    B.bsp_pack(scheme, B.BF16, w, mask, vals, idx, rp, tiles, other)
    y = torch.zeros(layer.y_shape, dtype=torch.bfloat16, device="cuda")
    B.bsp_conv2d(scheme, shape, B.BF16, B.BF16, to_dev(d["x"], "bf16"), tiles, None, True, y)
    torch.cuda.synchronize()
    assert torch.isnan(y.float()).all()


@pytest.mark.parametrize("reg,bh,bw,rate_pack,rate_run,batch", [
    (COL, 32, 32, 4, 2, 64),    # gathered lists, split K loop
    (COL, 16, 64, 4, 8, 512),   # gathered lists, unsplit
    (ROW, 32, 32, 2, 4, 64),    # identity list, split K loop
])
def test_linear_tiles_of_another_scheme_give_nan(B, reg, bh, bw, rate_pack, rate_run, batch):
    """A linear layer run with dev_tiles packed for another rate: every output is NaN
    (the kernel reads nothing of such tiles past their header)."""
    import torch
    R, C = 192, 256
    pack = B.Scheme(R, C, bh, bw, reg, rate_pack, 0)
    run = B.Scheme(R, C, bh, bw, reg, rate_run, 0)
    rng = np.random.default_rng(7)
    w = torch.from_numpy(rng.normal(0, 0.05, (R, C)).astype(np.float32)).to(torch.bfloat16).cuda()
    x = torch.from_numpy(rng.uniform(-1, 1, (C, batch)).astype(np.float32)).to(torch.bfloat16).cuda()
    mask = torch.empty(R * C, dtype=torch.uint8, device="cuda")
    B.bsp_prune(pack, B.BF16, w, mask)
    nv, ni, nr, nb = B.bsp_packed_sizes(pack, None, B.BF16)
    nb_run = B.bsp_packed_sizes(run, None, B.BF16)[3]
    vals = torch.empty(max(nv, 1), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty(max(ni, 1), dtype=torch.int32, device="cuda")
    rp = torch.empty(max(nr, 1), dtype=torch.int32, device="cuda")
    tiles = torch.zeros(max(nb, nb_run), dtype=torch.uint8, device="cuda")
    B.bsp_pack(pack, B.BF16, w, mask, vals, idx, rp, tiles)
    y = torch.zeros(R, batch, dtype=torch.bfloat16, device="cuda")
    bias = torch.ones(R, dtype=torch.float32, device="cuda")
    B.bsp_linear(run, batch, B.BF16, B.BF16, x, tiles, bias, True, y)
    torch.cuda.synchronize()
    assert torch.isnan(y.float()).all()


def test_small_plane_conv_tiles_of_another_scheme_give_nan(B):
    """The im2col route (gathered lists, split K loop) run with dev_tiles packed for
    another rate gives NaN everywhere.  (Tiles of a 1x1 plan over the expanded input do
    not depend on the image size, so a rate, not a geometry, makes the mismatch.)"""
    import torch
    cout, cin, n, hw = 64, 64, 2, 7
    shape = B.ConvShape(n, cin, hw, hw, 3, 3, 1, 1, 1, 1)
    pack = B.Scheme(cout, cin * 9, 16, 32, COL, 4, 0)
    run = B.Scheme(cout, cin * 9, 16, 32, COL, 2, 0)
    rng = np.random.default_rng(8)
    w = torch.from_numpy(rng.normal(0, 0.06, (cout, cin * 9)).astype(np.float32)).to(torch.bfloat16).cuda()
    x = torch.from_numpy(rng.normal(0, 1, (n, cin, hw, hw)).astype(np.float32)).to(torch.bfloat16).cuda()
    mask = torch.empty(cout * cin * 9, dtype=torch.uint8, device="cuda")
    B.bsp_prune(pack, B.BF16, w, mask)
    nv, ni, nr, nb = B.bsp_packed_sizes(pack, shape, B.BF16)
    nb_run = B.bsp_packed_sizes(run, shape, B.BF16)[3]
    vals = torch.empty(max(nv, 1), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty(max(ni, 1), dtype=torch.int32, device="cuda")
    rp = torch.empty(max(nr, 1), dtype=torch.int32, device="cuda")
    tiles = torch.zeros(max(nb, nb_run), dtype=torch.uint8, device="cuda")
    B.bsp_pack(pack, B.BF16, w, mask, vals, idx, rp, tiles, shape)
    y = torch.zeros(n, cout, hw, hw, dtype=torch.bfloat16, device="cuda")
    B.bsp_conv2d(run, shape, B.BF16, B.BF16, x, tiles, None, False, y)
    torch.cuda.synchronize()
    assert torch.isnan(y.float()).all()


# ------------------------------------------------- full-size workloads, sampled ---
def _c3_distinct():
    seen, out = set(), []
    for i, l in enumerate(workload(3)):
        if l.kind != "conv":
            continue
        key = (l.cin, l.h, l.cout, l.kh, l.sh)
        if key not in seen:
            seen.add(key)
            out.append((i, l))
    return out


C3 = _c3_distinct()


C3_IMAGES = [0, 21, 22, 63]   # first, last, and two neighbours whose boundary falls inside pixel tiles


@pytest.mark.parametrize("idx,layer", C3, ids=[l.name for _, l in C3])
def test_resnet50_layer_full_batch_sampled_images(B, idx, layer):
    """Batch-64 ResNet-50 layer in the launch configuration the benchmark times;
    the oracle checks images 0, 21, 22 and 63 in full (21 | 22: a tile and a
    workgroup range that straddle two images)."""
    d = draw_layer(layer, 3, idx)
    L, y = run_conv(B, layer, d["x"], d["w"], "bf16", "bf16")
    m = L.mask.cpu().numpy().reshape(layer.cout, -1)
    assert np.array_equal(m, oracle_mask(d["w"], "bf16", layer.scheme))
    got = out_to_f64(from_dev(y, "bf16"), "bf16")[C3_IMAGES]
    gate_conv(got, d["x"], d["w"], m, "bf16", "bf16", layer, images=C3_IMAGES)


def test_resnet50_fc_at_batch_64(B):
    """The fc layer of the ResNet-50 pass (2048 -> 1000, dense, batch 64), every output."""
    idx, layer = [(i, l) for i, l in enumerate(workload(3)) if l.kind != "conv"][0]
    d = draw_layer(layer, 3, idx)
    L, y = run_linear(B, layer, d["x"], d["w"], "bf16", "bf16")
    m = L.mask.cpu().numpy().reshape(layer.out_f, layer.in_f)
    assert m.all()
    gate_linear(out_to_f64(from_dev(y, "bf16"), "bf16"), d["x"], d["w"], m, "bf16", "bf16", name=layer.name)


def _sweep_settings():
    from paper_2111_11581_amd.latency import sweep_settings
    return sweep_settings(references=True)


SWEEP = _sweep_settings()


@pytest.fixture(scope="module")
def sweep_input(B):
    """The sweep layer's input (64 x 256 x 56 x 56 bf16), drawn once for every setting."""
    st = SWEEP[0]
    from synthetic import draw, seed_for, SEED_X
    x = draw(seed_for(5, 0, SEED_X), (st.batch, st.cin, st.h, st.w), ("normal", 0.0, 1.0), "bf16")
    return x, to_dev(x, "bf16")


@pytest.mark.parametrize("i", range(len(SWEEP)), ids=[s.key() for s in SWEEP])
def test_sweep_setting_full_batch_sampled_image(B, sweep_input, i):
    """Every setting the latency model times (3x3 256->256 at 56x56, batch 64: block
    size x regularity x rate, unstructured, pattern-based and dense references) at its
    full size in its timed launch configuration; one image per setting (rotating over
    the batch) is gated against the oracle in full."""
    import torch
    from synthetic import draw, seed_for, SEED_W
    s = SWEEP[i]
    x_host, x_dev = sweep_input
    rows, cols = s.cout, s.cin * s.kh * s.kw
    w = draw(seed_for(5, 100 + i, SEED_W), (rows, cols), ("normal", 0.0, (2.0 / cols) ** 0.5), "bf16")
    scheme = B.Scheme(rows, cols, s.bh, s.bw, s.regularity, s.rate, s.kh * s.kw)
    conv = B.ConvShape(s.batch, s.cin, s.h, s.w, s.kh, s.kw, s.stride, s.stride, s.pad, s.pad)
    L = _layers().PackedLayer(scheme, B.BF16, to_dev(w, "bf16"), conv=conv)
    y = torch.full((s.batch, s.cout, s.ho, s.wo), float("nan"), dtype=torch.bfloat16, device="cuda")
    L.conv2d(x_dev, y, s.batch, B.BF16)
    torch.cuda.synchronize()
    m = L.mask.cpu().numpy().reshape(rows, cols)
    assert np.array_equal(m, oracle_mask(w, "bf16", scheme))
    img = (7 * i + 3) % s.batch
    layer = ConvLayer(s.key(), s.batch, s.cin, s.h, s.w, s.cout, s.kh, s.kw, s.stride, s.stride, s.pad, s.pad,
                      s.bh, s.bw, s.regularity, s.rate, "bf16", ("normal", 0.0, 1.0), ("normal", 0.0, 1.0))
    got = out_to_f64(from_dev(y[img:img + 1], "bf16"), "bf16")
    gate_conv(got, x_host, w, m, "bf16", "bf16", layer, images=[img])


def test_c1_full(B):
    layer = workload(1)[0]
    d = draw_layer(layer, 1, 0)
    L, y = run_conv(B, layer, d["x"], d["w"], "f32", "f32")
    m = L.mask.cpu().numpy().reshape(layer.cout, -1)
    assert np.array_equal(m, oracle_mask(d["w"], "f32", layer.scheme))
    gate_conv(from_dev(y, "f32").astype(np.float64), d["x"], d["w"], m, "f32", "f32", layer)


# --------------------------------------------------------------------- linear ---
def run_linear(B, layer, x, w, dtype, out_dt, bias=None, relu=False):
    import torch
    L = _layers().PackedLayer(layer.scheme, DT[dtype], to_dev(w, dtype))
    tdt = torch.float32 if out_dt == "f32" else torch.bfloat16
    y = torch.full(layer.y_shape, float("nan"), dtype=tdt, device="cuda")
    bd = None if bias is None else torch.from_numpy(bias.astype(np.float32)).cuda()
    L.linear(to_dev(x, dtype), y, layer.batch, DT[out_dt], bd, relu)
    torch.cuda.synchronize()
    return L, y


def test_c4_fc_layer_every_column(B):
    """One 4096 -> 4096 layer of the FC stack at batch 512 (32x32 blocks, rate 10),
    every output gated."""
    layer = workload(4)[0]
    d = draw_layer(layer, 4, 0)
    L, y = run_linear(B, layer, d["x"], d["w"], "bf16", "bf16")
    m = L.mask.cpu().numpy().reshape(layer.out_f, layer.in_f)
    assert np.array_equal(m, oracle_mask(d["w"], "bf16", layer.scheme))
    gate_linear(out_to_f64(from_dev(y, "bf16"), "bf16"), d["x"], d["w"], m, "bf16", "bf16", name=layer.name)


@pytest.mark.parametrize("batch,reg,bh,bw,rate,out_dt,relu", [
    (37, COL, 32, 32, 10, "bf16", False), (100, ROW, 32, 32, 2, "f32", True),
    (64, DENSE, 0, 0, 1, "bf16", True), (130, COL, 16, 64, 4, "bf16", False),
    (100, ROW, 0, 0, 4, "bf16", True), (70, ROW, 32, 0, 2, "f32", False), (90, ROWCOL, 32, 32, 2, "bf16", True),
    (64, COL, 64, 32, 4, "bf16", True), (48, COL, 8, 16, 8, "f32", False), (96, COL, 0, 32, 4, "bf16", False),
    (203, COL, 16, 32, 4, "bf16", True)])
def test_linear_small(B, batch, reg, bh, bw, rate, out_dt, relu):
    layer = LinearLayer("fc", batch, 320, 200, bh, bw, reg, rate, "bf16", ("uniform", -1, 1),
                        ("normal", 0, 0.05), relu=relu)
    d = draw_layer(layer, 8, 90 + batch % 7, with_bias=True)
    L, y = run_linear(B, layer, d["x"], d["w"], "bf16", out_dt, d["bias"], relu)
    m = L.mask.cpu().numpy().reshape(200, 320)
    gate_linear(out_to_f64(from_dev(y, out_dt), out_dt), d["x"], d["w"], m, "bf16", out_dt, bias=d["bias"],
                relu=relu, name=f"fc b{batch}")


# -------------------------------------------------------------- VGG-16 stack ---
@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_maxpool_bit_exact(B, dt):
    """2x2 max pooling: odd sizes (floor), ties, -inf and NaN (NaN propagates)."""
    import torch
    from oracle import glue
    x = draw(seed_for(8, 99, 0), (3, 5, 11, 15), ("normal", 0, 1), "f32")
    x = np.round(x * 2) / 2                                   # many ties
    flat = x.reshape(-1)
    rng = np.random.default_rng(4)
    idx = rng.permutation(flat.size)
    flat[idx[:60]] = -np.inf
    flat[idx[60:90]] = np.nan
    bits = x if dt == "f32" else (x.view(np.uint32) >> 16).astype(np.uint16)   # exact: halves fit in bf16
    xd = to_dev(bits, dt)
    y = torch.empty((3, 5, 5, 7), dtype=torch.float32 if dt == "f32" else torch.bfloat16, device="cuda")
    B.bsp_maxpool2x2(DT[dt], 3, 5, 11, 15, xd, y)
    torch.cuda.synchronize()
    ref = glue.maxpool2x2(as_f64(bits, dt))
    assert np.array_equal(out_to_f64(from_dev(y, dt), dt), ref, equal_nan=True)


def test_vgg16_stack_per_layer_and_end_to_end(B):
    """Each layer of the VGG-16 stack at its batch of 32 is gated on its own seeded
    input (every output); the chained stack is compared end to end against the
    oracle run with bf16 storage between layers (reported, loosely gated)."""
    import torch
    from oracle import glue
    from synthetic import f32_to_bf16_bits
    layers = workload(2)
    nimg = layers[0].n
    assert nimg == 32
    x0 = draw(seed_for(2, 0, 0), (nimg, 3, 32, 32), ("normal", 0, 1), "bf16")
    cur_gpu = to_dev(x0, "bf16")
    cur_ref = as_f64(x0, "bf16")
    for i, full in enumerate(layers):
        layer = ConvLayer(full.name, nimg, full.cin, full.h, full.w, full.cout, 3, 3, 1, 1, 1, 1, full.bh,
                          full.bw, full.regularity, full.rate, "bf16", full.x_dist, full.w_dist, relu=True)
        d = draw_layer(layer, 2, i)
        # per-layer gate on a seeded input
        L, y = run_conv(B, layer, d["x"], d["w"], "bf16", "bf16", relu=True)
        m = L.mask.cpu().numpy().reshape(layer.cout, -1)
        assert np.array_equal(m, oracle_mask(d["w"], "bf16", layer.scheme))
        gate_conv(out_to_f64(from_dev(y, "bf16"), "bf16"), d["x"], d["w"], m, "bf16", "bf16", layer, relu=True)
        # chained stack
        yc = torch.empty(layer.y_shape, dtype=torch.bfloat16, device="cuda")
        L.conv2d(cur_gpu, yc, nimg, B.BF16, None, True)
        wm = as_f64(d["w"], "bf16") * m.reshape(layer.w_shape)
        from oracle import direct
        r = direct.conv2d(cur_ref, wm, None, (1, 1), (1, 1), relu=True)
        r = as_f64(f32_to_bf16_bits(r.astype(np.float32)), "bf16")
        if full.pool_after:
            h = layer.h
            yp = torch.empty((nimg, layer.cout, h // 2, h // 2), dtype=torch.bfloat16, device="cuda")
            B.bsp_maxpool2x2(B.BF16, nimg, layer.cout, h, h, yc, yp)
            yc, r = yp, glue.maxpool2x2(r)
        cur_gpu, cur_ref = yc, r
    torch.cuda.synchronize()
    e2e = rel_l2(out_to_f64(from_dev(cur_gpu, "bf16"), "bf16"), cur_ref)
    print(f"VGG-16 stack end-to-end rel-L2 {e2e:.3e}")
    assert e2e <= 3e-2


# ----------------------------------------------------- per-block kept counts ---
# Sec. 4.1.1: each block may keep its own number of rows / columns / locations; the
# counts come with the scheme (random here, including empty and full blocks).

def _block_groups(R, C, bh, bw, reg, khw):
    rr = OP.block_ranges(R, bh)
    cc = OP.block_ranges(C // khw if reg == PUNCHED else C, bw)
    return [[khw if reg == PUNCHED else ((c1 - c0) if reg == COL else (r1 - r0)) for c0, c1 in cc]
            for r0, r1 in rr]


def _counts(R, C, bh, bw, reg, khw, seed):
    g = np.asarray(_block_groups(R, C, bh, bw, reg, khw))
    rng = np.random.default_rng(seed)
    cnt = rng.integers(0, g + 1).astype(np.int32)
    cnt.flat[0] = 0                      # one empty block
    cnt.flat[-1] = g.flat[-1]            # one full block
    return cnt


COUNT_CASES = [  # name, n, cin, h, w, cout, k, s, p, bh, bw, reg, dtype, bias+relu
    ("3x3 col16x32", 2, 64, 12, 11, 64, 3, 1, 1, 16, 32, COL, "bf16", False),
    ("3x3 col8x16 s2 f32", 2, 32, 13, 13, 40, 3, 2, 1, 8, 16, COL, "f32", True),
    ("1x1 col32x32", 2, 128, 14, 14, 96, 1, 1, 0, 32, 32, COL, "bf16", False),
    ("1x1 row32x32", 2, 96, 14, 14, 160, 1, 1, 0, 32, 32, ROW, "bf16", True),
    ("3x3 row 16xwhole", 2, 24, 9, 11, 70, 3, 1, 1, 16, 0, ROW, "bf16", True),
    ("3x3 punched 16x8", 2, 64, 12, 12, 64, 3, 1, 1, 16, 8, PUNCHED, "bf16", False),
    ("3x3 col 16xwhole", 1, 32, 10, 10, 48, 3, 1, 1, 16, 0, COL, "bf16", False),
]


@pytest.mark.parametrize("case", COUNT_CASES, ids=[c[0] for c in COUNT_CASES])
def test_per_block_counts_prune_pack_and_conv(B, case):
    import torch
    name, n, cin, h, w_, cout, k, s, p, bh, bw, reg, dtype, br = case
    layer = ConvLayer(name, n, cin, h, w_, cout, k, k, s, s, p, p, bh, bw, reg, 4, dtype, ("normal", 0, 1.0),
                      ("normal", 0, (2.0 / (cin * k * k)) ** 0.5), relu=br)
    R, C, khw = cout, cin * k * k, k * k
    cnt = _counts(R, C, bh, bw, reg, khw, 300 + COUNT_CASES.index(case))
    d = draw_layer(layer, 8, 200 + COUNT_CASES.index(case), with_bias=br)
    scheme = B.Scheme(R, C, bh, bw, reg, 4, khw).set_counts(cnt)
    conv = B.ConvShape(n, cin, h, w_, k, k, s, s, p, p)
    L = _layers().PackedLayer(scheme, DT[dtype], to_dev(d["w"].reshape(R, C), dtype), conv=conv)
    m_ref = OP.prune_mask(as_f64(d["w"], dtype).reshape(R, C), bh, bw, reg, 4, khw=khw, counts=cnt)
    assert np.array_equal(L.mask.cpu().numpy().reshape(R, C), m_ref)
    pk = OP.pack(d["w"].reshape(R, C), m_ref, bh, bw, reg, 4)
    assert np.array_equal(L.indices[:L.n_indices].cpu().numpy(), pk["indices"])
    assert np.array_equal(L.rowptr[:L.n_rowptr].cpu().numpy(), pk["rowptr"])
    vals = from_dev(L.values[:L.n_values], dtype)
    assert np.array_equal(vals.view(np.uint8), np.ascontiguousarray(pk["values"]).view(np.uint8))
    back = from_dev(L.unpack(), dtype).reshape(R, C)
    assert np.array_equal(back.view(np.uint8), np.where(m_ref == 1, d["w"].reshape(R, C), 0).astype(back.dtype)
                          .view(np.uint8))
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    y = torch.full(layer.y_shape, float("nan"), dtype=tdt, device="cuda")
    bias = d.get("bias")
    bd = None if bias is None else torch.from_numpy(bias.astype(np.float32)).cuda()
    L.conv2d(to_dev(d["x"], dtype), y, n, DT[dtype], bd, br)
    torch.cuda.synchronize()
    gate_conv(out_to_f64(from_dev(y, dtype), dtype), d["x"], d["w"], m_ref, dtype, dtype, layer, bias=bias, relu=br,
              name=name)


def test_per_block_counts_linear_and_fingerprint(B):
    import torch
    layer = LinearLayer("fc", 100, 320, 200, 32, 32, COL, 4, "bf16", ("uniform", -1, 1), ("normal", 0, 0.05))
    d = draw_layer(layer, 8, 250, with_bias=True)
    cnt = _counts(200, 320, 32, 32, COL, 1, 77)
    scheme = B.Scheme(200, 320, 32, 32, COL, 4).set_counts(cnt)
    L = _layers().PackedLayer(scheme, B.BF16, to_dev(d["w"], "bf16"))
    m = OP.prune_mask(as_f64(d["w"], "bf16"), 32, 32, COL, 4, counts=cnt)
    assert np.array_equal(L.mask.cpu().numpy().reshape(200, 320), m)
    y = torch.full(layer.y_shape, float("nan"), dtype=torch.bfloat16, device="cuda")
    bd = torch.from_numpy(d["bias"].astype(np.float32)).cuda()
    L.linear(to_dev(d["x"], "bf16"), y, 100, B.BF16, bd, False)
    torch.cuda.synchronize()
    gate_linear(out_to_f64(from_dev(y, "bf16"), "bf16"), d["x"], d["w"], m, "bf16", "bf16", bias=d["bias"],
                name="fc counts")
    # the same tiles used with other counts of the same list length bound: NaN, never wrong numbers
    cnt2 = cnt.copy()
    i = int(np.argmax((cnt2 > 0) & (cnt2 < 32)))
    cnt2.flat[i] -= 1
    other = B.Scheme(200, 320, 32, 32, COL, 4).set_counts(cnt2)
    nb2 = B.bsp_packed_sizes(other, None, B.BF16)[3]
    if nb2 <= L.tiles.numel():
        y2 = torch.zeros(layer.y_shape, dtype=torch.bfloat16, device="cuda")
        B.bsp_linear(other, 100, B.BF16, B.BF16, to_dev(d["x"], "bf16"), L.tiles, None, False, y2)
        torch.cuda.synchronize()
        assert torch.isnan(y2.float()).all()


# ------------------------------------------------------------------- BCS ---
def _gpu_bcs(B, L, scheme):
    import torch
    nbr = L.n_rowptr - 1
    occ = torch.full((nbr + 1,), -1, dtype=torch.int32, device="cuda")
    st = torch.full((nbr + 1,), -1, dtype=torch.int32, device="cuda")
    cc = torch.full((max(L.n_indices, 1),), -1, dtype=torch.int32, device="cuda")
    ro = torch.full((scheme.rows + 1,), -1, dtype=torch.int32, device="cuda")
    nr = torch.zeros(1, dtype=torch.int32, device="cuda")
    B.bsp_to_bcs(scheme, L.indices, L.rowptr, occ, cc, st, ro, nr)
    torch.cuda.synchronize()
    n = int(nr.item())
    return {"occurrence": occ[:n + 1].cpu().numpy(), "col_stride": st[:n + 1].cpu().numpy(),
            "compact_cols": cc[:int(st[n].item())].cpu().numpy(), "row_offset": ro.cpu().numpy()}


@pytest.mark.parametrize("kind", ["col16x32", "col8x16 counts", "punched 16x8", "merged block-rows"])
def test_bcs_encoding_matches_oracle(B, kind):
    import torch
    rng = np.random.default_rng(len(kind))
    if kind == "punched 16x8":
        R, cin, khw = 64, 24, 9
        C = cin * khw
        scheme = B.Scheme(R, C, 16, 8, PUNCHED, 3, khw)
    else:
        R, C = 70, 160
        scheme = B.Scheme(R, C, 16, 32, COL, 4) if kind != "col8x16 counts" else B.Scheme(R, C, 8, 16, COL, 4)
    w = draw(seed_for(9, 80 + len(kind), 1), (R, C), ("normal", 0, 1), "bf16")
    mask = None
    if kind == "col8x16 counts":
        cnt = _counts(R, C, 8, 16, COL, 1, 5)
        scheme.set_counts(cnt)
        m = OP.prune_mask(as_f64(w, "bf16"), 8, 16, COL, 4, counts=cnt)
    elif kind == "merged block-rows":
        # block-rows 0-1 and 3-4 keep the same columns: BCS stores each list once
        m = OP.prune_mask(as_f64(w, "bf16"), 16, 32, COL, 4)
        m[16:32] = m[0]
        m[64:70] = m[48]
        mask = torch.from_numpy(m.reshape(-1)).cuda()
    else:
        m = oracle_mask(w, "bf16", scheme)
    L = _layers().PackedLayer(scheme, B.BF16, to_dev(w, "bf16"), mask=mask)
    assert np.array_equal(L.mask.cpu().numpy().reshape(R, C), m)
    ref = OP.bcs_encode(w, m)
    got = _gpu_bcs(B, L, scheme)
    for k in ("occurrence", "col_stride", "compact_cols", "row_offset"):
        assert np.array_equal(got[k], ref[k]), k
    # the BCS weights array is the canonical values array
    vals = from_dev(L.values[:L.n_values], "bf16")
    assert np.array_equal(vals, ref["weights"])
    if kind == "merged block-rows":
        assert len(ref["occurrence"]) - 1 == 3


# --------------------------------------------------- pattern-based (3x3) ---
PATTERN_MATS = [  # name, R, cin, n_patterns, rate, dtype, dist
    ("64x64 8 patterns r4", 64, 64, 8, 4, "bf16", ("normal", 0, 0.05)),
    ("37x20 16 patterns r2 f32", 37, 20, 16, 2, "f32", ("normal", 0, 1.0)),
    ("256x256 8 patterns r8", 256, 256, 8, 8, "bf16", ("normal", 0, 0.03)),
    ("ties 48x16 4 patterns r3", 48, 16, 4, 3, "bf16", ("ties",)),
]


@pytest.mark.parametrize("i", range(len(PATTERN_MATS)), ids=[m[0] for m in PATTERN_MATS])
def test_pattern_prune_and_pack_bit_exact(B, i):
    name, R, cin, npat, rate, dtype, dist = PATTERN_MATS[i]
    C = cin * 9
    w = _mat(70 + i, R, C, dtype, dist)
    scheme = B.Scheme(R, C, npat, 0, PATTERN, rate, 9)
    layer = _layers().PackedLayer(scheme, DT[dtype], to_dev(w, dtype))
    m_ref = oracle_mask(w, dtype, scheme)
    m_gpu = layer.mask.cpu().numpy().reshape(R, C)
    assert np.array_equal(m_gpu, m_ref), f"{name}: {int((m_gpu != m_ref).sum())} mask entries differ"
    assert OP.mask_is_valid(m_gpu, npat, 0, PATTERN, rate, khw=9)
    back = from_dev(layer.unpack(), dtype).reshape(R, C)
    assert np.array_equal(back.view(np.uint8), np.where(m_ref == 1, w, np.zeros_like(w)).view(np.uint8))


def test_pattern_conv_matches_oracle_and_pack_rejects_a_three_weight_kernel(B):
    import torch
    layer = ConvLayer("pattern", 2, 32, 12, 12, 48, 3, 3, 1, 1, 1, 1, 8, 0, PATTERN, 4, "bf16", ("normal", 0, 1.0),
                      ("normal", 0, (2.0 / 288) ** 0.5), relu=True)
    d = draw_layer(layer, 8, 300, with_bias=True)
    L, y = run_conv(B, layer, d["x"], d["w"], "bf16", "bf16", d["bias"], True)
    m = L.mask.cpu().numpy().reshape(48, -1)
    assert np.array_equal(m, oracle_mask(d["w"], "bf16", layer.scheme))
    gate_conv(out_to_f64(from_dev(y, "bf16"), "bf16"), d["x"], d["w"], m, "bf16", "bf16", layer, bias=d["bias"],
              relu=True)
    bad = m.copy().reshape(-1, 9)
    k = int(np.argmax(bad.sum(axis=1)))
    bad[k, np.nonzero(bad[k])[0][0]] = 0
    with pytest.raises(B.BspError) as e:
        _layers().PackedLayer(layer.scheme, B.BF16, to_dev(d["w"].reshape(48, -1), "bf16"),
                              conv=B.ConvShape(2, 32, 12, 12, 3, 3, 1, 1, 1, 1),
                              mask=torch.from_numpy(bad.reshape(-1)).cuda())
    assert e.value.status == -4
