"""Planted mistakes in the oracle are caught by its pins (CPU only).

Each case copies an oracle source, plants one plausible mistake in the copy (a
dropped term, a wrong sign, swapped or transposed indices, a wrong tie rule, a
floor for a ceiling), builds or loads the copy from a temporary folder, and
checks that at least one independent pin (pure-Python brute force, torch conv
in fp64, k-subset enumeration, hand-worked examples) rejects it.  The oracle
itself is never modified.
"""

import ctypes
import importlib.util
import itertools
import json
import math
import os
import subprocess

import numpy as np
import pytest
import torch

from oracle import brute

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_examples.json")))


# ------------------------------------------------------------ direct conv ---
DIRECT_MUTATIONS = {
    "dropped_filter_column": ("for (int s = 0; s < KW; ++s)", "for (int s = 0; s < KW - 1; ++s)"),
    "wrong_sign_of_padding": ("const int ih = oh * SH - PH + r;", "const int ih = oh * SH + PH + r;"),
    "swapped_filter_taps": ("w[(((size_t)o * C + c) * KH + r) * KW + s]",
                            "w[(((size_t)o * C + c) * KH + s) * KW + r]"),
    "relu_inverted": ("if (relu && acc < 0.0) acc = 0.0;\n                y[",
                      "if (relu && acc > 0.0) acc = 0.0;\n                y["),
    "linear_transposed_input": ("x[(size_t)k * B + b]", "x[(size_t)b * K + k]"),
    "dropped_bias": ("double acc = bias ? bias[o] : 0.0;\n                for (int c",
                     "double acc = 0.0;\n                for (int c"),
}


def _build_direct(tmp_path, name, old, new):
    src = open(os.path.join(ROOT, "oracle", "direct.c")).read()
    assert src.count(old) == 1, name
    path = tmp_path / ("direct_%s.c" % name)
    path.write_text(src.replace(old, new))
    so = tmp_path / ("libdirect_%s.so" % name)
    subprocess.run(["gcc", "-O1", "-ffp-contract=off", "-shared", "-fPIC", "-o", str(so), str(path)],
                   check=True)
    lib = ctypes.CDLL(str(so))
    d = ctypes.POINTER(ctypes.c_double)
    lib.oracle_conv2d_f64.argtypes = [d, d, d, d] + [ctypes.c_int] * 13
    lib.oracle_linear_f64.argtypes = [d, d, d, d] + [ctypes.c_int] * 5
    return lib


def _p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _conv(lib, x, w, b, s, p, relu):
    N, C, H, W = x.shape
    O, _, KH, KW = w.shape
    Ho, Wo = (H + 2 * p - KH) // s + 1, (W + 2 * p - KW) // s + 1
    y = np.zeros((N, O, Ho, Wo))
    x, w, b = (np.ascontiguousarray(v, dtype=np.float64) for v in (x, w, b))
    assert lib.oracle_conv2d_f64(_p(x), _p(w), _p(b), _p(y), N, C, H, W, O, KH, KW, s, s, p, p,
                                 int(relu), 1) == 0
    return y


def _linear(lib, x, w, b, relu):
    K, B = x.shape
    O = w.shape[0]
    y = np.zeros((O, B))
    x, w, b = (np.ascontiguousarray(v, dtype=np.float64) for v in (x, w, b))
    assert lib.oracle_linear_f64(_p(x), _p(w), _p(b), _p(y), K, B, O, int(relu), 1) == 0
    return y


def _direct_pins_pass(lib) -> bool:
    """The direct-conv pins of tests/test_oracle_direct.py, on a few shapes."""
    rng = np.random.default_rng(5)
    for k, s, p, relu in ((3, 1, 1, False), (3, 2, 1, True), (1, 1, 0, False), (3, 1, 0, True)):
        x = rng.standard_normal((2, 3, 6, 5))
        w = rng.standard_normal((4, 3, k, k))
        b = rng.standard_normal(4)
        y = _conv(lib, x, w, b, s, p, relu)
        yb = np.array(brute.conv2d(x.tolist(), w.tolist(), b.tolist(), (s, s), (p, p), relu=relu))
        if y.shape != yb.shape or not np.allclose(y, yb, rtol=1e-12, atol=1e-12):
            return False
        ref = torch.nn.functional.conv2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b),
                                         stride=s, padding=p)
        if relu:
            ref = torch.relu(ref)
        if not np.allclose(y, ref.numpy(), rtol=1e-11, atol=1e-11):
            return False
    for relu in (False, True):
        x, w, b = rng.standard_normal((5, 5)), rng.standard_normal((3, 5)), rng.standard_normal(3)
        yl = _linear(lib, x, w, b, relu)
        yb = np.array(brute.linear(x.tolist(), w.tolist(), b.tolist(), relu=relu))
        if not np.allclose(yl, yb, rtol=1e-12, atol=1e-12):
            return False
    return True


def test_unmodified_direct_copy_passes_the_pins(tmp_path):
    assert _direct_pins_pass(_build_direct(tmp_path, "none", "int oracle_conv2d_f64", "int oracle_conv2d_f64"))


@pytest.mark.parametrize("name", sorted(DIRECT_MUTATIONS))
def test_planted_direct_mistake_is_caught(tmp_path, name):
    old, new = DIRECT_MUTATIONS[name]
    assert not _direct_pins_pass(_build_direct(tmp_path, name, old, new))


# ----------------------------------------------------------------- prune ---
PRUNE_MUTATIONS = {
    "scores_over_wrong_axis": ("return np.cumsum(sq, axis=0)[-1]", "return np.cumsum(sq, axis=1)[:, -1]"),
    "ties_to_higher_index": ('order = np.argsort(-scores, kind="stable")',
                             'order = (len(scores) - 1 - np.argsort(-scores[::-1], kind="stable"))'),
    "kept_count_floors": ("return (int(extent) + int(rate) - 1) // int(rate)",
                          "return max(1, int(extent) // int(rate))"),
    "abs_instead_of_square": ("sq = block * block", "sq = np.abs(block)"),
    "keeps_smallest": ("order = np.argsort(-scores, kind=\"stable\")", "order = np.argsort(scores, kind=\"stable\")"),
    "ragged_block_anchored_at_the_end": (
        "return [(s, min(s + b, extent)) for s in range(0, extent, b)]",
        "return [(max(0, e - b), e) for e in range(int(extent), 0, -b)][::-1]"),
}


def _load_prune(tmp_path, name, old, new):
    src = open(os.path.join(ROOT, "oracle", "prune.py")).read()
    assert src.count(old) == 1, name
    path = tmp_path / ("prune_%s.py" % name)
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("planted_prune_%s" % name, str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _brute_keep(scores, k):
    best, best_set = None, None
    for sub in itertools.combinations(range(len(scores)), k):
        s = math.fsum(scores[i] for i in sub)
        if best is None or s > best:
            best, best_set = s, sub
    return list(best_set)


def _prune_pins_pass(P) -> bool:
    """Golden hand examples + k-subset enumeration of tests/test_oracle_prune.py."""
    g = GOLD["matrix_4x8"]
    W = np.array(g["W"], dtype=np.float64)
    if P.prune_mask(W, 2, 4, P.COL, 2).tolist() != g["col_2x4_rate2"]["mask"]:
        return False
    if P.prune_mask(W, 2, 4, P.ROW, 2).tolist() != g["row_2x4_rate2"]["mask"]:
        return False
    gr = GOLD["ragged_5x7"]
    Wr = np.array(gr["W"], dtype=np.float64)
    if P.prune_mask(Wr, 2, 3, P.COL, 2).tolist() != gr["col_2x3_rate2"]["mask"]:
        return False
    if P.prune_mask(Wr, 2, 3, P.ROW, 2).tolist() != gr["row_2x3_rate2"]["mask"]:
        return False
    rng = np.random.default_rng(11)
    for trial in range(40):
        bh, bw = int(rng.integers(1, 5)), int(rng.integers(1, 7))
        R, C = bh * int(rng.integers(1, 3)), bw * int(rng.integers(1, 3))
        Wt = rng.integers(-2, 3, size=(R, C)).astype(np.float64)
        rate = int(rng.integers(1, 5))
        for reg in (P.COL, P.ROW):
            m = P.prune_mask(Wt, bh, bw, reg, rate)
            for r0, r1 in P.block_ranges(R, bh):
                for c0, c1 in P.block_ranges(C, bw):
                    blk = Wt[r0:r1, c0:c1]
                    if reg == P.COL:
                        sc = [math.fsum(float(v) ** 2 for v in blk[:, j]) for j in range(c1 - c0)]
                        want = _brute_keep(sc, (c1 - c0 + rate - 1) // rate)
                        got = np.nonzero(m[r0, c0:c1])[0].tolist()
                    else:
                        sc = [math.fsum(float(v) ** 2 for v in blk[i, :]) for i in range(r1 - r0)]
                        want = _brute_keep(sc, (r1 - r0 + rate - 1) // rate)
                        got = np.nonzero(m[r0:r1, c0])[0].tolist()
                    if got != want:
                        return False
    return True


def test_unmodified_prune_copy_passes_the_pins(tmp_path):
    assert _prune_pins_pass(_load_prune(tmp_path, "none", "import numpy as np", "import numpy as np"))


@pytest.mark.parametrize("name", sorted(PRUNE_MUTATIONS))
def test_planted_prune_mistake_is_caught(tmp_path, name):
    old, new = PRUNE_MUTATIONS[name]
    assert not _prune_pins_pass(_load_prune(tmp_path, name, old, new))


# ----------------- block-punched, row + column, per-block counts, BCS ---
# The planted copy replaces the oracle module seen by the pins of
# tests/test_oracle_prune.py (hand-worked examples, the paper's BCS fragment,
# brute force, reductions to column / row pruning); at least one must fail.
EXT_MUTATIONS = {
    "punched_location_axis_transposed": ("w3 = wg.reshape(R, cin, khw)",
                                         "w3 = wg.reshape(R, khw, cin).transpose(0, 2, 1)"),
    "punched_count_from_channels": ("k = _count(counts, i, j, kept_count(khw, rate))",
                                    "k = _count(counts, i, j, kept_count(c1 - c0, rate))"),
    "rowcol_rows_by_reversed_scores": (
        "rows = top_k(group_scores(blk, ROW), kept_count(r1 - r0, rate))",
        "rows = top_k(group_scores(blk, ROW)[::-1], kept_count(r1 - r0, rate))"),
    "counts_ignored": ("    if counts is None:\n        return default", "    return default"),
    "bcs_runs_never_merge": ("if r == 0 or not np.array_equal(cols[r], cols[r - 1]):", "if True:"),
    "bcs_stride_holds_run_starts": ("            stride.append(len(compact))",
                                    "            stride.append(len(compact) - len(cols[r]))"),
    "pattern_library_least_frequent": ("library = sorted(counts, key=lambda code: (-counts[code], code))[:n_patterns]",
                                       "library = sorted(counts, key=lambda code: (counts[code], code))[:n_patterns]"),
    "pattern_connectivity_floors": ("return min(n_kernels, (n_kernels * khw + 4 * rate - 1) // (4 * rate))",
                                    "return min(n_kernels, (n_kernels * khw) // (4 * rate))"),
    "pattern_keeps_weakest_kernels": ("    keep = top_k(best, pattern_kept_kernels(R * cin, rate, khw))",
                                      "    keep = top_k(-best, pattern_kept_kernels(R * cin, rate, khw))"),
}


def _ext_pins_pass(P):
    import tests.test_oracle_prune as T
    saved = T.P
    T.P = P
    checks = [
        lambda: [T.test_punched_golden_masks(c) for c in ("whole_block_rate2", "filter_blocks_rate2",
                                                             "channel_blocks_rate4")],
        lambda: [T.test_punched_brute_force_on_small_integer_blocks(s) for s in range(3)],
        lambda: T.test_punched_with_one_channel_blocks_is_column_pruning(2, 2, 9),
        T.test_rowcol_golden_mask,
        lambda: T.test_rowcol_reduces_to_column_and_row_blocks(4, 8, 2),
        lambda: [T.test_counts_brute_force_on_small_integer_blocks(r) for r in (T.P.COL, T.P.ROW)],
        T.test_counts_pack_lengths_and_edge_counts,
        T.test_bcs_matches_the_paper_example_and_its_completion,
        lambda: T.test_bcs_is_csr_with_shared_column_runs(16, 32, T.P.COL, 4),
        lambda: T.test_pattern_with_every_pattern_allowed_keeps_each_kernels_best_four(False),
        T.test_pattern_library_is_the_most_frequent_sets_and_kernels_take_their_best_pattern,
        lambda: [T.test_pattern_connectivity_keeps_the_strongest_kernels(r) for r in (3, 4, 8)],
    ]
    try:
        for c in checks:
            try:
                c()
            except Exception:
                return False
        return True
    finally:
        T.P = saved


def test_extended_pins_pass_on_the_oracle():
    from oracle import prune as P
    assert _ext_pins_pass(P)


@pytest.mark.parametrize("name", sorted(EXT_MUTATIONS))
def test_planted_mistake_in_extended_schemes_is_caught(tmp_path, name):
    old, new = EXT_MUTATIONS[name]
    assert not _ext_pins_pass(_load_prune(tmp_path, name, old, new))


# ------------------------------------------------- parity gates themselves ---
# The forward parity tests gate every output three ways (tests/helpers.check_output):
# global rel-L2, rel-L2 per (image, output channel) plane, and an element-wise
# rounding bound.  A stand-in for the kernel that accumulates in fp32 and rounds to
# bf16 must pass all three; the same stand-in with one kept column of one output row
# left out passes the global norm but must fail the other two.

def _fp32_conv_bf16(x_bits, w_bits, mask, layer):
    """fp32-accumulating conv (torch on the CPU) of the bf16 inputs, rounded to bf16."""
    from tests.helpers import as_f64
    x = torch.from_numpy(as_f64(x_bits, "bf16").astype(np.float32))
    wm = (as_f64(w_bits, "bf16").reshape(layer.cout, -1) * mask).reshape(layer.w_shape).astype(np.float32)
    y = torch.nn.functional.conv2d(x, torch.from_numpy(wm), stride=(layer.sh, layer.sw),
                                   padding=(layer.ph, layer.pw))
    return y.to(torch.bfloat16).to(torch.float64).numpy()


def test_one_dropped_kept_column_fails_the_plane_and_element_gates(oracle_direct):
    from synthetic import ConvLayer, COL, draw_layer
    from tests.helpers import gate_conv, oracle_conv, oracle_mask, rel_l2
    layer = ConvLayer("3x3 256@14 col16x32 r4", 1, 256, 14, 14, 256, 3, 3, 1, 1, 1, 1, 16, 32, COL, 4, "bf16",
                      ("normal", 0, 1.0), ("normal", 0, (2.0 / 2304) ** 0.5))
    d = draw_layer(layer, 9, 0)
    m = oracle_mask(d["w"], "bf16", layer.scheme)
    good = _fp32_conv_bf16(d["x"], d["w"], m, layer)
    gate_conv(good, d["x"], d["w"], m, "bf16", "bf16", layer)
    # output row 77 loses a kept column of median weight magnitude
    m2 = m.reshape(layer.cout, -1).copy()
    o = 77
    kept = np.nonzero(m2[o])[0]
    wo = np.abs(as_f64_bits(d["w"]).reshape(layer.cout, -1)[o, kept])
    q = kept[np.argsort(wo)[len(kept) // 2]]
    m2[o, q] = 0
    bad = _fp32_conv_bf16(d["x"], d["w"], m2, layer)
    ref = oracle_conv(d["x"], d["w"], m, "bf16", layer)
    assert rel_l2(bad, ref) <= 5e-3        # the global norm alone lets it through
    with pytest.raises(AssertionError, match="plane rel-L2|error bound"):
        gate_conv(bad, d["x"], d["w"], m, "bf16", "bf16", layer)


def as_f64_bits(w_bits):
    from tests.helpers import as_f64
    return as_f64(w_bits, "bf16")


# --------------------------------------------------------------- maxpool ---
GLUE_MUTATIONS = {
    "window_one_row_down": ("x[:, :, 2 * i + 1, 2 * j], x[:, :, 2 * i + 1, 2 * j + 1]",
                            "x[:, :, 2 * i + 2 - (2 * i + 2 >= H), 2 * j], x[:, :, 2 * i + 1, 2 * j + 1]"),
    "nan_ignored": ("out[:, :, i, j] = np.maximum(np.maximum(", "out[:, :, i, j] = np.fmax(np.fmax("),
    "ceil_instead_of_floor": ("Ho, Wo = H // 2, W // 2", "Ho, Wo = (H + 1) // 2, (W + 1) // 2"),
    "min_for_one_pair": ("np.maximum(x[:, :, 2 * i + 1, 2 * j]", "np.minimum(x[:, :, 2 * i + 1, 2 * j]"),
}


def _load_glue(tmp_path, name, old, new):
    src = open(os.path.join(ROOT, "oracle", "glue.py")).read()
    assert src.count(old) == 1, name
    if name == "nan_ignored":
        src = src.replace(old, new).replace("np.maximum(x[:, :, 2 * i + 1", "np.fmax(x[:, :, 2 * i + 1")
    else:
        src = src.replace(old, new)
    path = tmp_path / ("glue_%s.py" % name)
    path.write_text(src)
    spec = importlib.util.spec_from_file_location("planted_glue_%s" % name, str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _glue_pins_pass(G) -> bool:
    import tests.test_oracle_direct as T
    import oracle
    saved = oracle.glue if hasattr(oracle, "glue") else None
    import sys
    saved_mod = sys.modules.get("oracle.glue")
    sys.modules["oracle.glue"] = G
    oracle.glue = G
    try:
        try:
            T.test_maxpool_golden_example()
            for shape in [(2, 3, 4, 4), (1, 2, 5, 7), (3, 1, 9, 2), (1, 1, 1, 6)]:
                T.test_maxpool_matches_brute_force_with_nonfinite_values(shape)
        except Exception:
            return False
        return True
    finally:
        if saved_mod is not None:
            sys.modules["oracle.glue"] = saved_mod
        if saved is not None:
            oracle.glue = saved


def test_unmodified_glue_copy_passes_the_pins(tmp_path):
    assert _glue_pins_pass(_load_glue(tmp_path, "none", "import numpy as np", "import numpy as np"))


@pytest.mark.parametrize("name", sorted(GLUE_MUTATIONS))
def test_planted_maxpool_mistake_is_caught(tmp_path, name):
    old, new = GLUE_MUTATIONS[name]
    assert not _glue_pins_pass(_load_glue(tmp_path, name, old, new))
