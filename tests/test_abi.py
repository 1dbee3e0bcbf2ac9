"""The C-ABI library loads and exports every declared symbol; host-only logic
(sizes, argument validation, fast division, row staging) is right.  CPU only:
no call here launches a kernel."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bsp.h")


@pytest.fixture(scope="module")
def bsp():
    import paper_2111_11581_amd as B
    if not os.path.exists(B.lib_path()):
        from paper_2111_11581_amd import build
        build.build()
    B.lib()
    return B


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bsp_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(bsp):
    syms = declared_symbols()
    assert len(syms) >= 9
    for s in syms:
        assert hasattr(bsp.lib(), s), s


def test_status_strings_and_version(bsp):
    assert bsp.bsp_status_string(0) == "ok"
    assert "block structure" in bsp.bsp_status_string(-4)
    assert bsp.bsp_version() == 100


def _sizes_from_oracle(R, C, bh, bw, reg, rate, khw=1):
    from oracle import prune as OP
    w = np.random.default_rng(R + C).standard_normal((R, C))
    m = OP.prune_mask(w, bh, bw, reg, rate, khw=khw)
    pk = OP.pack(w.astype(np.float32), m, bh, bw, reg, rate)
    return pk["values"].size, pk["indices"].size, pk["rowptr"].size


@pytest.mark.parametrize("R,C,bh,bw,reg,rate", [
    (64, 576, 16, 16, 1, 4), (64, 576, 8, 16, 1, 8), (256, 64, 32, 32, 0, 2), (37, 53, 8, 16, 1, 3),
    (37, 53, 8, 16, 0, 3), (40, 40, 0, 0, 1, 4), (40, 40, 0, 0, 0, 4), (96, 100, 32, 32, 1, 10),
    (64, 147, 0, 0, 3, 1), (30, 20, 1, 1, 2, 4), (64, 576, 16, 32, 5, 2), (37, 53, 8, 16, 5, 3)])
def test_packed_sizes_match_oracle_packing(bsp, R, C, bh, bw, reg, rate):
    s = bsp.Scheme(R, C, bh, bw, reg, rate)
    nv, ni, nr, nb = bsp.bsp_packed_sizes(s, None, bsp.BF16)
    assert (nv, ni, nr) == _sizes_from_oracle(R, C, bh, bw, reg, rate)
    assert nb > 256


@pytest.mark.parametrize("R,cin,khw,bh,bw,rate", [
    (64, 64, 9, 16, 8, 2), (37, 20, 9, 8, 0, 3), (48, 12, 25, 0, 5, 4), (32, 32, 4, 4, 4, 2), (20, 7, 9, 3, 2, 9)])
def test_packed_sizes_match_oracle_packing_block_punched(bsp, R, cin, khw, bh, bw, rate):
    s = bsp.Scheme(R, cin * khw, bh, bw, bsp.PUNCHED, rate, khw)
    nv, ni, nr, nb = bsp.bsp_packed_sizes(s, None, bsp.BF16)
    assert (nv, ni, nr) == _sizes_from_oracle(R, cin * khw, bh, bw, bsp.PUNCHED, rate, khw)
    k = int(np.sqrt(khw))
    conv = bsp.ConvShape(1, cin, 12, 12, k, k, 1, 1, k // 2, k // 2)
    assert bsp.bsp_packed_sizes(s, conv, bsp.BF16)[:3] == (nv, ni, nr)


def test_block_punched_argument_errors(bsp):
    L = bsp.lib()
    out = [ctypes.c_int64() for _ in range(4)]
    EINVAL = -1
    bad = bsp.Scheme(64, 64 * 9 + 1, 16, 8, bsp.PUNCHED, 2, 9)      # columns not Cin * khw
    assert L.bsp_packed_sizes(ctypes.byref(bad), None, 1, *[ctypes.byref(o) for o in out]) == EINVAL
    s = bsp.Scheme(64, 64 * 9, 16, 8, bsp.PUNCHED, 2, 9)
    conv = bsp.ConvShape(1, 144, 12, 12, 2, 2, 1, 1, 0, 0)           # 144 x 2 x 2 columns, khw 4 != 9
    assert L.bsp_packed_sizes(ctypes.byref(s), ctypes.byref(conv), 1, *[ctypes.byref(o) for o in out]) == EINVAL


def test_argument_errors_are_reported_before_any_launch(bsp):
    L = bsp.lib()
    s = bsp.Scheme(64, 576, 16, 16, 1, 4)
    conv = bsp.ConvShape(1, 64, 32, 32, 3, 3, 1, 1, 1, 1)
    EINVAL = -1
    # null pointers
    assert L.bsp_prune(ctypes.byref(s), 1, None, None, None) == EINVAL
    assert L.bsp_conv2d(ctypes.byref(s), ctypes.byref(conv), 1, 1, None, None, None, 0, None, None) == EINVAL
    # bad scheme: rate 0, negative block, bad regularity
    for bad in (bsp.Scheme(64, 576, 16, 16, 1, 0), bsp.Scheme(64, 576, -1, 16, 1, 4),
                bsp.Scheme(64, 576, 16, 16, 7, 4), bsp.Scheme(0, 576, 16, 16, 1, 4)):
        out = [ctypes.c_int64() for _ in range(4)]
        assert L.bsp_packed_sizes(ctypes.byref(bad), None, 1, *[ctypes.byref(o) for o in out]) == EINVAL
    # conv geometry that does not match the GEMM form (cols != cin*kh*kw)
    wrong = bsp.ConvShape(1, 32, 32, 32, 3, 3, 1, 1, 1, 1)
    out = [ctypes.c_int64() for _ in range(4)]
    assert L.bsp_packed_sizes(ctypes.byref(s), ctypes.byref(wrong), 1, *[ctypes.byref(o) for o in out]) == EINVAL
    # bad dtype
    assert L.bsp_packed_sizes(ctypes.byref(s), None, 5, *[ctypes.byref(o) for o in out]) == EINVAL
    # bad maxpool sizes
    assert L.bsp_maxpool2x2(1, -1, 1, 2, 2, ctypes.c_void_p(16), ctypes.c_void_p(16), None) == EINVAL


HOST_TEST = r"""
#include <cstdio>
#include <cstdlib>
#include "bsp_common.h"
using namespace bsp;
int main() {
  // fast division against the hardware divide
  unsigned ds[] = {1,2,3,5,7,9,10,13,49,56,64,100,196,3136,12544,65535,1000003};
  for (unsigned d : ds) {
    FastDiv f = make_fastdiv(d);
    for (unsigned n = 0; n < 300000; n += 1) if (fdiv(n, f) != n / d) { printf("fdiv %u %u\n", n, d); return 1; }
    for (unsigned n = 2147483647u; n > 2147000000u; n -= 97) if (fdiv(n, f) != n / d) { printf("fdiv hi %u %u\n", n, d); return 1; }
  }
  // slot staging: every (tile row, filter row) pair must name the input row it needs
  int Hs[] = {7, 14, 28, 56, 3};
  for (int Ho : Hs) for (int KH = 1; KH <= 7; KH += 2) for (int SH = 1; SH <= 2; ++SH)
  for (int TRW : {1, 2, 4, 8, 16}) for (int g0 = 0; g0 < 3 * Ho; g0 += TRW) {
    int rb[16], im[256], ih[256];
    for (int i = 0; i < 256; ++i) { im[i] = -7; ih[i] = -7; }
    int PH = KH / 2;
    int ns = slot_layout(g0, TRW, Ho, 2 * Ho + 1, KH, SH, PH, rb, im, ih);
    for (int tr = 0; tr < TRW; ++tr) {
      int g = g0 + tr; if (g >= 2 * Ho + 1) { if (rb[tr] != 0) return 2; continue; }
      // the forward kernel computes each row's base in closed form
      int k = g / Ho - g0 / Ho;
      int closed = (tr - k) * (SH < KH ? SH : KH) + k * KH;
      if (closed != rb[tr]) { printf("closed form %d %d %d %d %d\n", Ho, KH, SH, g0, tr); return 4; }
      int img = g / Ho, oh = g % Ho;
      for (int r = 0; r < KH; ++r) {
        int sl = rb[tr] + r;
        if (sl >= ns || im[sl] != img || ih[sl] != oh * SH - PH + r) { printf("slot %d %d %d %d\n", Ho, KH, SH, g0); return 3; }
      }
    }
  }
  printf("ok\n");
  return 0;
}
"""


def test_fastdiv_and_slot_layout_host(tmp_path):
    src = tmp_path / "t.cpp"
    src.write_text(HOST_TEST)
    exe = tmp_path / "t"
    subprocess.run(["g++", "-O2", "-std=c++17", f"-I{ROOT}/include",
                    f"-I{ROOT}/paper_2111_11581_amd/csrc", str(src), "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout


def test_every_tested_and_benchmarked_layer_gets_a_plan(bsp):
    """The planner finds a tiling (host only) for every configuration the GPU parity
    tests and the benchmark workloads run."""
    from synthetic import workload
    from tests.test_gpu_parity import CONV_CASES, MATS
    missing = []
    for c in CONV_CASES:
        l = c["layer"]
        conv = bsp.ConvShape(l.n, l.cin, l.h, l.w, l.kh, l.kw, l.sh, l.sw, l.ph, l.pw)
        try:
            bsp.bsp_packed_sizes(l.scheme, conv, bsp.F32 if l.dtype == "f32" else bsp.BF16)
        except bsp.BspError as e:
            missing.append((c["name"], str(e)))
    for name, R, C, bh, bw, reg, rate, dtype, _ in MATS:
        try:
            bsp.bsp_packed_sizes(bsp.Scheme(R, C, bh, bw, reg, rate), None, bsp.F32 if dtype == "f32" else bsp.BF16)
        except bsp.BspError as e:
            missing.append((name, str(e)))
    for cfg in (1, 2, 3, 4):
        for l in workload(cfg):
            conv = None if l.kind != "conv" else bsp.ConvShape(l.n, l.cin, l.h, l.w, l.kh, l.kw, l.sh, l.sw, l.ph, l.pw)
            try:
                bsp.bsp_packed_sizes(l.scheme, conv, bsp.F32 if l.dtype == "f32" else bsp.BF16)
            except bsp.BspError as e:
                missing.append((l.name, str(e)))
    assert not missing, missing


def _random_counts(nbr, nbc, groups, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, np.asarray(groups) + 1, size=(nbr, nbc)).astype(np.int32)


@pytest.mark.parametrize("R,C,bh,bw,reg,khw", [
    (64, 576, 16, 32, 1, 1), (37, 53, 8, 16, 1, 1), (37, 53, 8, 16, 0, 1), (48, 96, 0, 32, 0, 1),
    (40, 90, 16, 0, 1, 1), (20, 7 * 9, 6, 3, 4, 9)])
def test_packed_sizes_with_per_block_counts_match_oracle_packing(bsp, R, C, bh, bw, reg, khw):
    from oracle import prune as OP
    rr = OP.block_ranges(R, bh)
    cc = OP.block_ranges(C // khw if reg == 4 else C, bw)
    groups = [[khw if reg == 4 else ((c1 - c0) if reg == 1 else (r1 - r0)) for c0, c1 in cc] for r0, r1 in rr]
    cnt = _random_counts(len(rr), len(cc), groups, R * C + reg)
    s = bsp.Scheme(R, C, bh, bw, reg, 3, khw).set_counts(cnt)
    nv, ni, nr, nb = bsp.bsp_packed_sizes(s, None, bsp.BF16)
    w = np.random.default_rng(1).standard_normal((R, C))
    m = OP.prune_mask(w, bh, bw, reg, 3, khw=khw, counts=cnt)
    pk = OP.pack(w.astype(np.float32), m, bh, bw, reg, 3)
    assert (nv, ni, nr) == (pk["values"].size, pk["indices"].size, pk["rowptr"].size)
    # other counts give another fingerprint: the dev_tiles size or header differs
    cnt2 = cnt.copy()
    cnt2.flat[0] = (cnt2.flat[0] + 1) % (groups[0][0] + 1)
    s2 = bsp.Scheme(R, C, bh, bw, reg, 3, khw).set_counts(cnt2)
    assert bsp.bsp_packed_sizes(s2, None, bsp.BF16)[:2] != (nv, ni) or cnt2.flat[0] == cnt.flat[0]


def test_pattern_scheme_sizes_and_errors(bsp):
    s = bsp.Scheme(64, 64 * 9, 8, 0, bsp.PATTERN, 4, 9)
    nv, ni, nr, nb = bsp.bsp_packed_sizes(s, None, bsp.BF16)
    assert (nv, ni, nr) == _sizes_from_oracle(64, 64 * 9, 8, 0, bsp.PATTERN, 4, 9)
    L = bsp.lib()
    out = [ctypes.c_int64() for _ in range(4)]
    for bad in (bsp.Scheme(64, 64 * 9, 8, 0, bsp.PATTERN, 4, 4), bsp.Scheme(64, 64 * 9, 127, 0, bsp.PATTERN, 4, 9)):
        assert L.bsp_packed_sizes(ctypes.byref(bad), None, 1, *[ctypes.byref(o) for o in out]) == -1


def test_per_block_counts_out_of_range_are_rejected(bsp):
    L = bsp.lib()
    out = [ctypes.c_int64() for _ in range(4)]
    s = bsp.Scheme(32, 64, 16, 32, 1, 2).set_counts([[3, 33], [0, 1]])     # 33 > 32 columns
    assert L.bsp_packed_sizes(ctypes.byref(s), None, 1, *[ctypes.byref(o) for o in out]) == -1
    s = bsp.Scheme(32, 64, 16, 32, 1, 2).set_counts([[3, -1], [0, 1]])
    assert L.bsp_packed_sizes(ctypes.byref(s), None, 1, *[ctypes.byref(o) for o in out]) == -1


def test_prune_noalloc_rejects_before_any_launch(bsp):
    """The allocation-free prune validates on the host: too large an unstructured
    layer gives BSP_ETOOLARGE, pattern-based pruning and per-block counts
    BSP_EUNSUPPORTED, and nothing is launched (the pointers are never touched)."""
    L = bsp.lib()
    fake = ctypes.c_void_p(16)
    big = bsp.Scheme(1 << 15, (1 << 13) + 1, 1, 1, bsp.UNSTRUCTURED, 4)       # 2^28 + 2^15 weights
    assert L.bsp_prune_noalloc(ctypes.byref(big), bsp.BF16, fake, fake, None) == -5
    assert "fixed scratch" in bsp.bsp_status_string(-5)
    pat = bsp.Scheme(64, 64 * 9, 8, 0, bsp.PATTERN, 4, 9)
    assert L.bsp_prune_noalloc(ctypes.byref(pat), bsp.BF16, fake, fake, None) == -2
    cnt = bsp.Scheme(64, 64, 32, 32, bsp.COL, 4).set_counts([[4, 5], [6, 7]])
    assert L.bsp_prune_noalloc(ctypes.byref(cnt), bsp.BF16, fake, fake, None) == -2
    assert L.bsp_prune_noalloc(None, bsp.BF16, fake, fake, None) == -1
