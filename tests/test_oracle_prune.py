"""Pins of the pruning / packing oracle (CPU only).

The oracle follows Sec. 4.1.1 and Eqs. 2-3 (block rows / columns as groups,
squared Frobenius norm) with the readings: keep ceil(extent/rate) groups per
block, ties to the lower index, fp64 sequential scores.  These tests check it
against things other than itself: hand-worked examples, brute-force subset
enumeration, exact sums, structural invariants and scale invariance.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import prune as P
from synthetic import f32_to_bf16_bits, bf16_bits_to_f32

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")))


# ---------------------------------------------------------------- golden ---
def test_golden_col_mask_and_pack():
    g = GOLD["matrix_4x8"]
    W = np.array(g["W"], dtype=np.float32)
    ex = g["col_2x4_rate2"]
    m = P.prune_mask(W.astype(np.float64), 2, 4, P.COL, 2)
    assert m.tolist() == ex["mask"]
    pk = P.pack(W, m, 2, 4, P.COL, 2)
    assert pk["indices"].tolist() == ex["indices"]
    assert pk["rowptr"].tolist() == ex["rowptr"]
    assert pk["values"].tolist() == ex["values"]


def test_golden_row_mask_and_pack():
    g = GOLD["matrix_4x8"]
    W = np.array(g["W"], dtype=np.float32)
    ex = g["row_2x4_rate2"]
    m = P.prune_mask(W.astype(np.float64), 2, 4, P.ROW, 2)
    assert m.tolist() == ex["mask"]
    pk = P.pack(W, m, 2, 4, P.ROW, 2)
    assert pk["indices"].tolist() == ex["indices"]
    assert pk["rowptr"].tolist() == ex["rowptr"]
    assert pk["values"].tolist() == ex["values"]


@pytest.mark.parametrize("reg", [P.COL, P.ROW])
def test_golden_ragged_blocks_mask_and_pack(reg):
    """Blocks anchored at (0, 0) with a ragged last block-row and block-column, worked
    by hand (5x7 matrix, 2x3 blocks, rate 2)."""
    g = GOLD["ragged_5x7"]
    W = np.array(g["W"], dtype=np.float32)
    ex = g["col_2x3_rate2" if reg == P.COL else "row_2x3_rate2"]
    m = P.prune_mask(W.astype(np.float64), 2, 3, reg, 2)
    assert m.tolist() == ex["mask"]
    pk = P.pack(W, m, 2, 3, reg, 2)
    assert pk["indices"].tolist() == ex["indices"]
    assert pk["rowptr"].tolist() == ex["rowptr"]
    assert pk["values"].tolist() == ex["values"]
    assert P.mask_is_valid(m, 2, 3, reg, 2)


def test_ragged_block_edges_without_the_oracles_block_ranges():
    """The last block starts at a multiple of the block size: a column that the
    last (ragged) block holds alone is always kept, whatever its score; a column of
    a full block with the lowest score of its block is removed (rate 2, bw 3)."""
    rng = np.random.default_rng(3)
    for R, C, bh, bw in ((5, 7, 2, 3), (9, 10, 4, 3), (37, 53, 8, 16)):
        W = rng.standard_normal((R, C))
        W[:, C - 1] *= 1e-6                    # weakest column of all
        m = P.prune_mask(W, bh, bw, P.COL, 2)
        last0 = (C - 1) // bw * bw             # first column of the last block
        width = C - last0
        assert m[:, C - 1].all() == (width == 1)
        assert m[:, last0:].sum(axis=1).tolist() == [-(-width // 2)] * R
        Wr = rng.standard_normal((R, C))
        Wr[R - 1, :] *= 1e-6
        mr = P.prune_mask(Wr, bh, bw, P.ROW, 2)
        first_last_row = (R - 1) // bh * bh
        assert mr[R - 1, :].all() == (R - first_last_row == 1)


def test_golden_whole_matrix_conv_taps():
    g = GOLD["conv_plus_3x3"]
    wg = np.array(g["w"], dtype=np.float64).reshape(1, 9)
    m = P.prune_mask(wg, 0, 0, P.COL, 3)
    assert m.reshape(-1).tolist() == g["col_whole_rate3"]["mask"]


# ------------------------------------------------------------- brute force ---
def _brute_keep(scores, k):
    """Max-sum k-subset; among equal sums the lexicographically smallest."""
    best, best_set = None, None
    for sub in itertools.combinations(range(len(scores)), k):
        s = math.fsum(scores[i] for i in sub)
        if best is None or s > best:
            best, best_set = s, sub
    return list(best_set)


@pytest.mark.parametrize("reg", [P.COL, P.ROW])
def test_topk_equals_subset_enumeration(reg):
    rng = np.random.default_rng(7)
    for trial in range(60):
        bh, bw = int(rng.integers(1, 5)), int(rng.integers(1, 7))
        R, C = bh * int(rng.integers(1, 3)), bw * int(rng.integers(1, 3))
        # small integers: many exact ties
        W = rng.integers(-2, 3, size=(R, C)).astype(np.float64)
        rate = int(rng.integers(1, 5))
        m = P.prune_mask(W, bh, bw, reg, rate)
        for r0, r1 in P.block_ranges(R, bh):
            for c0, c1 in P.block_ranges(C, bw):
                blk = W[r0:r1, c0:c1]
                if reg == P.COL:
                    sc = [math.fsum(float(v) ** 2 for v in blk[:, j]) for j in range(c1 - c0)]
                    kept = _brute_keep(sc, P.kept_count(c1 - c0, rate))
                    got = np.nonzero(m[r0, c0:c1])[0].tolist()
                else:
                    sc = [math.fsum(float(v) ** 2 for v in blk[i, :]) for i in range(r1 - r0)]
                    kept = _brute_keep(sc, P.kept_count(r1 - r0, rate))
                    got = np.nonzero(m[r0:r1, c0])[0].tolist()
                assert got == kept, (trial, reg, r0, c0)


def test_scores_equal_exact_sums_for_bf16():
    """Squares of bf16 values are exact in fp64 and a few dozen of them sum
    exactly, so the sequential fp64 score equals math.fsum."""
    rng = np.random.default_rng(3)
    a = bf16_bits_to_f32(f32_to_bf16_bits(rng.standard_normal((32, 16)).astype(np.float32)))
    blk = a.astype(np.float64)
    s_col = P.group_scores(blk, P.COL)
    s_row = P.group_scores(blk, P.ROW)
    for j in range(16):
        assert s_col[j] == math.fsum(float(v) * float(v) for v in blk[:, j])
    for i in range(32):
        assert s_row[i] == math.fsum(float(v) * float(v) for v in blk[i, :])


# -------------------------------------------------------------- invariants ---
CASES = [  # R, C, bh, bw, rate
    (64, 576, 16, 16, 4), (64, 576, 8, 16, 8), (128, 1152, 16, 32, 4), (256, 64, 32, 32, 2),
    (96, 100, 32, 32, 10), (37, 53, 8, 16, 3), (40, 40, 0, 0, 4), (40, 40, 0, 8, 2),
    (33, 70, 16, 0, 5), (16, 16, 4, 4, 16), (10, 7, 3, 2, 1),
]


@pytest.mark.parametrize("R,C,bh,bw,rate", CASES)
@pytest.mark.parametrize("reg", [P.COL, P.ROW])
def test_block_structure_invariants(R, C, bh, bw, rate, reg):
    rng = np.random.default_rng(R * 131 + C + rate)
    W = rng.standard_normal((R, C))
    m = P.prune_mask(W, bh, bw, reg, rate)
    assert P.mask_is_valid(m, bh, bw, reg, rate)
    for r0, r1 in P.block_ranges(R, bh):
        for c0, c1 in P.block_ranges(C, bw):
            blk = m[r0:r1, c0:c1]
            if reg == P.COL:
                assert np.all(blk == blk[0])               # whole columns kept or removed
                assert blk[0].sum() == -(-(c1 - c0) // rate)
            else:
                assert np.all(blk == blk[:, :1])           # whole rows kept or removed
                assert blk[:, 0].sum() == -(-(r1 - r0) // rate)
    # scaling by a power of two is exact in fp64 and cannot change the mask
    assert np.array_equal(P.prune_mask(W * 2.0 ** 7, bh, bw, reg, rate), m)
    assert np.array_equal(P.prune_mask(W * 2.0 ** -9, bh, bw, reg, rate), m)
    # the mask only depends on magnitudes
    assert np.array_equal(P.prune_mask(-W, bh, bw, reg, rate), m)


def test_rate_one_and_dense_keep_everything():
    W = np.random.default_rng(1).standard_normal((24, 40))
    for reg in (P.COL, P.ROW):
        assert P.prune_mask(W, 8, 8, reg, 1).all()
    assert P.prune_mask(W, 0, 0, P.DENSE, 1).all()


def test_duplicate_columns_tie_to_lower_index():
    W = np.zeros((4, 8))
    W[:, 2] = W[:, 5] = [1.0, -2.0, 0.5, 3.0]     # identical columns
    W[:, 7] = 10.0
    m = P.prune_mask(W, 4, 8, P.COL, 4)             # keep 2 of 8
    assert np.nonzero(m[0])[0].tolist() == [2, 7]
    Wr = W.T.copy()
    mr = P.prune_mask(Wr, 8, 4, P.ROW, 4)
    assert np.nonzero(mr[:, 0])[0].tolist() == [2, 7]


def test_whole_matrix_is_structured_pruning():
    """Whole-matrix column blocks remove the same columns for every row
    (channel-style pruning); row blocks remove whole filters (Sec. 4.4)."""
    W = np.random.default_rng(5).standard_normal((12, 30))
    m = P.prune_mask(W, 0, 0, P.COL, 3)
    norms = (W ** 2).sum(axis=0)
    assert sorted(np.nonzero(m[0])[0].tolist()) == sorted(np.argsort(-norms)[:10].tolist())
    mr = P.prune_mask(W, 0, 0, P.ROW, 4)
    rn = (W ** 2).sum(axis=1)
    assert sorted(np.nonzero(mr[:, 0])[0].tolist()) == sorted(np.argsort(-rn)[:3].tolist())


def test_block_1x1_saturates_under_uniform_rate():
    """With 1x1 blocks every weight is its own group and a uniform integer
    rate keeps ceil(1/r) = 1 of 1: nothing is pruned.  (The paper's 1x1 =
    unstructured equivalence needs per-block rates; unstructured magnitude
    pruning is therefore its own regularity here.)"""
    W = np.random.default_rng(2).standard_normal((5, 6))
    assert P.prune_mask(W, 1, 1, P.COL, 4).all()


# ------------------------------------------------------------ unstructured ---
def test_unstructured_threshold_and_ties():
    rng = np.random.default_rng(11)
    for rate in (2, 3, 4, 8, 16):
        W = rng.integers(-4, 5, size=(13, 17)).astype(np.float64)   # many ties
        m = P.unstructured_mask(W, rate)
        k = -(-W.size // rate)
        assert m.sum() == k
        a = np.abs(W).reshape(-1)
        kept, drop = a[m.reshape(-1) == 1], a[m.reshape(-1) == 0]
        if drop.size:
            assert kept.min() >= drop.max()
            thr = kept.min()
            # among entries equal to the threshold, kept ones precede dropped ones
            flat = m.reshape(-1)
            eq = np.nonzero(a == thr)[0]
            ks = eq[flat[eq] == 1]
            ds = eq[flat[eq] == 0]
            if ks.size and ds.size:
                assert ks.max() < ds.min()


# ------------------------------------------------------------------ packing ---
@pytest.mark.parametrize("R,C,bh,bw,rate", CASES)
@pytest.mark.parametrize("reg", [P.COL, P.ROW])
def test_pack_unpack_roundtrip(R, C, bh, bw, rate, reg):
    rng = np.random.default_rng(R + 7 * C)
    wf = rng.standard_normal((R, C)).astype(np.float32)
    wb = f32_to_bf16_bits(wf)
    for stored, dt in ((wf, "f32"), (wb, "bf16")):
        m = P.prune_mask(P.as_f64(stored, dt), bh, bw, reg, rate)
        pk = P.pack(stored, m, bh, bw, reg, rate)
        back = P.unpack(pk, R, C, bh, bw, reg, stored)
        expect = np.where(m == 1, stored, np.zeros_like(stored))
        assert back.dtype == stored.dtype
        assert np.array_equal(back.view(np.uint8), expect.view(np.uint8))
        assert pk["values"].size == int(m.sum())
        ptr, idx = pk["rowptr"], pk["indices"]
        assert np.all(np.diff(ptr) >= 0) and ptr[0] == 0 and ptr[-1] == idx.size
        if reg == P.COL:
            for i in range(len(ptr) - 1):
                seg = idx[ptr[i]:ptr[i + 1]]
                assert np.all(np.diff(seg) > 0) and seg.min() >= 0 and seg.max() < C
        else:
            for b in range(len(ptr) - 1):
                seg = idx[ptr[b]:ptr[b + 1]]
                assert np.all(np.diff(seg) > 0) and seg.min() >= 0 and seg.max() < R


def test_invalid_masks_are_rejected():
    rng = np.random.default_rng(4)
    W = rng.standard_normal((16, 32))
    m = P.prune_mask(W, 8, 16, P.COL, 4)
    assert P.mask_is_valid(m, 8, 16, P.COL, 4)
    bad = m.copy(); bad[3, np.nonzero(m[3])[0][0]] = 0            # a hole in a kept column
    assert not P.mask_is_valid(bad, 8, 16, P.COL, 4)
    bad = m.copy(); bad[:8, np.nonzero(m[0] == 0)[0][0]] = 1      # one column too many
    assert not P.mask_is_valid(bad, 8, 16, P.COL, 4)
    bad = m.copy(); bad[0, 0] = 2
    assert not P.mask_is_valid(bad, 8, 16, P.COL, 4)
    mr = P.prune_mask(W, 8, 16, P.ROW, 2)
    assert P.mask_is_valid(mr, 8, 16, P.ROW, 2)
    bad = mr.copy(); bad[np.nonzero(mr[:, 0])[0][0], 5] = 0
    assert not P.mask_is_valid(bad, 8, 16, P.ROW, 2)


# --------------------------------------------------------- block-punched ---
# Sec. 4.1.2 and Eq. 4: blocks of filters x input channels; the group of a kernel
# location is that location in every kernel of the block.

def _gemm(w_oihw):
    w = np.asarray(w_oihw, dtype=np.float64)
    return w.reshape(w.shape[0], -1)


@pytest.mark.parametrize("case", ["whole_block_rate2", "filter_blocks_rate2", "channel_blocks_rate4"])
def test_punched_golden_masks(case):
    g = GOLD["punched_2x2x2x2"]
    ex = g[case]
    m = P.prune_mask(_gemm(g["W_oihw"]), ex["bh"], ex["bw"], P.PUNCHED, ex["rate"], khw=4)
    assert m.tolist() == ex["mask"]
    assert P.mask_is_valid(m, ex["bh"], ex["bw"], P.PUNCHED, ex["rate"], khw=4)
    if "indices" in ex:
        pk = P.pack(_gemm(g["W_oihw"]), m, ex["bh"], ex["bw"], P.PUNCHED, ex["rate"])
        assert pk["indices"].tolist() == ex["indices"]
        assert pk["rowptr"].tolist() == ex["rowptr"]
        assert pk["values"].tolist() == ex["values"]


@pytest.mark.parametrize("bh,rate,khw", [(2, 2, 9), (4, 3, 9), (0, 9, 9), (3, 2, 25), (0, 4, 4)])
def test_punched_with_one_channel_blocks_is_column_pruning(bh, rate, khw):
    """A block of one input channel holds that channel's khw GEMM columns: punched
    locations are then the columns of a (bh x khw) column block (Eq. 3)."""
    rng = np.random.default_rng(bh * 100 + rate * 10 + khw)
    wg = rng.standard_normal((12, 5 * khw))
    m = P.prune_mask(wg, bh, 1, P.PUNCHED, rate, khw=khw)
    assert np.array_equal(m, P.prune_mask(wg, bh, khw, P.COL, rate))


@pytest.mark.parametrize("seed", range(6))
def test_punched_brute_force_on_small_integer_blocks(seed):
    """Integer weights make every sum exact; the kept locations of each block must
    be the k-subset of largest total score, lexicographically smallest on ties."""
    rng = np.random.default_rng(40 + seed)
    R, cin, khw = 5, 7, 4 + seed % 3 * 2          # khw 4, 6, 8
    bh, bw, rate = [(2, 3, 2), (0, 2, 3), (3, 0, 2)][seed % 3]
    w = rng.integers(-3, 4, size=(R, cin, khw)).astype(np.float64)
    m = P.prune_mask(w.reshape(R, -1), bh, bw, P.PUNCHED, rate, khw=khw).reshape(R, cin, khw)
    k = P.kept_count(khw, rate)
    for r0, r1 in P.block_ranges(R, bh):
        for c0, c1 in P.block_ranges(cin, bw):
            s = [sum(w[o, c, l] ** 2 for o in range(r0, r1) for c in range(c0, c1)) for l in range(khw)]
            best = max(itertools.combinations(range(khw), k), key=lambda t: (sum(s[i] for i in t),
                                                                              [-i for i in t]))
            kept = tuple(np.nonzero(m[r0, c0])[0])
            assert kept == best, (r0, c0, s)
            assert np.all(m[r0:r1, c0:c1] == m[r0, c0])


def test_punched_invariants_and_degenerate_cases():
    rng = np.random.default_rng(7)
    R, cin, khw = 16, 12, 9
    wg = rng.standard_normal((R, cin * khw))
    for bh, bw, rate in [(4, 4, 2), (8, 5, 3), (0, 0, 4), (3, 7, 9), (16, 1, 5)]:
        m = P.prune_mask(wg, bh, bw, P.PUNCHED, rate, khw=khw)
        assert P.mask_is_valid(m, bh, bw, P.PUNCHED, rate, khw=khw)
        # every kernel keeps ceil(khw / rate) locations
        assert np.all(m.reshape(R, cin, khw).sum(axis=2) == P.kept_count(khw, rate))
        # scale by a power of two and sign flip: same mask (exact in fp64)
        assert np.array_equal(P.prune_mask(-wg * 2.0 ** 5, bh, bw, P.PUNCHED, rate, khw=khw), m)
    assert P.prune_mask(wg, 4, 4, P.PUNCHED, 1, khw=khw).all()              # rate 1 keeps all
    assert P.prune_mask(wg, 4, 4, P.PUNCHED, 3, khw=1).all()                # 1x1 kernels: one location
    # a mask with one kernel off its block's pattern is rejected
    m = P.prune_mask(wg, 4, 4, P.PUNCHED, 3, khw=khw)
    bad = m.copy().reshape(R, cin, khw)
    bad[1, 2] = np.roll(bad[1, 2], 1)
    assert not P.mask_is_valid(bad.reshape(R, -1), 4, 4, P.PUNCHED, 3, khw=khw)


def test_punched_is_invariant_to_kernel_order_inside_a_block():
    """Integer weights (exact sums): permuting the filters or channels of a block
    permutes nothing in its kept locations."""
    rng = np.random.default_rng(11)
    R, cin, khw = 6, 4, 9
    w = rng.integers(-4, 5, size=(R, cin, khw)).astype(np.float64)
    m = P.prune_mask(w.reshape(R, -1), 0, 0, P.PUNCHED, 3, khw=khw).reshape(R, cin, khw)
    wp = w[rng.permutation(R)][:, rng.permutation(cin)]
    mp = P.prune_mask(wp.reshape(R, -1), 0, 0, P.PUNCHED, 3, khw=khw).reshape(R, cin, khw)
    assert np.array_equal(m[0, 0], mp[0, 0])


def test_punched_pack_unpack_roundtrip_bitwise():
    rng = np.random.default_rng(5)
    R, cin, khw = 20, 9, 9
    wb = f32_to_bf16_bits(rng.standard_normal((R, cin * khw)).astype(np.float32))
    wg = P.as_f64(wb, "bf16")
    for bh, bw, rate in [(8, 4, 3), (0, 2, 2), (6, 0, 9)]:
        m = P.prune_mask(wg, bh, bw, P.PUNCHED, rate, khw=khw)
        pk = P.pack(wb, m, bh, bw, P.PUNCHED, rate)
        # a block-row keeps cin * ceil(khw / rate) whole columns
        L = cin * P.kept_count(khw, rate)
        assert np.all(np.diff(pk["rowptr"]) == L)
        back = P.unpack(pk, R, cin * khw, bh, bw, P.PUNCHED, wb)
        assert np.array_equal(back, np.where(m == 1, wb, 0).astype(wb.dtype))


# ---------------------------------------------------- per-block kept counts ---
# Sec. 4.1.1: a block may keep the same or a different number of rows / columns;
# the counts (from the reweighted method of Sec. 4.2) are the caller's input.

def _uniform_counts(R, C, bh, bw, reg, rate, khw=1):
    rr = P.block_ranges(R, bh)
    if reg == P.PUNCHED:
        cc = P.block_ranges(C // khw, bw)
        return np.full((len(rr), len(cc)), P.kept_count(khw, rate), dtype=np.int32)
    cc = P.block_ranges(C, bw)
    return np.array([[P.kept_count((c1 - c0) if reg == P.COL else (r1 - r0), rate) for c0, c1 in cc]
                     for r0, r1 in rr], dtype=np.int32)


@pytest.mark.parametrize("R,C,bh,bw,reg,rate,khw", [
    (37, 53, 8, 16, P.COL, 3, 1), (37, 53, 8, 16, P.ROW, 3, 1), (64, 72, 16, 0, P.COL, 4, 1),
    (20, 7 * 9, 6, 3, P.PUNCHED, 2, 9), (48, 96, 0, 32, P.ROW, 5, 1)])
def test_counts_equal_to_the_uniform_rule_give_the_uniform_mask(R, C, bh, bw, reg, rate, khw):
    w = np.random.default_rng(R * C).standard_normal((R, C))
    cnt = _uniform_counts(R, C, bh, bw, reg, rate, khw)
    assert np.array_equal(P.prune_mask(w, bh, bw, reg, rate, khw=khw, counts=cnt),
                          P.prune_mask(w, bh, bw, reg, rate, khw=khw))


@pytest.mark.parametrize("reg", [P.COL, P.ROW])
def test_counts_brute_force_on_small_integer_blocks(reg):
    rng = np.random.default_rng(3 + reg)
    R, C, bh, bw = 6, 8, 3, 4
    W = rng.integers(-3, 4, size=(R, C)).astype(np.float64)
    cnt = np.array([[0, 3], [4, 1]], dtype=np.int32) if reg == P.COL else np.array([[2, 0], [3, 1]], np.int32)
    m = P.prune_mask(W, bh, bw, reg, 2, counts=cnt)
    assert P.mask_is_valid(m, bh, bw, reg, 2, counts=cnt)
    for i, (r0, r1) in enumerate(P.block_ranges(R, bh)):
        for j, (c0, c1) in enumerate(P.block_ranges(C, bw)):
            blk = W[r0:r1, c0:c1]
            s = (blk ** 2).sum(axis=0) if reg == P.COL else (blk ** 2).sum(axis=1)
            k = int(cnt[i, j])
            best = max(itertools.combinations(range(len(s)), k), key=lambda t: (sum(s[q] for q in t),
                                                                                [-q for q in t]))
            sub = m[r0:r1, c0:c1]
            kept = tuple(np.nonzero(sub[0] if reg == P.COL else sub[:, 0])[0])
            assert kept == best


def test_counts_pack_lengths_and_edge_counts():
    rng = np.random.default_rng(9)
    R, C, bh, bw = 40, 96, 16, 32
    w = rng.standard_normal((R, C)).astype(np.float32)
    cnt = np.array([[0, 32, 5], [1, 2, 3], [7, 0, 0]], dtype=np.int32)   # ragged last block-row of 8 rows
    m = P.prune_mask(w.astype(np.float64), bh, bw, P.COL, 4, counts=cnt)
    assert P.mask_is_valid(m, bh, bw, P.COL, 4, counts=cnt)
    assert not P.mask_is_valid(m, bh, bw, P.COL, 4)                    # not the uniform rule
    assert m[0:16, 0:32].sum() == 0 and m[0:16, 32:64].all()           # 0 and all columns kept
    pk = P.pack(w, m, bh, bw, P.COL, 4)
    assert np.diff(pk["rowptr"]).tolist() == cnt.sum(axis=1).tolist()
    back = P.unpack(pk, R, C, bh, bw, P.COL, w)
    assert np.array_equal(back, np.where(m == 1, w, 0).astype(np.float32))
    with pytest.raises(ValueError):
        P.prune_mask(w.astype(np.float64), bh, bw, P.COL, 4, counts=np.full((3, 3), 33))


# ------------------------------------------------------------------- BCS ---
def test_bcs_matches_the_paper_example_and_its_completion():
    """Sec. 4.3 prints a fragment of a BCS example; the fixture completes it by hand."""
    g = GOLD["bcs_sec43"]
    W = np.array(g["W"], dtype=np.float32)
    b = P.bcs_encode(W, (W != 0).astype(np.uint8))
    for k, pref in g["paper_prefix"].items():
        assert b[k][:len(pref)].tolist() == pref, k
    for k in ("weights", "row_offset", "occurrence", "compact_cols", "col_stride"):
        assert b[k].tolist() == g[k], k


@pytest.mark.parametrize("bh,bw,reg,rate", [(16, 32, P.COL, 4), (8, 16, P.COL, 3), (0, 0, P.COL, 2), (4, 4, P.ROW, 2)])
def test_bcs_is_csr_with_shared_column_runs(bh, bw, reg, rate):
    rng = np.random.default_rng(bh + bw + reg)
    R, C = 40, 96
    w = rng.standard_normal((R, C)).astype(np.float32)
    m = P.prune_mask(w.astype(np.float64), bh, bw, reg, rate)
    b = P.bcs_encode(w, m)
    # CSR equivalence: row offsets are CSR's indptr, runs expand to CSR's column indices
    indptr = np.concatenate([[0], np.cumsum(m.sum(axis=1))])
    assert np.array_equal(b["row_offset"], indptr)
    rows_cols = []
    for gi in range(len(b["occurrence"]) - 1):
        cols = b["compact_cols"][b["col_stride"][gi]:b["col_stride"][gi + 1]]
        rows_cols += [cols] * (b["occurrence"][gi + 1] - b["occurrence"][gi])
    assert np.array_equal(np.concatenate(rows_cols), np.nonzero(m)[1])
    assert np.array_equal(P.bcs_decode(b, R, C, w), np.where(m == 1, w, 0).astype(np.float32))
    if reg == P.COL and bh:
        # column blocks: every block-row is one run at most (more rows merge only if equal)
        assert len(b["occurrence"]) - 1 <= len(P.block_ranges(R, bh))
        # BCS weights are the canonical column packing's values
        assert np.array_equal(b["weights"], P.pack(w, m, bh, bw, reg, rate)["values"])


# ------------------------------------------ simultaneous row + column pruning ---
def test_rowcol_golden_mask():
    g = GOLD["matrix_4x8"]
    m = P.prune_mask(np.array(g["W"], dtype=np.float64), 2, 4, P.ROWCOL, 2)
    assert m.tolist() == g["rowcol_2x4_rate2"]["mask"]
    assert P.mask_is_valid(m, 2, 4, P.ROWCOL, 2)


@pytest.mark.parametrize("bh,bw,rate", [(4, 8, 2), (0, 16, 3), (5, 0, 4), (8, 8, 8)])
def test_rowcol_reduces_to_column_and_row_blocks(bh, bw, rate):
    """One-row blocks keep their row: column pruning; one-column blocks: row pruning."""
    rng = np.random.default_rng(bh * 7 + bw + rate)
    w = rng.standard_normal((24, 40))
    assert np.array_equal(P.prune_mask(w, 1, bw, P.ROWCOL, rate), P.prune_mask(w, 1, bw, P.COL, rate))
    assert np.array_equal(P.prune_mask(w, bh, 1, P.ROWCOL, rate), P.prune_mask(w, bh, 1, P.ROW, rate))
    m = P.prune_mask(w, bh, bw, P.ROWCOL, rate)
    assert P.mask_is_valid(m, bh, bw, P.ROWCOL, rate)
    # the kept set is the product of the row choice and the column choice
    assert np.array_equal(m, P.prune_mask(w, bh, bw, P.ROW, rate) & P.prune_mask(w, bh, bw, P.COL, rate))


def test_rowcol_pack_roundtrip_and_invalid_mask():
    rng = np.random.default_rng(21)
    R, C, bh, bw = 37, 53, 8, 16
    wb = f32_to_bf16_bits(rng.standard_normal((R, C)).astype(np.float32))
    m = P.prune_mask(P.as_f64(wb, "bf16"), bh, bw, P.ROWCOL, 3)
    pk = P.pack(wb, m, bh, bw, P.ROWCOL, 3)
    back = P.unpack(pk, R, C, bh, bw, P.ROWCOL, wb)
    assert np.array_equal(back, np.where(m == 1, wb, 0).astype(wb.dtype))
    bad = m.copy()
    r, c = np.argwhere(m == 1)[0]
    bad[r, c] = 0                               # no longer a product of a row and a column set
    assert not P.mask_is_valid(bad, bh, bw, P.ROWCOL, 3)


# ---------------------------------------------------- pattern-based (3x3) ---
# Sec. 2.1 / Sec. 5.2.3: 4 weights per kernel in one of a library of patterns, and
# connectivity pruning of whole kernels beyond 9/4.

@pytest.mark.parametrize("integer", [False, True])
def test_pattern_with_every_pattern_allowed_keeps_each_kernels_best_four(integer):
    rng = np.random.default_rng(31)
    w = (rng.integers(-4, 5, size=(6, 5, 9)).astype(np.float64) if integer    # exact sums, many ties
         else rng.standard_normal((6, 5, 9)))
    m = P.prune_mask(w.reshape(6, -1), 126, 0, P.PATTERN, 2, khw=9).reshape(30, 9)
    for k, kern in enumerate(w.reshape(30, 9)):
        s = kern ** 2
        best = max(itertools.combinations(range(9), 4), key=lambda t: (sum(s[i] for i in t), [-i for i in t]))
        got = tuple(np.nonzero(m[k])[0])
        if integer:   # ties: any maximising set of the library may be taken
            assert len(got) == 4 and sum(s[i] for i in got) == sum(s[i] for i in best)
        else:
            assert got == best


def test_pattern_library_is_the_most_frequent_sets_and_kernels_take_their_best_pattern():
    A, Bs, Cs = (0, 1, 2, 4), (4, 5, 7, 8), (1, 3, 4, 6)
    kern = []
    for n, pat in ((10, A), (6, Bs), (3, Cs)):
        for i in range(n):
            k = np.full(9, 0.1 + 0.01 * i)
            k[list(pat)] = 2.0 + 0.1 * i
            kern.append(k)
    w = np.array(kern)                                                   # 19 kernels: 19 filters x 1 channel
    m = P.prune_mask(w, 2, 0, P.PATTERN, 2, khw=9)
    codes = {tuple(np.nonzero(r)[0]) for r in m}
    assert codes <= {A, Bs}                                              # library = the two most frequent
    for r, k in zip(m, kern):                                            # each kernel: its best library pattern
        best = max((A, Bs), key=lambda t: sum(k[i] ** 2 for i in t))
        assert tuple(np.nonzero(r)[0]) == best


@pytest.mark.parametrize("rate", [2, 3, 4, 8, 16])
def test_pattern_connectivity_keeps_the_strongest_kernels(rate):
    rng = np.random.default_rng(rate)
    R, cin = 12, 10
    w = rng.standard_normal((R, cin * 9))
    m = P.prune_mask(w, 8, 0, P.PATTERN, rate, khw=9)
    assert P.mask_is_valid(m, 8, 0, P.PATTERN, rate, khw=9)
    per = m.reshape(-1, 9).sum(axis=1)
    n_keep = P.pattern_kept_kernels(R * cin, rate)
    assert (per == 4).sum() == n_keep and set(per.tolist()) <= {0, 4}
    assert n_keep == min(R * cin, math.ceil(R * cin * 9 / (4 * rate)))
    kept_norm = ((w.reshape(-1, 9) ** 2) * m.reshape(-1, 9)).sum(axis=1)
    # every dropped kernel's best library pattern is no stronger than any kept kernel's
    lib = {tuple(np.nonzero(r)[0]) for r in m.reshape(-1, 9) if r.sum()}
    best = np.array([max(sum(k[i] ** 2 for i in t) for t in lib) for k in w.reshape(-1, 9)])
    if n_keep < R * cin:
        assert best[per == 0].max() <= kept_norm[per == 4].min() + 1e-12
