"""Oracle: block-structured pruning masks and canonical packing (numpy, fp64).

TEST INFRASTRUCTURE ONLY - the product path never imports this module.

Paper passages followed:
* Sec. 4.1.1 (block-based pruning): the weight matrix is split into equal
  blocks and rows / columns are pruned independently inside each block.
* Sec. 4.2: the GEMM form of layer i, W_i in R^{P x Q (x Kh x Kw)}, split into
  J blocks; Eq. 2 uses the rows of each block as groups, Eq. 3 the columns,
  each measured by its squared Frobenius norm.
* Sec. 5.1: one-shot pruning by weight magnitude.
* Sec. 4.4: a 1x1 block is unstructured pruning, the whole matrix as one block
  is structured (filter / channel) pruning.
* Sec. 6 (tables): the compression rate is the parameter reduction factor.
* Sec. 4.1.2 and Eq. 4 (block-punched pruning for CONV layers): the weight
  tensor is cut into blocks of filters x input channels; inside a block the
  group of kernel location (m, n) is the weight at (m, n) of every kernel of
  the block, measured by its squared Frobenius norm, and a pruned location is
  removed from all kernels of the block.

Readings where the paper is silent (each listed in the design notes):
* kept groups per block = ceil(extent / rate) with an integer rate;
* ties in the group score go to the lower index;
* scores are accumulated in fp64 in ascending order (the squares of fp32 /
  bf16 values are exact in fp64, so the order is the only rounding choice);
* blocks are anchored at (0, 0); a ragged last block keeps
  ceil(its own extent / rate);
* a block size of 0 means the whole extent;
* block-punched: blocks of bh filters x bw input channels; kept locations per
  block = ceil(kh*kw / rate); the score of a location sums over the block's
  (filter, channel) pairs in ascending (filter, channel) order;
* simultaneous row and column pruning (Sec. 4.2: Eqs. 2 and 3 solved together):
  every block keeps ceil(bh / rate) rows and ceil(bw / rate) columns, each set
  chosen by its own group norm on the block's weights; the block keeps their
  product (so the kept fraction is about 1 / rate^2);
* pattern-based pruning of 3x3 kernels (Sec. 2.1 and Sec. 5.2.3, the comparison
  point of block-punched pruning): every kept kernel keeps 4 weights in one of
  a library of P patterns (the P most frequent top-4 location sets of the
  layer's kernels, ties to the smaller location bit mask); a kernel takes the
  library pattern with the largest kept squared norm (ties to the earlier
  pattern); connectivity pruning keeps the ceil(n_kernels * 9 / (4 * rate))
  kernels with the largest kept norm (ties to the lower kernel index o*Cin+c),
  all of them when rate <= 9/4;
* per-block kept counts (Sec. 4.1.1: the same or a different number per block;
  Sec. 4.2: the reweighted method sets a rate per block) are given by the
  caller as an array over the blocks in row-major order, replacing
  ceil(extent / rate).

Pins: tests/test_oracle_prune.py (brute-force subset enumeration, invariants,
ties, ragged edges, scale invariance, hand-derived golden masks).
"""

from __future__ import annotations

import numpy as np

ROW, COL, UNSTRUCTURED, DENSE, PUNCHED, ROWCOL, PATTERN = 0, 1, 2, 3, 4, 5, 6


def kept_count(extent: int, rate: int) -> int:
    """ceil(extent / rate) in integers."""
    return (int(extent) + int(rate) - 1) // int(rate)


def block_ranges(extent: int, b: int):
    """Half-open ranges of the blocks along one dimension (b = 0: whole)."""
    if b == 0 or b >= extent:
        return [(0, int(extent))]
    return [(s, min(s + b, extent)) for s in range(0, extent, b)]


def as_f64(w_stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of stored fp32 values or bf16 bit patterns."""
    if dtype == "f32":
        return np.asarray(w_stored, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        u = np.asarray(w_stored, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def group_scores(block: np.ndarray, regularity: int) -> np.ndarray:
    """Squared Frobenius norm of every column (COL) or row (ROW) of one block.

    Eqs. 2-3 group a block's weights by row / column; the score is the sum of
    squares, accumulated sequentially in ascending index order in fp64
    (np.cumsum is a left-to-right running sum; its last entry is the total).
    """
    sq = block * block
    if regularity == COL:
        return np.cumsum(sq, axis=0)[-1]
    if regularity == ROW:
        return np.cumsum(sq, axis=1)[:, -1]
    raise ValueError(regularity)


def top_k(scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest scores, ties to the lower index (stable)."""
    order = np.argsort(-scores, kind="stable")
    return np.sort(order[:k])


def _count(counts, i: int, j: int, default: int) -> int:
    """Kept groups of block (i, j): the caller's count, else the uniform rule."""
    if counts is None:
        return default
    k = int(np.asarray(counts)[i, j])
    if k < 0:
        raise ValueError("kept counts must be >= 0")
    return k


def punched_mask(wg: np.ndarray, khw: int, bh: int, bw: int, rate: int, counts=None) -> np.ndarray:
    """Block-punched mask (Sec. 4.1.2, Eq. 4) of a GEMM-form fp64 conv weight
    (R filters x Cin*khw columns, column = c*khw + location).

    Blocks are bh filters x bw input channels (0: all).  The score of location
    l in a block is the sum of w[o, c*khw + l]^2 over the block's kernels,
    taken in ascending (o, c) order; the ceil(khw / rate) best locations are
    kept in every kernel of the block (ties to the lower location).
    """
    wg = np.asarray(wg, dtype=np.float64)
    R, C = wg.shape
    if khw < 1 or C % khw:
        raise ValueError("columns must be Cin * khw")
    cin = C // khw
    w3 = wg.reshape(R, cin, khw)
    mask = np.zeros((R, cin, khw), dtype=np.uint8)
    for i, (r0, r1) in enumerate(block_ranges(R, bh)):
        for j, (c0, c1) in enumerate(block_ranges(cin, bw)):
            k = _count(counts, i, j, kept_count(khw, rate))
            if k > khw:
                raise ValueError("kept count exceeds the block's groups")
            groups = w3[r0:r1, c0:c1, :].reshape(-1, khw)    # rows: kernels (o, c) in order
            s = np.cumsum(groups * groups, axis=0)[-1]
            mask[r0:r1, c0:c1, top_k(s, k)] = 1
    return mask.reshape(R, C)


def pattern_kept_kernels(n_kernels: int, rate: int, khw: int = 9) -> int:
    """Kernels kept by connectivity pruning: ceil(n * khw / (4 * rate)), at most n."""
    return min(n_kernels, (n_kernels * khw + 4 * rate - 1) // (4 * rate))


def pattern_mask(wg: np.ndarray, khw: int, n_patterns: int, rate: int) -> np.ndarray:
    """Pattern-based mask of a GEMM-form fp64 conv weight (R x Cin*khw), 4 kept
    weights per kept kernel (Sec. 2.1), library and connectivity as in the header."""
    wg = np.asarray(wg, dtype=np.float64)
    R, C = wg.shape
    cin = C // khw
    sq = (wg * wg).reshape(R * cin, khw)                  # kernel k = o * Cin + c
    own = [int(sum(1 << int(l) for l in top_k(sq[k], 4))) for k in range(R * cin)]
    counts = {}
    for code in own:
        counts[code] = counts.get(code, 0) + 1
    library = sorted(counts, key=lambda code: (-counts[code], code))[:n_patterns]
    locs = [[l for l in range(khw) if (code >> l) & 1] for code in library]
    best_pat = np.zeros(R * cin, dtype=np.int64)
    best = np.zeros(R * cin)
    for k in range(R * cin):
        vals = [sum(sq[k, l] for l in ls) for ls in locs]   # ascending location order
        best_pat[k] = int(np.argmax(vals))                 # first maximum: the earlier pattern
        best[k] = vals[best_pat[k]]
    keep = top_k(best, pattern_kept_kernels(R * cin, rate, khw))
    mask = np.zeros((R * cin, khw), dtype=np.uint8)
    for k in keep:
        mask[k, locs[best_pat[k]]] = 1
    return mask.reshape(R, C)


def prune_mask(wg: np.ndarray, bh: int, bw: int, regularity: int, rate: int, khw: int = 1,
               counts=None) -> np.ndarray:
    """Mask (uint8, R x C) of the kept weights of a GEMM-form fp64 matrix
    (khw: kernel locations per input channel, used by block-punched pruning;
    counts: optional kept groups per block, an (n_block_rows, n_block_cols)
    array, for ROW, COL and PUNCHED)."""
    wg = np.asarray(wg, dtype=np.float64)
    R, C = wg.shape
    mask = np.zeros((R, C), dtype=np.uint8)
    if regularity == PUNCHED:
        return punched_mask(wg, max(int(khw), 1), bh, bw, rate, counts)
    if regularity == PATTERN:   # bh: library size (0: 8)
        return pattern_mask(wg, int(khw), int(bh) or 8, rate)
    if regularity == ROWCOL:
        if counts is not None:
            raise ValueError("per-block counts are not defined for simultaneous row and column pruning")
        for r0, r1 in block_ranges(R, bh):
            for c0, c1 in block_ranges(C, bw):
                blk = wg[r0:r1, c0:c1]
                rows = top_k(group_scores(blk, ROW), kept_count(r1 - r0, rate))
                cols = top_k(group_scores(blk, COL), kept_count(c1 - c0, rate))
                mask[np.ix_(r0 + rows, c0 + cols)] = 1
        return mask
    if regularity == DENSE:
        mask[:] = 1
        return mask
    if regularity == UNSTRUCTURED:
        return unstructured_mask(wg, rate)
    for i, (r0, r1) in enumerate(block_ranges(R, bh)):
        for j, (c0, c1) in enumerate(block_ranges(C, bw)):
            blk = wg[r0:r1, c0:c1]
            s = group_scores(blk, regularity)
            ng = (c1 - c0) if regularity == COL else (r1 - r0)
            k = _count(counts, i, j, kept_count(ng, rate))
            if k > ng:
                raise ValueError("kept count exceeds the block's groups")
            keep = top_k(s, k)
            if regularity == COL:
                mask[r0:r1, c0 + keep] = 1
            else:
                mask[r0 + keep, c0:c1] = 1
    return mask


def unstructured_mask(wg: np.ndarray, rate: int) -> np.ndarray:
    """Magnitude pruning over the whole layer: keep ceil(R*C/rate) entries
    with the largest |w|, ties to the smaller flat index p*C + q."""
    R, C = wg.shape
    a = np.abs(np.asarray(wg, dtype=np.float64)).reshape(-1)
    k = kept_count(R * C, rate)
    keep = np.argsort(-a, kind="stable")[:k]
    m = np.zeros(R * C, dtype=np.uint8)
    m[keep] = 1
    return m.reshape(R, C)


def mask_is_valid(mask: np.ndarray, bh: int, bw: int, regularity: int, rate: int, khw: int = 1,
                  counts=None) -> bool:
    """True iff the mask has the block structure of the scheme: every block
    keeps whole columns (COL) or whole rows (ROW), exactly ceil(extent/rate);
    block-punched: the same ceil(khw/rate) locations in every kernel of a block."""
    mask = np.asarray(mask, dtype=np.uint8)
    R, C = mask.shape
    if not np.all((mask == 0) | (mask == 1)):
        return False
    if regularity == PUNCHED:
        khw = max(int(khw), 1)
        if C % khw:
            return False
        m3 = mask.reshape(R, C // khw, khw)
        for i, (r0, r1) in enumerate(block_ranges(R, bh)):
            for j, (c0, c1) in enumerate(block_ranges(C // khw, bw)):
                blk = m3[r0:r1, c0:c1, :]
                if not np.all(blk == blk[0:1, 0:1, :]):
                    return False
                if int(blk[0, 0].sum()) != _count(counts, i, j, kept_count(khw, rate)):
                    return False
        return True
    if regularity == DENSE:
        return bool(np.all(mask == 1))
    if regularity == UNSTRUCTURED:
        return int(mask.sum()) == kept_count(R * C, rate)
    if regularity == PATTERN:
        per = mask.reshape(-1, khw).sum(axis=1)
        codes = {tuple(r) for r in mask.reshape(-1, khw) if r.sum()}
        return bool(np.all((per == 0) | (per == 4)) and (per == 4).sum() == pattern_kept_kernels(len(per), rate, khw)
                    and len(codes) <= (bh or 8))
    if regularity == ROWCOL:
        for r0, r1 in block_ranges(R, bh):
            for c0, c1 in block_ranges(C, bw):
                blk = mask[r0:r1, c0:c1]
                rows, cols = blk.any(axis=1), blk.any(axis=0)
                if not np.array_equal(blk, np.outer(rows, cols).astype(np.uint8)):
                    return False
                if rows.sum() != kept_count(r1 - r0, rate) or cols.sum() != kept_count(c1 - c0, rate):
                    return False
        return True
    for i, (r0, r1) in enumerate(block_ranges(R, bh)):
        for j, (c0, c1) in enumerate(block_ranges(C, bw)):
            blk = mask[r0:r1, c0:c1]
            if regularity == COL:
                if not np.all(blk == blk[0:1, :]):
                    return False
                if int(blk[0].sum()) != _count(counts, i, j, kept_count(c1 - c0, rate)):
                    return False
            else:
                if not np.all(blk == blk[:, 0:1]):
                    return False
                if int(blk[:, 0].sum()) != _count(counts, i, j, kept_count(r1 - r0, rate)):
                    return False
    return True


def pack(w_stored: np.ndarray, mask: np.ndarray, bh: int, bw: int, regularity: int, rate: int) -> dict:
    """Canonical packing of a masked GEMM-form matrix (stored dtype kept as is).

    COL: for block-row i, ``indices[rowptr[i]:rowptr[i+1]]`` are its kept
         columns, block by block left to right, ascending inside a block (so
         ascending overall); ``values[rowptr[i]*bh + p*len + t]`` is
         W[i*bh + p, indices[rowptr[i] + t]].
    PUNCHED: as COL (a block-row keeps whole GEMM columns: the kept locations
         of each of its channel blocks).
    ROWCOL: as COL over the columns any row of the block-row keeps; the values
         of the rows a block removed are zero.
    ROW: for block (i, j) in row-major order, ``indices[rowptr[b]:rowptr[b+1]]``
         are its kept rows ascending; its values are rows of the block,
         ``[t][q_local]``, stored one block after the other.
    DENSE / UNSTRUCTURED: no indices, ``values`` = W * mask, R x C.
    """
    w_stored = np.asarray(w_stored)
    mask = np.asarray(mask, dtype=np.uint8)
    R, C = mask.shape
    if regularity in (DENSE, UNSTRUCTURED, PATTERN):
        vals = np.where(mask == 1, w_stored, np.zeros_like(w_stored))
        return {"indices": np.zeros(0, np.int32), "rowptr": np.zeros(0, np.int32),
                "values": vals.reshape(-1).copy()}
    idx, ptr, vals = [], [0], []
    if regularity in (COL, PUNCHED, ROWCOL):
        for r0, r1 in block_ranges(R, bh):
            kept = np.nonzero(mask[r0:r1].any(axis=0))[0].astype(np.int32)
            idx.append(kept)
            ptr.append(ptr[-1] + len(kept))
            sub = np.where(mask[r0:r1][:, kept] == 1, w_stored[r0:r1][:, kept], np.zeros_like(w_stored[:1, :1]))
            vals.append(sub.reshape(-1))
    else:
        for r0, r1 in block_ranges(R, bh):
            for c0, c1 in block_ranges(C, bw):
                kept = (r0 + np.nonzero(mask[r0:r1, c0])[0]).astype(np.int32)
                idx.append(kept)
                ptr.append(ptr[-1] + len(kept))
                vals.append(w_stored[kept][:, c0:c1].reshape(-1))
    return {"indices": np.concatenate(idx).astype(np.int32),
            "rowptr": np.asarray(ptr, dtype=np.int32),
            "values": np.concatenate(vals)}


def unpack(packed: dict, R: int, C: int, bh: int, bw: int, regularity: int, like: np.ndarray) -> np.ndarray:
    """Inverse of ``pack``: the masked dense matrix in the stored dtype."""
    out = np.zeros((R, C), dtype=np.asarray(like).dtype)
    vals, idx, ptr = packed["values"], packed["indices"], packed["rowptr"]
    if regularity in (DENSE, UNSTRUCTURED, PATTERN):
        return vals.reshape(R, C).copy()
    off = 0
    if regularity in (COL, PUNCHED, ROWCOL):
        for i, (r0, r1) in enumerate(block_ranges(R, bh)):
            kept = idx[ptr[i]:ptr[i + 1]]
            n = (r1 - r0) * len(kept)
            out[r0:r1][:, kept] = vals[off:off + n].reshape(r1 - r0, len(kept))
            off += n
    else:
        b = 0
        for r0, r1 in block_ranges(R, bh):
            for c0, c1 in block_ranges(C, bw):
                kept = idx[ptr[b]:ptr[b + 1]]
                n = len(kept) * (c1 - c0)
                out[kept, c0:c1] = vals[off:off + n].reshape(len(kept), c1 - c0)
                off += n
                b += 1
    return out


def gemm_form(w: np.ndarray) -> np.ndarray:
    """(Cout, Cin, kh, kw) -> (Cout, Cin*kh*kw) with column q = (c*kh + r)*kw + s."""
    w = np.asarray(w)
    return w.reshape(w.shape[0], -1)


def bcs_encode(w_stored: np.ndarray, mask: np.ndarray) -> dict:
    """Blocked Compressed Storage (Sec. 4.3) of a masked matrix, from its definition.

    Like CSR, but the column indices of consecutive rows that keep the same columns
    are stored once:
      weights      the kept weights, row by row, ascending columns (CSR order);
      row_offset   start of each row in ``weights`` (R + 1 entries);
      occurrence   first row of each run of consecutive rows with identical kept
                   columns, then R (runs + 1 entries);
      compact_cols the kept columns of each run, run after run;
      col_stride   start of each run's columns in ``compact_cols``, then its length
                   (runs + 1 entries).
    Kept means kept by the mask (a kept weight may be numerically zero).
    """
    w_stored = np.asarray(w_stored)
    mask = np.asarray(mask, dtype=np.uint8)
    R, C = mask.shape
    cols = [np.nonzero(mask[r])[0] for r in range(R)]
    weights = [w_stored[r, cols[r]] for r in range(R)]
    row_offset = [0]
    for r in range(R):
        row_offset.append(row_offset[-1] + len(cols[r]))
    occurrence, compact, stride = [], [], [0]
    for r in range(R):
        if r == 0 or not np.array_equal(cols[r], cols[r - 1]):
            occurrence.append(r)
            compact.extend(cols[r].tolist())
            stride.append(len(compact))
    occurrence.append(R)
    return {"weights": np.concatenate(weights) if R else np.zeros(0, w_stored.dtype),
            "row_offset": np.asarray(row_offset, np.int32), "occurrence": np.asarray(occurrence, np.int32),
            "compact_cols": np.asarray(compact, np.int32), "col_stride": np.asarray(stride, np.int32)}


def bcs_decode(bcs: dict, R: int, C: int, like: np.ndarray) -> np.ndarray:
    """Dense matrix (stored dtype) of a BCS encoding: row r of run g takes the run's
    columns and its weights from row_offset[r]."""
    out = np.zeros((R, C), dtype=np.asarray(like).dtype)
    occ, st, cc = bcs["occurrence"], bcs["col_stride"], bcs["compact_cols"]
    for g in range(len(occ) - 1):
        cols = cc[st[g]:st[g + 1]]
        for r in range(occ[g], occ[g + 1]):
            o = bcs["row_offset"][r]
            out[r, cols] = bcs["weights"][o:o + len(cols)]
    return out
