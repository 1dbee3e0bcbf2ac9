// Packing of pruned weights on the device.
//
// Canonical packing (checked bit-exact against the oracle): per block-row kept
// column lists (column pruning) or per block kept row lists (row pruning) plus the
// kept values - the same information as the paper's compact storage of Sec. 4.3
// (kept weights and the column indices shared by the rows of a block), in this
// library's own layout.  The private dev_tiles layout for the forward kernel adds
// pre-decoded LDS gather offsets per kept column, MFMA-ordered weight tiles (8
// consecutive kept columns per lane, zero padded to steps of 32), and the channel
// windows ("chunks") the forward stages through LDS.
#include <hip/hip_runtime.h>

#include <vector>

#include "bsp_kernels.h"

namespace bsp {

namespace {

constexpr int kFlagOffset = 32;   // TileHeader::reserved[0]: error flag
constexpr int kCountOffset = 36;  // TileHeader::reserved[1]: kept counter

__device__ __forceinline__ int block_excl_scan_256(int v, int *wave_tot, int *total) {
    // exclusive prefix of v (0/1) over a 256-thread workgroup, using ballots
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const unsigned long long b = __ballot(v != 0);
    const int pre = __builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32),
                                              __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0));
    if (lane == 0) wave_tot[wv] = __popcll(b);
    __syncthreads();
    int off = 0, tot = 0;
    for (int i = 0; i < 4; ++i) {
        if (i < wv) off += wave_tot[i];
        tot += wave_tot[i];
    }
    *total = tot;
    __syncthreads();
    return off + pre;
}

__global__ void k_validate_blocks(const uint8_t *__restrict__ mask, int R, int C, int bh, int bw,
                                  int nbc, int col, int rate, const int32_t *__restrict__ counts, int *flag) {
    __shared__ int cnt;
    if (threadIdx.x == 0) cnt = 0;
    __syncthreads();
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw, c1 = min(C, c0 + bw);
    const int ng = col ? c1 - c0 : r1 - r0;
    int bad = 0, local = 0;
    for (int g = threadIdx.x; g < ng; g += blockDim.x) {
        if (col) {
            const uint8_t v0 = mask[(size_t)r0 * C + c0 + g];
            bad |= v0 > 1;
            for (int p = r0 + 1; p < r1; ++p) bad |= mask[(size_t)p * C + c0 + g] != v0;
            local += v0 == 1;
        } else {
            const uint8_t *mr = mask + (size_t)(r0 + g) * C;
            const uint8_t v0 = mr[c0];
            bad |= v0 > 1;
            for (int q = c0 + 1; q < c1; ++q) bad |= mr[q] != v0;
            local += v0 == 1;
        }
    }
    if (local) atomicAdd(&cnt, local);
    if (bad) atomicOr(flag, 1);
    __syncthreads();
    if (threadIdx.x == 0 && cnt != (counts ? counts[b] : (ng + rate - 1) / rate)) atomicOr(flag, 1);
}

// Block-punched structure (Sec. 4.1.2): in block (filters [r0, r1) x channels
// [c0, c1)) every kernel keeps the locations of the block's first kernel, and that
// kernel keeps exactly k of its khw locations.
__global__ void k_validate_punched(const uint8_t *__restrict__ mask, int R, int C, int khw, int bh,
                                   int bw, int nbc, int k, const int32_t *__restrict__ counts, int *flag) {
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int cin = C / khw;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw, c1 = min(cin, c0 + bw);
    const int nk = (r1 - r0) * (c1 - c0);   // kernels of the block
    const uint8_t *ref = mask + (size_t)r0 * C + (size_t)c0 * khw;
    int bad = 0;
    for (int e = threadIdx.x; e < nk * khw; e += blockDim.x) {
        const int kr = e / khw, l = e - kr * khw;
        const int o = r0 + kr / (c1 - c0), c = c0 + kr % (c1 - c0);
        const uint8_t v = mask[(size_t)o * C + (size_t)c * khw + l];
        bad |= (v > 1) | (v != ref[l]);
    }
    if (threadIdx.x == 0) {
        int cnt = 0;
        for (int l = 0; l < khw; ++l) cnt += ref[l] == 1;
        bad |= cnt != (counts ? counts[b] : k);
    }
    if (bad) atomicOr(flag, 1);
}

// Row + column structure: inside a block the mask is the product of its kept rows
// (rows with any kept entry) and kept columns, with ceil(extent / rate) of each.
__global__ void k_validate_rowcol(const uint8_t *__restrict__ mask, int R, int C, int bh, int bw, int nbc, int rate,
                                  int *flag) {
    extern __shared__ uint8_t kf[];   // kept rows [bh], kept columns [bw]
    __shared__ int nrk, nck;
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw, c1 = min(C, c0 + bw);
    const int nr = r1 - r0, nc = c1 - c0;
    if (threadIdx.x == 0) nrk = nck = 0;
    __syncthreads();
    int bad = 0, lr = 0, lc = 0;
    for (int g = threadIdx.x; g < nr + nc; g += blockDim.x) {
        uint8_t any = 0;
        if (g < nr)
            for (int q = c0; q < c1; ++q) any |= mask[(size_t)(r0 + g) * C + q];
        else
            for (int p = r0; p < r1; ++p) any |= mask[(size_t)p * C + c0 + (g - nr)];
        bad |= any > 1;
        kf[g < nr ? g : bh + (g - nr)] = any;
        if (g < nr) lr += any == 1;
        else lc += any == 1;
    }
    if (lr) atomicAdd(&nrk, lr);
    if (lc) atomicAdd(&nck, lc);
    __syncthreads();
    for (int e = threadIdx.x; e < nr * nc; e += blockDim.x) {
        const int p = e / nc, q = e - p * nc;
        bad |= mask[(size_t)(r0 + p) * C + c0 + q] != (kf[p] & kf[bh + q]);
    }
    if (threadIdx.x == 0) bad |= nrk != (nr + rate - 1) / rate || nck != (nc + rate - 1) / rate;
    if (bad) atomicOr(flag, 1);
}

__global__ void k_validate_all(const uint8_t *__restrict__ mask, size_t n, int need_ones,
                               int *flag, unsigned int *count) {
    int bad = 0;
    unsigned int c = 0;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        const uint8_t v = mask[i];
        bad |= v > 1;
        if (need_ones) bad |= v != 1;
        c += v == 1;
    }
    if (bad) atomicOr(flag, 1);
    if (c) atomicAdd(count, c);
}

// Pattern-based masks: every 3x3 kernel keeps 0 or 4 weights.
__global__ void k_validate_kernels4(const uint8_t *__restrict__ mask, int n_kernels, int *flag) {
    for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n_kernels; k += gridDim.x * blockDim.x) {
        int c = 0;
        for (int l = 0; l < 9; ++l) c += mask[(size_t)k * 9 + l];
        if (c != 0 && c != 4) atomicOr(flag, 1);
    }
}

__global__ void k_check_count(const unsigned int *count, unsigned int k, int *flag) {
    if (*count != k) atomicOr(flag, 1);
}

// Kept-column list of block-row i, written at rowptr[i] (offsets computed on the host
// from the scheme); the block-row's first row holds its kept columns.
__global__ void k_col_lists(const uint8_t *__restrict__ mask, int R, int C, int bh, int any_row,
                            const int32_t *__restrict__ rowptr, int32_t *__restrict__ indices, int *flag) {
    __shared__ int wave_tot[4];
    const int i = blockIdx.x;
    const uint8_t *mr = mask + (size_t)i * bh * C;
    const int rows = any_row ? min(R - i * bh, bh) : 1;   // row + column blocks: a column is kept by any row
    const int off = rowptr[i], L = rowptr[i + 1] - off;
    int base = 0;
    for (int q0 = 0; q0 < C; q0 += 256) {
        const int q = q0 + threadIdx.x;
        int v = 0;
        if (q < C)
            for (int r = 0; r < rows && !v; ++r) v = mr[(size_t)r * C + q];
        int tot;
        const int pos = base + block_excl_scan_256(v, wave_tot, &tot);
        if (v) {
            if (pos < L) indices[off + pos] = q;
            else atomicOr(flag, 1);
        }
        base += tot;
    }
    if (threadIdx.x == 0 && base != L) atomicOr(flag, 1);
}

// Values of block-row i: [row][t] at rowptr[i] * bh (earlier block-rows are full).
template <typename E>
__global__ void k_col_values(const E *__restrict__ w, const uint8_t *__restrict__ mask,
                             const int32_t *__restrict__ indices, const int32_t *__restrict__ rowptr,
                             E *__restrict__ values, int R, int C, int bh) {
    const int i = blockIdx.x;
    const int off = rowptr[i], L = rowptr[i + 1] - off;
    const int r0 = i * bh, rows = min(R, r0 + bh) - r0;
    const size_t vbase = (size_t)off * bh;
    for (int e = threadIdx.x; e < rows * L; e += blockDim.x) {
        const int p = e / L, t = e - p * L;
        const size_t wi = (size_t)(r0 + p) * C + indices[off + t];
        values[vbase + e] = mask[wi] ? w[wi] : (E)0;   // zero in the rows a row + column block removed
    }
}

// Value offset of row block b: its values follow those of every earlier block, kept
// rows x block width (only the last block column may be narrower).
__device__ __forceinline__ size_t row_voff(const int32_t *__restrict__ rowptr, int b, int nbc, int bw,
                                           int last_w) {
    size_t v = (size_t)bw * rowptr[b];
    if (last_w != bw) {
        const int bi = b / nbc;
        for (int i = 0; i < bi; ++i)
            v -= (size_t)(bw - last_w) * (rowptr[i * nbc + nbc] - rowptr[i * nbc + nbc - 1]);
    }
    return v;
}

// Kept-row list of block b, written at rowptr[b]; the block's first column holds its
// kept rows.
__global__ void k_row_lists(const uint8_t *__restrict__ mask, int R, int C, int bh, int bw, int nbc,
                            const int32_t *__restrict__ rowptr, int32_t *__restrict__ indices, int *flag) {
    __shared__ int wave_tot[4];
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw;
    const int off = rowptr[b], ki = rowptr[b + 1] - off;
    int base = 0;
    for (int p0 = r0; p0 < r1; p0 += 256) {
        const int p = p0 + threadIdx.x;
        const int v = p < r1 ? mask[(size_t)p * C + c0] : 0;
        int tot;
        const int t = base + block_excl_scan_256(v, wave_tot, &tot);
        if (v) {
            if (t < ki) indices[off + t] = p;
            else atomicOr(flag, 1);
        }
        base += tot;
    }
    if (threadIdx.x == 0 && base != ki) atomicOr(flag, 1);
}

template <typename E>
__global__ void k_row_values(const E *__restrict__ w, const int32_t *__restrict__ indices,
                             const int32_t *__restrict__ rowptr, E *__restrict__ values, int C, int bw,
                             int nbc) {
    const int b = blockIdx.x;
    const int bj = b % nbc;
    const int c0 = bj * bw, c1 = min(C, c0 + bw);
    const int wj = c1 - c0, last_w = C - (nbc - 1) * bw;
    const int off = rowptr[b], ki = rowptr[b + 1] - off;
    const size_t voff = row_voff(rowptr, b, nbc, bw, last_w);
    for (int e = threadIdx.x; e < ki * wj; e += blockDim.x) {
        const int t = e / wj, q = e - t * wj;
        values[voff + e] = w[(size_t)indices[off + t] * C + c0 + q];
    }
}

template <typename E>
__global__ void k_masked_copy(const E *__restrict__ w, const uint8_t *__restrict__ mask,
                              E *__restrict__ out, size_t n) {
    for (size_t e = blockIdx.x * (size_t)blockDim.x + threadIdx.x; e < n;
         e += (size_t)gridDim.x * blockDim.x)
        out[e] = mask[e] ? w[e] : (E)0;
}

struct DescArgs {
    int shared, n_groups, L, LP, C, KH, KW, CH_STRIDE, RS, VS, V;
    CountTables ct;   // per-block counts (ct.P null: uniform lists)
    int nbc, blk_cols;
};

// Kept list of group g: offset and length (shared identity list: 0, L).
__device__ __forceinline__ int2 group_list(const int32_t *__restrict__ rowptr, int shared, int L, int g) {
    return shared ? int2{0, L} : int2{rowptr[g], rowptr[g + 1] - rowptr[g]};
}

// Slot t of group g's forward list when blocks have their own kept counts: block
// column j owns slots [P[j], P[j+1]) in every group (as many as its largest count),
// and group g's n kept columns of that block are spread evenly over them (kept column
// e at slot floor(e * W / n)); the other slots repeat the kept column before them with
// zero weight, so a step covers the same blocks in every group.  Returns the column
// and whether the slot carries a kept weight.
__device__ __forceinline__ int2 slot_col(const CountTables &ct, const int32_t *__restrict__ indices,
                                         const int32_t *__restrict__ rowptr, int nbc, int blk_cols, int g, int t) {
    const int j = ct.slot_block[t];
    const int W = ct.P[j + 1] - ct.P[j], l = t - ct.P[j];
    const int n = ct.ncols[g * nbc + j];
    if (n == 0 || W == 0) return int2{j * blk_cols, 0};
    const int e = (int)(((int64_t)(l + 1) * n - 1) / W);
    const int real = (int)((int64_t)e * W / n) == l;
    return int2{indices[rowptr[g] + ct.start[g * nbc + j] + e], real};
}

__global__ void k_desc(DescArgs a, const int32_t *__restrict__ indices, const int32_t *__restrict__ rowptr,
                       int32_t *__restrict__ desc) {
    const int n = a.n_groups * a.LP;
    const int khw = a.KH * a.KW;
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) {
        const int g = e / a.LP, t = e - g * a.LP;
        int q;
        if (a.ct.P) {
            q = slot_col(a.ct, indices, rowptr, a.nbc, a.blk_cols, g, min(t, a.L - 1)).x;
        } else {
            const int2 gl = group_list(rowptr, a.shared, a.L, g);
            // padding repeats the last kept column (column 0 for an empty list); its weights are zero
            const int tt = t < gl.y ? t : gl.y - 1;
            q = gl.y == 0 ? 0 : (a.shared ? tt : indices[gl.x + tt]);
        }
        const int c = q / khw, rs = q - c * khw;
        const int r = rs / a.KW, s = rs - r * a.KW;
        desc[e] = c * a.CH_STRIDE + (s % a.V) * a.VS + r * a.RS + (s / a.V) * a.V;
    }
}

struct ATileArgs {
    int shared, n_groups, mt_per_group, n_mt_pad, group_rows, S, L, R, C;
    int rowmap;   // 1: computed row i is weight row indices[i] (kept filters, ascending)
    CountTables ct;
    int nbc, blk_cols;
};

template <typename E>
__global__ void k_atiles(ATileArgs a, const E *__restrict__ w, const uint8_t *__restrict__ mask,
                         const int32_t *__restrict__ indices, const int32_t *__restrict__ rowptr,
                         E *__restrict__ A) {
    const int64_t per_mt = (int64_t)a.S * 512;
    const int64_t n = (int64_t)a.n_mt_pad * per_mt;   // m-tiles past the last group are zero
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int j = (int)(e & 7), lane = (int)((e >> 3) & 63);
        const int64_t rest = e >> 9;
        const int s = (int)(rest % a.S);
        const int64_t gm = rest / a.S;
        const int mt = (int)(gm % a.mt_per_group);
        const int g = (int)(gm / a.mt_per_group);
        const int rig = mt * 16 + (lane & 15);
        const int row = g * a.group_rows + rig;
        const int t = s * 32 + 8 * (lane >> 4) + j;
        E v = (E)0;
        int2 gl = int2{0, 0};   // (column, carries a weight)
        if (g < a.n_groups && t < a.L) {
            if (a.ct.P) {
                gl = slot_col(a.ct, indices, rowptr, a.nbc, a.blk_cols, g, t);
            } else {
                const int2 li = group_list(rowptr, a.shared, a.L, g);
                if (t < li.y) gl = int2{a.shared ? t : indices[li.x + t], 1};
            }
        }
        if (gl.y && rig < a.group_rows && row < a.R) {
            const int q = gl.x;
            const int src = a.rowmap ? indices[row] : row;
            const size_t wi = (size_t)src * a.C + q;
            if (mask[wi]) v = w[wi];
        }
        A[e] = v;
    }
}

// Row map of whole-width row pruning.  The kept filters are `kept` ascending
// (the canonical row lists of the block-rows, in order); output row o is kept iff it
// is found there, and then it is computed row pos = (kept rows below o).  Otherwise it
// is pruned row o - pos.  One thread per output row, no atomics.
__global__ void k_rowmap(const int32_t *__restrict__ kept, int RK, int R, int32_t *__restrict__ rowmap,
                         int32_t *__restrict__ pruned) {
    for (int o = blockIdx.x * blockDim.x + threadIdx.x; o < R; o += gridDim.x * blockDim.x) {
        int lo = 0, hi = RK;   // first position with kept[pos] >= o
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (kept[mid] < o) lo = mid + 1;
            else hi = mid;
        }
        if (lo < RK && kept[lo] == o) rowmap[lo] = o;
        else pruned[o - lo] = o;
    }
}

__global__ void k_step_spans(const int32_t *__restrict__ desc, int n_groups, int LP, int S,
                             int CH_STRIDE, int4 *table) {
    for (int s = blockIdx.x * blockDim.x + threadIdx.x; s < S; s += gridDim.x * blockDim.x) {
        int lo = 0x7fffffff, hi = -1;
        for (int g = 0; g < n_groups; ++g) {
            const int a = desc[(size_t)g * LP + 32 * s] / CH_STRIDE;
            const int b = desc[(size_t)g * LP + 32 * s + 31] / CH_STRIDE;
            lo = min(lo, a);
            hi = max(hi, b);
        }
        table[s] = make_int4(lo, hi, 0, 0);
    }
}

__global__ void k_build_chunks(int4 *table, int S, int CC, int smax, int *n_chunks, int *flag) {
    extern __shared__ int spans[];  // 2*S
    for (int s = threadIdx.x; s < S; s += blockDim.x) {
        spans[2 * s] = table[s].x;
        spans[2 * s + 1] = table[s].y;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    int nc = 0, s = 0;
    while (s < S) {
        const int lo = spans[2 * s];
        int hi = spans[2 * s + 1];
        if (hi - lo + 1 > CC) {
            atomicOr(flag, 2);
            break;
        }
        int e = s + 1;
        while (e < S && (smax == 0 || e - s < smax)) {
            const int h2 = max(hi, spans[2 * e + 1]);
            if (spans[2 * e] < lo || h2 - lo + 1 > CC) break;
            hi = h2;
            ++e;
        }
        table[nc++] = make_int4(s, e, lo, hi - lo + 1);
        s = e;
    }
    *n_chunks = nc;
}

// 16-bit chunk-relative gather offsets: each step belongs to one chunk (a range of
// steps); the offset of a kept column relative to the chunk's first channel is
// below CC * CH_STRIDE, which fits 16 bits by the LDS budget.
__global__ void k_desc16(const int32_t *__restrict__ desc, const int4 *__restrict__ table,
                         const int *n_chunks_p, int n_groups, int LP, int CH_STRIDE,
                         uint16_t *__restrict__ desc16, int *flag) {
    const int n = n_groups * LP;
    const int nch = *n_chunks_p;
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) {
        const int s = (e % LP) / 32;
        int lo = -1;
        for (int c = 0; c < nch; ++c) {
            const int4 t = table[c];
            if (s >= t.x && s < t.y) { lo = t.z; break; }
        }
        const int off = desc[e] - lo * CH_STRIDE;
        if (lo < 0 || off < 0 || off > 0xffff) {
            atomicOr(flag, 2);
            desc16[e] = 0;
        } else {
            desc16[e] = (uint16_t)off;
        }
    }
}

// 16-bit channels of the pointwise kernel's gathered lists (the lists' channel
// numbers themselves; no chunks).
__global__ void k_desc16_abs(const int32_t *__restrict__ desc, int n, uint16_t *__restrict__ desc16, int *flag) {
    for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < n; e += gridDim.x * blockDim.x) {
        const int v = desc[e];
        if (v < 0 || v > 0xffff) {
            atomicOr(flag, 2);
            desc16[e] = 0;
        } else {
            desc16[e] = (uint16_t)v;
        }
    }
}

template <typename E>
__global__ void k_fill(E *p, size_t n, E v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

template <typename E>
__global__ void k_col_unpack(const E *__restrict__ values, const int32_t *__restrict__ indices,
                             const int32_t *__restrict__ rowptr, E *__restrict__ out, int R, int C, int bh) {
    const int i = blockIdx.x;
    const int off = rowptr[i], L = rowptr[i + 1] - off;
    const int r0 = i * bh, rows = min(R, r0 + bh) - r0;
    const size_t vbase = (size_t)off * bh;
    for (int e = threadIdx.x; e < rows * L; e += blockDim.x) {
        const int p = e / L, t = e - p * L;
        out[(size_t)(r0 + p) * C + indices[off + t]] = values[vbase + e];
    }
}

template <typename E>
__global__ void k_row_unpack(const E *__restrict__ values, const int32_t *__restrict__ indices,
                             const int32_t *__restrict__ rowptr, E *__restrict__ out, int C, int bw, int nbc) {
    const int b = blockIdx.x;
    const int bj = b % nbc;
    const int c0 = bj * bw, c1 = min(C, c0 + bw);
    const int wj = c1 - c0, last_w = C - (nbc - 1) * bw;
    const int off = rowptr[b], ki = rowptr[b + 1] - off;
    const size_t voff = row_voff(rowptr, b, nbc, bw, last_w);
    for (int e = threadIdx.x; e < ki * wj; e += blockDim.x) {
        const int t = e / wj, q = e - t * wj;
        out[(size_t)indices[off + t] * C + c0 + q] = values[voff + e];
    }
}

// Blocked Compressed Storage (Sec. 4.3) from the canonical column packing: runs of
// consecutive block-rows with identical kept-column lists share one copy of the list.
// One workgroup walks the block-rows in order (prep-time work, no inter-workgroup
// synchronisation): it compares each list with the previous one, appends the lists
// that start a run, and writes every row's start in the values array.
__global__ void k_bcs(const int32_t *__restrict__ indices, const int32_t *__restrict__ rowptr, int nbr, int bh,
                      int R, int32_t *__restrict__ occurrence, int32_t *__restrict__ compact,
                      int32_t *__restrict__ col_stride, int32_t *__restrict__ row_offset, int32_t *__restrict__ n_runs) {
    __shared__ int s_same, s_runs, s_cpos;
    if (threadIdx.x == 0) {
        s_runs = 0;
        s_cpos = 0;
    }
    __syncthreads();
    for (int i = 0; i < nbr; ++i) {
        const int off = rowptr[i], len = rowptr[i + 1] - off;
        const int r0 = i * bh, r1 = min(R, r0 + bh);
        for (int r = r0 + threadIdx.x; r < r1; r += blockDim.x) row_offset[r] = off * bh + (r - r0) * len;
        if (threadIdx.x == 0) s_same = i > 0 && len == off - rowptr[i - 1];
        __syncthreads();
        if (s_same) {
            const int prev = rowptr[i - 1];
            for (int t = threadIdx.x; t < len; t += blockDim.x)
                if (indices[off + t] != indices[prev + t]) s_same = 0;   // every writer stores 0
        }
        __syncthreads();
        if (!s_same) {
            const int run = s_runs, cpos = s_cpos;
            for (int t = threadIdx.x; t < len; t += blockDim.x) compact[cpos + t] = indices[off + t];
            if (threadIdx.x == 0) {
                occurrence[run] = r0;
                col_stride[run] = cpos;
            }
        }
        __syncthreads();
        if (threadIdx.x == 0 && !s_same) {
            s_runs += 1;
            s_cpos += len;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        occurrence[s_runs] = R;
        col_stride[s_runs] = s_cpos;
        row_offset[R] = rowptr[nbr - 1] * bh + (R - (nbr - 1) * bh) * (rowptr[nbr] - rowptr[nbr - 1]);
        *n_runs = s_runs;
    }
}

inline int grid_for(size_t n) { return (int)std::max<size_t>(1, std::min<size_t>(8192, (n + 255) / 256)); }

template <typename E>
bsp_status pack_t(const Plan &p, const E *w, const uint8_t *mask, E *values, int32_t *indices,
                  int32_t *rowptr, uint8_t *tiles, hipStream_t st) {
    int *flag = (int *)(tiles + kFlagOffset);
    unsigned int *count = (unsigned int *)(tiles + kCountOffset);
    TileHeader h;
    memset(&h, 0, sizeof(h));
    h.magic = kMagic;
    h.fp_lo = (uint32_t)p.fingerprint;
    h.fp_hi = (uint32_t)(p.fingerprint >> 32);
    h.n_groups = p.n_groups;
    h.mt_per_group = p.mt_per_group;
    h.LP = p.LP;
    h.S = p.S;
    if (hipMemcpyAsync(tiles, &h, sizeof(h), hipMemcpyHostToDevice, st) != hipSuccess)
        return BSP_EDEVICE;
    const size_t n = (size_t)p.R * p.C;
    const bool blocked = p.reg != BSP_DENSE && p.reg != BSP_UNSTRUCTURED && p.reg != BSP_PATTERN;
    // canonical list offsets (from the scheme and its counts) and the counts, for the
    // kernels below; both copies complete before this call returns (it synchronises)
    std::vector<int32_t> rp(blocked ? (size_t)p.n_rowptr : 0);
    if (blocked) {
        plan_rowptr(p, rp.data());
        if (hipMemcpyAsync(rowptr, rp.data(), sizeof(int32_t) * rp.size(), hipMemcpyHostToDevice, st) !=
            hipSuccess)
            return BSP_EDEVICE;
    }
    const int32_t *counts = nullptr;
    CountTables ct{};
    std::vector<int32_t> tab;
    if (p.counts) {
        // counts, slot runs, block of each slot, per-block start and length in the lists
        const int nb = p.nbr * p.nbc;
        const bool lists = p.reg == BSP_COL || p.reg == BSP_PUNCHED;
        tab.assign((size_t)count_tables_bytes(p.nbr, p.nbc, p.L) / 4, 0);
        int32_t *tc = tab.data(), *tP = tc + nb, *tsb = tP + p.nbc + 1, *tst = tsb + p.L, *tn = tst + nb;
        for (int b = 0; b < nb; ++b) tc[b] = p.counts[b];
        if (lists) {
            count_slots(p, tP);
            for (int j = 0; j < p.nbc; ++j)
                for (int t = tP[j]; t < tP[j + 1]; ++t) tsb[t] = j;
            for (int i = 0; i < p.nbr; ++i) {
                int off = 0;
                for (int j = 0; j < p.nbc; ++j) {
                    tst[i * p.nbc + j] = off;
                    tn[i * p.nbc + j] = block_cols(p, i, j);
                    off += tn[i * p.nbc + j];
                }
            }
        }
        const int32_t *dt = (const int32_t *)(tiles + p.off_counts);
        if (hipMemcpyAsync((void *)dt, tab.data(), sizeof(int32_t) * tab.size(), hipMemcpyHostToDevice, st) !=
            hipSuccess)
            return BSP_EDEVICE;
        counts = dt;
        if (lists) ct = CountTables{dt, dt + nb, dt + nb + p.nbc + 1, dt + nb + p.nbc + 1 + p.L,
                                    dt + 2 * nb + p.nbc + 1 + p.L};
    }
    const int blk_cols = p.reg == BSP_PUNCHED ? p.bw_eff * p.khw : p.bw_eff;
    // 1. validate the block structure
    if (p.reg == BSP_ROWCOL) {
        k_validate_rowcol<<<p.nbr * p.nbc, 256, p.bh_eff + p.bw_eff, st>>>(mask, p.R, p.C, p.bh_eff, p.bw_eff,
                                                                          p.nbc, p.rate, flag);
    } else if (p.reg == BSP_PUNCHED) {
        k_validate_punched<<<p.nbr * p.nbc, 256, 0, st>>>(mask, p.R, p.C, p.khw, p.bh_eff, p.bw_eff, p.nbc,
                                                         (p.khw + p.rate - 1) / p.rate, counts, flag);
    } else if (p.reg == BSP_COL || p.reg == BSP_ROW) {
        const int ng = p.reg == BSP_COL ? p.bw_eff : p.bh_eff;
        const int threads = std::min(256, ((ng + 63) / 64) * 64);
        k_validate_blocks<<<p.nbr * p.nbc, threads, 0, st>>>(mask, p.R, p.C, p.bh_eff, p.bw_eff,
                                                            p.nbc, p.reg == BSP_COL, p.rate, counts, flag);
    } else {
        k_validate_all<<<grid_for(n), 256, 0, st>>>(mask, n, p.reg == BSP_DENSE, flag, count);
        if (p.reg == BSP_UNSTRUCTURED)
            k_check_count<<<1, 1, 0, st>>>(count, (unsigned int)((n + p.rate - 1) / p.rate), flag);
        if (p.reg == BSP_PATTERN) {
            const int nk = (int)(n / 9);
            k_validate_kernels4<<<grid_for(nk), 256, 0, st>>>(mask, nk, flag);
            k_check_count<<<1, 1, 0, st>>>(count, 4u * (unsigned int)pattern_kept(nk, p.rate), flag);
        }
    }
    int hflag = 0;
    if (hipMemcpyAsync(&hflag, flag, sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return BSP_EDEVICE;
    if (hflag) return BSP_EMASK;
    // 2. canonical packing
    if (p.reg == BSP_COL || p.reg == BSP_PUNCHED || p.reg == BSP_ROWCOL) {
        k_col_lists<<<p.nbr, 256, 0, st>>>(mask, p.R, p.C, p.bh_eff, p.reg == BSP_ROWCOL, rowptr, indices, flag);
        k_col_values<E><<<p.nbr, 256, 0, st>>>(w, mask, indices, rowptr, values, p.R, p.C, p.bh_eff);
    } else if (p.reg == BSP_ROW) {
        k_row_lists<<<p.nbr * p.nbc, 256, 0, st>>>(mask, p.R, p.C, p.bh_eff, p.bw_eff, p.nbc, rowptr,
                                                    indices, flag);
        k_row_values<E><<<p.nbr * p.nbc, 256, 0, st>>>(w, indices, rowptr, values, p.C, p.bw_eff, p.nbc);
    } else {
        k_masked_copy<E><<<grid_for(n), 256, 0, st>>>(w, mask, values, n);
    }
    // 3. forward layout
    int32_t *desc = (int32_t *)(tiles + p.off_desc);
    DescArgs da{p.shared, p.n_groups, p.L, p.LP, p.C, p.KH, p.KW, p.CH_STRIDE, p.RS, p.VS, std::max(p.V, 1),
                ct, p.nbc, blk_cols};
    k_desc<<<grid_for((size_t)p.n_groups * p.LP), 256, 0, st>>>(da, indices, rowptr, desc);
    ATileArgs aa{p.shared, p.n_groups, p.mt_per_group, p.n_mt_pad, p.group_rows, p.S, p.L, p.RK, p.C, p.rowmap,
                 ct, p.nbc, blk_cols};
    const size_t na = (size_t)p.n_mt_pad * p.S * 512;
    k_atiles<E><<<grid_for(na), 256, 0, st>>>(aa, w, mask, indices, rowptr, (E *)(tiles + p.off_a));
    if (p.rowmap) {
        int32_t *rm = (int32_t *)(tiles + p.off_rowmap);
        const size_t nrm = (size_t)p.n_mt_pad * kMT;
        k_fill<int32_t><<<grid_for(nrm), 256, 0, st>>>(rm, nrm, 0);
        k_rowmap<<<grid_for(p.R), 256, 0, st>>>(indices, p.RK, p.R, rm, (int32_t *)(tiles + p.off_pruned));
    }
    if (p.pl && !p.shared) {
        // the pointwise kernel with gathered lists reads the channels of the lists (its
        // plan's channel stride is 1) and no chunk table
        k_desc16_abs<<<grid_for((size_t)p.n_groups * p.LP), 256, 0, st>>>(
            desc, p.n_groups * p.LP, (uint16_t *)(tiles + p.off_desc16), flag);
    } else {
        int4 *table = (int4 *)(tiles + p.off_chunks);
        k_step_spans<<<grid_for(p.S), 256, 0, st>>>(desc, p.n_groups, p.LP, p.S, p.CH_STRIDE, table);
        k_build_chunks<<<1, 256, sizeof(int) * 2 * p.S, st>>>(
            table, p.S, p.CC, p.SMAX, (int *)(tiles + offsetof(TileHeader, n_chunks)), flag);
        k_desc16<<<grid_for((size_t)p.n_groups * p.LP), 256, 0, st>>>(
            desc, table, (const int *)(tiles + offsetof(TileHeader, n_chunks)), p.n_groups, p.LP,
            p.CH_STRIDE, (uint16_t *)(tiles + p.off_desc16), flag);
    }
    if (p.n_g_pad > p.n_groups) {
        // offsets of the padding groups of the last m-block: 0 (a valid patch position)
        const size_t nd = (size_t)(p.n_g_pad - p.n_groups) * p.LP;
        k_fill<uint16_t><<<grid_for(nd), 256, 0, st>>>(
            (uint16_t *)(tiles + p.off_desc16) + (size_t)p.n_groups * p.LP, nd, (uint16_t)0);
    }
    if (hipGetLastError() != hipSuccess) return BSP_EDEVICE;
    if (hipMemcpyAsync(&hflag, flag, sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return BSP_EDEVICE;
    if (hflag & 2) return BSP_EUNSUPPORTED;
    if (hflag) return BSP_EMASK;
    return BSP_OK;
}

template <typename E>
hipError_t unpack_t(const Plan &p, const E *values, const int32_t *indices, const int32_t *rowptr, E *out,
                    hipStream_t st) {
    const size_t n = (size_t)p.R * p.C;
    if (p.reg == BSP_DENSE || p.reg == BSP_UNSTRUCTURED || p.reg == BSP_PATTERN) {
        return hipMemcpyAsync(out, values, n * sizeof(E), hipMemcpyDeviceToDevice, st);
    }
    k_fill<E><<<grid_for(n), 256, 0, st>>>(out, n, (E)0);
    if (p.reg == BSP_COL || p.reg == BSP_PUNCHED || p.reg == BSP_ROWCOL)
        k_col_unpack<E><<<p.nbr, 256, 0, st>>>(values, indices, rowptr, out, p.R, p.C, p.bh_eff);
    else
        k_row_unpack<E><<<p.nbr * p.nbc, 256, 0, st>>>(values, indices, rowptr, out, p.C, p.bw_eff, p.nbc);
    return hipGetLastError();
}

}  // namespace

bsp_status run_pack(const Plan &p, const void *w, const uint8_t *mask, void *values,
                    int32_t *indices, int32_t *rowptr, uint8_t *tiles, hipStream_t st) {
    if (p.dt == BSP_F32)
        return pack_t<float>(p, (const float *)w, mask, (float *)values, indices, rowptr, tiles, st);
    return pack_t<uint16_t>(p, (const uint16_t *)w, mask, (uint16_t *)values, indices, rowptr,
                            tiles, st);
}

hipError_t launch_bcs(const Plan &p, const int32_t *indices, const int32_t *rowptr, int32_t *occurrence,
                      int32_t *compact, int32_t *col_stride, int32_t *row_offset, int32_t *n_runs, hipStream_t st) {
    k_bcs<<<1, 256, 0, st>>>(indices, rowptr, p.nbr, p.bh_eff, p.R, occurrence, compact, col_stride, row_offset,
                             n_runs);
    return hipGetLastError();
}

hipError_t launch_unpack(const Plan &p, const void *values, const int32_t *indices,
                         const int32_t *rowptr, void *w_out, hipStream_t st) {
    if (p.dt == BSP_F32)
        return unpack_t<float>(p, (const float *)values, indices, rowptr, (float *)w_out, st);
    return unpack_t<uint16_t>(p, (const uint16_t *)values, indices, rowptr, (uint16_t *)w_out, st);
}

}  // namespace bsp
