// Internal definitions shared by the host planner and the gfx950 kernels.
//
// Execution model of the forward (implicit GEMM, Y[R x P] = Wpruned[R x K] * B[K x P],
// B = im2col of x, P = output pixels):
//  * A "list group" is a set of 16-row MFMA m-tiles that share one list of kept
//    GEMM columns.  Column pruning (Sec. 4.1.1 / Eq. 3) gives one list per block-row;
//    row pruning, dense and unstructured layers use one identity list (all columns)
//    shared by every m-tile, with pruned weights zero in the weight tiles.
//  * Output pixels are taken in groups of 4 adjacent pixels of one output row (rows
//    padded to a multiple of 4); groups are numbered row after row over all images,
//    so a run of consecutive groups is a run of consecutive output pixels in memory.
//    A sub-tile is 16 groups (64 pixels); a workgroup tile is NSUB sub-tiles.
//  * A workgroup (4 waves) owns one tile and one m-block of m-tiles.  Wave w works on
//    sub-tile w % NSUB; the 4 / NSUB waves of a sub-tile split either the m-block's
//    m-tiles or the 32-wide steps of the kept lists (then they sum their partial
//    results at the end).
//  * The K loop walks "chunks": ranges of steps whose kept columns fall in at most CC
//    consecutive input channels.  The input rows of a chunk's channels (the patch)
//    are staged in LDS by asynchronous direct-to-LDS copies while the previous chunk
//    computes (two buffers); weights and gather offsets come from LDS too.
#pragma once

#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "bsp.h"

#if defined(__HIPCC__)
#define BSP_HD __host__ __device__
#else
#define BSP_HD
#endif

namespace bsp {

constexpr int kMT = 16;            // MFMA tile rows (M) and pixels per n-tile (N)
constexpr int kKS = 32;            // kept columns per step
constexpr int kGroups = 16;        // 4-pixel groups per sub-tile (64 pixels)
constexpr int kWaves = 4;
constexpr int kThreads = 256;
constexpr int kMaxTileRows = 72;   // output rows one workgroup tile may span
constexpr int kMaxSlots = 192;     // staged input rows per workgroup tile
constexpr int kMaxCC = 2047;       // channels of one chunk (11 bits of a granule's decode)
constexpr int kMaxChunks = 512;    // chunk table entries staged in LDS
constexpr int kLdsStatic = 17 * 1024;  // static LDS tables of the general kernel (16.1 KB) and slack
constexpr uint32_t kMagic = 0x34505342u;  // "BSP4"
constexpr int kHeaderBytes = 256;
constexpr int kZeroOffset = 128;   // 128 zero bytes inside the header: source of padding loads
constexpr int kNominalImages = 64; // batch the planner tunes conv tilings for
constexpr int kNominalVectors = 512;  // batch the planner tunes linear tilings for
constexpr int kLinRow = 64;        // a linear layer's batch is staged as rows of 64 vectors

// Unsigned division by a run-time constant with a multiply-high and a shift
// (round-up method of Granlund and Montgomery, "Division by invariant integers
// using multiplication", 1994), valid for 0 <= n < 2^31 and 1 <= d < 2^31.
struct FastDiv {
    uint32_t d, m, s;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.d = d;
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    f.s = l;
    // m = floor(2^32 * (2^l - d) / d) + 1
    f.m = (uint32_t)(((((uint64_t)1 << l) - d) << 32) / d + 1);
    return f;
}

BSP_HD inline uint32_t fdiv(uint32_t n, const FastDiv &f) {
    const uint32_t t = (uint32_t)(((uint64_t)n * f.m) >> 32);  // v_mul_hi_u32 on the device
    return (t + n) >> f.s;
}

// Staging of input rows for one tile of output rows g0 .. g0+TRW-1 (g = img*Ho + oh).
// Rows of one image share slots (slot = base(row) + r for filter row r; the base
// advances by min(SH, KH) inside an image and by KH at an image boundary).  Returns
// the number of slots; fills rowbase[TRW] (0 for rows past the end) and, when slot_ih
// is not null, slot_img/slot_ih for every slot (ih may be outside [0, H): zero row).
BSP_HD inline int slot_layout(int g0, int TRW, int Ho, int n_rows_total, int KH, int SH, int PH,
                              int *rowbase, int *slot_img, int *slot_ih) {
    int base = 0, prev_img = -1, nslot = 0;
    const int step = SH < KH ? SH : KH;
    for (int tr = 0; tr < TRW; ++tr) {
        const int g = g0 + tr;
        if (g >= n_rows_total) {
            if (rowbase) rowbase[tr] = 0;
            continue;
        }
        const int img = g / Ho, oh = g - img * Ho;
        if (prev_img >= 0) base += (img == prev_img) ? step : KH;
        if (rowbase) rowbase[tr] = base;
        if (slot_ih) {
            for (int r = 0; r < KH; ++r) {
                slot_img[base + r] = img;
                slot_ih[base + r] = oh * SH - PH + r;
            }
        }
        prev_img = img;
        nslot = base + KH;
    }
    return nslot;
}

// Header at the start of dev_tiles.  Written by the host, except n_chunks
// (device chunk builder).  Bytes [kZeroOffset, kHeaderBytes) stay zero.
struct TileHeader {
    uint32_t magic;
    uint32_t fp_lo, fp_hi;       // plan fingerprint
    int32_t n_chunks;
    int32_t n_groups, mt_per_group, LP, S;
    int32_t reserved[kHeaderBytes / 4 - 8];
};

struct Plan {
    // scheme
    int R, C, bh, bw, reg, rate, dt, esize;
    int nbr, nbc;                 // number of block-rows / block-cols (PUNCHED: channel blocks)
    int khw;                      // kernel locations per input channel (PUNCHED), else 1
    const int32_t *counts;        // caller's kept groups per block (host, valid during the call), or null
    uint32_t counts_hash;         // hash of the counts (part of the fingerprint)
    int bh_eff, bw_eff;           // block size with 0 resolved to the extent
    // lists
    int shared;                   // 1 = identity list shared by all m-tiles
    int n_groups, group_rows, mt_per_group;
    int RK;                       // rows the kernels compute (R, or the kept filters with a row map)
    int im2col;                   // 1: a conv planned as a 1x1 layer over its im2col input
                                  // (channels cin * kh * kw, image Ho x Wo)
    int xplane;                   // input plane stride (elements) of a stride-1 pointwise plan
                                  // when not H * W: im2col planes padded to whole granules
    int rowmap;                   // 1: row pruning with whole-width blocks (filter pruning): the
                                  // kernels compute the kept rows only, the epilogue writes row
                                  // rowmap[i] of the output, a fill writes the pruned rows
    int L, LP, S;                 // kept per list, padded to 32, steps
    // geometry (linear: Cin = C, H = ceil(batch / 64) rows of W = 64 vectors, 1x1)
    int is_linear;
    int Cin, H, W, KH, KW, SH, SW, PH, PW, Ho, Wo;
    int Wop, GPR;                 // output row width padded to 4, 4-pixel groups per row
    int NSUB;                     // 64-pixel sub-tiles per workgroup tile
    int TRWMAX;                   // output rows a tile may span
    int NSLOT;                    // staged input rows per tile (worst case)
    int GE;                       // elements per 16-byte granule
    int LEFT, RS, RG, CH_STRIDE;  // patch row: left pad (0), row stride (elements, granules), channel stride
    int V;                        // copies of each staged row (stride 1: min(KW, 4), shifted by 0..V-1)
    int VS;                       // patch stride between the copies of one channel
    int POFF;                     // patch offset of output column 0 for filter column 0 (V == 1)
    int CC;                       // channels of one chunk
    int gather;                   // 1: stride-1 vector reads, 2: stride-2 16-byte reads, 0: per element
    // waves and m-blocks
    int qmode;                    // 0: the 4 / NSUB waves of a sub-tile split m-tiles, 1: split steps
    int KS;                       // step split (qmode 1), else 1
    int TM, TPG;                  // m-tiles per wave, m-tiles per list group inside a wave
    int MBT, MBG, n_mb;           // m-tiles / list groups per workgroup, m-blocks
    int n_mt_pad, n_g_pad;        // m-tiles / groups with tiles in dev_tiles (padded to whole m-blocks)
    int resident;                 // 1: the m-block's weights stay in LDS; 0: staged per chunk
    int NB;                       // LDS buffers of the K loop (2 or 3)
    int SMAX;                     // steps per chunk when weights are staged (0 = unlimited)
    int FR;                       // patch granules per thread and chunk
    int lds_d, lds_a, lds_patch, lds_astage, lds_buf, lds_total;   // dynamic LDS bytes
    // pointwise kernel (1x1 without padding, stride 1 or 2; linear layers)
    int pw;                       // 1: the pointwise kernel runs this layer
    int pl;                       // 1: the identity-list pointwise kernel (k_pl) runs it
    int NGR;                      // 16-byte granules per patch row (one channel of a tile)
    int gpg;                      // 4-pixel groups per granule
    int occ;                      // workgroups per CU the plan is sized for
    // dev_tiles layout (bytes); with a row map, off_rowmap holds int32 rowmap[n_mt_pad * 16]
    // (kept output row of each computed row, 0 past RK) followed by the R - RK pruned rows
    int64_t off_chunks, off_desc, off_desc16, off_a, off_rowmap, off_pruned, off_counts, tile_bytes;
    uint64_t fingerprint;
    // canonical sizes (elements)
    int64_t n_values, n_indices, n_rowptr;
};

// Computes the plan; the geometry part ignores conv->n.  With conv_or_null == NULL
// and batch_for_linear < 0 only the scheme and list structure are resolved.
// Returns BSP_OK or an error.
bsp_status make_plan(const bsp_scheme *s, const bsp_conv_shape *conv_or_null, bsp_dtype wdt,
                     int batch_for_linear, Plan *p);

// Per-call launch arguments of the forward kernel.
struct ConvArgs {
    const void *x;
    void *y;
    const uint8_t *tiles;
    const float *bias;
    int relu, out_bf16;
    int N, Cin, H, W, R, Ho, Wo, KH, KW, SH, SW, PH, PW;
    int64_t x_cs, y_cs;           // channel strides of x and y (elements)
    int64_t x_total;              // elements of x (loads never reach past it)
    int w_last;                   // valid width of the last input row of an image (linear: batch tail)
    int w_last_out;               // valid width of the last output row of an image
    int GPR, NSUB, NSLOT, LEFT, RS, RG, CH_STRIDE, CC, GE, FR;
    int n_groups, group_rows, mt_per_group, LP, S;
    int KS, MBT, MBG, n_mb;
    int resident, NB;
    int lds_d, lds_a, lds_patch, lds_astage, lds_buf;
    int64_t n_groups_total;       // 4-pixel groups over all images
    int n_pt;                     // pixel tiles
    int tiles_per_wg;             // consecutive pixel tiles one workgroup walks
    int grid_valid;               // number of real workgroups (grid is padded to 8)
    int64_t off_chunks, off_desc16, off_a;
    uint32_t fp_lo, fp_hi;
    FastDiv div_GPR;              // group -> (row, group in row)
    FastDiv div_Ho;               // flattened output row -> (image, oh)
    FastDiv div_RG;               // patch granule -> (row, granule in row)
    FastDiv div_CHG;              // patch granule -> (channel, granule in channel)
    FastDiv div_VSG;              // granule in channel -> (filter column, granule in copy)
    int CHG, VSG;                 // granules per channel, per shifted copy
    int V, POFF;                  // copies per staged row, patch offset of output column 0
    FastDiv div_nmb;              // workgroup -> (pixel tile, m-block)
    const int32_t *rowmap;        // output row of each computed row (row-mapped kernels only)
    int Rout;                     // output channels (R is the number of computed rows)
};

// Launch arguments of the pointwise kernel.  Output pixels are numbered in groups
// of 4: at stride 1 the pixels of an image are one row of Ho * Wo pixels; at stride
// 2 each output row is a row of groups.  Rows hold GPR groups.
struct PwArgs {
    const void *x;
    void *y;
    const uint8_t *tiles;
    const float *bias;
    int relu, out_bf16;
    int R;                        // computed rows of the GEMM (filters, out features)
    int Ho;                       // group rows per image
    int Wo;                       // output pixels per group row
    int GPR;                      // groups per group row
    int in_row;                   // input elements from one group row to the next
    int SW;                       // stride
    int64_t x_is, y_is;           // image strides of x and y (elements)
    int64_t x_cs, y_cs;           // channel strides of x and y (elements)
    int64_t x_total;              // elements of x (copies never reach past it)
    int64_t n_groups_total;       // groups over all images
    int NSUB, lg_nsub, NGR, lg_ngr, gpg, FR;
    int n_groups, group_rows, mt_per_group, LP, S;
    int MBT, MBG, n_mb, resident, NB;
    int lds_d, lds_a, lds_patch, lds_astage, lds_buf;
    int n_pt;                     // pixel tiles
    int tiles_per_wg;             // consecutive pixel tiles one workgroup walks
    int grid_valid;
    int64_t off_chunks, off_desc16, off_a;
    uint32_t fp_lo, fp_hi;
    FastDiv div_GPR;              // group -> (group row, group in row)
    FastDiv div_Ho;               // group row -> (image, row in image)
    FastDiv div_nmb;              // workgroup -> (pixel tile, m-block)
    const int32_t *rowmap;        // output row of each computed row (row-mapped kernels only)
    int Rout;                     // output channels (R is the number of computed rows)
    int Cin;                      // input channels (in_features)
    int SMAX;                     // steps per stage (identity-list kernel)
    // K loop split over workgroups (pipelined kernel): ks parts of s_per steps, kpart_wgs
    // workgroups each; part kp stores fp32 partial sums at y + kp * part_stride
    int ks, s_per, kpart_wgs;
    FastDiv div_kpart;
    int64_t part_stride;
};

// Workgroups per CU the pointwise kernel's register budget allows (its launch
// bound): element size, gather mode (1: stride 1, 2: stride 2), m-tiles per wave.
BSP_HD constexpr int pw_occ(int esize, int mode, int tm) {
    return esize == 4 ? (tm == 1 ? 3 : 2) : (tm == 4 ? 2 : (tm == 2 || mode == 2 ? 3 : 4));
}

// The general kernel runs workgroups of 8 waves: 4 that multiply and 4 that copy the
// next chunks into LDS and clear their pads.  Two waves per SIMD leave each wave 256
// registers: one workgroup per CU (arguments kept for the plan's gather mode and shape).
constexpr int kFwdThreads = 512;
BSP_HD constexpr int fwd_occ(int gather, int tm, int tpg) { return (void)gather, (void)tm, (void)tpg, 1; }

inline int div_up(int a, int b) { return (a + b - 1) / b; }
inline int64_t div_up64(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int kept_count(int extent, int rate) { return (extent + rate - 1) / rate; }

// Kernels kept by the connectivity pruning of pattern-based pruning (3x3 kernels,
// 4 weights each): ceil(n * 9 / (4 * rate)), at most n.
inline int pattern_kept(int n, int rate) {
    return (int)std::min<int64_t>(n, ((int64_t)n * 9 + 4 * rate - 1) / (4 * (int64_t)rate));
}

// Kept groups of block b (row-major over block-rows x block-columns): the caller's
// count, else ceil(groups / rate).
int block_count(const Plan &p, int b);

// Canonical rowptr of the plan (COL / PUNCHED: per block-row list offsets; ROW: per
// block offsets), n_rowptr entries.
void plan_rowptr(const Plan &p, int32_t *rowptr);

// Kept GEMM columns of block (i, j) of a COL / PUNCHED plan.
int block_cols(const Plan &p, int i, int j);

// Slot runs of the forward lists of a COL / PUNCHED plan with per-block counts:
// block column j owns slots [P[j], P[j+1]) of every block-row's list, as many as its
// largest kept-column count; P has nbc + 1 entries and P[nbc] = L.
void count_slots(const Plan &p, int32_t *P);

// Device tables of a plan with per-block counts (in dev_tiles at off_counts):
// counts[nbr*nbc], slot run starts P[nbc+1], block of each slot [L], and per block
// (i, j) the offset of its kept columns inside list i and their number.
struct CountTables {
    const int32_t *counts, *P, *slot_block, *start, *ncols;
};
inline int64_t count_tables_bytes(int nbr, int nbc, int L) {
    return 4 * ((int64_t)3 * nbr * nbc + nbc + 1 + L);
}

}  // namespace bsp
