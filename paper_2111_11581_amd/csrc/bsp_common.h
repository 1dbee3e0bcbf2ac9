// Internal definitions shared by the host planner and the gfx950 kernels.
//
// Execution model of the forward (implicit GEMM, Y[R x P] = Wpruned[R x K] * B[K x P],
// B = im2col of x, P = output pixels):
//  * A "list group" is a set of 16-row MFMA m-tiles that share one list of kept
//    GEMM columns.  Column pruning (Sec. 4.1.1 / Eq. 3) gives one list per block-row;
//    row pruning, dense and unstructured layers use one identity list (all columns)
//    shared by every m-tile, with pruned weights zero in the weight tiles.
//  * Pixels are cut into sub-tiles of 64 outputs (TRW output rows x TW columns, rows
//    flattened over images).  A workgroup (4 waves) owns NSUB vertically stacked
//    sub-tiles and one "m-block" of m-tiles; wave w works on sub-tile w % NSUB for the
//    m-set w / NSUB of the m-block.  Workgroups are persistent: each walks a
//    contiguous range of pixel tiles for its m-block.
//  * Work items are (tile, chunk): a chunk is a range of 32-wide steps of the kept
//    lists whose columns fall in at most CC consecutive input channels (and, when
//    weights are streamed, at most SMAX steps).  Items are double buffered in LDS:
//    the input patch (and streamed weight / offset slices) of item i+1 load with
//    asynchronous direct-to-LDS copies while item i computes.
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
constexpr int kNPIX = 64;          // output pixels per sub-tile
constexpr int kWaves = 4;
constexpr int kThreads = 256;
constexpr int kMaxTileRows = 64;   // NSUB * TRW
constexpr int kMaxSlots = 160;     // staged input rows per workgroup tile
constexpr int kLdsPerWG = 76 * 1024;  // dynamic LDS per workgroup (two per CU with the static tables)
constexpr int kLdsOneWG = 152 * 1024; // dynamic LDS when one workgroup per CU is needed
constexpr int kSmaxStreamed = 4;   // steps per item when weights are streamed
constexpr uint32_t kMagic = 0x32505342u;  // "BSP2"
constexpr int kHeaderBytes = 256;
constexpr int kZeroOffset = 128;   // 128 zero bytes inside the header: source of padding loads
constexpr int kTargetWGs = 512;    // two resident workgroups per CU

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
    int nbr, nbc;                 // number of block-rows / block-cols
    int bh_eff, bw_eff;           // block size with 0 resolved to the extent
    // lists
    int shared;                   // 1 = identity list shared by all m-tiles
    int n_groups, group_rows, mt_per_group;
    int L, LP, S;                 // kept per list, padded to 32, steps
    // geometry (linear: Cin = C, H = 1, W = batch, KH = KW = 1)
    int is_linear;
    int Cin, H, W, KH, KW, SH, SW, PH, PW, Ho, Wo;
    int TW, TRW, Wop;             // sub-tile width/rows, padded output width
    int NSUB;                     // sub-tiles per workgroup tile (stacked rows)
    int VEC, LEFT, RL, NSLOT, CH_STRIDE, CC;
    int gran;                     // patch fill: 16 / 4 = direct-to-LDS granule bytes, 0 = register path
    int gather;                   // 1: stride-1 8-byte reads, 2: stride-2 16-byte reads, 0: per element
    // m-blocks: wave w of a workgroup handles m-set w / NSUB (4 / NSUB m-sets)
    int split;                    // 0: m-sets own G whole groups; 1: m-sets own T m-tiles of one group
    int T, G;                     // m-tiles per group per wave, groups per wave (powers of two)
    int msets, mb_tiles, mb_groups, mpg_blocks, n_mb;
    int resident;                 // 1: the m-block's weights stay in LDS; 0: streamed per item
    int SMAX;                     // steps per item (0 = unlimited)
    int lds_a, lds_d, lds_patch, lds_buf, lds_total;   // LDS bytes
    // dev_tiles layout (bytes)
    int64_t off_chunks, off_desc, off_desc16, off_a, tile_bytes;
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
    int TW, TRW, NSUB, RL, NSLOT, CH_STRIDE, LEFT;
    int n_groups, group_rows, mt_per_group, LP, S;
    int split, msets, mb_tiles, mb_groups, mpg_blocks, n_mb;
    int resident, gran, gather;
    int lds_a, lds_d, lds_patch, lds_buf;
    int n_ct, n_wt;               // column tiles, workgroup tiles
    int wg_per_mb, tiles_per_wg;  // persistent split of the tiles of one m-block
    int grid_valid;               // number of real workgroups (grid is padded to 8)
    int64_t off_chunks, off_desc16, off_a;
    uint32_t fp_lo, fp_hi;
    FastDiv div_nslot;            // row -> (channel, slot) in the patch loader
    FastDiv div_nv;               // granule index -> (row, granule in row)
    FastDiv div_Ho;               // flattened output row -> (image, oh)
};

inline int div_up(int a, int b) { return (a + b - 1) / b; }
inline int64_t div_up64(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int kept_count(int extent, int rate) { return (extent + rate - 1) / rate; }

}  // namespace bsp
