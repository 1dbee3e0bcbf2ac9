// Internal definitions shared by the host planner and the gfx950 kernels.
//
// Execution model of the forward (implicit GEMM, Y[R x P] = Wpruned[R x K] * B[K x P],
// B = im2col of x, P = output pixels):
//  * A "list group" is a set of 16-row MFMA m-tiles that share one list of kept
//    GEMM columns.  Column pruning (Sec. 4.1.1 / Eq. 3) gives one list per block-row;
//    row pruning, dense and unstructured layers use one identity list (all columns)
//    shared by every m-tile, with pruned weights zero in the weight tiles.
//  * A workgroup owns a tile of 64 output pixels (TRW output rows x TW columns,
//    rows flattened over images) and a block of m-tiles.  It stages an input patch
//    for a window of input channels in LDS, then each wave walks its lists in
//    steps of 32 kept columns: per lane, 8 kept columns x 4 neighbouring pixels are
//    gathered from LDS with one 8-byte read each, re-packed, and fed to
//    v_mfma_f32_16x16x32_bf16 (or 8 x v_mfma_f32_16x16x4_f32 for fp32).
//  * The channel windows ("chunks") are ranges of 32-wide steps whose kept columns
//    fall in at most CC consecutive input channels; they are built at pack time.
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

constexpr int kMT = 16;          // MFMA tile rows (M) and pixels per n-tile (N)
constexpr int kKS = 32;          // kept columns per step
constexpr int kNPIX = 64;        // output pixels per workgroup tile
constexpr int kWaves = 4;
constexpr int kThreads = 256;
constexpr int kMaxTileRows = 16; // TRW <= 64 / 4
constexpr int kMaxSlots = 64;    // input rows staged per tile (<= TRW * KH)
constexpr int kLdsBudget = 63 * 1024;  // patch; the small tile tables stay under 64 KiB
constexpr int kMaxAccTiles = 8;  // G * T m-tiles per wave
constexpr uint32_t kMagic = 0x31505342u;  // "BSP1"
constexpr int kHeaderBytes = 256;
constexpr int kZeroOffset = 128;  // 128 zero bytes inside the header: source of padding loads
constexpr int kTargetWGs = 512;   // aim for at least two workgroups per CU

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

// Header at the start of dev_tiles.  Written by the host (fields up to
// n_steps) and by the device chunk builder (n_chunks).
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
    int TW, TRW, Wop;             // tile width/rows, padded output width
    int VEC, LEFT, RL, NSLOT, CH_STRIDE, CC;
    int gran;                     // patch fill: 16 / 4 = direct-to-LDS granule bytes, 0 = register path
    int gather;                   // 1: stride-1 8-byte reads, 2: stride-2 16-byte reads, 0: per element
    // work split
    int T, G;                     // m-tiles per group per wave, groups per wave
    int split;                    // 0: waves own whole groups, 1: waves split one group's m-tiles
    int mpg_blocks;               // split mode: m-blocks per group (4*T m-tiles each)
    int n_mb;                     // m-blocks (workgroups along the output rows)
    // dev_tiles layout (bytes)
    int64_t off_chunks, off_desc, off_desc16, off_a, tile_bytes;
    uint64_t fingerprint;
    // canonical sizes (elements)
    int64_t n_values, n_indices, n_rowptr;
};

// Computes the plan; the geometry part ignores conv->n.  Returns BSP_OK or an error.
bsp_status make_plan(const bsp_scheme *s, const bsp_conv_shape *conv_or_null, bsp_dtype wdt,
                     int batch_for_linear, Plan *p);

// Chooses how the waves of a workgroup share the m-tiles for n_pt pixel tiles
// (fills p->T, G, split, mpg_blocks, n_mb).  T, G are powers of two with
// G * T <= 4.
void choose_split(Plan *p, int64_t n_pt);

// Per-call launch arguments of the forward kernel.
struct ConvArgs {
    const void *x;
    void *y;
    const uint8_t *tiles;
    const float *bias;
    int relu, out_bf16;
    int N, Cin, H, W, R, Ho, Wo, KH, KW, SH, SW, PH, PW;
    int TW, TRW, Wop, VEC, LEFT, RL, NSLOT, CH_STRIDE, CC;
    int n_groups, group_rows, mt_per_group, LP, S, T, G, split, mpg_blocks;
    int n_ct, n_pt, n_mb, total, gather, gran;
    int64_t off_chunks, off_desc16, off_a;
    uint32_t fp_lo, fp_hi;
    FastDiv div_nslot;   // row -> (channel, slot) in the patch loader
    FastDiv div_nv;      // vector index -> (row, vector in row) in the patch loader
    FastDiv div_Ho;      // flattened output row -> (image, oh)
};

inline int div_up(int a, int b) { return (a + b - 1) / b; }
inline int64_t div_up64(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int kept_count(int extent, int rate) { return (extent + rate - 1) / rate; }

}  // namespace bsp
