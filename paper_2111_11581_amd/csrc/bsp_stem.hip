// Stem convolutions: stride 2, filters at most 8 wide, few input channels (the 7x7/2
// first layer of ResNet-style networks), over the identity list of a shared plan
// (dense weights, or zero-expanded ones).  The implicit GEMM of Sec. 4.3 with output
// channels as the MFMA rows and output pixels as its columns:
//  - the k index of one MFMA lane is 8 consecutive filter columns of one (input
//    channel, filter row) pair, so a lane's B operand is 8 consecutive input elements
//    of one staged row: element iw of a row sits at LDS element iw + PW, and output
//    column ow reads elements 2 ow .. 2 ow + 7 (dwords ow .. ow + 3, always aligned);
//  - MFMA nt of a 64-column segment takes columns 4 n + nt (n = lane % 16), so the
//    4 windows of a lane come from 7 dwords read once, and the lane ends with 4
//    adjacent output columns of each of its channels (16 lanes store 128 bytes of a row);
//  - filter columns past KW and pairs past C * KH carry zero weights; their input
//    elements are masked (pairs: a zero row), so no Inf or NaN input leaks into them;
//  - a workgroup computes 4 output rows of one image (a wave each, every output
//    channel), staging the 2 * 3 + KH input rows of each channel once.
// The weight fragments are rebuilt from the packed MFMA tiles of the plan, so the
// packed layout is the same as for the general kernel.

#include "bsp_fwd.h"

namespace bsp {
namespace stem {

constexpr int kRows = 4;                 // output rows per workgroup, one per wave
constexpr int kStemThreads = 64 * kRows;
constexpr int kMaxKst = 8;              // k-steps of 4 (channel, filter row) pairs
constexpr int kMaxT = 6;                // staging tasks per thread (input granules of a row group)

struct StemArgs {
    const uint16_t *x;
    void *y;
    const uint8_t *tiles;
    const float *bias;
    int relu, out_bf16;
    int Cin, H, W, R, Ho, Wo, KH, KW, PH, PW;
    int S;              // 32-column steps of the packed weight tiles
    int64_t off_a;
    uint32_t fp_lo, fp_hi;
    int npair, kst;     // (channel, filter row) pairs; k-steps of 4 pairs
    int rw;             // staged input rows per channel
    int rsd;            // LDS row stride (dwords)
    int gt;             // staging tasks per row (16-byte granules + 1)
    int row_groups;     // row groups (kRows output rows) per image
    int n_rg;           // row groups of all images
    int lds_w;          // LDS bytes of the weight fragments
};

// One wave: output row oh0 + wave of image img, every output channel.
__device__ __forceinline__ void stem_rows(const StemArgs &a, const uint4 *s_w, const uint32_t *s_x,
                                          const float *s_bias, bool ok, int img, int oh0, int wave, int lane,
                                          int nrows) {
    const int oh = oh0 + wave;
    if (oh >= a.Ho) return;
    const int n = lane & 15, g = lane >> 4;
    // filter columns 2 q, 2 q + 1 of dword q that exist (the last dword of a window)
    const uint32_t km3 = (6 < a.KW ? 0xffffu : 0u) | (7 < a.KW ? 0xffff0000u : 0u);
    uint32_t km[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) km[q] = (2 * q < a.KW ? 0xffffu : 0u) | (2 * q + 1 < a.KW ? 0xffff0000u : 0u);
    const float qnan = __builtin_nanf("");
    // segments of 64 output columns; MFMA nt of a segment computes columns 4 n + nt, so
    // that a lane ends with 4 adjacent columns of each of its channels
    for (int seg = 0; seg * 64 < a.Wo; ++seg) {
        f32x4 acc[4][4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int ks = 0; ks < a.kst; ++ks) {
            s16x8 W[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) W[mt] = __builtin_bit_cast(s16x8, s_w[(ks * 4 + mt) * 64 + lane]);
            const int p = 4 * ks + g;
            const int c = p / a.KH, kh = p - c * a.KH;
            const int r = p < a.npair ? c * a.rw + 2 * wave + kh : nrows;
            // dwords 4 n .. 4 n + 7 of the segment: the windows of columns 4 n + 0..3
            const uint4 *wp = (const uint4 *)(s_x + r * a.rsd + 64 * seg + 4 * n);
            const uint4 lo = wp[0], hi = wp[1];
            const uint32_t d[7] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z};
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                const uint4 v = make_uint4(d[nt] & km[0], d[nt + 1] & km[1], d[nt + 2] & km[2], d[nt + 3] & km3);
                const s16x8 X = __builtin_bit_cast(s16x8, v);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(W[mt], X, acc[mt][nt], 0, 0, 0);
            }
        }
        // lane: channels 16 mt + 4 g + i, columns 64 seg + 4 n + 0..3 (16 lanes: 128 bytes
        // of one output row per store)
        const int px0 = 64 * seg + 4 * n;
        if (px0 < a.Wo) {
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int co = 16 * mt + 4 * g + i;
                    if (co >= a.R) continue;
                    float o[4];
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) {
                        float v = acc[mt][nt][i] + s_bias[co];
                        if (a.relu) v = v < 0.f ? 0.f : v;
                        o[nt] = ok ? v : qnan;
                    }
                    const size_t off = (((size_t)img * a.R + co) * a.Ho + oh) * a.Wo + px0;
                    if (a.out_bf16)
                        *(uint2 *)((uint16_t *)a.y + off) =
                            make_uint2(fwd::pk_bf16(o[0], o[1]), fwd::pk_bf16(o[2], o[3]));
                    else
                        *(float4 *)((float *)a.y + off) = make_float4(o[0], o[1], o[2], o[3]);
                }
        }
    }
}

__global__ __launch_bounds__(kStemThreads, 2) void k_stem(StemArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    __shared__ float s_bias[64];
    const uint4 *s_w = (const uint4 *)lds;
    uint32_t *s_x = (uint32_t *)(lds + a.lds_w);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid < 64) s_bias[tid] = (a.bias && tid < a.R) ? a.bias[tid] : 0.f;
    const TileHeader *hdr = (const TileHeader *)a.tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == a.fp_lo && hdr->fp_hi == a.fp_hi;
    const uint16_t *A = (const uint16_t *)(a.tiles + a.off_a);

    // input rows [c][r] (input row 2 oh0 - PH + r), then one zero row.  Task q of a row
    // writes dwords d_lo + 4 q .. + 3: elements 8 q - 1 .. 8 q + 6 of the row, realigned
    // by two bytes from granule q and the dword before it; the other dwords of a row
    // and the zero row are cleared once.
    const int nrows = a.Cin * a.rw;
    const int d_lo = (a.PW - 1) >> 1, d_hi = d_lo + 4 * a.gt;
    for (int i = tid; i < (nrows + 1) * a.rsd; i += kStemThreads) {
        const int r = i / a.rsd, d = i - r * a.rsd;
        if (r == nrows || d < d_lo || d >= d_hi) s_x[i] = 0u;
    }
    // a thread's staging tasks (at most kMaxT): the loads of the next row group are in
    // flight while the current one is computed and stored
    const int ntask = nrows * a.gt;
    uint4 cur[kMaxT];
    uint32_t prev[kMaxT];
    uint32_t sel = 0;   // bit 2 u: cur[u] holds input, bit 2 u + 1: prev[u] does
    auto load = [&](int rg) {
        sel = 0;
        const int img = rg / a.row_groups;
        const int oh0 = (rg - img * a.row_groups) * kRows;
#pragma unroll
        for (int u = 0; u < kMaxT; ++u) {
            const int i = tid + u * kStemThreads;
            const int row = i / a.gt, q = i - row * a.gt;
            const int c = row / a.rw, r = row - c * a.rw;
            const int ih = 2 * oh0 - a.PH + r;
            // loads always issued (outside the image: from the start of x), then selected
            const bool in = i < ntask && ih >= 0 && ih < a.H;
            const uint16_t *src = a.x + (in ? (((int64_t)img * a.Cin + c) * a.H + ih) * a.W : 0);
            const bool has_c = in && q < a.gt - 1, has_p = in && q > 0;
            const uint4 cv = *(const uint4 *)(has_c ? src + 8 * q : a.x);
            const uint32_t pv = *(const uint32_t *)(has_p ? src + 8 * q - 2 : a.x);
            cur[u] = cv;   // raw: the selects wait for the loads, so they happen at the writes
            prev[u] = pv;
            sel |= (has_c ? 1u : 0u) << (2 * u) | (has_p ? 2u : 0u) << (2 * u);
        }
    };
    int rg = blockIdx.x;
    if (rg < a.n_rg) load(rg);

    // weight fragments [ks][mt][lane]: filter columns 0..7 of pair p = 4 ks + lane / 16
    // and output channel co = 16 mt + lane % 16, i.e. GEMM columns p KW .. p KW + 7 of
    // row co.  The packed tiles hold 8 consecutive columns of a row in 16 bytes (chunk q:
    // m-tile co / 16, step q / 4, lane co % 16 + 16 (q % 4)), so a fragment is the two
    // chunks around its first column, shifted by that column's place in the chunk.  All
    // loads of a thread are issued first (zero fragments read the header).
    {
        const int nfrag = a.kst * 4 * 64;
        uint4 c0[kMaxKst], c1[kMaxKst];
        bool use[kMaxKst];
#pragma unroll
        for (int u = 0; u < kMaxKst; ++u) {
            const int f = tid + u * kStemThreads;
            const int l = f & 63, mt = (f >> 6) & 3, ks = f >> 8;
            const int p = 4 * ks + (l >> 4), co = 16 * mt + (l & 15);
            const int q0 = p * a.KW >> 3;
            use[u] = ok && f < nfrag && p < a.npair && co < a.R;
            const int64_t row = (int64_t)(co >> 4) * a.S;
            const bool v0 = use[u] && (q0 >> 2) < a.S, v1 = use[u] && ((q0 + 1) >> 2) < a.S;
            const uint16_t *s0 = v0 ? A + ((row + (q0 >> 2)) * 64 + (co & 15) + 16 * (q0 & 3)) * 8
                                    : (const uint16_t *)a.tiles;
            const uint16_t *s1 = v1 ? A + ((row + ((q0 + 1) >> 2)) * 64 + (co & 15) + 16 * ((q0 + 1) & 3)) * 8
                                    : (const uint16_t *)a.tiles;
            c0[u] = *(const uint4 *)s0;
            c1[u] = *(const uint4 *)s1;
            if (!v1) c1[u] = make_uint4(0u, 0u, 0u, 0u);
        }
        uint32_t km[4];   // filter columns 2 k, 2 k + 1 that exist
#pragma unroll
        for (int k = 0; k < 4; ++k) km[k] = (2 * k < a.KW ? 0xffffu : 0u) | (2 * k + 1 < a.KW ? 0xffff0000u : 0u);
        uint4 *s_wf = (uint4 *)lds;
#pragma unroll
        for (int u = 0; u < kMaxKst; ++u) {
            const int f = tid + u * kStemThreads;
            if (f >= nfrag) continue;
            const int l = f & 63, ks = f >> 8;
            const int t0 = (4 * ks + (l >> 4)) * a.KW;
            const int base = (t0 & 7) >> 1;        // first dword of the fragment in the chunk pair
            const bool odd = (t0 & 1) != 0;        // the fragment starts in the upper half of it
            const uint32_t d[8] = {c0[u].x, c0[u].y, c0[u].z, c0[u].w, c1[u].x, c1[u].y, c1[u].z, c1[u].w};
            auto pick = [&](int i) {   // d[i], i in 0..7
                const uint32_t a01 = i & 1 ? d[1] : d[0], a23 = i & 1 ? d[3] : d[2];
                const uint32_t a45 = i & 1 ? d[5] : d[4], a67 = i & 1 ? d[7] : d[6];
                const uint32_t b03 = i & 2 ? a23 : a01, b47 = i & 2 ? a67 : a45;
                return i & 4 ? b47 : b03;
            };
            uint32_t r[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint32_t lo = pick(base + k), hi = pick(min(base + k + 1, 7));
                r[k] = (odd ? __builtin_amdgcn_alignbyte(hi, lo, 2) : lo) & km[k];
            }
            s_wf[f] = use[u] ? make_uint4(r[0], r[1], r[2], r[3]) : make_uint4(0u, 0u, 0u, 0u);
        }
    }

    for (; rg < a.n_rg; rg += gridDim.x) {
#pragma unroll
        for (int u = 0; u < kMaxT; ++u) {
            const int i = tid + u * kStemThreads;
            if (i >= ntask) continue;
            const int row = i / a.gt, q = i - row * a.gt;
            const uint4 cv = (sel >> (2 * u)) & 1u ? cur[u] : make_uint4(0u, 0u, 0u, 0u);
            const uint32_t pv = (sel >> (2 * u)) & 2u ? prev[u] : 0u;
            uint32_t *dst = s_x + row * a.rsd + d_lo + 4 * q;
            dst[0] = __builtin_amdgcn_alignbyte(cv.x, pv, 2);
            dst[1] = __builtin_amdgcn_alignbyte(cv.y, cv.x, 2);
            dst[2] = __builtin_amdgcn_alignbyte(cv.z, cv.y, 2);
            dst[3] = __builtin_amdgcn_alignbyte(cv.w, cv.z, 2);
        }
        __syncthreads();
        if (rg + (int)gridDim.x < a.n_rg) load(rg + (int)gridDim.x);
        const int img = rg / a.row_groups;
        const int oh0 = (rg - img * a.row_groups) * kRows;
        stem_rows(a, s_w, s_x, s_bias, ok, img, oh0, wave, lane, nrows);
        __syncthreads();   // the next row group rewrites the rows
    }
}

}  // namespace stem

// LDS row stride (dwords) of the staged input: the dwords the staging writes and the
// windows of every 64-column segment (dwords up to 64 (segments - 1) + 67)
static int stem_rsd(const Plan &p) {
    const int d_hi = (p.PW - 1) / 2 + 4 * (p.W / 8 + 1);
    const int nseg = (p.Wo + 63) / 64;
    return (std::max(d_hi, 64 * nseg + 4) + 3) / 4 * 4;
}

static int64_t stem_lds(const Plan &p) {
    const int kst = (p.Cin * p.KH + 3) / 4;
    return (int64_t)kst * 4 * 64 * 16 + (int64_t)(p.Cin * (2 * (stem::kRows - 1) + p.KH) + 1) * stem_rsd(p) * 4;
}

bool stem_ok(const Plan &p, const void *x) {
    return !p.pw && !p.is_linear && !p.im2col && p.esize == 2 && p.shared && !p.rowmap && p.counts_hash == 0 &&
           p.SH == 2 && p.SW == 2 && p.KW >= 1 && p.KW <= 8 && p.KH >= 1 && (p.PW & 1) == 1 && p.PW < 8 &&
           p.PH >= 0 && p.W % 8 == 0 && p.Wo % 4 == 0 && p.Wo <= 1024 && p.R <= 64 && p.RK == p.R &&
           p.Cin * p.KH <= 4 * stem::kMaxKst && p.L == p.Cin * p.KH * p.KW && stem_lds(p) <= 64 * 1024 &&
           p.Cin * (2 * (stem::kRows - 1) + p.KH) * (p.W / 8 + 1) <= stem::kMaxT * stem::kStemThreads &&
           ((uintptr_t)x & 15) == 0;
}

hipError_t launch_stem(const Plan &p, int n, const void *x, const uint8_t *tiles, const float *bias, int relu,
                       int out_bf16, void *y, hipStream_t st) {
    using namespace stem;
    if (n <= 0 || p.Ho <= 0) return hipSuccess;
    StemArgs a;
    memset(&a, 0, sizeof(a));
    a.x = (const uint16_t *)x;
    a.y = y;
    a.tiles = tiles;
    a.bias = bias;
    a.relu = relu;
    a.out_bf16 = out_bf16;
    a.Cin = p.Cin; a.H = p.H; a.W = p.W; a.R = p.R; a.Ho = p.Ho; a.Wo = p.Wo;
    a.KH = p.KH; a.KW = p.KW; a.PH = p.PH; a.PW = p.PW;
    a.S = p.S;
    a.off_a = p.off_a;
    a.fp_lo = (uint32_t)p.fingerprint;
    a.fp_hi = (uint32_t)(p.fingerprint >> 32);
    a.npair = p.Cin * p.KH;
    a.kst = (a.npair + 3) / 4;
    a.rw = 2 * (kRows - 1) + p.KH;
    a.gt = p.W / 8 + 1;
    a.rsd = stem_rsd(p);
    a.row_groups = (p.Ho + kRows - 1) / kRows;
    a.lds_w = a.kst * 4 * 64 * 16;
    const int64_t lds = stem_lds(p);
    const int64_t n_rg = (int64_t)n * a.row_groups;
    if (lds > 160 * 1024 || n_rg > INT32_MAX) return hipErrorInvalidValue;
    a.n_rg = (int)n_rg;
    // persistent workgroups, two per CU (the kernel's register budget), each walking
    // the same number of row groups
    const int64_t per = (n_rg + 2 * 256 - 1) / (2 * 256);
    const int64_t grid = (n_rg + per - 1) / per;
    void (*fn)(StemArgs) = k_stem;
    if (lds > 48 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(kStemThreads), (size_t)lds, st, a);
    return hipGetLastError();
}

}  // namespace bsp
