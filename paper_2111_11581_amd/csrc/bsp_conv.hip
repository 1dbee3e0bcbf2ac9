// Launcher of the forward kernel: argument set-up and instantiation choice.  The
// kernel template lives in bsp_fwd.h; its instantiations are compiled in
// bsp_fwd_*.hip (one translation unit per element type and gather mode).
#include <mutex>

#include "bsp_pl.h"
#include "bsp_pw.h"

namespace bsp {
namespace pl {

pl_fn pick_1(int NSUB, int TM, bool map);
pl_fn pick_2(int NSUB, int TM, bool map);
pl_fn pick_g(int NSUB, int TM, int G);

}  // namespace pl
namespace pw {

pw_fn pick_b1(int TM, int TPG, int KS, bool map);
pw_fn pick_b2(int TM, int TPG, int KS, bool map);
pw_fn pick_f(int TM, int TPG, int KS, bool map);

}  // namespace pw

namespace fwd {

// instantiation sets, one per translation unit (bsp_fwd_*.hip)
fwd_fn pick_b1_k1(int TM, int TPG, int KS, bool map);
fwd_fn pick_b1_k24(int TM, int TPG, int KS, bool map);
fwd_fn pick_b2(int TM, int TPG, int KS, bool map);
fwd_fn pick_b3(int TM, int TPG, int KS, bool map);
fwd_fn pick_b0(int TM, int TPG, int KS, bool map);
fwd_fn pick_f(int mode, int TM, int TPG, int KS, bool map);

static fwd_fn pick(int dt, int mode, int TM, int TPG, int KS, bool map) {
    if (dt == BSP_F32) return pick_f(mode == 2 ? 0 : mode, TM, TPG, KS, map);
    if (mode == 1) return KS == 1 ? pick_b1_k1(TM, TPG, KS, map) : pick_b1_k24(TM, TPG, KS, map);
    if (mode == 2) return pick_b2(TM, TPG, KS, map);
    if (mode == 3) return pick_b3(TM, TPG, KS, map);
    return pick_b0(TM, TPG, KS, map);
}

}  // namespace fwd

// Output rows of the filters that whole-width row pruning removed: every element is
// the epilogue of a zero sum (bias, ReLU, rounding), as the forward kernels would write
// it.  A workgroup walks planes (image, pruned row) of `plane` contiguous elements;
// 16-byte stores where the plane allows them.  Tiles packed for another plan (header
// check): the list of pruned rows is not read; rows R - n_pruned .. R - 1 get NaN,
// the forward kernel fills the others with NaN, so the whole output is NaN.
__device__ __forceinline__ int fill_row(const int32_t *pruned, bool ok, int R, int n_pruned, int j) {
    return ok ? pruned[j] : R - n_pruned + j;
}
template <typename E>
__device__ __forceinline__ E fill_value(bool ok, const float *bias, int o, int relu) {
    const float v = ok ? fwd::epi(0.f, bias ? bias[o] : 0.f, relu) : __builtin_nanf("");
    if constexpr (sizeof(E) == 2) return (E)fwd::f32_to_bf16_rne(v);
    else return v;
}
// Planes smaller than a workgroup (small images): one thread per element of the
// flattened (plane, element) range, fewer than 2^32 elements.
template <typename E>
__global__ void k_fill_pruned_small(E *__restrict__ y, const uint8_t *__restrict__ tiles, int64_t off_pruned,
                                    uint32_t fp_lo, uint32_t fp_hi, const float *__restrict__ bias, int relu, int R,
                                    int n_pruned, uint32_t total, uint32_t plane, int64_t img_stride,
                                    int64_t ch_stride) {
    const TileHeader *hdr = (const TileHeader *)tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == fp_lo && hdr->fp_hi == fp_hi;
    const int32_t *pruned = (const int32_t *)(tiles + off_pruned);
    for (uint32_t idx = blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += gridDim.x * blockDim.x) {
        const uint32_t pi = idx / plane, e = idx - pi * plane;
        const uint32_t img = pi / (uint32_t)n_pruned, j = pi - img * (uint32_t)n_pruned;
        const int o = fill_row(pruned, ok, R, n_pruned, (int)j);
        if (o < 0 || o >= R) continue;   // not a row of the output
        y[(int64_t)img * img_stride + (int64_t)o * ch_stride + e] = fill_value<E>(ok, bias, o, relu);
    }
}
template <typename E>
__global__ void k_fill_pruned(E *__restrict__ y, const uint8_t *__restrict__ tiles, int64_t off_pruned, uint32_t fp_lo,
                              uint32_t fp_hi, const float *__restrict__ bias, int relu, int R, int n_pruned,
                              int64_t n_planes, int64_t plane, int64_t img_stride, int64_t ch_stride) {
    constexpr int VE = 16 / (int)sizeof(E);
    const TileHeader *hdr = (const TileHeader *)tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == fp_lo && hdr->fp_hi == fp_hi;
    const int32_t *pruned = (const int32_t *)(tiles + off_pruned);
    for (int64_t pi = blockIdx.x; pi < n_planes; pi += gridDim.x) {
        const int64_t img = pi / n_pruned;
        const int j = (int)(pi - img * n_pruned);
        const int o = fill_row(pruned, ok, R, n_pruned, j);
        if (o < 0 || o >= R) continue;   // not a row of the output
        const E ev = fill_value<E>(ok, bias, o, relu);
        E *base = y + img * img_stride + (int64_t)o * ch_stride;
        if (((uintptr_t)base & 15) == 0 && plane % VE == 0) {
            union { E e[VE]; uint4 u; } w;
#pragma unroll
            for (int k = 0; k < VE; ++k) w.e[k] = ev;
            uint4 *b4 = (uint4 *)base;
            for (int64_t k = threadIdx.x; k < plane / VE; k += blockDim.x) b4[k] = w.u;
        } else {
            for (int64_t k = threadIdx.x; k < plane; k += blockDim.x) base[k] = ev;
        }
    }
}

static hipError_t launch_fill_pruned(const Plan &p, int64_t n_img, int64_t plane, int64_t img_stride,
                                     int64_t ch_stride, const uint8_t *tiles, const float *bias, int relu,
                                     int out_bf16, void *y, hipStream_t st) {
    const int n_pruned = p.R - p.RK;
    const int64_t n_planes = n_img * n_pruned;
    if (!p.rowmap || n_planes <= 0 || plane <= 0) return hipSuccess;
    const uint32_t lo = (uint32_t)p.fingerprint, hi = (uint32_t)(p.fingerprint >> 32);
    const int64_t total = n_planes * plane;
    if (plane < 256 && total < ((int64_t)1 << 32)) {
        const int g = (int)std::min<int64_t>((total + 255) / 256, 16384);
        if (out_bf16)
            k_fill_pruned_small<uint16_t><<<g, 256, 0, st>>>((uint16_t *)y, tiles, p.off_pruned, lo, hi, bias, relu,
                                                             p.R, n_pruned, (uint32_t)total, (uint32_t)plane,
                                                             img_stride, ch_stride);
        else
            k_fill_pruned_small<float><<<g, 256, 0, st>>>((float *)y, tiles, p.off_pruned, lo, hi, bias, relu, p.R,
                                                          n_pruned, (uint32_t)total, (uint32_t)plane, img_stride,
                                                          ch_stride);
        return hipGetLastError();
    }
    const int grid = (int)std::min<int64_t>(n_planes, 16384);
    if (out_bf16)
        k_fill_pruned<uint16_t><<<grid, 256, 0, st>>>((uint16_t *)y, tiles, p.off_pruned, lo, hi, bias, relu, p.R,
                                                      n_pruned, n_planes, plane, img_stride, ch_stride);
    else
        k_fill_pruned<float><<<grid, 256, 0, st>>>((float *)y, tiles, p.off_pruned, lo, hi, bias, relu, p.R,
                                                   n_pruned, n_planes, plane, img_stride, ch_stride);
    return hipGetLastError();
}

static hipError_t workspace(size_t bytes, void **out);

// Sum of the K parts' fp32 partial sums (at most 16 parts), then bias, ReLU and
// rounding: one element of y per thread (output channel (i / plane) % R; fewer than
// 2^31 elements), the loads of every part issued before they are summed, so a thread
// waits once.
template <typename E>
__global__ void k_splitk_sum(const float *__restrict__ part, int ks, int64_t stride, uint32_t total,
                             FastDiv div_plane, FastDiv div_R, const float *__restrict__ bias, int relu,
                             E *__restrict__ y) {
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        float t[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) t[k] = k < ks ? part[(int64_t)k * stride + i] : 0.f;
        float v = 0.f;
#pragma unroll
        for (int k = 0; k < 16; ++k) v += t[k];
        const uint32_t q = fdiv(i, div_plane);
        const uint32_t o = q - fdiv(q, div_R) * div_R.d;
        const float r = fwd::epi(v, bias ? bias[o] : 0.f, relu);
        if constexpr (sizeof(E) == 2) y[i] = (E)fwd::f32_to_bf16_rne(r);
        else y[i] = r;
    }
}

// 4-pixel groups of a pointwise layer for n images (vectors), as launch_pw numbers them.
static int64_t pw_groups(const Plan &p, int n) {
    if (p.is_linear) return div_up64(div_up(n, 4), p.gpg) * p.gpg;
    if (p.SW == 1) return (int64_t)n * (div_up64(div_up(p.H * p.W, 4), p.gpg) * p.gpg);
    return (int64_t)n * p.Ho * div_up(p.Wo, 4);
}

// K-loop split of the pipelined kernel for n images: with at most half as many (tile,
// m-block) pairs as CUs, the steps are split into ks parts (at least 2 steps each, up
// to 16 parts, at most one workgroup per CU: the kernel holds a CU's LDS) whose fp32
// partial sums a second kernel adds.
struct PwSplit {
    int ks, s_per;
    int64_t yelems;   // elements of y (the stride between parts)
};
static PwSplit pw_split(const Plan &p, int n) {
    PwSplit r{1, p.S, 0};
    if (!p.pl || p.rowmap || n <= 0) return r;
    const int64_t n_pt = div_up64(pw_groups(p, n), (int64_t)kGroups * p.NSUB);
    const int64_t units = n_pt * p.n_mb;
    if (units > 128 || p.S < 4) return r;
    int ks = (int)std::min<int64_t>(16, 256 / units);
    ks = std::min(ks, p.S / 2);
    const int s_per = div_up(p.S, ks);
    ks = div_up(p.S, s_per);
    if (ks < 2) return r;
    r.ks = ks;
    r.s_per = s_per;
    r.yelems = p.is_linear ? (int64_t)p.R * n
                           : (int64_t)n * p.R * (p.SW == 1 ? (int64_t)p.H * p.W : (int64_t)p.Ho * p.Wo);
    return r;
}

size_t pw_part_bytes(const Plan &p, int n) {
    const PwSplit sp = pw_split(p, n);
    return sp.ks > 1 ? (size_t)sp.ks * sp.yelems * sizeof(float) : 0;
}

static int log2_int(int v) {
    int l = 0;
    while ((1 << l) < v) ++l;
    return l;
}

// Pointwise layers: the image (stride 1) or each output row (stride 2) is a run of
// 4-pixel groups; a linear layer's batch is one image of n pixels.
static hipError_t launch_pw(const Plan &p, int n, const void *x, const uint8_t *tiles, const float *bias,
                            int relu, int out_bf16, void *y, hipStream_t st, void *part) {
    PwArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.y = y;
    a.tiles = tiles;
    a.bias = bias;
    a.relu = relu;
    a.out_bf16 = out_bf16;
    a.R = p.RK;
    a.Rout = p.R;
    a.Cin = p.Cin;
    a.SMAX = p.SMAX;
    a.rowmap = p.rowmap ? (const int32_t *)(tiles + p.off_rowmap) : nullptr;
    a.SW = p.SW;
    int64_t images;
    if (p.is_linear) {
        images = 1;
        a.Ho = 1; a.Wo = n; a.in_row = 0;
        a.x_cs = n; a.y_cs = n; a.x_is = 0; a.y_is = 0;
    } else if (p.SW == 1) {
        images = n;
        a.Ho = 1; a.Wo = p.H * p.W; a.in_row = 0;
        a.x_cs = p.xplane ? p.xplane : (int64_t)p.H * p.W; a.y_cs = (int64_t)p.H * p.W;
        a.x_is = (int64_t)p.Cin * a.x_cs; a.y_is = (int64_t)p.R * a.y_cs;
    } else {
        images = n;
        a.Ho = p.Ho; a.Wo = p.Wo; a.in_row = p.SH * p.W;
        a.x_cs = (int64_t)p.H * p.W; a.y_cs = (int64_t)p.Ho * p.Wo;
        a.x_is = (int64_t)p.Cin * a.x_cs; a.y_is = (int64_t)p.R * a.y_cs;
    }
    a.GPR = p.SW == 1 ? (div_up(a.Wo, 4) + p.gpg - 1) / p.gpg * p.gpg : div_up(a.Wo, 4);
    a.x_total = (p.is_linear ? (int64_t)p.Cin * n : images * a.x_is);
    a.n_groups_total = images * a.Ho * a.GPR;
    const int64_t n_pt = div_up64(a.n_groups_total, (int64_t)kGroups * p.NSUB);
    if (n_pt <= 0) return hipSuccess;
    // persistent workgroups: about occ per CU; each walks a range of pixel tiles of
    // its m-block (one tile when the waves split the steps)
    int64_t wpm = std::max<int64_t>(1, div_up64((int64_t)256 * p.occ, p.n_mb));
    const PwSplit sp = pw_split(p, n);
    if (p.KS > 1 || sp.ks > 1 || wpm > n_pt) wpm = n_pt;
    const int64_t tpw = div_up64(n_pt, wpm);
    const int64_t gv = div_up64(n_pt, tpw) * p.n_mb;
    if (gv * sp.ks > INT32_MAX - 8 || n_pt > INT32_MAX || images * a.Ho > INT32_MAX ||
        a.n_groups_total + kGroups * 4 > INT32_MAX)
        return hipErrorInvalidValue;
    // a split K loop: the kernel stores fp32 partial sums (no bias, ReLU or rounding)
    a.ks = sp.ks;
    a.s_per = sp.s_per;
    a.kpart_wgs = (int)gv;
    a.div_kpart = make_fastdiv((uint32_t)gv);
    a.part_stride = sp.yelems;
    if (sp.ks > 1) {
        if (!part) {
            hipError_t e = workspace((size_t)sp.ks * sp.yelems * sizeof(float), &part);
            if (e != hipSuccess) return e;
        }
        a.y = part;
        a.out_bf16 = 0;
        a.bias = nullptr;
        a.relu = 0;
    }
    a.n_pt = (int)n_pt;
    a.tiles_per_wg = (int)tpw;
    a.NSUB = p.NSUB; a.lg_nsub = log2_int(p.NSUB);
    a.NGR = p.NGR; a.lg_ngr = log2_int(p.NGR);
    a.gpg = p.gpg; a.FR = p.FR;
    a.n_groups = p.n_groups; a.group_rows = p.group_rows; a.mt_per_group = p.mt_per_group;
    a.LP = p.LP; a.S = p.S;
    a.MBT = p.MBT; a.MBG = p.MBG; a.n_mb = p.n_mb; a.resident = p.resident; a.NB = p.NB;
    a.lds_d = p.lds_d; a.lds_a = p.lds_a; a.lds_patch = p.lds_patch; a.lds_astage = p.lds_astage;
    a.lds_buf = p.lds_buf;
    a.grid_valid = (int)(gv * sp.ks);
    a.off_chunks = p.off_chunks;
    a.off_desc16 = p.off_desc16;
    a.off_a = p.off_a;
    a.fp_lo = (uint32_t)p.fingerprint;
    a.fp_hi = (uint32_t)(p.fingerprint >> 32);
    a.div_GPR = make_fastdiv((uint32_t)a.GPR);
    a.div_Ho = make_fastdiv((uint32_t)a.Ho);
    a.div_nmb = make_fastdiv((uint32_t)p.n_mb);
    pw::pw_fn fn = nullptr;
    const bool map = p.rowmap != 0;
    int threads = kThreads;
    if (p.pl) {
        if (p.dt == BSP_BF16)
            fn = !p.shared ? (p.SW == 1 ? pl::pick_g(p.NSUB, p.TM, p.MBG) : nullptr)
                           : (p.SW == 1 ? pl::pick_1(p.NSUB, p.TM, map) : pl::pick_2(p.NSUB, p.TM, map));
        threads = pl::kPlThreads;
    } else if (p.dt == BSP_F32) {
        fn = p.SW == 1 ? pw::pick_f(p.TM, p.TPG, p.KS, map) : nullptr;
    } else {
        fn = p.SW == 1 ? pw::pick_b1(p.TM, p.TPG, p.KS, map) : pw::pick_b2(p.TM, p.TPG, p.KS, map);
    }
    if (!fn) return hipErrorInvalidValue;
    const int grid = (int)(div_up64(gv * sp.ks, 8) * 8);
    if (p.lds_total > 48 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           p.lds_total);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fn, dim3(grid), dim3(threads), (size_t)p.lds_total, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (sp.ks > 1) {
        const uint32_t total = (uint32_t)sp.yelems;   // the API keeps y below 2^31 elements
        const int64_t plane = p.is_linear ? n : a.y_cs;
        const int g = (int)std::min<int64_t>((sp.yelems + 255) / 256, 65536);
        if (out_bf16)
            k_splitk_sum<uint16_t><<<g, 256, 0, st>>>((const float *)part, sp.ks, sp.yelems, total,
                                                      make_fastdiv((uint32_t)plane), make_fastdiv((uint32_t)p.R),
                                                      bias, relu, (uint16_t *)y);
        else
            k_splitk_sum<float><<<g, 256, 0, st>>>((const float *)part, sp.ks, sp.yelems, total,
                                                   make_fastdiv((uint32_t)plane), make_fastdiv((uint32_t)p.R), bias,
                                                   relu, (float *)y);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return launch_fill_pruned(p, images, a.y_cs, a.y_is, a.y_cs, tiles, bias, relu, out_bf16, y, st);
}

hipError_t launch_conv(const Plan &p, int n, const void *x, const uint8_t *tiles, const float *bias,
                       int relu, int out_bf16, void *y, hipStream_t st, void *part) {
    if (p.pw) return launch_pw(p, n, x, tiles, bias, relu, out_bf16, y, st, part);
    if (stem_ok(p, x)) return launch_stem(p, n, x, tiles, bias, relu, out_bf16, y, st);
    ConvArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.y = y;
    a.tiles = tiles;
    a.bias = bias;
    a.relu = relu;
    a.out_bf16 = out_bf16;
    a.Cin = p.Cin; a.R = p.RK; a.Rout = p.R;
    a.rowmap = p.rowmap ? (const int32_t *)(tiles + p.off_rowmap) : nullptr;
    a.KH = p.KH; a.KW = p.KW; a.SH = p.SH; a.SW = p.SW; a.PH = p.PH; a.PW = p.PW;
    if (p.is_linear) {
        // batch n vectors of a feature-major [C][n] matrix: rows of 64 vectors
        const int rows = div_up(n, kLinRow);
        a.N = 1; a.H = rows; a.W = kLinRow; a.Ho = rows; a.Wo = kLinRow;
        a.x_cs = n; a.y_cs = n;
        a.w_last = n - (rows - 1) * kLinRow;
        a.w_last_out = a.w_last;
    } else {
        a.N = n; a.H = p.H; a.W = p.W; a.Ho = p.Ho; a.Wo = p.Wo;
        a.x_cs = (int64_t)p.H * p.W; a.y_cs = (int64_t)p.Ho * p.Wo;
        a.w_last = p.W;
        a.w_last_out = p.Wo;
    }
    a.x_total = (int64_t)a.N * a.Cin * a.x_cs;
    a.GPR = p.GPR; a.NSUB = p.NSUB; a.NSLOT = p.NSLOT; a.LEFT = p.LEFT; a.RS = p.RS; a.RG = p.RG;
    a.CH_STRIDE = p.CH_STRIDE; a.CC = p.CC; a.GE = p.GE; a.FR = p.FR;
    a.n_groups = p.n_groups; a.group_rows = p.group_rows; a.mt_per_group = p.mt_per_group;
    a.LP = p.LP; a.S = p.S;
    a.KS = p.KS; a.MBT = p.MBT; a.MBG = p.MBG; a.n_mb = p.n_mb;
    a.resident = p.resident;
    a.NB = p.NB;
    a.lds_d = p.lds_d; a.lds_a = p.lds_a; a.lds_patch = p.lds_patch; a.lds_astage = p.lds_astage;
    a.lds_buf = p.lds_buf;
    a.n_groups_total = (int64_t)a.N * a.Ho * p.GPR;
    const int64_t n_pt = div_up64(a.n_groups_total, (int64_t)kGroups * p.NSUB);
    if (n_pt <= 0) return hipSuccess;
    // persistent workgroups: about one wave of workgroups over the chip; each walks a
    // range of pixel tiles of its m-block (one tile when waves split the steps)
    const int occ = std::max(1, std::min(fwd_occ(p.gather, p.TM, p.TPG), (160 * 1024) / (p.lds_total + kLdsStatic)));
    int64_t wpm = std::max<int64_t>(1, div_up64((int64_t)256 * occ, p.n_mb));
    if (p.KS > 1 || wpm > n_pt) wpm = n_pt;
    const int64_t tpw = div_up64(n_pt, wpm);
    if (tpw > INT32_MAX) return hipErrorInvalidValue;
    const int64_t gv = div_up64(n_pt, tpw) * p.n_mb;
    if (gv > INT32_MAX - 8 || (int64_t)a.N * a.Ho > INT32_MAX / 2 || a.n_groups_total > INT32_MAX)
        return hipErrorInvalidValue;
    a.n_pt = (int)n_pt;
    a.tiles_per_wg = (int)tpw;
    a.grid_valid = (int)gv;
    a.off_chunks = p.off_chunks;
    a.off_desc16 = p.off_desc16;
    a.off_a = p.off_a;
    a.fp_lo = (uint32_t)p.fingerprint;
    a.fp_hi = (uint32_t)(p.fingerprint >> 32);
    a.div_GPR = make_fastdiv((uint32_t)p.GPR);
    a.div_Ho = make_fastdiv((uint32_t)a.Ho);
    a.div_RG = make_fastdiv((uint32_t)p.RG);

    a.VSG = p.NSLOT * p.RG;
    a.CHG = p.V * a.VSG;
    a.V = p.V;
    a.POFF = p.POFF;
    a.div_CHG = make_fastdiv((uint32_t)a.CHG);
    a.div_VSG = make_fastdiv((uint32_t)a.VSG);
    a.div_nmb = make_fastdiv((uint32_t)p.n_mb);
    fwd::fwd_fn fn = fwd::pick(p.dt, p.gather, p.TM, p.TPG, p.KS, p.rowmap != 0);
    if (!fn) return hipErrorInvalidValue;
    const int grid = (int)(div_up64(gv, 8) * 8);
    if (p.lds_total > 48 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           p.lds_total);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kFwdThreads), (size_t)p.lds_total, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // images of the output: conv NCHW planes of Ho * Wo; linear one [R][n] matrix
    return launch_fill_pruned(p, a.N, p.is_linear ? n : a.y_cs, (int64_t)p.R * a.y_cs, a.y_cs, tiles, bias,
                              relu, out_bf16, y, st);
}

// im2col of a conv for its 1x1 plan: ws[img][k][p], k = (c * kh + r) * kw + s (the GEMM
// form's column), p = oh * wo + ow; taps outside the image are zero.  One thread per
// element of the expanded input (fewer than 2^31).
template <typename E>
__global__ void k_im2col(const E *__restrict__ x, E *__restrict__ ws, int total, int cols, int cin, int h, int w,
                         int kh, int kw, int sh, int sw, int ph, int pw, int ho, int wo) {
    const int plane = ho * wo, khw = kh * kw;
    for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += gridDim.x * blockDim.x) {
        const int pix = idx % plane, k = (idx / plane) % cols, img = idx / (plane * cols);
        const int c = k / khw, rs = k - c * khw, r = rs / kw, s = rs - r * kw;
        const int oh = pix / wo, ow = pix - oh * wo;
        const int ih = oh * sh - ph + r, iw = ow * sw - pw + s;
        ws[idx] = (ih >= 0 && ih < h && iw >= 0 && iw < w) ? x[(((int64_t)img * cin + c) * h + ih) * w + iw] : (E)0;
    }
}

// As k_im2col for planes padded to whole 16-byte granules (xplane elements, a multiple
// of GE = 16 / sizeof(E)): one thread per granule of a row (img, k) of the expanded
// input (fewer than 2^31 granules), GE loads and one 16-byte store; padding elements
// are zero.  Divisions by the layer's sizes are multiply-shifts.
struct Im2colArgs {
    uint32_t n_gran;              // granules of the expanded input
    int cin, h, w, kh, kw, sh, sw, ph, pw, ho, wo, xplane;
    FastDiv div_gpr, div_cols, div_khw, div_kw, div_wo;
};

template <typename E>
__global__ void k_im2col_g(const E *__restrict__ x, E *__restrict__ ws, Im2colArgs a) {
    constexpr int GE = 16 / sizeof(E);
    const int plane = a.ho * a.wo, gpr = a.xplane / GE;
    for (uint32_t idx = blockIdx.x * blockDim.x + threadIdx.x; idx < a.n_gran; idx += gridDim.x * blockDim.x) {
        const uint32_t row = fdiv(idx, a.div_gpr);
        const int g = (int)(idx - row * (uint32_t)gpr);
        const uint32_t img = fdiv(row, a.div_cols);
        const int k = (int)(row - img * a.div_cols.d);
        const int c = (int)fdiv((uint32_t)k, a.div_khw), rs = k - c * a.kh * a.kw;
        const int r = (int)fdiv((uint32_t)rs, a.div_kw), s = rs - r * a.kw;
        const E *xc = x + ((int64_t)img * a.cin + c) * a.h * a.w;
        int pix = g * GE;
        int oh = (int)fdiv((uint32_t)pix, a.div_wo), ow = pix - oh * a.wo;
        E v[GE];
#pragma unroll
        for (int e = 0; e < GE; ++e) {
            const int ih = oh * a.sh - a.ph + r, iw = ow * a.sw - a.pw + s;
            v[e] = (pix < plane && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w) ? xc[ih * a.w + iw] : (E)0;
            ++pix;
            if (++ow == a.wo) { ow = 0; ++oh; }
        }
        *(uint4 *)(ws + (int64_t)row * a.xplane + g * GE) = *(const uint4 *)v;
    }
}

// One workspace per device, grown on demand and kept until the process ends.  Layers on
// the im2col path share it, so such calls that overlap on one device (other streams) race.
static hipError_t workspace(size_t bytes, void **out) {
    static std::mutex mu;
    static void *buf[64] = {};
    static size_t size[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (size[dev] < bytes) {
        if (buf[dev]) {
            e = hipFree(buf[dev]);
            buf[dev] = nullptr;
            size[dev] = 0;
            if (e != hipSuccess) return e;
        }
        e = hipMalloc(&buf[dev], bytes);
        if (e != hipSuccess) {
            buf[dev] = nullptr;
            return e;
        }
        size[dev] = bytes;
    }
    *out = buf[dev];
    return hipSuccess;
}

hipError_t launch_conv_im2col(const Plan &p, const bsp_conv_shape &c, const void *x, const uint8_t *tiles,
                              const float *bias, int relu, int out_bf16, void *y, hipStream_t st) {
    // the 1x1 plan: Cin = cin kh kw, H x W = Ho x Wo, planes of xplane elements when padded
    const int64_t plane = p.xplane ? p.xplane : (int64_t)p.H * p.W;
    const int64_t total = (int64_t)c.n * p.Cin * plane;
    if (total <= 0) return hipSuccess;
    if (total > INT32_MAX) return hipErrorInvalidValue;
    // one workspace: the expanded input, then the partial sums of a split K loop
    const size_t in_bytes = ((size_t)total * p.esize + 255) / 256 * 256;
    const size_t part_bytes = pw_part_bytes(p, c.n);
    void *ws = nullptr;
    hipError_t e = workspace(in_bytes + part_bytes, &ws);
    if (e != hipSuccess) return e;
    void *part = part_bytes ? (void *)((unsigned char *)ws + in_bytes) : nullptr;
    if (p.xplane) {
        Im2colArgs ia;
        ia.n_gran = (uint32_t)(total / (16 / p.esize));
        ia.cin = c.cin; ia.h = c.h; ia.w = c.w; ia.kh = c.kh; ia.kw = c.kw;
        ia.sh = c.stride_h; ia.sw = c.stride_w; ia.ph = c.pad_h; ia.pw = c.pad_w;
        ia.ho = p.H; ia.wo = p.W; ia.xplane = p.xplane;
        ia.div_gpr = make_fastdiv((uint32_t)(p.xplane / (16 / p.esize)));
        ia.div_cols = make_fastdiv((uint32_t)p.Cin);
        ia.div_khw = make_fastdiv((uint32_t)(c.kh * c.kw));
        ia.div_kw = make_fastdiv((uint32_t)c.kw);
        ia.div_wo = make_fastdiv((uint32_t)p.W);
        const int grid = (int)std::min<int64_t>(((int64_t)ia.n_gran + 255) / 256, 65536);
        if (p.esize == 2)
            k_im2col_g<uint16_t><<<grid, 256, 0, st>>>((const uint16_t *)x, (uint16_t *)ws, ia);
        else
            k_im2col_g<float><<<grid, 256, 0, st>>>((const float *)x, (float *)ws, ia);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        return launch_conv(p, c.n, ws, tiles, bias, relu, out_bf16, y, st, part);
    }
    const int grid = (int)std::min<int64_t>((total + 255) / 256, 16384);
    if (p.esize == 2)
        k_im2col<uint16_t><<<grid, 256, 0, st>>>((const uint16_t *)x, (uint16_t *)ws, (int)total, p.Cin, c.cin, c.h,
                                                 c.w, c.kh, c.kw, c.stride_h, c.stride_w, c.pad_h, c.pad_w, p.H, p.W);
    else
        k_im2col<float><<<grid, 256, 0, st>>>((const float *)x, (float *)ws, (int)total, p.Cin, c.cin, c.h, c.w,
                                              c.kh, c.kw, c.stride_h, c.stride_w, c.pad_h, c.pad_w, p.H, p.W);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_conv(p, c.n, ws, tiles, bias, relu, out_bf16, y, st, part);
}

}  // namespace bsp
