// Forward of block-pruned conv / FC layers on gfx950: implicit GEMM over the kept
// columns only.
//
// What is computed (Sec. 4.2, layer i with pruned weights): for every output pixel
// and every output row o, the sum over the kept GEMM columns q = (c, r, s) of o's
// list of W[o, q] * x[n, c, oh*sh - ph + r, ow*sw - pw + s], plus bias, then ReLU.
//
// How.  A persistent workgroup (4 waves) owns one m-block of output rows and walks a
// contiguous range of pixel tiles (NSUB stacked sub-tiles of 64 outputs).  Its work
// items are (tile, chunk); items are double buffered in LDS:
//  * fill: the input patch x[n, c_lo .. c_lo+cnt, staged rows, columns] of the next
//    item is copied with asynchronous direct-to-LDS loads (global_load_lds, 16- or
//    4-byte granules, lane-linear destinations; padding and out-of-image rows read a
//    zero block in the tile header; odd-width rows use batched register loads).  When
//    the m-block's weights and gather offsets do not stay resident in LDS, the item's
//    slice of them is copied the same way.
//  * compute: each wave walks its lists in steps of 32 kept columns.  Lane l owns
//    kept positions 8*(l/16) .. +7 and the 4 horizontally adjacent pixels
//    4*(l%16) .. +3 of its sub-tile: per kept column one 8-byte LDS read (stride 1;
//    16 bytes for stride 2) at the pre-decoded 16-bit offset plus the pixel offset,
//    then v_perm re-packs the 8 x 4 values into the B operands of 4 MFMAs (one per
//    pixel of the group).  Weights (A operand) are read from LDS, 16 bytes per lane,
//    and reused across the 4 pixel n-tiles; a list shared by several m-tiles (row
//    pruning, dense) also reuses the gathered B operands across them.
//  * epilogue (deferred by one item so its stores overlap the next fill and compute):
//    bias + ReLU + round-to-nearest-even bf16 (or fp32); each lane writes 4 adjacent
//    pixels of 4 output rows with 8-byte stores.
// Workgroup ids are remapped so that the workgroups of one pixel range (all its
// m-blocks) run on the same XCD and share its L2.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "bsp_kernels.h"

namespace bsp {

typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

namespace {

__device__ __forceinline__ uint32_t perm(uint32_t hi_src, uint32_t lo_src, uint32_t sel) {
    return __builtin_amdgcn_perm(hi_src, lo_src, sel);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    __bf16 h = (__bf16)f;
    return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void lds_load16(const void *src, unsigned char *dst) {
    __builtin_amdgcn_global_load_lds(src, (lds_void_t *)dst, 16, 0, 0);
}
__device__ __forceinline__ void lds_load4(const void *src, unsigned char *dst) {
    __builtin_amdgcn_global_load_lds(src, (lds_void_t *)dst, 4, 0, 0);
}

// Dense copy of n16 16-byte granules into LDS: granule q lands at dst + 16 q; its
// source is src_of(q).  One wave instruction moves 64 consecutive granules.
template <typename F>
__device__ __forceinline__ void copy_granules(unsigned char *dst, int n16, F src_of) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int q0 = wave * 64; q0 < n16; q0 += kThreads) {
        const int q = q0 + lane;
        if (q < n16) lds_load16(src_of(q), dst + (size_t)q0 * 16);
    }
}

// Patch fill.  Granule v (GB bytes) of the patch lands at byte v*GB.
template <typename E, int GB>
__device__ __forceinline__ void fill_patch_direct(const ConvArgs &a, unsigned char *patch,
                                                  const int *s_img, const int *s_ih, int c_lo,
                                                  int c_cnt, int a0) {
    constexpr int GE = GB / (int)sizeof(E);
    const int NV = a.RL / GE;
    const int total = c_cnt * a.NSLOT * NV;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const unsigned char *x = (const unsigned char *)a.x;
    const unsigned char *zero = a.tiles + kZeroOffset;
    for (int v0 = wave * 64; v0 < total; v0 += kThreads) {
        const int v = v0 + lane;
        if (v < total) {
            const int row = (int)fdiv((uint32_t)v, a.div_nv);
            const int vi = v - row * NV;
            const int c = (int)fdiv((uint32_t)row, a.div_nslot);
            const int sl = row - c * a.NSLOT;
            const int ih = s_ih[sl];
            const int iw = a0 + vi * GE;
            const unsigned char *src = zero;
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                src = x + (((size_t)(s_img[sl] * a.Cin + c_lo + c) * a.H + ih) * a.W + iw) * sizeof(E);
            if constexpr (GB == 16) lds_load16(src, patch + (size_t)v0 * GB);
            else lds_load4(src, patch + (size_t)v0 * GB);
        }
    }
}

// Register-path patch fill (2-byte elements of odd-width rows): 8 loads in flight
// per thread before the LDS stores.
__device__ __forceinline__ void fill_patch_regs(const ConvArgs &a, uint16_t *patch, const int *s_img,
                                                const int *s_ih, int c_lo, int c_cnt, int a0) {
    const int NV = a.RL;
    const int total = c_cnt * a.NSLOT * NV;
    const uint16_t *x = (const uint16_t *)a.x;
    for (int v0 = threadIdx.x; v0 < total; v0 += kThreads * 8) {
        uint16_t val[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int v = v0 + k * kThreads;
            val[k] = 0;
            if (v < total) {
                const int row = (int)fdiv((uint32_t)v, a.div_nv);
                const int iw = a0 + (v - row * NV);
                const int c = (int)fdiv((uint32_t)row, a.div_nslot);
                const int sl = row - c * a.NSLOT;
                const int ih = s_ih[sl];
                if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                    val[k] = x[((size_t)(s_img[sl] * a.Cin + c_lo + c) * a.H + ih) * a.W + iw];
            }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int v = v0 + k * kThreads;
            if (v < total) patch[v] = val[k];
        }
    }
}

template <typename E>
__device__ __forceinline__ void fill_patch(const ConvArgs &a, unsigned char *patch, const int *s_img,
                                           const int *s_ih, int c_lo, int c_cnt, int a0) {
    if (a.gran == 16) fill_patch_direct<E, 16>(a, patch, s_img, s_ih, c_lo, c_cnt, a0);
    else if (a.gran == 4) fill_patch_direct<E, 4>(a, patch, s_img, s_ih, c_lo, c_cnt, a0);
    else fill_patch_regs(a, (uint16_t *)patch, s_img, s_ih, c_lo, c_cnt, a0);
}

// ---- operand gathers -------------------------------------------------------------
// v[j] holds pixels 0..3 (16 bits each) of kept column j of this lane; B[nt] is the
// 8-wide k-vector of pixel nt.
__device__ __forceinline__ void repack_bf16(const uint2 *v, s16x8 *B) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint2 lo = v[2 * d], hi = v[2 * d + 1];
        ((uint32_t *)&B[0])[d] = perm(hi.x, lo.x, 0x05040100u);
        ((uint32_t *)&B[1])[d] = perm(hi.x, lo.x, 0x07060302u);
        ((uint32_t *)&B[2])[d] = perm(hi.y, lo.y, 0x05040100u);
        ((uint32_t *)&B[3])[d] = perm(hi.y, lo.y, 0x07060302u);
    }
}

__device__ __forceinline__ void offsets(uint4 d, int pixoff, int *ad) {
    ad[0] = (int)(d.x & 0xffffu) + pixoff; ad[1] = (int)(d.x >> 16) + pixoff;
    ad[2] = (int)(d.y & 0xffffu) + pixoff; ad[3] = (int)(d.y >> 16) + pixoff;
    ad[4] = (int)(d.z & 0xffffu) + pixoff; ad[5] = (int)(d.z >> 16) + pixoff;
    ad[6] = (int)(d.w & 0xffffu) + pixoff; ad[7] = (int)(d.w >> 16) + pixoff;
}

// Gathers, split in two halves so that the LDS reads of the next stage can be in
// flight while the current stage re-packs and multiplies.  MODE 1: stride 1 (one
// 8-byte read per kept column, 16 bytes for fp32), MODE 2: stride 2 (16-byte reads,
// even elements), MODE 0: any stride (one read per element).
template <typename E, int MODE>
struct Gat;

template <int MODE>
struct Gat<uint16_t, MODE> {
    typedef typename std::conditional<MODE == 2, uint4, uint2>::type R1;
    struct Raw { R1 v[8]; };
    typedef uint4 AReg;
    static __device__ __forceinline__ void read(Raw &r, const unsigned char *patch_b, uint4 d, int pixoff,
                                                int SW) {
        const uint16_t *patch = (const uint16_t *)patch_b;
        int ad[8];
        offsets(d, pixoff, ad);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if constexpr (MODE == 0) {
                const uint16_t *p = patch + ad[j];
                r.v[j].x = (uint32_t)p[0] | ((uint32_t)p[SW] << 16);
                r.v[j].y = (uint32_t)p[2 * SW] | ((uint32_t)p[3 * SW] << 16);
            } else {
                __builtin_memcpy(&r.v[j], patch + ad[j], sizeof(R1));
            }
        }
    }
    static __device__ __forceinline__ AReg read_a(const unsigned char *ap) { return *(const uint4 *)ap; }
    struct Frag {
        s16x8 b[4];
    };
    static __device__ __forceinline__ void finish(const Raw &r, Frag &f) {
        uint2 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if constexpr (MODE == 2) {
                v[j].x = perm(r.v[j].y, r.v[j].x, 0x05040100u);
                v[j].y = perm(r.v[j].w, r.v[j].z, 0x05040100u);
            } else {
                v[j] = r.v[j];
            }
        }
        repack_bf16(v, f.b);
    }
    static __device__ __forceinline__ void mma(const AReg &ar, const Frag &f, f32x4 *acc) {
        const s16x8 A = __builtin_bit_cast(s16x8, ar);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, f.b[nt], acc[nt], 0, 0, 0);
    }
};

template <int MODE>
struct Gat<float, MODE> {
    struct Raw { float4 v[8]; };
    struct AReg { float4 lo, hi; };
    static __device__ __forceinline__ void read(Raw &r, const unsigned char *patch_b, uint4 d, int pixoff,
                                                int SW) {
        const float *patch = (const float *)patch_b;
        int ad[8];
        offsets(d, pixoff, ad);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if constexpr (MODE == 1) {
                __builtin_memcpy(&r.v[j], patch + ad[j], 16);
            } else {
                const float *p = patch + ad[j];
                r.v[j] = make_float4(p[0], p[SW], p[2 * SW], p[3 * SW]);
            }
        }
    }
    static __device__ __forceinline__ AReg read_a(const unsigned char *ap) {
        AReg r;
        r.lo = *(const float4 *)ap;
        r.hi = *(const float4 *)(ap + 16);
        return r;
    }
    struct Frag {
        Raw r;
    };
    static __device__ __forceinline__ void finish(const Raw &r, Frag &f) { f.r = r; }
    static __device__ __forceinline__ void mma(const AReg &ar, const Frag &f, f32x4 *acc) {
        const float A[8] = {ar.lo.x, ar.lo.y, ar.lo.z, ar.lo.w, ar.hi.x, ar.hi.y, ar.hi.z, ar.hi.w};
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const float4 &v = f.r.v[u];
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], v.x, acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], v.y, acc[1], 0, 0, 0);
            acc[2] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], v.z, acc[2], 0, 0, 0);
            acc[3] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], v.w, acc[3], 0, 0, 0);
        }
    }
};

__device__ __forceinline__ float epi(float v, float b, int relu) {
    v += b;
    return (relu && v < 0.f) ? 0.f : v;
}

template <int T, int G>
__device__ __forceinline__ void store_tile(const ConvArgs &a, f32x4 (&acc)[G][T][4], bool ok, int gr,
                                           int ow, int gbase, int gcount, int t0, int tcount, int kg) {
    if (gr >= a.N * a.Ho || ow >= a.Wo) return;
    const int img = (int)fdiv((uint32_t)gr, a.div_Ho), oh = gr - img * a.Ho;
    const bool full = (ow + 3 < a.Wo) && ((a.Wo & 3) == 0);
    const size_t plane = (size_t)a.Ho * a.Wo;
    const int row0 = gbase * a.group_rows + t0 * kMT + 4 * kg;   // first row of this lane
    const size_t y0 = ((size_t)img * a.R + row0) * plane + (size_t)oh * a.Wo + ow;
    const float qnan = __builtin_nanf("");
    const bool plain = ok && !a.bias && !a.relu;
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
        if (gi >= gcount) continue;
#pragma unroll
        for (int ti = 0; ti < T; ++ti) {
            if (ti >= tcount) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rig = (t0 + ti) * kMT + 4 * kg + i;
                const int row = row0 + gi * a.group_rows + ti * kMT + i;
                if (rig >= a.group_rows || row >= a.R) continue;
                float o[4];
                if (plain) {
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) o[nt] = acc[gi][ti][nt][i];
                } else {
                    const float bv = a.bias ? a.bias[row] : 0.f;
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) o[nt] = ok ? epi(acc[gi][ti][nt][i], bv, a.relu) : qnan;
                }
                const size_t yo = y0 + (size_t)(gi * a.group_rows + ti * kMT + i) * plane;
                if (a.out_bf16) {
                    uint16_t *y = (uint16_t *)a.y + yo;
                    if (full) {
                        uint2 pk;
                        pk.x = (uint32_t)f32_to_bf16_rne(o[0]) | ((uint32_t)f32_to_bf16_rne(o[1]) << 16);
                        pk.y = (uint32_t)f32_to_bf16_rne(o[2]) | ((uint32_t)f32_to_bf16_rne(o[3]) << 16);
                        *(uint2 *)y = pk;
                    } else {
                        for (int nt = 0; nt < 4; ++nt)
                            if (ow + nt < a.Wo) y[nt] = f32_to_bf16_rne(o[nt]);
                    }
                } else {
                    float *y = (float *)a.y + yo;
                    if (full) {
                        *(float4 *)y = make_float4(o[0], o[1], o[2], o[3]);
                    } else {
                        for (int nt = 0; nt < 4; ++nt)
                            if (ow + nt < a.Wo) y[nt] = o[nt];
                    }
                }
            }
        }
    }
}

template <typename E, int T, int G, int MODE>
__global__ __launch_bounds__(kThreads, 2) void k_conv(ConvArgs a) {
    typedef Gat<E, MODE> GT;
    extern __shared__ __attribute__((aligned(256))) unsigned char lds[];
    __shared__ int s_rowbase[2][kMaxTileRows];
    __shared__ int s_img[2][kMaxSlots];
    __shared__ int s_ih[2][kMaxSlots];
    constexpr int AB = 8 * (int)sizeof(E);   // weight bytes per lane, one m-tile and step
    constexpr int ASTEP = 64 * AB;           // one m-tile, one step

    // workgroup -> (pixel-tile range j, m-block mb); ids remapped so that each XCD
    // (hardware places workgroup id on XCD id % 8) gets a contiguous logical range
    const int per = gridDim.x >> 3;
    const int lid = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (lid >= a.grid_valid) return;
    const int j = lid / a.n_mb, mb = lid - j * a.n_mb;
    const int wt_begin = j * a.tiles_per_wg;
    const int wt_end = min(a.n_wt, wt_begin + a.tiles_per_wg);
    if (wt_begin >= wt_end) return;

    const TileHeader *hdr = (const TileHeader *)a.tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == a.fp_lo && hdr->fp_hi == a.fp_hi;
    const int n_chunks = ok ? hdr->n_chunks : 0;
    const int4 *table = (const int4 *)(a.tiles + a.off_chunks);
    const uint16_t *desc_g = (const uint16_t *)(a.tiles + a.off_desc16);
    const unsigned char *A_g = a.tiles + a.off_a;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n16 = lane & 15, kg = lane >> 4;
    const int sub = wave % a.NSUB, mset = wave / a.NSUB;
    const int tr = sub * a.TRW + (4 * n16) / a.TW;     // row of this lane's pixels in the tile
    const int cx = (4 * n16) % a.TW;

    // this wave's groups / m-tiles, and the m-block's weight range
    int gbase, gcount, t0, tcount, g_first, g_count, mt_first, mt_count;
    if (!a.split) {
        g_first = mb * a.mb_groups;
        g_count = min(a.mb_groups, a.n_groups - g_first);
        gbase = g_first + mset * G;
        gcount = max(0, min(G, a.n_groups - gbase));
        t0 = 0;
        tcount = a.mt_per_group;
        mt_first = g_first * a.mt_per_group;
        mt_count = g_count * a.mt_per_group;
    } else {
        g_first = mb / a.mpg_blocks;
        g_count = 1;
        const int tb = (mb - g_first * a.mpg_blocks) * a.mb_tiles;
        gbase = g_first;
        gcount = 1;
        t0 = tb + mset * T;
        tcount = max(0, min(T, a.mt_per_group - t0));
        mt_first = g_first * a.mt_per_group + tb;
        mt_count = min(a.mb_tiles, a.mt_per_group - tb);
    }
    const bool active = gcount > 0 && tcount > 0;
    // local index (inside the m-block) of this wave's first m-tile and group
    const int m_loc0 = (gbase * a.mt_per_group + t0) - mt_first;
    const int g_loc0 = gbase - g_first;

    unsigned char *A_res = lds;
    unsigned char *D_res = lds + a.lds_a;
    unsigned char *bufs = lds + a.lds_a + a.lds_d;

    if (a.resident && n_chunks > 0) {
        const unsigned char *asrc = A_g + (size_t)mt_first * a.S * ASTEP;
        copy_granules(A_res, mt_count * a.S * ASTEP / 16,
                      [&](int q) { return (const void *)(asrc + (size_t)q * 16); });
        const unsigned char *dsrc = (const unsigned char *)(desc_g + (size_t)g_first * a.LP);
        copy_granules(D_res, g_count * a.LP * 2 / 16,
                      [&](int q) { return (const void *)(dsrc + (size_t)q * 16); });
    }

    // row staging of a workgroup tile into slot buffer sb
    auto setup_slots = [&](int wt, int sb) {
        const int rt = wt / a.n_ct;
        const int g0 = rt * a.TRW * a.NSUB;
        const int rows = a.TRW * a.NSUB, n_rows = a.N * a.Ho;
        if ((int)threadIdx.x < a.NSLOT) {
            s_img[sb][threadIdx.x] = 0;
            s_ih[sb][threadIdx.x] = -1;
        }
        __syncthreads();
        if ((int)threadIdx.x < rows) {
            const int r0 = threadIdx.x, g = g0 + r0;
            int base = 0;
            if (g < n_rows) {
                const int img = (int)fdiv((uint32_t)g, a.div_Ho), oh = g - img * a.Ho;
                const int k = img - (int)fdiv((uint32_t)g0, a.div_Ho);   // image boundaries crossed
                base = (r0 - k) * min(a.SH, a.KH) + k * a.KH;
                for (int r = 0; r < a.KH; ++r) {
                    s_img[sb][base + r] = img;
                    s_ih[sb][base + r] = oh * a.SH - a.PH + r;
                }
            }
            s_rowbase[sb][r0] = base;
        }
        __syncthreads();
    };

    // issue the loads of item (wt, ch) into buffer pb using slot buffer sb
    auto fill = [&](int wt, int ch, int pb, int sb) {
        const int4 cd = table[ch];  // first step, end step, first channel, channel count
        const int ct = wt % a.n_ct;
        const int a0 = ct * a.TW * a.SW - a.PW - a.LEFT;
        unsigned char *buf = bufs + (size_t)pb * a.lds_buf;
        fill_patch<E>(a, buf, s_img[sb], s_ih[sb], cd.z, cd.w, a0);
        if (!a.resident) {
            const int ns = cd.y - cd.x;
            unsigned char *Ai = buf + a.lds_patch;
            const int a16 = ns * ASTEP / 16;   // granules per m-tile
            const unsigned char *asrc = A_g + (size_t)mt_first * a.S * ASTEP + (size_t)cd.x * ASTEP;
            copy_granules(Ai, mt_count * a16, [&](int q) {
                const int m = q / a16, o = q - m * a16;
                return (const void *)(asrc + (size_t)m * a.S * ASTEP + (size_t)o * 16);
            });
            unsigned char *Di = Ai + (size_t)a.mb_tiles * ns * ASTEP;
            const int d16 = ns * 4;            // granules per group (32 x 2 bytes per step)
            const unsigned char *dsrc = (const unsigned char *)(desc_g + (size_t)g_first * a.LP + cd.x * kKS);
            copy_granules(Di, g_count * d16, [&](int q) {
                const int g = q / d16, o = q - g * d16;
                return (const void *)(dsrc + (size_t)g * a.LP * 2 + (size_t)o * 16);
            });
        }
    };

    f32x4 acc[G][T][4];
#pragma unroll
    for (int gi = 0; gi < G; ++gi)
#pragma unroll
        for (int ti = 0; ti < T; ++ti)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[gi][ti][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nch = max(n_chunks, 1);
    const int n_items = (wt_end - wt_begin) * nch;
    if (n_chunks > 0) {
        setup_slots(wt_begin, 0);
        fill(wt_begin, 0, 0, 0);
    }
    int pixoff = 0, ep_gr = 0, ep_ow = 0;
    for (int i = 0; i < n_items; ++i) {
        const int wt = wt_begin + i / nch;
        const int ch = i - (wt - wt_begin) * nch;
        wait_vm_all();
        __syncthreads();
        if (ch == 0) {
            if (i > 0) {
                store_tile<T, G>(a, acc, ok, ep_gr, ep_ow, gbase, gcount, t0, tcount, kg);
#pragma unroll
                for (int gi = 0; gi < G; ++gi)
#pragma unroll
                    for (int ti = 0; ti < T; ++ti)
#pragma unroll
                        for (int nt = 0; nt < 4; ++nt) acc[gi][ti][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            const int sbc = (wt - wt_begin) & 1;
            pixoff = s_rowbase[sbc][tr] * a.RL + cx * a.SW;
            ep_gr = (wt / a.n_ct) * a.TRW * a.NSUB + tr;
            ep_ow = (wt % a.n_ct) * a.TW + cx;
        }
        if (n_chunks == 0) continue;
        const int4 cd = table[ch];   // read before the next item's loads are queued
        if (i + 1 < n_items) {
            const int wt_n = wt_begin + (i + 1) / nch;
            const int ch_n = (i + 1) - (wt_n - wt_begin) * nch;
            const int sbn = (wt_n - wt_begin) & 1;
            if (ch_n == 0) setup_slots(wt_n, sbn);
            fill(wt_n, ch_n, (i + 1) & 1, sbn);
        }
        // compute item i: stages (s, gi) walk a two-deep software pipeline - the
        // gathers and weights of the next stage are read while this stage re-packs
        // and multiplies, and the offsets two stages ahead are read meanwhile
        const int ns = cd.y - cd.x;
        const unsigned char *buf = bufs + (size_t)(i & 1) * a.lds_buf;
        if (active) {
            const uint16_t *Dbase = a.resident
                ? (const uint16_t *)D_res + kg * 8
                : (const uint16_t *)(buf + a.lds_patch + (size_t)a.mb_tiles * ns * ASTEP) + kg * 8;
            const size_t dstr_g = a.resident ? (size_t)a.LP : (size_t)ns * kKS;   // per group
            const int dsoff = a.resident ? 0 : cd.x;                               // step origin
            const unsigned char *Abase = (a.resident ? A_res : buf + a.lds_patch) + lane * AB;
            const size_t astr_m = a.resident ? (size_t)a.S * ASTEP : (size_t)ns * ASTEP;
            auto dptr = [&](int s, int gi) {
                return *(const uint4 *)(Dbase + (size_t)(g_loc0 + gi) * dstr_g + (size_t)(s - dsoff) * kKS);
            };
            auto aptr = [&](int s, int gi, int ti) {
                return GT::read_a(Abase + (size_t)(m_loc0 + gi * a.mt_per_group + ti) * astr_m +
                                  (size_t)(s - dsoff) * ASTEP);
            };
            // weights of the next stage are prefetched too when registers allow
            constexpr bool kPipeA = T * (int)sizeof(E) <= 4;
            typename GT::Raw rn;
            typename GT::AReg an[T];
            uint4 dn;
            {
                const uint4 d0 = dptr(cd.x, 0);
                GT::read(rn, buf, d0, pixoff, a.SW);
                if constexpr (kPipeA)
#pragma unroll
                    for (int ti = 0; ti < T; ++ti)
                        if (ti < tcount) an[ti] = aptr(cd.x, 0, ti);
                int s1 = cd.x, g1 = 1;
                if (g1 >= gcount) { g1 = 0; ++s1; }
                if (s1 < cd.y) dn = dptr(s1, g1);
            }
            for (int s = cd.x; s < cd.y; ++s) {
#pragma unroll
                for (int gi = 0; gi < G; ++gi) {
                    if (gi < gcount) {
                        const typename GT::Raw rc = rn;
                        typename GT::AReg ac[T];
                        if constexpr (kPipeA) {
#pragma unroll
                            for (int ti = 0; ti < T; ++ti) ac[ti] = an[ti];
                        }
                        int sn = s, gn = gi + 1;
                        if (gn >= gcount) { gn = 0; ++sn; }
                        if (sn < cd.y) {
                            GT::read(rn, buf, dn, pixoff, a.SW);
                            if constexpr (kPipeA)
#pragma unroll
                                for (int ti = 0; ti < T; ++ti)
                                    if (ti < tcount) an[ti] = aptr(sn, gn, ti);
                            int snn = sn, gnn = gn + 1;
                            if (gnn >= gcount) { gnn = 0; ++snn; }
                            if (snn < cd.y) dn = dptr(snn, gnn);
                        }
                        typename GT::Frag f;
                        GT::finish(rc, f);
#pragma unroll
                        for (int ti = 0; ti < T; ++ti) {
                            if (ti < tcount) {
                                if constexpr (!kPipeA) ac[ti] = aptr(s, gi, ti);
                                GT::mma(ac[ti], f, acc[gi][ti]);
                            }
                        }
                    }
                }
            }
        }
    }
    wait_vm_all();
    store_tile<T, G>(a, acc, ok, ep_gr, ep_ow, gbase, gcount, t0, tcount, kg);
}

typedef void (*conv_fn)(ConvArgs);

template <typename E, int MODE>
conv_fn pick_tg(int T, int G) {
    switch (T * 16 + G) {
        case 0x11: return k_conv<E, 1, 1, MODE>;
        case 0x12: return k_conv<E, 1, 2, MODE>;
        case 0x21: return k_conv<E, 2, 1, MODE>;
        case 0x41:   // four tiles per wave: bf16 with 8-byte gathers only (register budget)
            if constexpr (sizeof(E) == 2 && MODE != 2) return k_conv<E, 4, 1, MODE>;
            return nullptr;
        default: return nullptr;
    }
}

template <typename E>
conv_fn pick(int T, int G, int mode) {
    if (mode == 1) return pick_tg<E, 1>(T, G);
    if (mode == 2) return pick_tg<E, 2>(T, G);
    return pick_tg<E, 0>(T, G);
}

}  // namespace

hipError_t launch_conv(const Plan &p, int n, const void *x, const uint8_t *tiles, const float *bias,
                       int relu, int out_bf16, void *y, hipStream_t st) {
    ConvArgs a;
    memset(&a, 0, sizeof(a));
    a.n_ct = p.Wop / p.TW;
    const int64_t n_rt = div_up64((int64_t)n * p.Ho, (int64_t)p.TRW * p.NSUB);
    const int64_t n_wt = n_rt * a.n_ct;
    if (n_wt <= 0) return hipSuccess;
    if (n_wt > INT32_MAX / 2) return hipErrorInvalidValue;
    a.n_wt = (int)n_wt;
    int64_t wpm = std::min<int64_t>(n_wt, std::max<int64_t>(1, div_up64(kTargetWGs, p.n_mb)));
    a.tiles_per_wg = (int)div_up64(n_wt, wpm);
    a.wg_per_mb = (int)div_up64(n_wt, a.tiles_per_wg);
    const int64_t gv = (int64_t)a.wg_per_mb * p.n_mb;
    if (gv > INT32_MAX - 8) return hipErrorInvalidValue;
    a.grid_valid = (int)gv;
    a.x = x;
    a.y = y;
    a.tiles = tiles;
    a.bias = bias;
    a.relu = relu;
    a.out_bf16 = out_bf16;
    a.N = n;
    a.Cin = p.Cin; a.H = p.H; a.W = p.W; a.R = p.R; a.Ho = p.Ho; a.Wo = p.Wo;
    a.KH = p.KH; a.KW = p.KW; a.SH = p.SH; a.SW = p.SW; a.PH = p.PH; a.PW = p.PW;
    a.TW = p.TW; a.TRW = p.TRW; a.NSUB = p.NSUB; a.RL = p.RL; a.NSLOT = p.NSLOT;
    a.CH_STRIDE = p.CH_STRIDE; a.LEFT = p.LEFT;
    a.n_groups = p.n_groups; a.group_rows = p.group_rows; a.mt_per_group = p.mt_per_group;
    a.LP = p.LP; a.S = p.S;
    a.split = p.split; a.msets = p.msets; a.mb_tiles = p.mb_tiles; a.mb_groups = p.mb_groups;
    a.mpg_blocks = p.mpg_blocks; a.n_mb = p.n_mb;
    a.resident = p.resident; a.gran = p.gran; a.gather = p.gather;
    a.lds_a = p.lds_a; a.lds_d = p.lds_d; a.lds_patch = p.lds_patch; a.lds_buf = p.lds_buf;
    a.off_chunks = p.off_chunks;
    a.off_desc16 = p.off_desc16;
    a.off_a = p.off_a;
    a.fp_lo = (uint32_t)p.fingerprint;
    a.fp_hi = (uint32_t)(p.fingerprint >> 32);
    const int ge = p.gran ? p.gran / p.esize : 1;   // elements per fill granule
    a.div_nslot = make_fastdiv((uint32_t)p.NSLOT);
    a.div_nv = make_fastdiv((uint32_t)(p.RL / ge));
    a.div_Ho = make_fastdiv((uint32_t)p.Ho);
    conv_fn fn = p.dt == BSP_F32 ? pick<float>(p.T, p.G, p.gather == 2 ? 0 : p.gather)
                                  : pick<uint16_t>(p.T, p.G, p.gather);
    if (!fn) return hipErrorInvalidValue;
    const int grid = (int)(div_up64(gv, 8) * 8);
    if (p.lds_total > 48 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           p.lds_total);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kThreads), (size_t)p.lds_total, st, a);
    return hipGetLastError();
}

}  // namespace bsp
