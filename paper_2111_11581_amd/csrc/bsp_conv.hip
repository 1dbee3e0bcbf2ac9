// Forward of block-pruned conv / FC layers on gfx950: implicit GEMM over the kept
// columns only.
//
// What is computed (Sec. 4.2, layer i with pruned weights): for every output pixel
// and every output row o, the sum over the kept GEMM columns q = (c, r, s) of o's
// list of W[o, q] * x[n, c, oh*sh - ph + r, ow*sw - pw + s], plus bias, then ReLU.
//
// How (one workgroup = 4 waves = one tile of 64 output pixels x a block of m-tiles):
//  1. The tile's output rows are mapped to staged input rows ("slots"), one row per
//     thread, in closed form.
//  2. For each channel window of the kept lists ("chunk", built at pack time), the
//     workgroup copies the input patch x[n, c_lo .. c_lo+cnt, slot rows, columns]
//     into LDS with asynchronous direct-to-LDS loads (global_load_lds, 16- or 4-byte
//     granules, lane-linear destinations); padding and out-of-image rows are read from
//     a zero block in the tile header.  Odd-width images fall back to batched
//     register loads.
//  3. Each wave walks its lists in steps of 32 kept columns.  Lane l owns kept
//     positions 8*(l/16) .. +7 and the 4 horizontally adjacent pixels 4*(l%16) ..+3
//     of the tile: per kept column it issues one 8-byte LDS read (stride 1; 16 bytes
//     for stride 2) at the pre-decoded 16-bit offset plus its pixel offset, and
//     v_perm re-packs the 8 x 4 values into the B operands of 4 MFMAs (one per pixel
//     of the group).  The weights (A operand) come pre-tiled, 16 bytes per lane, and
//     are reused across the 4 pixel n-tiles; a list shared by several m-tiles (row
//     pruning, dense) also reuses the gathered B operands across them.  Offsets and
//     weights of step s+1 are loaded while step s computes.
//  4. Epilogue: bias + ReLU + round-to-nearest-even bf16 (or fp32); each lane writes
//     4 adjacent pixels of 4 output rows with 8-byte stores.
// Workgroup ids are remapped so that consecutive logical tiles (which share input
// rows and weights) run on the same XCD and its L2.
#include <hip/hip_runtime.h>

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

// Direct-to-LDS patch fill.  Granule g (GB bytes) of the patch lands at byte g*GB;
// with LDS destinations lane-linear per instruction, 64 consecutive granules per
// wave instruction.
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
            lds_void_t *dst = (lds_void_t *)(patch + (size_t)v0 * GB);
            if constexpr (GB == 16) __builtin_amdgcn_global_load_lds((const void *)src, dst, 16, 0, 0);
            else __builtin_amdgcn_global_load_lds((const void *)src, dst, 4, 0, 0);
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

template <typename E>
struct Frag;

template <>
struct Frag<uint16_t> {
    typedef uint4 AReg;   // 8 bf16 weights of this lane
    s16x8 b[4];
    __device__ __forceinline__ void gather(const unsigned char *patch_b, uint4 d, int pixoff, int mode,
                                           int SW) {
        const uint16_t *patch = (const uint16_t *)patch_b;
        int ad[8];
        offsets(d, pixoff, ad);
        uint2 v[8];
        if (mode == 1) {
#pragma unroll
            for (int j = 0; j < 8; ++j) __builtin_memcpy(&v[j], patch + ad[j], 8);
        } else if (mode == 2) {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                uint4 u;
                __builtin_memcpy(&u, patch + ad[j], 16);
                v[j].x = perm(u.y, u.x, 0x05040100u);
                v[j].y = perm(u.w, u.z, 0x05040100u);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const uint16_t *p = patch + ad[j];
                v[j].x = (uint32_t)p[0] | ((uint32_t)p[SW] << 16);
                v[j].y = (uint32_t)p[2 * SW] | ((uint32_t)p[3 * SW] << 16);
            }
        }
        repack_bf16(v, b);
    }
    static __device__ __forceinline__ AReg load_a(const unsigned char *ap) {
        return *(const uint4 *)ap;
    }
    __device__ __forceinline__ void mma(const AReg &ar, f32x4 *acc) const {
        const s16x8 A = __builtin_bit_cast(s16x8, ar);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, b[nt], acc[nt], 0, 0, 0);
    }
};

struct F32x8 {
    float4 lo, hi;
};

template <>
struct Frag<float> {
    typedef F32x8 AReg;
    float b[4][8];
    __device__ __forceinline__ void gather(const unsigned char *patch_b, uint4 d, int pixoff, int mode,
                                           int SW) {
        const float *patch = (const float *)patch_b;
        int ad[8];
        offsets(d, pixoff, ad);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (mode == 1) {
                float4 f;
                __builtin_memcpy(&f, patch + ad[j], 16);
                b[0][j] = f.x; b[1][j] = f.y; b[2][j] = f.z; b[3][j] = f.w;
            } else {
                const float *p = patch + ad[j];
                b[0][j] = p[0]; b[1][j] = p[SW]; b[2][j] = p[2 * SW]; b[3][j] = p[3 * SW];
            }
        }
    }
    static __device__ __forceinline__ AReg load_a(const unsigned char *ap) {
        AReg r;
        r.lo = *(const float4 *)ap;
        r.hi = *(const float4 *)(ap + 16);
        return r;
    }
    __device__ __forceinline__ void mma(const AReg &ar, f32x4 *acc) const {
        const float A[8] = {ar.lo.x, ar.lo.y, ar.lo.z, ar.lo.w, ar.hi.x, ar.hi.y, ar.hi.z, ar.hi.w};
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int u = 0; u < 8; ++u)
                acc[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[u], b[nt][u], acc[nt], 0, 0, 0);
    }
};

__device__ __forceinline__ float epi(float v, float b, int relu) {
    v += b;
    return (relu && v < 0.f) ? 0.f : v;
}

template <typename E, int T, int G>
__global__ __launch_bounds__(kThreads, 2) void k_conv(ConvArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char patch[];
    __shared__ int s_rowbase[kMaxTileRows];
    __shared__ int s_img[kMaxSlots];
    __shared__ int s_ih[kMaxSlots];
    typedef typename Frag<E>::AReg AReg;
    constexpr int ABYTES = 8 * (int)sizeof(E);   // weight bytes per lane per m-tile and step

    // XCD-aware remap: hardware places workgroup id on XCD (id % 8); give each XCD a
    // contiguous range of logical tiles.
    const int per = gridDim.x >> 3;
    const int lid = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (lid >= a.total) return;
    const int pt = lid / a.n_mb, mb = lid - pt * a.n_mb;
    const int rt = pt / a.n_ct, ct = pt - rt * a.n_ct;
    const int g0 = rt * a.TRW, ow0 = ct * a.TW;
    const int n_rows = a.N * a.Ho;

    // staged input rows: row tr of the tile uses slots rowbase[tr] + r (r < KH)
    if ((int)threadIdx.x < a.NSLOT) {
        s_img[threadIdx.x] = 0;
        s_ih[threadIdx.x] = -1;
    }
    __syncthreads();
    if ((int)threadIdx.x < a.TRW) {
        const int tr = threadIdx.x, g = g0 + tr;
        int base = 0;
        if (g < n_rows) {
            const int img = (int)fdiv((uint32_t)g, a.div_Ho), oh = g - img * a.Ho;
            const int k = img - (int)fdiv((uint32_t)g0, a.div_Ho);   // image boundaries crossed
            base = (tr - k) * min(a.SH, a.KH) + k * a.KH;
            for (int r = 0; r < a.KH; ++r) {
                s_img[base + r] = img;
                s_ih[base + r] = oh * a.SH - a.PH + r;
            }
        }
        s_rowbase[tr] = base;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n16 = lane & 15, kg = lane >> 4;
    const int tr = (4 * n16) / a.TW, cx = 4 * n16 - tr * a.TW;
    const int pixoff = s_rowbase[tr] * a.RL + cx * a.SW;

    int gbase, t0, tcount, gcount;
    if (!a.split) {
        gbase = mb * kWaves * G + wave * G;
        t0 = 0;
        tcount = a.mt_per_group;
        gcount = min(G, a.n_groups - gbase);
    } else {
        gbase = mb / a.mpg_blocks;
        t0 = (mb - gbase * a.mpg_blocks) * kWaves * T + wave * T;
        tcount = min(T, a.mt_per_group - t0);
        gcount = 1;
    }
    const bool active = gcount > 0 && tcount > 0;

    const TileHeader *hdr = (const TileHeader *)a.tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == a.fp_lo && hdr->fp_hi == a.fp_hi;
    const int n_chunks = ok ? hdr->n_chunks : 0;
    const int4 *table = (const int4 *)(a.tiles + a.off_chunks);
    const uint16_t *desc = (const uint16_t *)(a.tiles + a.off_desc16);
    const unsigned char *At = a.tiles + a.off_a;
    const int a0 = ow0 * a.SW - a.PW - a.LEFT;
    const size_t a_step = (size_t)64 * ABYTES;               // one m-tile, one step
    const size_t a_mt = (size_t)a.S * a_step;                // one m-tile, all steps

    f32x4 acc[G][T][4];
#pragma unroll
    for (int gi = 0; gi < G; ++gi)
#pragma unroll
        for (int ti = 0; ti < T; ++ti)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[gi][ti][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    uint4 dn[G];
    AReg an[G][T];
    auto fetch = [&](int s) {
#pragma unroll
        for (int gi = 0; gi < G; ++gi) {
            if (gi < gcount && active) {
                const int g = gbase + gi;
                dn[gi] = *(const uint4 *)(desc + (size_t)g * a.LP + s * kKS + kg * 8);
                const unsigned char *ap = At + ((size_t)g * a.mt_per_group + t0) * a_mt +
                                          (size_t)s * a_step + (size_t)lane * ABYTES;
#pragma unroll
                for (int ti = 0; ti < T; ++ti)
                    if (ti < tcount) an[gi][ti] = Frag<E>::load_a(ap + ti * a_mt);
            }
        }
    };

    for (int ch = 0; ch < n_chunks; ++ch) {
        const int4 cd = table[ch];  // first step, end step, first channel, channel count
        __syncthreads();            // previous chunk's gathers are done
        fill_patch<E>(a, patch, s_img, s_ih, cd.z, cd.w, a0);
        fetch(cd.x);
        wait_vm_all();
        __syncthreads();
        for (int s = cd.x; s < cd.y; ++s) {
            uint4 dc[G];
            AReg ac[G][T];
#pragma unroll
            for (int gi = 0; gi < G; ++gi) {
                dc[gi] = dn[gi];
#pragma unroll
                for (int ti = 0; ti < T; ++ti) ac[gi][ti] = an[gi][ti];
            }
            if (s + 1 < cd.y) fetch(s + 1);
#pragma unroll
            for (int gi = 0; gi < G; ++gi) {
                if (gi < gcount && active) {
                    Frag<E> f;
                    f.gather(patch, dc[gi], pixoff, a.gather, a.SW);
#pragma unroll
                    for (int ti = 0; ti < T; ++ti)
                        if (ti < tcount) f.mma(ac[gi][ti], acc[gi][ti]);
                }
            }
        }
    }

    // epilogue
    const int gr = g0 + tr;
    if (gr >= n_rows) return;
    const int img = (int)fdiv((uint32_t)gr, a.div_Ho), oh = gr - img * a.Ho;
    const int ow = ow0 + cx;
    if (ow >= a.Wo) return;
    const bool full = (ow + 3 < a.Wo) && ((a.Wo & 3) == 0);
    const float qnan = __builtin_nanf("");
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
        if (gi >= gcount) continue;
        const int g = gbase + gi;
#pragma unroll
        for (int ti = 0; ti < T; ++ti) {
            if (ti >= tcount) continue;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rig = (t0 + ti) * kMT + 4 * kg + i;
                const int row = g * a.group_rows + rig;
                if (rig >= a.group_rows || row >= a.R) continue;
                const float bv = a.bias ? a.bias[row] : 0.f;
                float o[4];
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) o[nt] = ok ? epi(acc[gi][ti][nt][i], bv, a.relu) : qnan;
                const size_t yo = ((size_t)(img * a.R + row) * a.Ho + oh) * a.Wo + ow;
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

typedef void (*conv_fn)(ConvArgs);

template <typename E>
conv_fn pick(int T, int G) {
    switch (T * 16 + G) {
        case 0x11: return k_conv<E, 1, 1>;
        case 0x12: return k_conv<E, 1, 2>;
        case 0x14: return k_conv<E, 1, 4>;
        case 0x21: return k_conv<E, 2, 1>;
        case 0x22: return k_conv<E, 2, 2>;
        case 0x41: return k_conv<E, 4, 1>;
        default: return nullptr;
    }
}

}  // namespace

hipError_t launch_conv(const Plan &plan, int n, const void *x, const uint8_t *tiles, const float *bias,
                       int relu, int out_bf16, void *y, hipStream_t st) {
    Plan p = plan;
    ConvArgs a;
    memset(&a, 0, sizeof(a));
    a.n_ct = p.Wop / p.TW;
    const int64_t n_rt = div_up64((int64_t)n * p.Ho, p.TRW);
    const int64_t n_pt = n_rt * a.n_ct;
    if (n_pt <= 0) return hipSuccess;
    choose_split(&p, n_pt);
    a.x = x;
    a.y = y;
    a.tiles = tiles;
    a.bias = bias;
    a.relu = relu;
    a.out_bf16 = out_bf16;
    a.N = n;
    a.Cin = p.Cin; a.H = p.H; a.W = p.W; a.R = p.R; a.Ho = p.Ho; a.Wo = p.Wo;
    a.KH = p.KH; a.KW = p.KW; a.SH = p.SH; a.SW = p.SW; a.PH = p.PH; a.PW = p.PW;
    a.TW = p.TW; a.TRW = p.TRW; a.Wop = p.Wop; a.VEC = p.VEC; a.LEFT = p.LEFT; a.RL = p.RL;
    a.NSLOT = p.NSLOT; a.CH_STRIDE = p.CH_STRIDE; a.CC = p.CC;
    a.n_groups = p.n_groups; a.group_rows = p.group_rows; a.mt_per_group = p.mt_per_group;
    a.LP = p.LP; a.S = p.S; a.T = p.T; a.G = p.G; a.split = p.split; a.mpg_blocks = p.mpg_blocks;
    a.gather = p.gather;
    a.gran = p.gran;
    a.n_pt = (int)n_pt;
    a.n_mb = p.n_mb;
    const int64_t total = n_pt * a.n_mb;
    if (total > (int64_t)INT32_MAX - 8) return hipErrorInvalidValue;
    a.total = (int)total;
    a.off_chunks = p.off_chunks;
    a.off_desc16 = p.off_desc16;
    a.off_a = p.off_a;
    a.fp_lo = (uint32_t)p.fingerprint;
    a.fp_hi = (uint32_t)(p.fingerprint >> 32);
    const int ge = p.gran ? p.gran / p.esize : 1;   // elements per fill granule
    a.div_nslot = make_fastdiv((uint32_t)p.NSLOT);
    a.div_nv = make_fastdiv((uint32_t)(p.RL / ge));
    a.div_Ho = make_fastdiv((uint32_t)p.Ho);
    conv_fn fn = p.dt == BSP_F32 ? pick<float>(p.T, p.G) : pick<uint16_t>(p.T, p.G);
    if (!fn) return hipErrorInvalidValue;
    const size_t lds = (size_t)p.CC * p.CH_STRIDE * p.esize;
    const int grid = (int)(div_up64(total, 8) * 8);
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kThreads), lds, st, a);
    return hipGetLastError();
}

}  // namespace bsp
