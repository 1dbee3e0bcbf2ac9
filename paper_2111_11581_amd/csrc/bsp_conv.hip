// Forward of block-pruned conv / FC layers on gfx950: implicit GEMM over the kept
// columns only.
//
// What is computed (Sec. 4.2, layer i with pruned weights): for every output pixel
// and every output row o, the sum over the kept GEMM columns q = (c, r, s) of o's
// list of W[o, q] * x[n, c, oh*sh - ph + r, ow*sw - pw + s], plus bias, then ReLU.
//
// How (one workgroup = 4 waves = one tile of 64 output pixels x a block of m-tiles):
//  1. Thread 0 maps the tile's output rows to staged input rows ("slots").
//  2. For each channel window of the kept lists ("chunk", built at pack time), the
//     workgroup copies the input patch x[n, c_lo .. c_lo+cnt, slot rows, columns]
//     into LDS with 2..16-byte coalesced loads; padding and out-of-image rows are 0.
//  3. Each wave walks its lists in steps of 32 kept columns.  Lane l owns kept
//     positions 8*(l/16) .. +7 and the 4 horizontally adjacent pixels 4*(l%16) ..+3
//     of the tile: per kept column it issues one 8-byte LDS read (stride 1; 16 bytes
//     for stride 2) at the pre-decoded offset plus its pixel offset, and v_perm
//     re-packs the 8 x 4 values into the B operands of 4 MFMAs (one per pixel of the
//     group).  The A operand (weights) comes pre-tiled from dev_tiles, 16 bytes per
//     lane, and is reused across the 4 pixel n-tiles; when a list is shared by
//     several m-tiles (row pruning, dense) the gathered B operands are reused across
//     them too.
//  4. Epilogue: bias + ReLU + round-to-nearest-even bf16 (or fp32), each lane writes
//     4 adjacent pixels of 4 output rows with 8-byte stores.
// Workgroup ids are remapped so that consecutive logical tiles (which share input
// rows and weights) run on the same XCD and its L2.
#include <hip/hip_runtime.h>

#include "bsp_kernels.h"

namespace bsp {

typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

__device__ __forceinline__ uint32_t perm(uint32_t hi_src, uint32_t lo_src, uint32_t sel) {
    return __builtin_amdgcn_perm(hi_src, lo_src, sel);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    __bf16 h = (__bf16)f;
    return __builtin_bit_cast(uint16_t, h);
}

template <int VB>
struct VecT;
template <> struct VecT<2> { typedef uint16_t type; };
template <> struct VecT<4> { typedef uint32_t type; };
template <> struct VecT<8> { typedef uint2 type; };
template <> struct VecT<16> { typedef uint4 type; };

template <typename E, int VB>
__device__ __forceinline__ void load_patch_vec(const ConvArgs &a, E *patch, const int *s_img,
                                               const int *s_ih, int c_lo, int c_cnt, int a0) {
    typedef typename VecT<VB>::type V;
    constexpr int VEC = VB / (int)sizeof(E);
    const int NV = a.RL / VEC;
    const int total = c_cnt * a.NSLOT * NV;
    const E *x = (const E *)a.x;
    for (int v = threadIdx.x; v < total; v += kThreads) {
        const int row = (int)fdiv((uint32_t)v, a.div_nv);
        const int vi = v - row * NV;
        const int c = (int)fdiv((uint32_t)row, a.div_nslot);
        const int sl = row - c * a.NSLOT;
        const int ih = s_ih[sl];
        const int iw = a0 + vi * VEC;
        V val;
        if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) {
            const size_t off = ((size_t)(s_img[sl] * a.Cin + c_lo + c) * a.H + ih) * a.W + iw;
            val = *(const V *)(x + off);
        } else {
            val = V{};
        }
        *(V *)(patch + c * a.CH_STRIDE + sl * a.RL + vi * VEC) = val;
    }
}

template <typename E>
__device__ __forceinline__ void load_patch(const ConvArgs &a, E *patch, const int *s_img,
                                           const int *s_ih, int c_lo, int c_cnt, int a0) {
    switch (a.VEC * (int)sizeof(E)) {
        case 16: load_patch_vec<E, 16>(a, patch, s_img, s_ih, c_lo, c_cnt, a0); break;
        case 8: load_patch_vec<E, 8>(a, patch, s_img, s_ih, c_lo, c_cnt, a0); break;
        case 4: load_patch_vec<E, 4>(a, patch, s_img, s_ih, c_lo, c_cnt, a0); break;
        default: load_patch_vec<E, 2>(a, patch, s_img, s_ih, c_lo, c_cnt, a0); break;
    }
}

// ---- bf16 operand gathers -----------------------------------------------------------
// v[j] holds pixels 0..3 (16 bits each) of kept column j of this lane; B[nt] is the
// 8-wide k-vector of pixel nt.
__device__ __forceinline__ void repack_bf16(const uint2 *v, s16x8 *B) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint2 lo = v[2 * d], hi = v[2 * d + 1];
        uint32_t w0 = perm(hi.x, lo.x, 0x05040100u);
        uint32_t w1 = perm(hi.x, lo.x, 0x07060302u);
        uint32_t w2 = perm(hi.y, lo.y, 0x05040100u);
        uint32_t w3 = perm(hi.y, lo.y, 0x07060302u);
        ((uint32_t *)&B[0])[d] = w0;
        ((uint32_t *)&B[1])[d] = w1;
        ((uint32_t *)&B[2])[d] = w2;
        ((uint32_t *)&B[3])[d] = w3;
    }
}

__device__ __forceinline__ void gather_bf16(const uint16_t *patch, const int *ad, int mode, int SW,
                                            s16x8 *B) {
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
    repack_bf16(v, B);
}

__device__ __forceinline__ void gather_f32(const float *patch, const int *ad, int mode, int SW,
                                           float (*B)[8]) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (mode == 1) {
            float4 f;
            __builtin_memcpy(&f, patch + ad[j], 16);
            B[0][j] = f.x;
            B[1][j] = f.y;
            B[2][j] = f.z;
            B[3][j] = f.w;
        } else {
            const float *p = patch + ad[j];
            B[0][j] = p[0];
            B[1][j] = p[SW];
            B[2][j] = p[2 * SW];
            B[3][j] = p[3 * SW];
        }
    }
}

template <typename E>
struct Frag;

template <>
struct Frag<uint16_t> {
    s16x8 b[4];
    __device__ __forceinline__ void gather(const uint16_t *patch, const int *ad, int mode, int SW) {
        gather_bf16(patch, ad, mode, SW, b);
    }
    __device__ __forceinline__ void mma(const uint16_t *ap, f32x4 *acc) const {
        const s16x8 A = *(const s16x8 *)ap;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, b[nt], acc[nt], 0, 0, 0);
    }
};

template <>
struct Frag<float> {
    float b[4][8];
    __device__ __forceinline__ void gather(const float *patch, const int *ad, int mode, int SW) {
        gather_f32(patch, ad, mode, SW, b);
    }
    __device__ __forceinline__ void mma(const float *ap, f32x4 *acc) const {
        const float4 a0 = *(const float4 *)ap;
        const float4 a1 = *(const float4 *)(ap + 4);
        const float A[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
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
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    __shared__ int s_rowbase[kMaxTileRows];
    __shared__ int s_img[kMaxSlots];
    __shared__ int s_ih[kMaxSlots];
    E *patch = (E *)smem;

    // XCD-aware remap: hardware places workgroup id on XCD id % 8; give each XCD a
    // contiguous range of logical tiles.
    const int per = gridDim.x >> 3;
    const int lid = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (lid >= a.total) return;
    const int pt = lid / a.n_mb, mb = lid - pt * a.n_mb;
    const int rt = pt / a.n_ct, ct = pt - rt * a.n_ct;
    const int g0 = rt * a.TRW, ow0 = ct * a.TW;
    const int n_rows = a.N * a.Ho;

    if (threadIdx.x == 0) {
        for (int i = 0; i < a.NSLOT; ++i) {
            s_img[i] = 0;
            s_ih[i] = -1;
        }
        slot_layout(g0, a.TRW, a.Ho, n_rows, a.KH, a.SH, a.PH, s_rowbase, s_img, s_ih);
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

    const TileHeader *hdr = (const TileHeader *)a.tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == a.fp_lo && hdr->fp_hi == a.fp_hi;
    const int n_chunks = ok ? hdr->n_chunks : 0;
    const int4 *table = (const int4 *)(a.tiles + a.off_chunks);
    const int32_t *desc = (const int32_t *)(a.tiles + a.off_desc);
    const E *At = (const E *)(a.tiles + a.off_a);
    const int a0 = ow0 * a.SW - a.PW - a.LEFT;

    f32x4 acc[G][T][4];
#pragma unroll
    for (int gi = 0; gi < G; ++gi)
#pragma unroll
        for (int ti = 0; ti < T; ++ti)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[gi][ti][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int ch = 0; ch < n_chunks; ++ch) {
        const int4 cd = table[ch];  // first step, end step, first channel, channel count
        __syncthreads();
        load_patch<E>(a, patch, s_img, s_ih, cd.z, cd.w, a0);
        __syncthreads();
        const int cbase = cd.z * a.CH_STRIDE - pixoff;
        for (int s = cd.x; s < cd.y; ++s) {
#pragma unroll
            for (int gi = 0; gi < G; ++gi) {
                if (gi < gcount && tcount > 0) {
                    const int g = gbase + gi;
                    const int32_t *dp = desc + (size_t)g * a.LP + s * kKS + kg * 8;
                    const int4 d0 = *(const int4 *)dp, d1 = *(const int4 *)(dp + 4);
                    const int ad[8] = {d0.x - cbase, d0.y - cbase, d0.z - cbase, d0.w - cbase,
                                       d1.x - cbase, d1.y - cbase, d1.z - cbase, d1.w - cbase};
                    Frag<E> f;
                    f.gather(patch, ad, a.gather, a.SW);
                    const E *ap = At + (((size_t)g * a.mt_per_group + t0) * a.S + s) * 512 + lane * 8;
#pragma unroll
                    for (int ti = 0; ti < T; ++ti)
                        if (ti < tcount) f.mma(ap + (size_t)ti * a.S * 512, acc[gi][ti]);
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
        case 0x18: return k_conv<E, 1, 8>;
        case 0x21: return k_conv<E, 2, 1>;
        case 0x22: return k_conv<E, 2, 2>;
        case 0x24: return k_conv<E, 2, 4>;
        case 0x41: return k_conv<E, 4, 1>;
        case 0x42: return k_conv<E, 4, 2>;
        case 0x81: return k_conv<E, 8, 1>;
        default: return nullptr;
    }
}

}  // namespace

hipError_t launch_conv(const Plan &p, int n, const void *x, const uint8_t *tiles, const float *bias,
                       int relu, int out_bf16, void *y, hipStream_t st) {
    ConvArgs a;
    memset(&a, 0, sizeof(a));
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
    a.n_ct = p.Wop / p.TW;
    const int n_rt = div_up(n * p.Ho, p.TRW);
    a.n_pt = n_rt * a.n_ct;
    a.n_mb = p.n_mb;
    const int64_t total = (int64_t)a.n_pt * a.n_mb;
    if (total <= 0) return hipSuccess;
    if (total > (int64_t)INT32_MAX - 8) return hipErrorInvalidValue;
    a.total = (int)total;
    a.off_chunks = p.off_chunks;
    a.off_desc = p.off_desc;
    a.off_a = p.off_a;
    a.fp_lo = (uint32_t)p.fingerprint;
    a.fp_hi = (uint32_t)(p.fingerprint >> 32);
    a.div_nslot = make_fastdiv((uint32_t)p.NSLOT);
    a.div_nv = make_fastdiv((uint32_t)(p.RL / p.VEC));
    a.div_Ho = make_fastdiv((uint32_t)p.Ho);
    conv_fn fn = p.dt == BSP_F32 ? pick<float>(p.T, p.G) : pick<uint16_t>(p.T, p.G);
    if (!fn) return hipErrorInvalidValue;
    const size_t lds = (size_t)p.CC * p.CH_STRIDE * p.esize;
    const int grid = (int)(div_up64(total, 8) * 8);
    hipLaunchKernelGGL(fn, dim3(grid), dim3(kThreads), lds, st, a);
    return hipGetLastError();
}

}  // namespace bsp
