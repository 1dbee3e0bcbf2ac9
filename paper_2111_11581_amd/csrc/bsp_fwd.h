// Forward kernel of block-pruned conv / FC layers on gfx950 (template; instantiated
// in bsp_fwd_*.hip): implicit GEMM over the kept columns only.
//
// What is computed (Sec. 4.2, layer i with pruned weights): for every output pixel
// and every output row o, the sum over the kept GEMM columns q = (c, r, s) of o's
// list of W[o, q] * x[n, c, oh*sh - ph + r, ow*sw - pw + s], plus bias, then ReLU.
//
// How.  One workgroup (4 waves) computes one tile of output pixels (NSUB runs of 64
// consecutive pixels, in groups of 4 adjacent pixels of one output row) for one
// m-block of output rows.  Its K loop walks chunks of the kept lists:
//  * fill: the input rows of the chunk's channels (every staged row is an input row
//    of the tile, whole width, zero-padded left and right) are copied into LDS with
//    asynchronous 16-byte direct-to-LDS loads, issued from inline assembly and awaited
//    explicitly, in batches between the steps of the previous chunk's compute (other
//    LDS buffer).  Each thread's granules of the patch are decoded once per tile;
//    padding and out-of-image rows are zeroed once.  When the m-block's weights do not
//    stay resident in LDS, the chunk's slice of them is copied the same way.
//  * compute: each wave walks its steps of 32 kept columns.  Lane l owns kept
//    positions 8*(l/16) .. +7 and the 4 pixels of group l % 16 of its sub-tile: per
//    kept column aligned LDS reads at the pre-decoded 16-bit offset plus the group's
//    offset (see Gat below), then v_perm re-packs the 8 x 4 values into the B operands
//    of 4 MFMAs.  A list shared by several m-tiles (row pruning, dense) reuses the
//    gathered operands across them.
//  * when the 4 / NSUB waves of a sub-tile split the steps, they add their partial
//    sums through LDS at the end;
//  * epilogue: bias + ReLU + round-to-nearest-even bf16 (or fp32); each lane writes
//    its group's 4 pixels of 4 output rows with 8-byte stores, so a wave writes 128
//    contiguous bytes per output row.
// Workgroup ids are remapped so that the m-blocks of one pixel tile and neighbouring
// tiles run on the same XCD (workgroup id % 8) and share its L2.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "bsp_kernels.h"

namespace bsp {

typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(4))) const int const_int;

namespace fwd {

__device__ __forceinline__ uint32_t perm(uint32_t hi_src, uint32_t lo_src, uint32_t sel) {
    return __builtin_amdgcn_perm(hi_src, lo_src, sel);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    __bf16 h = (__bf16)f;
    return __builtin_bit_cast(uint16_t, h);
}

// Two floats rounded to bf16 (RNE, as f32_to_bf16_rne) in one instruction: lo in bits
// 15..0, hi in bits 31..16.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
    return (uint32_t)(uintptr_t)(lds_void_t *)p;
}

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Chunk k of the table (first step, end step, first channel, channel count), read
// through the scalar data cache as wave-uniform values.
__device__ __forceinline__ int4 chunk_at(const const_int *t, int k) {
    return make_int4(uni(t[4 * k]), uni(t[4 * k + 1]), uni(t[4 * k + 2]), uni(t[4 * k + 3]));
}

// Asynchronous 16-byte copy global -> LDS: lane l writes LDS byte lds_base + 16 l
// (lds_base is wave-uniform).  Issued from inline assembly so that the compiler does
// not hold later LDS reads back behind it; callers await it with wait_vm_all().  M0
// (the LDS base of the copy) is saved and restored around it.
__device__ __forceinline__ void dma16(const void *src, uint32_t lds_base) {
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(src), "s"(uni((int)lds_base))
                 : "memory");
}

// Pointer made wave-uniform (held in scalar registers).
__device__ __forceinline__ const void *uni_ptr(const void *p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return (const void *)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// As dma16 with the source split into a wave-uniform base (scalar registers) and a
// per-lane 32-bit byte offset: lane l copies 16 bytes at sbase + voff to LDS byte
// m0 + 16 l.  No 64-bit address arithmetic per copy.
__device__ __forceinline__ void dma_sv(const void *sbase, uint32_t voff, uint32_t m0) {
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
                 : "=&s"(saved)
                 : "v"(voff), "s"(uni_ptr(sbase)), "s"(uni((int)m0))
                 : "memory");
}

// Contiguous copy of n16 16-byte granules from src to the LDS byte address dst.
__device__ __forceinline__ void dma_run(const unsigned char *src, uint32_t dst, int n16) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int q0 = wave * 64; q0 < n16; q0 += kThreads) {
        if (q0 + lane < n16) dma16(src + (size_t)(q0 + lane) * 16, dst + (uint32_t)q0 * 16);
    }
}

// Batches of asynchronous 16-byte copies global -> LDS with one M0 (LDS base) for up
// to four copies: copy k of a batch writes LDS bytes m0 + 1024 k + 16 l for lane l and
// reads 16 bytes at its own source address.  The immediate offset 1024 k moves both
// the LDS destination and the source, so each source is passed lowered by it.  Every
// lane takes part; each copy is one vector memory operation of the wave, so waits can
// count them.  Rewriting M0 before every copy would stall issue on the previous copy.
__device__ __forceinline__ void dma_b4(const unsigned char *s0, const unsigned char *s1, const unsigned char *s2,
                                       const unsigned char *s3, uint32_t m0, int n) {
    uint32_t sv;
    const int base = uni((int)m0);
    switch (uni(n)) {
        case 1:
            asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
                         "global_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
                         : "=&s"(sv) : "v"(s0), "s"(base) : "memory");
            break;
        case 2:
            asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\t"
                         "global_load_lds_dwordx4 %1, off\n\tglobal_load_lds_dwordx4 %2, off offset:1024\n\t"
                         "s_mov_b32 m0, %0"
                         : "=&s"(sv) : "v"(s0), "v"(s1 - 1024), "s"(base) : "memory");
            break;
        case 3:
            asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %4\n\ts_nop 0\n\t"
                         "global_load_lds_dwordx4 %1, off\n\tglobal_load_lds_dwordx4 %2, off offset:1024\n\t"
                         "global_load_lds_dwordx4 %3, off offset:2048\n\ts_mov_b32 m0, %0"
                         : "=&s"(sv) : "v"(s0), "v"(s1 - 1024), "v"(s2 - 2048), "s"(base) : "memory");
            break;
        default:
            asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %5\n\ts_nop 0\n\t"
                         "global_load_lds_dwordx4 %1, off\n\tglobal_load_lds_dwordx4 %2, off offset:1024\n\t"
                         "global_load_lds_dwordx4 %3, off offset:2048\n\tglobal_load_lds_dwordx4 %4, off offset:3072\n\t"
                         "s_mov_b32 m0, %0"
                         : "=&s"(sv) : "v"(s0), "v"(s1 - 1024), "v"(s2 - 2048), "v"(s3 - 3072), "s"(base) : "memory");
            break;
    }
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
// flight while the current stage re-packs and multiplies.  Every LDS read is aligned
// to its own size: on gfx950 a misaligned multi-dword LDS read costs about twenty
// aligned ones.  MODE 1: stride 1, reads start at a multiple of 4 elements (one 8-byte
// read per kept column, 16 bytes for fp32); MODE 3: stride 1 at any element (the
// dwords holding the 4 elements, joined by a byte shift of 0 or 2); MODE 2: stride 2,
// 16-byte reads at a multiple of 8 elements (even elements kept); MODE 4: stride 2 at
// any element (the 4 dwords holding elements e, e + 2, e + 4, e + 6, halves picked by
// the parity of e); MODE 0: any stride (one read per element).
template <typename E, int MODE>
struct Gat;

struct U3 { uint32_t x, y, z; };

template <int MODE>
struct Gat<uint16_t, MODE> {
    typedef typename std::conditional<MODE == 2 || MODE == 4, uint4,
                                      typename std::conditional<MODE == 3, U3, uint2>::type>::type R1;
    struct Raw { R1 v[8]; uint32_t sh; };
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
            } else if constexpr (MODE == 3) {
                // dwords ad/2 .. ad/2 + 2 (the third is needed when ad is odd); bit 2j + 1
                // of sh: ad odd, i.e. a byte shift of 2 in bits 1..0 of sh >> 2j
                const uint32_t *w = (const uint32_t *)patch_b + (ad[j] >> 1);
                r.v[j] = U3{w[0], w[1], w[2]};
                if (j == 0) r.sh = 0;
                r.sh |= (uint32_t)(ad[j] & 1) << (2 * j + 1);
            } else if constexpr (MODE == 4) {
                // dwords ad/2 .. ad/2 + 3; bit j of sh: ad odd (elements in the high halves)
                const uint32_t *w = (const uint32_t *)patch_b + (ad[j] >> 1);
                r.v[j] = make_uint4(w[0], w[1], w[2], w[3]);
                if (j == 0) r.sh = 0;
                r.sh |= (uint32_t)(ad[j] & 1) << j;
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
            } else if constexpr (MODE == 4) {
                const uint32_t sel = ((r.sh >> j) & 1) ? 0x07060302u : 0x05040100u;
                v[j].x = perm(r.v[j].y, r.v[j].x, sel);
                v[j].y = perm(r.v[j].w, r.v[j].z, sel);
            } else if constexpr (MODE == 3) {
                const uint32_t bs = r.sh >> (2 * j);   // alignbyte uses bits 1..0
                v[j].x = __builtin_amdgcn_alignbyte(r.v[j].y, r.v[j].x, bs);
                v[j].y = __builtin_amdgcn_alignbyte(r.v[j].z, r.v[j].y, bs);
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

// Stores of one wave with an explicit lane mask (wave-uniform), issued from inline
// assembly so that the wave knows exactly how many vector memory operations it has
// in flight (waits for later copies then need not wait for these stores).  Inactive
// lanes' address and data are ignored.
__device__ __forceinline__ void st_mask_b16(void *addr, uint32_t v, uint64_t mask) {
    uint64_t saved;
    asm volatile("s_mov_b64 %0, exec\n\ts_mov_b64 exec, %3\n\tglobal_store_short %1, %2, off\n\ts_mov_b64 exec, %0"
                 : "=&s"(saved) : "v"(addr), "v"(v), "s"(mask) : "memory");
}
__device__ __forceinline__ void st_mask_b32(void *addr, uint32_t v, uint64_t mask) {
    uint64_t saved;
    asm volatile("s_mov_b64 %0, exec\n\ts_mov_b64 exec, %3\n\tglobal_store_dword %1, %2, off\n\ts_mov_b64 exec, %0"
                 : "=&s"(saved) : "v"(addr), "v"(v), "s"(mask) : "memory");
}
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st_mask_b64(void *addr, u32x2 v, uint64_t mask) {
    uint64_t saved;
    asm volatile("s_mov_b64 %0, exec\n\ts_mov_b64 exec, %3\n\tglobal_store_dwordx2 %1, %2, off\n\ts_mov_b64 exec, %0"
                 : "=&s"(saved) : "v"(addr), "v"(v), "s"(mask) : "memory");
}
__device__ __forceinline__ void st_mask_b128(void *addr, u32x4 v, uint64_t mask) {
    uint64_t saved;
    asm volatile("s_mov_b64 %0, exec\n\ts_mov_b64 exec, %3\n\tglobal_store_dwordx4 %1, %2, off\n\ts_mov_b64 exec, %0"
                 : "=&s"(saved) : "v"(addr), "v"(v), "s"(mask) : "memory");
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// One stage (step k, list group GWI) of a wave's K loop.  Issue order: the weights of
// the next stage (when APF, into an; else this stage's into ac), the gather offsets
// two stages ahead (into dn), the gathers of the next stage (into rn, at offsets dc);
// then re-pack this stage's gathers (rc) and multiply.  Waiting for this stage's
// weights and gathers thus never waits for reads issued in this stage (APF) or only
// for the weights (no APF: many m-tiles per list make the stage long anyway).
template <typename E, int MODE, int TM, int TPG, int GWI, bool APF>
__device__ __forceinline__ void stage(f32x4 (&acc)[TM][4], const unsigned char *patch,
                                      const unsigned char *Ak, const unsigned char *Anext, int a_mstr,
                                      const unsigned char *dnext2, int pixoff, int SW,
                                      typename Gat<E, MODE>::Raw &rc, typename Gat<E, MODE>::Raw &rn,
                                      const uint4 &dc, uint4 &dn, typename Gat<E, MODE>::AReg (&ac)[TPG],
                                      typename Gat<E, MODE>::AReg (&an)[TPG]) {
    typedef Gat<E, MODE> GT;
    if constexpr (APF) {
#pragma unroll
        for (int t = 0; t < TPG; ++t) an[t] = GT::read_a(Anext + t * a_mstr);
    } else {
#pragma unroll
        for (int t = 0; t < TPG; ++t) ac[t] = GT::read_a(Ak + (GWI * TPG + t) * a_mstr);
    }
    __builtin_amdgcn_sched_barrier(0);
    dn = *(const uint4 *)dnext2;
    __builtin_amdgcn_sched_barrier(0);
    GT::read(rn, patch, dc, pixoff, SW);
    __builtin_amdgcn_sched_barrier(0);
    typename GT::Frag f;
    GT::finish(rc, f);
#pragma unroll
    for (int t = 0; t < TPG; ++t) GT::mma(ac[t], f, acc[GWI * TPG + t]);
}

// One chunk of a wave's K loop: stages (step, list group) in order, steps KS apart.
// While stage i multiplies, the gathers (and, for one or two m-tiles per list, the
// weights) of stage i + 1 and the gather offsets of stage i + 2 are in flight; two
// register sets alternate by stage parity, so no copies force early waits.  Reads
// past the last stage re-read the last stage.
//   Ab: LDS weights of the wave's first m-tile at its first step (+ lane offset);
//       m-tile t at step k: Ab + t * a_mstr + k * KS * ASTEP
//   Db: LDS gather offsets (this lane's 8) of the first list group at the first step;
//       group gw: + gw * d_gstr bytes, step k: + k * KS * 64 bytes
//   hook(): called after each step (other work of the wave, e.g. copy batches)
template <typename E, int MODE, int TM, int TPG, int KS, typename Hook>
__device__ __forceinline__ void compute_chunk(f32x4 (&acc)[TM][4], const unsigned char *patch,
                                              const unsigned char *Ab, int a_mstr,
                                              const unsigned char *Db, int d_gstr, int nsteps,
                                              int pixoff, int SW, Hook &&hook) {
    typedef Gat<E, MODE> GT;
    constexpr int GW = TM / TPG;
    constexpr bool APF = TPG <= 2;
    constexpr int ASTEP = 64 * 8 * (int)sizeof(E);
    const int nst = nsteps * GW;   // stages
    auto dptr = [&](int st) {
        st = min(st, nst - 1);
        const int k = st / GW, gw = st - k * GW;
        return Db + gw * d_gstr + k * (KS * kKS * 2);
    };
    auto aptr = [&](int st) {   // weights of the first m-tile of stage st
        st = min(st, nst - 1);
        const int k = st / GW, gw = st - k * GW;
        return Ab + gw * TPG * a_mstr + k * (KS * ASTEP);
    };
    typename GT::Raw r0, r1;
    typename GT::AReg a0[TPG], a1[TPG];
    uint4 d0, d1;
    d0 = *(const uint4 *)dptr(0);
    GT::read(r0, patch, d0, pixoff, SW);
    if constexpr (APF) {
#pragma unroll
        for (int t = 0; t < TPG; ++t) a0[t] = GT::read_a(aptr(0) + t * a_mstr);
    }
    d1 = *(const uint4 *)dptr(1);
    if constexpr (GW % 2 == 0) {
        for (int k = 0; k < nsteps; ++k) {
            const unsigned char *Ak = Ab + k * (KS * ASTEP);
            const int st = k * GW;
#define BSP_STAGE2(G)                                                                                     \
            stage<E, MODE, TM, TPG, G, APF>(acc, patch, Ak, aptr(st + G + 1), a_mstr, dptr(st + G + 2),     \
                                            pixoff, SW, r0, r1, d1, d0, a0, a1);                          \
            stage<E, MODE, TM, TPG, G + 1, APF>(acc, patch, Ak, aptr(st + G + 2), a_mstr, dptr(st + G + 3), \
                                                pixoff, SW, r1, r0, d0, d1, a1, a0);
            BSP_STAGE2(0)
            if constexpr (GW >= 4) { BSP_STAGE2(2) }
            if constexpr (GW >= 8) { BSP_STAGE2(4) BSP_STAGE2(6) }
#undef BSP_STAGE2
            hook();
        }
    } else {
        int k = 0;
        for (; k + 1 < nsteps; k += 2) {
            stage<E, MODE, TM, TPG, 0, APF>(acc, patch, Ab + k * (KS * ASTEP), aptr(k + 1), a_mstr, dptr(k + 2),
                                            pixoff, SW, r0, r1, d1, d0, a0, a1);
            hook();
            stage<E, MODE, TM, TPG, 0, APF>(acc, patch, Ab + (k + 1) * (KS * ASTEP), aptr(k + 2), a_mstr,
                                            dptr(k + 3), pixoff, SW, r1, r0, d0, d1, a1, a0);
            hook();
        }
        if (k < nsteps) {
            stage<E, MODE, TM, TPG, 0, APF>(acc, patch, Ab + k * (KS * ASTEP), aptr(k + 1), a_mstr, dptr(k + 2),
                                            pixoff, SW, r0, r1, d1, d0, a0, a1);
            hook();
        }
    }
}

// Waits until at most n of this wave's vector memory operations are outstanding
// (they complete in issue order).  s_waitcnt takes an immediate, so the wave-uniform
// count selects one of the encodings; counts above 63 wait for 63.
__device__ __forceinline__ void wait_vm(int n) {
    switch (uni(n)) {
        case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(1)" ::: "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(2)" ::: "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(3)" ::: "memory"); break;
        case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
        case 5: asm volatile("s_waitcnt vmcnt(5)" ::: "memory"); break;
        case 6: asm volatile("s_waitcnt vmcnt(6)" ::: "memory"); break;
        case 7: asm volatile("s_waitcnt vmcnt(7)" ::: "memory"); break;
        case 8: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
        case 9: asm volatile("s_waitcnt vmcnt(9)" ::: "memory"); break;
        case 10: asm volatile("s_waitcnt vmcnt(10)" ::: "memory"); break;
        case 11: asm volatile("s_waitcnt vmcnt(11)" ::: "memory"); break;
        case 12: asm volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
        case 13: asm volatile("s_waitcnt vmcnt(13)" ::: "memory"); break;
        case 14: asm volatile("s_waitcnt vmcnt(14)" ::: "memory"); break;
        case 15: asm volatile("s_waitcnt vmcnt(15)" ::: "memory"); break;
        case 16: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
        case 17: asm volatile("s_waitcnt vmcnt(17)" ::: "memory"); break;
        case 18: asm volatile("s_waitcnt vmcnt(18)" ::: "memory"); break;
        case 19: asm volatile("s_waitcnt vmcnt(19)" ::: "memory"); break;
        case 20: asm volatile("s_waitcnt vmcnt(20)" ::: "memory"); break;
        case 21: asm volatile("s_waitcnt vmcnt(21)" ::: "memory"); break;
        case 22: asm volatile("s_waitcnt vmcnt(22)" ::: "memory"); break;
        case 23: asm volatile("s_waitcnt vmcnt(23)" ::: "memory"); break;
        case 24: asm volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
        case 25: asm volatile("s_waitcnt vmcnt(25)" ::: "memory"); break;
        case 26: asm volatile("s_waitcnt vmcnt(26)" ::: "memory"); break;
        case 27: asm volatile("s_waitcnt vmcnt(27)" ::: "memory"); break;
        case 28: asm volatile("s_waitcnt vmcnt(28)" ::: "memory"); break;
        case 29: asm volatile("s_waitcnt vmcnt(29)" ::: "memory"); break;
        case 30: asm volatile("s_waitcnt vmcnt(30)" ::: "memory"); break;
        case 31: asm volatile("s_waitcnt vmcnt(31)" ::: "memory"); break;
        case 32: asm volatile("s_waitcnt vmcnt(32)" ::: "memory"); break;
        case 33: asm volatile("s_waitcnt vmcnt(33)" ::: "memory"); break;
        case 34: asm volatile("s_waitcnt vmcnt(34)" ::: "memory"); break;
        case 35: asm volatile("s_waitcnt vmcnt(35)" ::: "memory"); break;
        case 36: asm volatile("s_waitcnt vmcnt(36)" ::: "memory"); break;
        case 37: asm volatile("s_waitcnt vmcnt(37)" ::: "memory"); break;
        case 38: asm volatile("s_waitcnt vmcnt(38)" ::: "memory"); break;
        case 39: asm volatile("s_waitcnt vmcnt(39)" ::: "memory"); break;
        case 40: asm volatile("s_waitcnt vmcnt(40)" ::: "memory"); break;
        case 41: asm volatile("s_waitcnt vmcnt(41)" ::: "memory"); break;
        case 42: asm volatile("s_waitcnt vmcnt(42)" ::: "memory"); break;
        case 43: asm volatile("s_waitcnt vmcnt(43)" ::: "memory"); break;
        case 44: asm volatile("s_waitcnt vmcnt(44)" ::: "memory"); break;
        case 45: asm volatile("s_waitcnt vmcnt(45)" ::: "memory"); break;
        case 46: asm volatile("s_waitcnt vmcnt(46)" ::: "memory"); break;
        case 47: asm volatile("s_waitcnt vmcnt(47)" ::: "memory"); break;
        case 48: asm volatile("s_waitcnt vmcnt(48)" ::: "memory"); break;
        case 49: asm volatile("s_waitcnt vmcnt(49)" ::: "memory"); break;
        case 50: asm volatile("s_waitcnt vmcnt(50)" ::: "memory"); break;
        case 51: asm volatile("s_waitcnt vmcnt(51)" ::: "memory"); break;
        case 52: asm volatile("s_waitcnt vmcnt(52)" ::: "memory"); break;
        case 53: asm volatile("s_waitcnt vmcnt(53)" ::: "memory"); break;
        case 54: asm volatile("s_waitcnt vmcnt(54)" ::: "memory"); break;
        case 55: asm volatile("s_waitcnt vmcnt(55)" ::: "memory"); break;
        case 56: asm volatile("s_waitcnt vmcnt(56)" ::: "memory"); break;
        case 57: asm volatile("s_waitcnt vmcnt(57)" ::: "memory"); break;
        case 58: asm volatile("s_waitcnt vmcnt(58)" ::: "memory"); break;
        case 59: asm volatile("s_waitcnt vmcnt(59)" ::: "memory"); break;
        case 60: asm volatile("s_waitcnt vmcnt(60)" ::: "memory"); break;
        case 61: asm volatile("s_waitcnt vmcnt(61)" ::: "memory"); break;
        case 62: asm volatile("s_waitcnt vmcnt(62)" ::: "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(63)" ::: "memory"); break;
    }
}

constexpr int kTableSets = 4;      // tiles in flight: computing, landing, filling, being set up
constexpr int kMaxMBRows = 256;    // rows of an m-block (bias staged in LDS)
constexpr int kMaxCHG = 512;       // patch granules per channel (per-tile lookup table)
constexpr int kNoData = -2147483647 - 1;   // lookup entry of a granule holding no input
static_assert(kTableSets * kMaxTileRows * 4 + kTableSets * kMaxSlots * 8 + kMaxMBRows * 4 + 2 * kMaxCHG * 8 <=
                  kLdsStatic, "static LDS tables exceed the planner's reserve");

// Granule kinds of the per-thread patch decode.
constexpr int kKindNone = 0, kKindZero = 1, kKindData = 2;

template <typename E, int MODE, int TM, int TPG, int KS, bool MAP = false>
__global__ __launch_bounds__(kFwdThreads, 1) void k_fwd(ConvArgs a) {
    constexpr int AB = 8 * (int)sizeof(E);   // weight bytes per lane, one m-tile and step
    constexpr int ASTEP = 64 * AB;           // one m-tile, one step
    constexpr int AI = ASTEP / 1024;         // 1 KB copies per m-tile and step
    extern __shared__ __attribute__((aligned(256))) unsigned char lds[];
    __shared__ int s_rowbase[kTableSets][kMaxTileRows];
    __shared__ int2 s_slot[kTableSets][kMaxSlots];   // (element offset of the slot's input row or -1, valid width)
    __shared__ float s_bias[kMaxMBRows];
    __shared__ int2 s_lut[2][kMaxCHG];

    // workgroup -> (range of pixel tiles, m-block); ids remapped so that each XCD
    // (hardware places workgroup id on XCD id % 8) gets a contiguous logical range
    const int per = gridDim.x >> 3;
    const int lid = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (lid >= a.grid_valid) return;
    const int jr = (int)fdiv((uint32_t)lid, a.div_nmb);
    const int mb = lid - jr * a.n_mb;
    const int t_begin = jr * a.tiles_per_wg;
    const int t_end = min(a.n_pt, t_begin + a.tiles_per_wg);
    if (t_begin >= t_end) return;

    const TileHeader *hdr = (const TileHeader *)a.tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == a.fp_lo && hdr->fp_hi == a.fp_hi;
    const int nch = ok ? uni(hdr->n_chunks) : 0;
    const const_int *table = (const const_int *)(a.tiles + a.off_chunks);
    const unsigned char *A_g = a.tiles + a.off_a;
    const unsigned char *zero = a.tiles + kZeroOffset;
    const unsigned char *xb = (const unsigned char *)a.x;

    // waves 0-3 multiply (and store), waves 4-7 produce: copies, tables, pad fixups
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const bool prod = wave >= kWaves;
    const int pw = wave - kWaves;             // producer wave 0 .. 3
    const int ptid = tid - kThreads;          // producer thread 0 .. 255
    const int n16 = lane & 15, kg = lane >> 4;
    const int ps = wave & (a.NSUB - 1), q = wave / a.NSUB;
    const int m_loc0 = KS > 1 ? 0 : q * TM;   // first m-tile of this wave in the m-block
    const int s_off = KS > 1 ? q : 0;         // first step of this wave in a chunk

    // m-block: global m-tiles [mt_first, mt_first + MBT); its list groups from g_first
    const int mt_first = mb * a.MBT;
    const int g_first = a.n_groups == 1 ? 0 : mt_first / a.mt_per_group;

    unsigned char *D_res = lds;
    unsigned char *A_res = lds + a.lds_d;
    unsigned char *bufs = lds + a.lds_d + a.lds_a;
    const uint32_t lds0 = lds_addr(lds);               // LDS byte address of the dynamic area
    auto ldsa = [&](const unsigned char *p) { return lds0 + (uint32_t)(p - lds); };
    const int NB = a.NB;                                // LDS buffers: copies run NB - 1 items ahead
    auto bufp = [&](int i) { return bufs + (size_t)(i % NB) * a.lds_buf; };
    const int64_t tg = (int64_t)kGroups * a.NSUB;
    auto tset = [&](int t) { return (t - t_begin) & (kTableSets - 1); };

    // ---- staged input rows of tile t into its table set (one pass, no barrier: every
    // slot below the tile's last is written by one of its rows, the rest by others) ----
    auto setup_tile = [&](int t) {
        const int sb = tset(t);
        const int64_t G0 = (int64_t)t * tg;
        const int64_t G1 = min(G0 + tg, a.n_groups_total) - 1;
        const int g0 = (int)fdiv((uint32_t)G0, a.div_GPR), g1 = (int)fdiv((uint32_t)G1, a.div_GPR);
        const int nrows = g1 - g0 + 1;
        const int img0 = (int)fdiv((uint32_t)g0, a.div_Ho);
        const int kl = (int)fdiv((uint32_t)g1, a.div_Ho) - img0;   // image boundaries crossed
        const int used = (nrows - 1 - kl) * min(a.SH, a.KH) + kl * a.KH + a.KH;
        if (ptid >= 0 && ptid < nrows) {
            const int g = g0 + ptid;
            const int img = (int)fdiv((uint32_t)g, a.div_Ho), oh = g - img * a.Ho;
            const int k = img - img0;
            const int base = (ptid - k) * min(a.SH, a.KH) + k * a.KH;
            for (int r = 0; r < a.KH; ++r) {
                const int ih = oh * a.SH - a.PH + r;
                const bool in = ih >= 0 && ih < a.H;
                s_slot[sb][base + r] = in ? make_int2((int)((int64_t)img * a.Cin * a.x_cs + (int64_t)ih * a.W),
                                                      ih == a.H - 1 ? a.w_last : a.W)
                                          : make_int2(-1, 0);
            }
            s_rowbase[sb][ptid] = base;
        }
        for (int i = used + ptid; i < a.NSLOT; i += kThreads) s_slot[sb][i] = make_int2(-1, 0);
    };

    // ---- patch granules.  A chunk's patch holds, per channel, V copies of the tile's
    // staged input rows: at stride 1 copy m starts at input column m - PW, so the reads
    // of filter column s (copy s % V) start at a multiple of 4 elements; otherwise one
    // copy with LEFT zeros before input column 0.  Wave w issues copy slots
    // w * FR .. + FR - 1; slot u fills granules 64 u .. + 63, lane l granule 64 u + l
    // (channel v / CHG of the chunk, granule v % CHG of that channel's patch, looked up
    // in the tile's table below at each use).
    const int total_g = a.CC * a.CHG;                    // granules of a full chunk
    // Per tile, granule r of a channel's patch -> (element offset of its first element in
    // x for channel 0, or kNoData when it holds only pads / rows outside the image;
    // elements before the row start | elements past the row end << 3).  Two tables,
    // by tile parity: the tile being filled and the one being fixed up.
    auto build_lut = [&](int t) {
        const int sb = tset(t), ls = t & 1;
        for (int r = ptid; r < a.CHG; r += kThreads) {
            const int s = (int)fdiv((uint32_t)r, a.div_VSG), rem2 = r - s * a.VSG;
            const int slot = (int)fdiv((uint32_t)rem2, a.div_RG), gi = rem2 - slot * a.RG;
            const int2 so = s_slot[sb][slot];
            const int col0 = gi * a.GE + (a.V > 1 ? s - a.PW : -a.LEFT);
            int2 e = make_int2(kNoData, 0);
            if (so.x >= 0 && col0 < so.y && col0 + a.GE > 0)
                e = make_int2(so.x + col0, max(0, -col0) | (max(0, col0 + a.GE - so.y) << 3));
            s_lut[ls][r] = e;
        }
    };
    auto decode = [&](int ls, int j, int &off, int &meta) {
        const int v = (pw * a.FR + j) * 64 + lane;
        const int c_rel = (int)fdiv((uint32_t)v, a.div_CHG), r = v - c_rel * a.CHG;
        int kind = kKindNone, pads = 0;
        off = 0;
        if (v < total_g) {
            const int2 e = s_lut[ls][r];
            kind = e.x == kNoData ? kKindZero : kKindData;
            off = e.x + c_rel * (int)a.x_cs;
            pads = e.y;
        }
        meta = c_rel | ((pads >> 3) << 11) | ((pads & 7) << 14) | (kind << 17);
    };
    auto tail_of = [&](int m) { return (m >> 11) & 7; };
    auto head_of = [&](int m) { return (m >> 14) & 7; };

    // issue the copies of one chunk into buf (patch: data; zero rows, pads, channels past
    // the chunk's count and slots past the patch read zeros; weights when staged);
    // returns the wave's count
    // fmask: bit j set when this lane's granule j of the chunk needs fixup() after it
    // landed (pads inside the granule, or a copy that would read outside x).  Element
    // offsets fit 32 bits (x holds fewer than 2^31 elements).
    const uint32_t x_last = (uint32_t)(a.x_total - a.GE);   // last granule start inside x
    // The copies of one chunk go out in batches (four copies per lane) from a small
    // per-wave state: fill_begin() sets it up, each fill_step() issues one batch.
    int fj = 0, fc = 0, fc_end = 0, fcount = 0, fls = 0, fper_m = 1;
    int4 fcd = make_int4(0, 0, 0, 0);
    uint32_t fpbase = 0, fab = 0, fmask_acc = 0;
    int fFR = 0;   // patch copies of the chunk in progress (0: none)
    auto fill_begin = [&](int t, int4 cd, unsigned char *buf) {
        fls = t & 1;
        fcd = cd;
        fpbase = ldsa(buf) + (uint32_t)(pw * a.FR * 1024);
        fj = 0;
        fFR = a.FR;
        fmask_acc = 0;
        fcount = 0;
        fc = fc_end = 0;
        if (!a.resident) {
            // weight copies: per m-tile a contiguous run of ns * AI KB in both places;
            // wave w takes copies w * naw .. + naw - 1, in batches inside one run
            fper_m = (cd.y - cd.x) * AI;
            const int na = a.MBT * fper_m;
            const int naw = (na + kWaves - 1) / kWaves;
            fc = pw * naw;
            fc_end = min(na, fc + naw);
            fab = ldsa(buf + a.lds_patch);
        }
    };
    auto fill_step = [&]() -> bool {
        const bool patch = fj < fFR;
        if (!patch && fc >= fc_end) return false;
        const unsigned char *src[4];
        uint32_t dst;
        int nb;
        if (patch) {
            const int xcs = (int)a.x_cs;
            int2 le[4];
            int crel[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int v = (pw * a.FR + fj + u) * 64 + lane;
                crel[u] = (int)fdiv((uint32_t)v, a.div_CHG);
                const int r = v - crel[u] * a.CHG;
                le[u] = s_lut[fls][min(r, a.CHG - 1)];
                if (v >= total_g) crel[u] = fcd.w;   // past the patch: no data
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool live = (le[u].x != kNoData) & (crel[u] < fcd.w);
                const int e = le[u].x + (fcd.z + crel[u]) * xcs;
                const bool inside = (uint32_t)e <= x_last;
                src[u] = (live & inside) ? xb + (int64_t)e * (int)sizeof(E) : zero;
                const uint32_t need = (uint32_t)(live & (fj + u < fFR) & ((le[u].y != 0) | !inside));
                fmask_acc |= need << (fj + u);
            }
            nb = min(4, fFR - fj);
            dst = fpbase + (uint32_t)(fj * 1024);
        } else {
            const int m = fc / fper_m, r = fc - m * fper_m;
            nb = min(4, min(fc_end - fc, fper_m - r));
            src[0] = A_g + ((size_t)(mt_first + m) * a.S + fcd.x) * ASTEP + (size_t)r * 1024 + lane * 16;
            src[1] = src[0] + 1024;
            src[2] = src[0] + 2048;
            src[3] = src[0] + 3072;
            dst = fab + (uint32_t)fc * 1024;
        }
        dma_b4(src[0], src[1], src[2], src[3], dst, nb);
        fcount += nb;
        fj += patch ? 4 : 0;
        fc += patch ? 0 : nb;
        return true;
    };
    // all copies of one chunk at once; returns the wave's count
    auto fill = [&](int t, int4 cd, unsigned char *buf, uint32_t &fmask) {
        fill_begin(t, cd, buf);
        while (fill_step()) {
        }
        fmask = fmask_acc;
        fFR = 0;
        return fcount;
    };
    // after the copies landed: zero the elements of a granule before the row start and
    // past the row end, and load granules that would read outside x element by element;
    // only the granules flagged by fill() are decoded again
    auto fixup = [&](int t, int4 cd, unsigned char *buf, uint32_t fmask) {
        const int ls = t & 1;
        const int64_t cbase = (int64_t)cd.z * a.x_cs;
        while (fmask) {
            const int j = __builtin_ctz(fmask);
            fmask &= fmask - 1;
            int off, meta;
            decode(ls, j, off, meta);
            const int tail = tail_of(meta), head = head_of(meta);
            unsigned char *gp = buf + ((size_t)(pw * a.FR + j) * 64 + lane) * 16;
            E *dst = (E *)gp;
            const int64_t e = (int64_t)off + cbase;
            if (e < 0 || e + a.GE > a.x_total) {
                // all loads first, then the writes: one wait for the granule
                constexpr int kGE = 16 / (int)sizeof(E);
                const E *src = (const E *)a.x + e;
                E v[kGE];
#pragma unroll
                for (int i2 = 0; i2 < kGE; ++i2)
                    v[i2] = (i2 >= head && i2 < kGE - tail && e + i2 >= 0 && e + i2 < a.x_total) ? src[i2] : (E)0;
#pragma unroll
                for (int i2 = 0; i2 < kGE; ++i2) dst[i2] = v[i2];
            } else {
                // keep bytes [head, GE - tail) elements of the 16-byte granule, zero the rest
                const int lo = head * (int)sizeof(E), hi = 16 - tail * (int)sizeof(E);
                uint4 v = *(uint4 *)gp;
                uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    uint32_t keep = 0;
#pragma unroll
                    for (int b = 0; b < 4; ++b) keep |= (4 * d + b >= lo && 4 * d + b < hi) ? (0xffu << (8 * b)) : 0u;
                    w[d] &= keep;
                }
                *(uint4 *)gp = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
    };

    // this lane's pixel group of tile t: patch offset, group index
    auto lane_geom = [&](int t, int &pixoff, int64_t &grp) {
        const int sb = tset(t);
        const int64_t G0 = (int64_t)t * tg;
        const int64_t G1 = min(G0 + tg, a.n_groups_total) - 1;
        const int g0 = (int)fdiv((uint32_t)G0, a.div_GPR), g1 = (int)fdiv((uint32_t)G1, a.div_GPR);
        grp = G0 + ps * kGroups + n16;
        const int64_t gc = min(grp, G1);
        const int grow = (int)fdiv((uint32_t)gc, a.div_GPR);
        const int col4 = (int)(gc - (int64_t)grow * a.GPR);
        pixoff = s_rowbase[sb][min(grow - g0, g1 - g0)] * a.RS + a.POFF + 4 * col4 * a.SW;
    };

    f32x4 acc[TM][4];
    auto clear_acc = [&]() {
#pragma unroll
        for (int t = 0; t < TM; ++t)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[t][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    clear_acc();

    // bias + ReLU + rounding, stores of the lane's 4 pixels of its output rows.  No
    // divergent branches: lane masks are ballots and every store carries its mask;
    // returns the number of stores the wave issued.
    auto epilogue = [&](int64_t grp) {
        const bool pix_ok = grp < a.n_groups_total;
        const int64_t gq = pix_ok ? grp : 0;
        const int grow = (int)fdiv((uint32_t)gq, a.div_GPR);
        const int col4 = (int)(gq - (int64_t)grow * a.GPR);
        const int img = (int)fdiv((uint32_t)grow, a.div_Ho), oh = grow - img * a.Ho;
        const int ow = 4 * col4;
        const int lim = oh == a.Ho - 1 ? a.w_last_out : a.Wo;
        const int nvalid = pix_ok ? max(0, min(4, lim - ow)) : 0;
        const float qnan = __builtin_nanf("");
        // row map (kept filter of each computed row): loaded, and waited for, before the
        // first store, since the kernel counts its outstanding stores by hand
        // (tiles of another plan: no map is read and the rows below stay in range)
        int omap[TM][4] = {};
        if constexpr (MAP) {
            if (ok) {
#pragma unroll
                for (int t = 0; t < TM; ++t) {
                    const int gm = mt_first + m_loc0 + t;
                    const int mt_in = gm - (gm / a.mt_per_group) * a.mt_per_group;
#pragma unroll
                    for (int i = 0; i < 4; ++i) omap[t][i] = a.rowmap[mt_in * kMT + 4 * kg + i];
                }
                wait_vm_all();
            }
        }
        // lane masks of the tile: whole 4-pixel groups, and element e of partial groups
        const uint64_t full_px = ballot(nvalid == 4);
        const uint64_t part_px = ballot(nvalid > 0 && nvalid < 4);
        uint64_t part_e[3];
#pragma unroll
        for (int e = 0; e < 3; ++e) part_e[e] = part_px & ballot(e < nvalid);
        const size_t ybase = (size_t)img * a.Rout * a.y_cs + (size_t)oh * a.Wo + ow;   // row 0 at the lane's pixels
        int n = 0;
#pragma unroll
        for (int t = 0; t < TM; ++t) {
            const int gm = mt_first + m_loc0 + t;                      // global m-tile
            const int gidx = gm / a.mt_per_group, mt_in = gm - gidx * a.mt_per_group;
            const int rig0 = mt_in * kMT + 4 * kg;                     // the lane's first row inside the list group
            const int row0 = gidx * a.group_rows + rig0;
            const bool all_rows = uni((mt_in + 1) * kMT <= a.group_rows &&
                                      gidx * a.group_rows + (mt_in + 1) * kMT <= a.R ? 1 : 0) != 0;
            // bias, ReLU and the header check on the accumulators, each only when it applies
            if (!ok) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) acc[t][nt][i] = qnan;
            } else {
                if (a.bias) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float bv = s_bias[(m_loc0 + t) * kMT + 4 * kg + i];
#pragma unroll
                        for (int nt = 0; nt < 4; ++nt) acc[t][nt][i] += bv;
                    }
                }
                if (a.relu) {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int nt = 0; nt < 4; ++nt) acc[t][nt][i] = acc[t][nt][i] < 0.f ? 0.f : acc[t][nt][i];
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rig = rig0 + i, row = row0 + i;
                const bool row_ok = rig < a.group_rows && row < a.R;
                const uint64_t rmask = all_rows ? ~0ull : ballot(row_ok);
                size_t yo;
                if constexpr (MAP) {
                    const int orow = ok ? min(max(omap[t][i], 0), a.Rout - 1) : min(row, a.Rout - 1);
                    yo = ybase + (size_t)(row_ok ? orow : 0) * a.y_cs;
                } else {
                    yo = ybase + (size_t)(row_ok ? row : 0) * a.y_cs;
                }
                float o[4];
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) o[nt] = acc[t][nt][i];
                const uint64_t full = full_px & rmask;
                if (a.out_bf16) {
                    uint16_t *y = (uint16_t *)a.y + yo;
                    const uint32_t w01 = pk_bf16(o[0], o[1]), w23 = pk_bf16(o[2], o[3]);
                    const uint32_t h[3] = {w01 & 0xffffu, w01 >> 16, w23 & 0xffffu};
                    if (full) {
                        st_mask_b64(y, u32x2{w01, w23}, full);
                        ++n;
                    }
                    if (part_px) {
#pragma unroll
                        for (int e = 0; e < 3; ++e) {
                            const uint64_t me = part_e[e] & rmask;
                            if (me) {
                                st_mask_b16(y + e, h[e], me);
                                ++n;
                            }
                        }
                    }
                } else {
                    float *y = (float *)a.y + yo;
                    if (full) {
                        st_mask_b128(y, u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                                              __float_as_uint(o[3])}, full);
                        ++n;
                    }
                    if (part_px) {
#pragma unroll
                        for (int e = 0; e < 3; ++e) {
                            const uint64_t me = part_e[e] & rmask;
                            if (me) {
                                st_mask_b32(y + e, __float_as_uint(o[e]), me);
                                ++n;
                            }
                        }
                    }
                }
            }
        }
        return n;
    };

    // compute one chunk from buf for the lane's pixel group at pixoff
    auto compute = [&](int4 cd, const unsigned char *buf, int pixoff) {
        const int s0 = cd.x, s1 = cd.y;
        const int sf = s0 + s_off;
        if (sf >= s1) return;
        // weights of the wave's first m-tile at step sf, bytes per m-tile
        const unsigned char *Ab;
        int a_mstr;
        if (a.resident) {
            Ab = A_res + (m_loc0 * a.S + sf) * ASTEP;
            a_mstr = a.S * ASTEP;
        } else {
            Ab = buf + a.lds_patch + (m_loc0 * (s1 - s0) + s_off) * ASTEP;
            a_mstr = (s1 - s0) * ASTEP;
        }
        const int gl0 = a.n_groups == 1 ? 0 : (mt_first + m_loc0) / a.mt_per_group - g_first;
        const unsigned char *Db = D_res + (gl0 * a.LP + sf * kKS + kg * 8) * 2;
        const int d_gstr = TPG >= a.mt_per_group ? a.LP * 2 : 0;   // next list group of the wave
        compute_chunk<E, MODE, TM, TPG, KS>(acc, buf, Ab + lane * AB, a_mstr, Db, d_gstr,
                                            (s1 - sf + KS - 1) / KS, pixoff, a.SW, [] {});
    };

    // ---- work items (tile, chunk): NB buffers, copies NB - 1 items ahead ----
    const int nchx = max(nch, 1);
    const int n_items = (t_end - t_begin) * nchx;
    auto item_tile = [&](int i) { return t_begin + i / nchx; };
    auto item_chunk = [&](int i) { return i - (i / nchx) * nchx; };
    // Every barrier below is reached by all 8 waves (conditions are uniform over the
    // workgroup); the roles differ only in the work between barriers.
    if (prod) {
        for (int i = 0; i < NB && i < n_items; ++i)
            if (i == 0 || item_chunk(i) == 0) setup_tile(item_tile(i));
    } else if (a.bias) {
        for (int r = tid; r < a.MBT * kMT; r += kThreads) {
            const int gm = mt_first + r / kMT;
            const int gidx = gm / a.mt_per_group;
            const int row = gidx * a.group_rows + (gm - gidx * a.mt_per_group) * kMT + r % kMT;
            const int orow = MAP ? (ok ? min(max(a.rowmap[row], 0), a.Rout - 1) : min(row, a.Rout - 1)) : row;
            s_bias[r] = row < a.R ? a.bias[orow] : 0.f;
        }
    }
    __syncthreads();
    uint32_t fm0 = 0, fm1 = 0;   // fixup masks of the next two items in flight (producers)
    if (prod && nch > 0) {
        build_lut(item_tile(0));
        if (NB == 3 && n_items > 1 && item_chunk(1) == 0) build_lut(item_tile(1));
    }
    __syncthreads();
    if (prod && nch > 0) {
        // offsets and resident weights: contiguous runs over the producer waves
        auto run = [&](const unsigned char *src, uint32_t dst, int n16) {
            for (int q0 = pw * 64; q0 < n16; q0 += kThreads)
                if (q0 + lane < n16) dma16(src + (size_t)(q0 + lane) * 16, dst + (uint32_t)q0 * 16);
        };
        run(a.tiles + a.off_desc16 + (size_t)g_first * a.LP * 2, ldsa(D_res), a.MBG * a.LP * 2 / 16);
        if (a.resident) run(A_g + (size_t)mt_first * a.S * ASTEP, ldsa(A_res), a.MBT * a.S * ASTEP / 16);
        const int4 cd0 = chunk_at(table, 0);
        fill(item_tile(0), cd0, bufp(0), fm0);
        int n1 = 0;
        if (NB == 3 && n_items > 1) n1 = fill(item_tile(1), chunk_at(table, item_chunk(1)), bufp(1), fm1);
        wait_vm(n1);
        fixup(item_tile(0), cd0, bufp(0), fm0);
        fm0 = fm1;
    }
    __syncthreads();

    int pixoff = 0;
    int64_t grp = 0;
    for (int i = 0; i < n_items; ++i) {
        const int t = item_tile(i), c = item_chunk(i);
        if (!prod && c == 0) lane_geom(t, pixoff, grp);
        const int ia = i + NB - 1;   // item whose copies go out now
        if (nch > 0 && ia < n_items && item_chunk(ia) == 0) {   // first copies of a tile
            if (prod) build_lut(item_tile(ia));
            __syncthreads();
        }
        if (prod) {
            // copies of item ia (NB - 1 ahead); then item i + 1 landed: wait for every copy
            // issued before its last one, clear its pads
            int n2 = 0;
            if (nch > 0 && ia < n_items) {
                uint32_t fm;
                const int nf = fill(item_tile(ia), chunk_at(table, item_chunk(ia)), bufp(ia), fm);
                fm1 = NB == 3 ? fm : fm1;
                fm0 = NB == 3 ? fm0 : fm;
                n2 = NB == 3 ? nf : 0;
            }
            if (i + NB < n_items && item_chunk(i + NB) == 0) setup_tile(item_tile(i + NB));
            if (nch > 0 && i + 1 < n_items) {
                wait_vm(n2);
                fixup(item_tile(i + 1), chunk_at(table, item_chunk(i + 1)), bufp(i + 1), fm0);
                fm0 = fm1;
            }
        } else if (nch > 0) {
            compute(chunk_at(table, c), bufp(i), pixoff);
        }
        __syncthreads();
        // output of a finished tile: its stores overlap the next items
        if constexpr (KS == 1) {
            if (!prod && c == nchx - 1) {
                epilogue(grp);
                clear_acc();
            }
        }
    }

    // ---- partial sums of the waves that split the steps (one tile per workgroup) ----
    if constexpr (KS > 1) {
        f32x4 *red = (f32x4 *)lds;    // [region][TM][4][64 lanes]; the K loop is done with LDS
        const int region = TM * 4 * 64;
        if constexpr (KS == 4) {
            if (!prod && q >= 2) {
#pragma unroll
                for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) red[(q - 2) * region + (t2 * 4 + nt) * 64 + lane] = acc[t2][nt];
            }
            __syncthreads();
            if (!prod && q < 2) {
#pragma unroll
                for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) acc[t2][nt] += red[q * region + (t2 * 4 + nt) * 64 + lane];
            }
            __syncthreads();
        }
        if (!prod && q == 1) {
#pragma unroll
            for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) red[ps * region + (t2 * 4 + nt) * 64 + lane] = acc[t2][nt];
        }
        __syncthreads();
        if (prod || q != 0) return;
#pragma unroll
        for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[t2][nt] += red[ps * region + (t2 * 4 + nt) * 64 + lane];
        epilogue(grp);
    }
}

typedef void (*fwd_fn)(ConvArgs);

// Instantiation choice for one element type and gather mode; KSM is the set of step
// splits (bit KS) instantiated in the including translation unit.  MAP: the layer
// computes kept filters only and writes them through the row map.
template <typename E, int MODE, int TM, int TPG, int KSM, bool MAP = false>
fwd_fn pick_ks(int KS) {
    if constexpr ((KSM & 2) != 0) if (KS == 1) return k_fwd<E, MODE, TM, TPG, 1, MAP>;
    if constexpr ((KSM & 4) != 0) if (KS == 2) return k_fwd<E, MODE, TM, TPG, 2, MAP>;
    if constexpr ((KSM & 16) != 0) if (KS == 4) return k_fwd<E, MODE, TM, TPG, 4, MAP>;
    return nullptr;
}

// TMMAX: most m-tiles per wave instantiated (register budget of the gather mode).
// Row-mapped layers share one list over all m-tiles, so only TPG == TM exists for them.
template <typename E, int MODE, int KSM, int TMMAX>
fwd_fn pick_tm(int TM, int TPG, int KS, bool map) {
    if (map) {
        if (TPG != TM) return nullptr;
        switch (TM) {
            case 1: return pick_ks<E, MODE, 1, 1, KSM, true>(KS);
            case 2: if constexpr (TMMAX >= 2) return pick_ks<E, MODE, 2, 2, KSM, true>(KS); return nullptr;
            case 4: if constexpr (TMMAX >= 4) return pick_ks<E, MODE, 4, 4, KSM, true>(KS); return nullptr;
            default: return nullptr;
        }
    }
    switch (TM * 16 + TPG) {
        case 0x11: return pick_ks<E, MODE, 1, 1, KSM>(KS);
        case 0x21: if constexpr (TMMAX >= 2) return pick_ks<E, MODE, 2, 1, KSM>(KS); return nullptr;
        case 0x22: if constexpr (TMMAX >= 2) return pick_ks<E, MODE, 2, 2, KSM>(KS); return nullptr;
        case 0x41: if constexpr (TMMAX >= 4) return pick_ks<E, MODE, 4, 1, KSM>(KS); return nullptr;
        case 0x42: if constexpr (TMMAX >= 4) return pick_ks<E, MODE, 4, 2, KSM>(KS); return nullptr;
        case 0x44: if constexpr (TMMAX >= 4) return pick_ks<E, MODE, 4, 4, KSM>(KS); return nullptr;
        case 0x81: if constexpr (TMMAX >= 8) return pick_ks<E, MODE, 8, 1, KSM>(KS); return nullptr;
        case 0x82: if constexpr (TMMAX >= 8) return pick_ks<E, MODE, 8, 2, KSM>(KS); return nullptr;
        case 0x88: if constexpr (TMMAX >= 8) return pick_ks<E, MODE, 8, 8, KSM>(KS); return nullptr;
        default: return nullptr;
    }
}

}  // namespace fwd
}  // namespace bsp
