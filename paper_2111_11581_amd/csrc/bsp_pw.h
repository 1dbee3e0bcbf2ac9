// Forward kernel of pruned pointwise layers on gfx950: 1x1 convolutions without
// padding at stride 1 or 2, and fully connected layers (Sec. 4.2: the GEMM form of a
// 1x1 layer has one column per input channel).  Template; instantiated in
// bsp_pw_*.hip.
//
// A kept GEMM column of a pointwise layer is an input channel, so every operand row
// of the implicit GEMM is a plain input row: no shifted windows and no padding.
//  * Output pixels are taken in groups of 4.  At stride 1 an image is one run of
//    pixels (padded to whole 16-byte granules); at stride 2 every output row is a
//    run of groups.  Groups are numbered over all images; a workgroup tile is NSUB
//    runs of 16 groups (64 pixels each), for one m-block of output rows.
//  * The patch of a chunk is, for every channel of the chunk, the tile's input
//    granules: 16 bytes holding two groups (bf16, stride 1), one group (fp32, stride
//    1) or one group's 8 input pixels of which the even ones are used (bf16, stride
//    2).  Granules are copied with asynchronous direct-to-LDS loads; a thread always
//    copies the same granule position of the tile, for channels NGR apart, so its
//    source address is set up once per workgroup.  A granule past the end of the
//    image run only feeds output pixels that are never stored: 1x1 outputs depend on
//    their own pixel alone.
//  * Two LDS buffers: the copies of chunk c + 1 run while chunk c multiplies.  Gather
//    offsets and (when they fit) the m-block's weights stay in LDS for the whole K
//    loop; otherwise each chunk's slice of weights is copied with its patch.
//  * The multiply, the gathers and the epilogue are those of the general kernel:
//    lane l owns kept positions 8 (l / 16) .. + 7 and group l % 16 of its run.
// One tile per workgroup; several workgroups share a CU, so one workgroup's copies
// overlap another's multiply and stores.  Workgroup ids are remapped so that the
// m-blocks of one tile and neighbouring tiles run on one XCD and share its L2.
#pragma once

#include "bsp_fwd.h"

namespace bsp {
namespace pw {

using namespace bsp::fwd;

template <typename E, int MODE, int TM, int TPG, int KS, bool MAP = false>
__global__ __launch_bounds__(kThreads, pw_occ((int)sizeof(E), MODE, TM)) void k_pw(PwArgs a) {
    constexpr int AB = 8 * (int)sizeof(E);   // weight bytes per lane, one m-tile and step
    constexpr int ASTEP = 64 * AB;           // one m-tile, one step
    constexpr int AI = ASTEP / 1024;         // 1 KB copies per m-tile and step
    constexpr int GE = 16 / (int)sizeof(E);  // elements per granule
    extern __shared__ __attribute__((aligned(256))) unsigned char lds[];
    __shared__ __attribute__((aligned(16))) float s_bias[kMaxMBRows];
    __shared__ int s_orow[MAP ? kMaxMBRows : 1];   // output row of each row of the m-block (row map)

    // workgroup -> (range of pixel tiles, m-block); each XCD (workgroup id % 8) gets
    // a contiguous range of logical ids, the m-blocks of a tile range adjacent
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
    const unsigned char *xb = (const unsigned char *)a.x;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int n16 = lane & 15, kg = lane >> 4;
    const int ps = wave & (a.NSUB - 1), q = wave >> a.lg_nsub;
    const int m_loc0 = KS > 1 ? 0 : q * TM;   // first m-tile of this wave in the m-block
    const int s_off = KS > 1 ? q : 0;         // first step of this wave in a chunk
    const int mt_first = mb * a.MBT;
    const int g_first = a.n_groups == 1 ? 0 : mt_first / a.mt_per_group;
    const int TG = kGroups * a.NSUB;          // groups per tile

    unsigned char *D_res = lds;
    unsigned char *A_res = lds + a.lds_d;
    unsigned char *bufs = lds + a.lds_d + a.lds_a;
    const uint32_t lds0 = lds_addr(lds);
    auto ldsa = [&](const unsigned char *p) { return lds0 + (uint32_t)(p - lds); };

    // ---- patch copies: wave w issues copy slots w * FRW .. + FRW - 1 of a chunk; slot v
    // fills LDS granules 64 v .. + 63, lane l granule 64 v + l, which is position
    // gr = l % NGR of the tile for channel v * (64 / NGR) + l / NGR of the chunk.
    const int gr = lane & (a.NGR - 1);
    const int c_lane = lane >> a.lg_ngr;
    const int c_slot = 64 >> a.lg_ngr;
    const int slot0 = wave * a.FR;
    const unsigned char *zero = a.tiles + kZeroOffset;
    // element offset in channel 0 of the granule at position gr of tile t
    auto granule = [&](int t, int64_t &off0) {
        const int64_t Gg = (int64_t)t * TG + gr * a.gpg;
        if (Gg >= a.n_groups_total) return false;
        const int row = (int)fdiv((uint32_t)Gg, a.div_GPR);
        const int gi = (int)Gg - row * a.GPR;
        const int img = (int)fdiv((uint32_t)row, a.div_Ho);
        const int oh = row - img * a.Ho;
        off0 = (int64_t)img * a.x_is + (int64_t)oh * a.in_row + gi * 4 * a.SW;
        return true;
    };

    // issue the copies of chunk cd of tile t into buf: patch granules (channels past
    // the chunk and positions past the last group read zeros; a granule that would read
    // past the end of x reads zeros here and is completed by tail()), then (when staged)
    // the chunk's weights.  Returns the number of copies the wave issued.
    // element offsets fit 32 bits (x holds fewer than 2^31 elements)
    const uint32_t x_last = (uint32_t)(a.x_total - GE);   // last granule start inside x
    auto fill = [&](int t, int4 cd, unsigned char *buf) {
        int64_t off0 = 0;
        const bool g_ok = granule(t, off0);
        const uint32_t pb = ldsa(buf);
        const int xcs = (int)a.x_cs;
        const int ebase = (int)off0 + (cd.z + c_lane) * xcs;   // channel c_lane of the chunk
        const int cw = g_ok ? cd.w : 0;
        auto src_of = [&](int v) {
            const int c_rel = v * c_slot + c_lane;
            const int e = ebase + v * c_slot * xcs;
            const bool data = c_rel < cw && (uint32_t)e <= x_last;
            return data ? xb + (int64_t)e * (int)sizeof(E) : zero;
        };
        for (int k = 0; k < a.FR; k += 4) {
            const int v = slot0 + k;
            dma_b4(src_of(v), src_of(v + 1), src_of(v + 2), src_of(v + 3), pb + (uint32_t)v * 1024,
                   min(4, a.FR - k));
        }
        int n = a.FR;
        if (!a.resident) {
            // weight copies: per m-tile a contiguous run of ns * AI KB in both places;
            // wave w takes copies w * naw .. + naw - 1, in batches inside one run
            const int per_m = (cd.y - cd.x) * AI;
            const int na = a.MBT * per_m;
            const int naw = (na + kWaves - 1) / kWaves;
            const uint32_t ab = ldsa(buf + a.lds_patch);
            int c = wave * naw;
            const int c_end = min(na, c + naw);
            while (c < c_end) {
                const int m = c / per_m, r = c - m * per_m;
                const int nb = min(4, min(c_end - c, per_m - r));
                const unsigned char *src = A_g + ((size_t)(mt_first + m) * a.S + cd.x) * ASTEP + (size_t)r * 1024 + lane * 16;
                dma_b4(src, src + 1024, src + 2048, src + 3072, ab + (uint32_t)c * 1024, nb);
                n += nb;
                c += nb;
            }
        }
        return n;
    };
    // after the copies of (t, cd) landed: granules that would read past the end of x,
    // element by element (only the last granules of the last image can)
    auto tail = [&](int t, int4 cd, unsigned char *buf) {
        int64_t off0 = 0;
        if (!granule(t, off0)) return;
        if (off0 + (int64_t)(cd.z + cd.w - 1) * a.x_cs + GE <= a.x_total) return;
        for (int k = 0; k < a.FR; ++k) {
            const int v = slot0 + k;
            const int c_rel = v * c_slot + c_lane;
            const int64_t e = off0 + (int64_t)(cd.z + c_rel) * a.x_cs;
            if (c_rel < cd.w && e + GE > a.x_total) {
                E *dst = (E *)(buf + ((size_t)v * 64 + lane) * 16);
                const E *src = (const E *)a.x + e;
                // all loads first, then the writes: one wait for the granule
                E w[GE];
#pragma unroll
                for (int i2 = 0; i2 < GE; ++i2) w[i2] = e + i2 < a.x_total ? src[i2] : (E)0;
#pragma unroll
                for (int i2 = 0; i2 < GE; ++i2) dst[i2] = w[i2];
            }
        }
    };

    f32x4 acc[TM][4];
    auto clear_acc = [&]() {
#pragma unroll
        for (int t = 0; t < TM; ++t)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[t][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    clear_acc();

    // the lane's group: patch offset of its pixels (elements), the same in every tile
    const int pixoff = (ps * kGroups + n16) * 4 * a.SW;

    auto compute = [&](int4 cd, const unsigned char *buf) {
        const int s0 = cd.x, s1 = cd.y;
        const int sf = s0 + s_off;
        if (sf >= s1) return;
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
        const int d_gstr = TPG >= a.mt_per_group ? a.LP * 2 : 0;
        compute_chunk<E, MODE, TM, TPG, KS>(acc, buf, Ab + lane * AB, a_mstr, Db, d_gstr,
                                            (s1 - sf + KS - 1) / KS, pixoff, a.SW, [] {});
    };

    // bias + ReLU + rounding; each lane stores its group's pixels of its 4 rows per
    // m-tile (8 or 16 contiguous bytes; 16 lanes cover 64 pixels).  Masked stores from
    // ballots; returns the number of stores the wave issued.
    auto epilogue = [&](int t) {
        const int64_t grp = (int64_t)t * TG + ps * kGroups + n16;
        const bool pix_ok = grp < a.n_groups_total;
        const int64_t gq = pix_ok ? grp : 0;
        const int row = (int)fdiv((uint32_t)gq, a.div_GPR);
        const int gi = (int)gq - row * a.GPR;
        const int img = (int)fdiv((uint32_t)row, a.div_Ho);
        const int oh = row - img * a.Ho;
        const int p0 = oh * a.Wo + 4 * gi;
        const int nvalid = pix_ok ? max(0, min(4, a.Wo - 4 * gi)) : 0;
        // tiles of another plan: every output NaN (a NaN bias makes every sum NaN, and
        // ReLU keeps NaN)
        const float bad = ok ? 0.f : __builtin_nanf("");
        // lane masks of the tile: whole 4-pixel groups, and element e of partial groups
        const uint64_t full_px = ballot(nvalid == 4);
        const uint64_t part_px = ballot(nvalid > 0 && nvalid < 4);
        uint64_t part_e[3];
#pragma unroll
        for (int e = 0; e < 3; ++e) part_e[e] = part_px & ballot(e < nvalid);
        const int64_t ybase = (int64_t)img * a.y_is + p0;   // output row 0 at the lane's pixels
        int n = 0;
#pragma unroll
        for (int t2 = 0; t2 < TM; ++t2) {
            const int gm = mt_first + m_loc0 + t2;   // global m-tile
            const int gidx = gm / a.mt_per_group, mt_in = gm - gidx * a.mt_per_group;
            const int r0 = (m_loc0 + t2) * kMT + 4 * kg;       // the lane's first row in the m-block
            const int rig0 = mt_in * kMT + 4 * kg;             // ... inside the list group
            const int crow0 = gidx * a.group_rows + rig0;      // its computed row
            const bool all_rows = uni((mt_in + 1) * kMT <= a.group_rows &&
                                      gidx * a.group_rows + (mt_in + 1) * kMT <= a.R ? 1 : 0) != 0;
            // bias, ReLU and the header check on the accumulators, each only when it applies
            // (uniform branches: most layers need one of them or none)
            if (!ok) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) acc[t2][nt][i] = bad;
            } else {
                if (a.bias) {
                    const float4 bv = *(const float4 *)&s_bias[r0];
                    const float bvs[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int nt = 0; nt < 4; ++nt) acc[t2][nt][i] += bvs[i];
                }
                if (a.relu) {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int nt = 0; nt < 4; ++nt) acc[t2][nt][i] = acc[t2][nt][i] < 0.f ? 0.f : acc[t2][nt][i];
                }
            }
            const int64_t yrow = ybase + (int64_t)(rig0 < a.group_rows && crow0 < a.R ? crow0 : 0) * a.y_cs;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rig = rig0 + i, crow = crow0 + i;
                const bool row_ok = rig < a.group_rows && crow < a.R;
                const uint64_t rmask = all_rows ? ~0ull : ballot(row_ok);
                int64_t yo = yrow + (int64_t)i * a.y_cs;
                if constexpr (MAP) yo = ybase + (int64_t)(row_ok ? s_orow[r0 + i] : 0) * a.y_cs;
                if (!all_rows && !row_ok) yo = ybase;
                float o[4];
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) o[nt] = acc[t2][nt][i];
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

    // ---- work items (tile, chunk), NB buffers, copies NB - 1 items ahead ----
    if (a.bias || MAP)
        for (int r = tid; r < a.MBT * kMT; r += kThreads) {
            const int gm = mt_first + r / kMT;
            const int gidx = gm / a.mt_per_group;
            const int orow = gidx * a.group_rows + (gm - gidx * a.mt_per_group) * kMT + r % kMT;
            // tiles of another plan (!ok): no map is read; output rows stay in range
            const int out = MAP ? (orow < a.R && ok ? min(max(a.rowmap[orow], 0), a.Rout - 1) : min(orow, a.Rout - 1))
                                : orow;
            if constexpr (MAP) s_orow[r] = out;
            if (a.bias) s_bias[r] = orow < a.R ? a.bias[out] : 0.f;   // out < Rout: in the bias array
        }
    const int NB = a.NB;
    const int nchx = max(nch, 1);
    const int n_items = (t_end - t_begin) * nchx;
    // item counters: (tile, chunk, buffer) of the item computed and of the next to copy
    int ct = t_begin, cc = 0, cb = 0;
    int ft = t_begin, fc = 0, fb = 0;
    auto advance = [&](int &t, int &c, int &b) {
        if (++c == nchx) { c = 0; ++t; }
        if (++b == NB) b = 0;
    };
    if (nch > 0) {
        dma_run(a.tiles + a.off_desc16 + (size_t)g_first * a.LP * 2, ldsa(D_res), a.MBG * a.LP * 2 / 16);
        if (a.resident) dma_run(A_g + (size_t)mt_first * a.S * ASTEP, ldsa(A_res), a.MBT * a.S * ASTEP / 16);
        fill(ft, chunk_at(table, fc), bufs + (size_t)fb * a.lds_buf);
        advance(ft, fc, fb);
        int n1 = 0;
        if (NB == 3 && n_items > 1) {
            n1 = fill(ft, chunk_at(table, fc), bufs + (size_t)fb * a.lds_buf);
            advance(ft, fc, fb);
        }
        wait_vm(n1);
        tail(ct, chunk_at(table, cc), bufs + (size_t)cb * a.lds_buf);
    }
    __syncthreads();
    int n_st = 0;   // stores issued by the previous item's epilogue
    for (int i = 0; i < n_items; ++i) {
        int n2 = 0;
        if (nch > 0 && i + NB - 1 < n_items) {
            const int nf = fill(ft, chunk_at(table, fc), bufs + (size_t)fb * a.lds_buf);
            advance(ft, fc, fb);
            if (NB == 3) n2 = nf;
        }
        if (nch > 0) compute(chunk_at(table, cc), bufs + (size_t)cb * a.lds_buf);
        // item i + 1 landed: wait for every copy and store issued before its last copy
        if (nch > 0 && i + 1 < n_items) {
            wait_vm(NB == 3 ? n_st + n2 : 0);
            int nt = ct, nc = cc, nb2 = cb;
            advance(nt, nc, nb2);
            tail(nt, chunk_at(table, nc), bufs + (size_t)nb2 * a.lds_buf);
        }
        __syncthreads();
        n_st = 0;
        if constexpr (KS == 1) {
            if (cc == nchx - 1) {
                n_st = epilogue(ct);
                clear_acc();
            }
        }
        advance(ct, cc, cb);
    }

    // ---- partial sums of the waves that split the steps (one tile per workgroup) ----
    if constexpr (KS > 1) {
        f32x4 *red = (f32x4 *)lds;   // [region][TM][4][64 lanes]; the K loop is done with LDS
        const int region = TM * 4 * 64;
        if constexpr (KS == 4) {
            if (q >= 2) {
#pragma unroll
                for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) red[(q - 2) * region + (t2 * 4 + nt) * 64 + lane] = acc[t2][nt];
            }
            __syncthreads();
            if (q < 2) {
#pragma unroll
                for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) acc[t2][nt] += red[q * region + (t2 * 4 + nt) * 64 + lane];
            }
            __syncthreads();
        }
        if (q == 1) {
#pragma unroll
            for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) red[ps * region + (t2 * 4 + nt) * 64 + lane] = acc[t2][nt];
        }
        __syncthreads();
        if (q != 0) return;
#pragma unroll
        for (int t2 = 0; t2 < TM; ++t2)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[t2][nt] += red[ps * region + (t2 * 4 + nt) * 64 + lane];
        epilogue(t_begin);
    }
}

typedef void (*pw_fn)(PwArgs);

template <typename E, int MODE, int TM, int TPG, int KSM, bool MAP = false>
pw_fn pw_pick_ks(int KS) {
    if constexpr ((KSM & 2) != 0) if (KS == 1) return k_pw<E, MODE, TM, TPG, 1, MAP>;
    if constexpr ((KSM & 4) != 0) if (KS == 2) return k_pw<E, MODE, TM, TPG, 2, MAP>;
    if constexpr ((KSM & 16) != 0) if (KS == 4) return k_pw<E, MODE, TM, TPG, 4, MAP>;
    return nullptr;
}

// TMMAX: most m-tiles per wave instantiated.  MAP (row-mapped layers: one list shared
// by all m-tiles) exists for TPG == TM only.
template <typename E, int MODE, int KSM, int TMMAX>
pw_fn pw_pick_tm(int TM, int TPG, int KS, bool map) {
    if (map) {
        if (TPG != TM) return nullptr;
        switch (TM) {
            case 1: return pw_pick_ks<E, MODE, 1, 1, KSM, true>(KS);
            case 2: if constexpr (TMMAX >= 2) return pw_pick_ks<E, MODE, 2, 2, KSM, true>(KS); return nullptr;
            case 4: if constexpr (TMMAX >= 4) return pw_pick_ks<E, MODE, 4, 4, KSM, true>(KS); return nullptr;
            default: return nullptr;
        }
    }
    switch (TM * 16 + TPG) {
        case 0x11: return pw_pick_ks<E, MODE, 1, 1, KSM>(KS);
        case 0x21: if constexpr (TMMAX >= 2) return pw_pick_ks<E, MODE, 2, 1, KSM>(KS); return nullptr;
        case 0x22: if constexpr (TMMAX >= 2) return pw_pick_ks<E, MODE, 2, 2, KSM>(KS); return nullptr;
        case 0x41: if constexpr (TMMAX >= 4) return pw_pick_ks<E, MODE, 4, 1, KSM>(KS); return nullptr;
        case 0x42: if constexpr (TMMAX >= 4) return pw_pick_ks<E, MODE, 4, 2, KSM>(KS); return nullptr;
        case 0x44: if constexpr (TMMAX >= 4) return pw_pick_ks<E, MODE, 4, 4, KSM>(KS); return nullptr;
        default: return nullptr;
    }
}

}  // namespace pw
}  // namespace bsp
