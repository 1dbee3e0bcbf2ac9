// Forward kernel of pointwise layers (1x1 convolutions without padding at stride 1 or
// 2, fully connected layers, and convolutions run over their im2col input; Sec. 4.2:
// the GEMM form of a 1x1 layer has one column per input channel).  Template;
// instantiated in bsp_pl_*.hip.
//
// Two kinds of K loop:
//  * identity list (G = 0: row blocks stored with zeros for their removed rows, dense
//    and unstructured layers): every 32-wide step is 32 consecutive input channels;
//  * gathered lists (G >= 1: column and block-punched blocks): the m-block holds G list
//    groups (block-rows) and step s of group g is the 32 channels of entries 32 s ..
//    32 s + 31 of g's list of kept columns (Sec. 4.1.1), each channel a row of the
//    input; the lists of the m-block sit in LDS for the whole run and every step
//    stages one patch per group.
// Either way a step's operands sit at fixed LDS offsets, so the multiplying waves
// need no gather offsets.  A workgroup has 8 waves and owns one m-block (MB rows)
// and a run of pixel tiles (NP = 64 NSUB output pixels each):
//  * waves 4-7 copy: per stage (SPS steps) each issues the same number of 16-byte
//    direct-to-LDS copies: for every step, its share of the stage's input granules
//    (G x 32 channels x NP pixels) and, unless the m-block's weights stay in LDS for
//    the whole run (copied once at the start), of its weight tiles (MB / 64 tiles of
//    1 KB); the sources are set up once per tile.  Copies run NB - 1 stages ahead, so
//    every wait is for a constant count;
//  * waves 0-3 multiply: wave w works on sub-tile w % NSUB and m-tiles
//    (w / NSUB) * TM .. + TM - 1 (one list group); per step it reads its weights (one
//    16-byte LDS read per m-tile) and the 8 channels x 4 pixels of its lane of its
//    group's patch (8-byte reads, 16-byte at stride 2) at compile-time offsets,
//    re-packs them with v_perm into the B operands of 4 MFMA 16x16x32 bf16 and
//    multiplies; steps of a stage are software-pipelined.  At the end of a tile they
//    add bias, apply ReLU, round to bf16 and store.
// One barrier per stage; the stores of a finished tile overlap the next tile.
#pragma once

#include "bsp_fwd.h"

namespace bsp {
namespace pl {

using namespace bsp::fwd;

constexpr int kPlThreads = 512;

// MODE 1: stride 1, a granule holds two 4-pixel groups; MODE 2: stride 2, a granule
// holds the 8 input pixels of one group (the even ones are used).
// G: list groups of an m-block (0: the identity list).  With G > 1 the m-block's MT
// m-tiles are G whole groups of MT / G m-tiles; with G = 1 the m-block lies inside one
// group.  A wave's TM m-tiles always lie in one group.
template <int MODE, int NSUB, int TM, bool MAP = false, int G = 0>
__global__ __launch_bounds__(kPlThreads, 1) void k_pl(PwArgs a) {
    typedef Gat<uint16_t, MODE> GT;
    constexpr int Q = kWaves / NSUB;              // multiplying waves per sub-tile
    constexpr int MT = TM * Q;                    // m-tiles of the m-block
    constexpr int NP = 64 * NSUB;                 // output pixels of a tile
    constexpr int RB = NP * 2 * MODE;             // patch bytes per channel
    constexpr int GPC = RB / 16;                  // granules per channel
    constexpr int GG = G == 0 ? 1 : G;            // patches per step
    constexpr int PCOPY = GG * 32 * GPC / kThreads;   // patch copies per producer wave and step
    constexpr int WCOPY = MT / kWaves;            // weight copies per producer wave and step
    static_assert(32 * GPC % kThreads == 0 && MT % kWaves == 0, "whole copies per wave");
    static_assert(G <= 1 || (MT % G == 0 && (MT / G) % TM == 0), "a wave's m-tiles lie in one group");
    static_assert(!MAP || G == 0, "row maps come with the identity list");
    constexpr int PB1 = 32 * RB;                  // LDS bytes of one group's patch of a step
    constexpr int PB = GG * PB1;                  // LDS bytes of one step's patches
    extern __shared__ __attribute__((aligned(256))) unsigned char lds[];
    __shared__ __attribute__((aligned(16))) float s_bias[kMaxMBRows];
    __shared__ int s_orow[MAP ? kMaxMBRows : 1];

    // workgroup -> (K part, range of pixel tiles, m-block); each XCD (workgroup id % 8)
    // gets a contiguous range of logical ids, the m-blocks of a tile range adjacent
    const int per = gridDim.x >> 3;
    const int lid0 = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    if (lid0 >= a.grid_valid) return;
    const int kp = a.ks > 1 ? (int)fdiv((uint32_t)lid0, a.div_kpart) : 0;
    const int lid = lid0 - kp * a.kpart_wgs;
    const int jr = (int)fdiv((uint32_t)lid, a.div_nmb);
    const int mb = lid - jr * a.n_mb;
    const int t_begin = jr * a.tiles_per_wg;
    const int t_end = min(a.n_pt, t_begin + a.tiles_per_wg);
    if (t_begin >= t_end) return;

    const TileHeader *hdr = (const TileHeader *)a.tiles;
    const bool ok = hdr->magic == kMagic && hdr->fp_lo == a.fp_lo && hdr->fp_hi == a.fp_hi;
    const unsigned char *A_g = a.tiles + a.off_a;
    const unsigned char *xb = (const unsigned char *)a.x;
    const unsigned char *zero = a.tiles + kZeroOffset;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const bool prod = wave >= kWaves;
    const int rw = wave & (kWaves - 1);   // wave index inside its role
    const int n16 = lane & 15, kg = lane >> 4;
    const int ps = rw % NSUB, q = rw / NSUB;
    const int m_loc0 = q * TM;
    const int mt_first = mb * MT;
    // steps (32 channels each) of the K loop: with the K loop split over workgroups
    // (ks parts) this workgroup runs steps s0 .. s0 + S - 1 and stores fp32 partial sums
    const int S_tot = a.S;                // steps of the whole loop (stride of the weight tiles)
    const int s0 = kp * a.s_per;
    const int S = a.ks > 1 ? min(a.s_per, S_tot - s0) : S_tot;
    const int SPS = a.SMAX;               // steps per stage
    const int NS = (S + SPS - 1) / SPS;   // stages per tile
    const int NB = a.NB;
    const bool res = a.resident;          // the m-block's weights stay in LDS ([m-tile][step], 1 KB each)
    const int wcopy = res ? 0 : WCOPY;
    const int stage_b = SPS * PB + (res ? 0 : SPS * MT * 1024);   // patches of the stage, then its weights
    unsigned char *const lds_w = lds + (G > 0 ? a.lds_d : 0);   // resident weights
    unsigned char *bufs = lds_w + (res ? MT * S * 1024 : 0);
    const uint32_t ldsw0 = lds_addr(lds_w);
    const uint32_t bufs0 = lds_addr(bufs);
    const int n_items = (t_end - t_begin) * (ok ? NS : 1);
    // gathered lists: the m-block's G lists (16-bit channels, LP entries each) at LDS
    // byte 0, before the weights and the buffers
    const uint16_t *s_list = (const uint16_t *)lds + s0 * 32;   // entries of the part's first step

    // ---- producers: copy k of a step fills LDS granules gid = (rw * PCOPY + k) * 64 + lane
    // of the step's patches (byte 16 gid): list group lg = gid / (32 GPC), channel
    // c = gid / GPC % 32 of the step, granule g = gid % GPC of the tile row; a wave's
    // copies are 1 KB apart, so four share one M0 ----
    const int xcs = (int)a.x_cs;
    const uint32_t x_last = (uint32_t)(a.x_total - 8);   // last granule start inside x
    int e_base[PCOPY];     // element offset of the copy's granule: at channel 0 of the step
                           // (identity list), at channel 0 of x (gathered lists)
    int c_of[PCOPY];       // its channel within a step (identity list), its list entry at step 0
    bool g_live[PCOPY];    // the granule holds output pixels
    int cur_tile = -1;
    // fast path: sources as a scalar base plus a 32-bit per-lane byte offset
    const int rwu = uni(rw);
    const unsigned char *xbu = (const unsigned char *)uni_ptr(xb);
    uint32_t w_voff[WCOPY];   // weight tile u of this wave: lane bytes, relative to tile 0
#pragma unroll
    for (int u = 0; u < WCOPY; ++u) w_voff[u] = (uint32_t)(lane * 16 + u * S_tot * 1024);
    auto set_tile = [&](int t) {
        if (t == cur_tile) return;
        cur_tile = t;
#pragma unroll
        for (int k = 0; k < PCOPY; ++k) {
            const int gid = (rw * PCOPY + k) * 64 + lane;
            const int c = gid / GPC % 32, g = gid % GPC;
            const int64_t Gg = (int64_t)t * (kGroups * NSUB) + (int64_t)g * a.gpg;
            g_live[k] = Gg < a.n_groups_total;
            int64_t off = 0;
            if (g_live[k]) {
                const int row = (int)fdiv((uint32_t)Gg, a.div_GPR);
                const int gi = (int)Gg - row * a.GPR;
                const int img = (int)fdiv((uint32_t)row, a.div_Ho);
                const int oh = row - img * a.Ho;
                off = (int64_t)img * a.x_is + (int64_t)oh * a.in_row + gi * 4 * a.SW +
                      (G == 0 ? (int64_t)c * a.x_cs : 0);
            }
            e_base[k] = (int)off;   // x holds fewer than 2^31 elements
            c_of[k] = G == 0 ? c : gid / (32 * GPC) * a.LP + c;
        }
    };
    // copies of stage st of tile t into buffer b; every producer wave issues exactly
    // SPS * (PCOPY + wcopy) copies (steps past the K loop read zeros)
    auto fill = [&](int t, int st, int b) {
        set_tile(t);
        const uint32_t buf = bufs0 + (uint32_t)(b * stage_b);
        if (t != a.n_pt - 1 && (st + 1) * SPS <= S && (G > 0 || (s0 + (st + 1) * SPS) * 32 <= a.Cin)) {
            // every granule of the stage is inside x and every channel exists (not the
            // last tile, not past the K loop): scalar bases, one VALU add per copy (a
            // multiply-add with the list's channel for gathered lists)
            int ch[PCOPY];
            if constexpr (G > 0) {
#pragma unroll
                for (int k = 0; k < PCOPY; ++k) ch[k] = s_list[c_of[k] + st * SPS * 32];
            }
            for (int j = 0; j < SPS; ++j) {
                const int s = st * SPS + j;
                const uint32_t pb = buf + (uint32_t)(j * PB);
                if constexpr (G > 0) {
                    // this step's channels, the next step's read ahead
                    int cur[PCOPY];
#pragma unroll
                    for (int k = 0; k < PCOPY; ++k) cur[k] = ch[k];
                    if (j + 1 < SPS) {
#pragma unroll
                        for (int k = 0; k < PCOPY; ++k) ch[k] = s_list[c_of[k] + (s + 1) * 32];
                    }
#pragma unroll
                    for (int k = 0; k < PCOPY; ++k)
                        dma_sv(xbu, (uint32_t)(e_base[k] + cur[k] * xcs) * 2u,
                               pb + (uint32_t)((rwu * PCOPY + k) * 1024));
                } else {
                    const uint32_t step_b = (uint32_t)(s0 + s) * 64u * (uint32_t)xcs;   // 32 channels, bytes
#pragma unroll
                    for (int k = 0; k < PCOPY; ++k)
                        dma_sv(xbu, (uint32_t)e_base[k] * 2u + step_b, pb + (uint32_t)((rwu * PCOPY + k) * 1024));
                }
                if (!res) {
                    const unsigned char *wbase = A_g + ((size_t)(mt_first + rwu * WCOPY) * S_tot + s0 + s) * 1024;
                    const uint32_t wb = buf + (uint32_t)(SPS * PB + j * MT * 1024);
#pragma unroll
                    for (int u = 0; u < WCOPY; ++u) dma_sv(wbase, w_voff[u], wb + (uint32_t)((rwu * WCOPY + u) * 1024));
                }
            }
            return;
        }
        for (int j = 0; j < SPS; ++j) {
            const int s = st * SPS + j;
            const uint32_t pb = buf + (uint32_t)(j * PB);
            const unsigned char *src[PCOPY];
#pragma unroll
            for (int k = 0; k < PCOPY; ++k) {
                int e;
                bool live;
                if constexpr (G > 0) {
                    e = e_base[k] + (s < S ? (int)s_list[c_of[k] + s * 32] : 0) * xcs;
                    live = g_live[k] && s < S && (uint32_t)e <= x_last;
                } else {
                    e = e_base[k] + (s0 + s) * 32 * xcs;
                    live = g_live[k] && s < S && (s0 + s) * 32 + c_of[k] < a.Cin && (uint32_t)e <= x_last;
                }
                src[k] = live ? xb + (int64_t)e * 2 : zero;
            }
#pragma unroll
            for (int k = 0; k < PCOPY; k += 4)
                dma_b4(src[k], src[min(k + 1, PCOPY - 1)], src[min(k + 2, PCOPY - 1)], src[min(k + 3, PCOPY - 1)],
                       pb + (uint32_t)((rw * PCOPY + k) * 1024), min(4, PCOPY - k));
            if (!res) {
                // weight tiles m = rw * WCOPY + u of the m-block
                const uint32_t wb = buf + (uint32_t)(SPS * PB + j * MT * 1024);
                const unsigned char *ws[WCOPY];
#pragma unroll
                for (int u = 0; u < WCOPY; ++u)
                    ws[u] = s < S ? A_g + ((size_t)(mt_first + rw * WCOPY + u) * S_tot + s0 + s) * 1024 + lane * 16
                                  : zero;
#pragma unroll
                for (int u = 0; u < WCOPY; u += 4)
                    dma_b4(ws[u], ws[min(u + 1, WCOPY - 1)], ws[min(u + 2, WCOPY - 1)], ws[min(u + 3, WCOPY - 1)],
                           wb + (uint32_t)((rw * WCOPY + u) * 1024), min(4, WCOPY - u));
            }
        }
    };
    // after stage st of tile t landed in buffer b: granules that would read past the
    // end of x, element by element.  Only the last channel of the last image ends
    // there, so only the last tile can hold such granules, and with the identity list
    // only its last stage; every other item returns at once (the element loads wait
    // for all copies in flight).
    auto tail = [&](int t, int st, int b) {
        if (t != a.n_pt - 1 || (G == 0 && st != NS - 1)) return;
        set_tile(t);
        for (int j = 0; j < SPS; ++j) {
            const int s = st * SPS + j;
#pragma unroll
            for (int k = 0; k < PCOPY; ++k) {
                int64_t e;
                bool chan;
                if constexpr (G > 0) {
                    e = (int64_t)e_base[k] + (int64_t)(s < S ? (int)s_list[c_of[k] + s * 32] : 0) * xcs;
                    chan = true;
                } else {
                    e = (int64_t)e_base[k] + (int64_t)(s0 + s) * 32 * xcs;
                    chan = (s0 + s) * 32 + c_of[k] < a.Cin;
                }
                if (g_live[k] && s < S && chan && e + 8 > a.x_total) {
                    uint16_t *dst = (uint16_t *)(bufs + b * stage_b + j * PB + ((rw * PCOPY + k) * 64 + lane) * 16);
                    const uint16_t *sx = (const uint16_t *)a.x + e;
                    // all loads first, then the writes: one wait for the granule
                    uint16_t v[8];
#pragma unroll
                    for (int i2 = 0; i2 < 8; ++i2) v[i2] = e + i2 < a.x_total ? sx[i2] : (uint16_t)0;
#pragma unroll
                    for (int i2 = 0; i2 < 8; ++i2) dst[i2] = v[i2];
                }
            }
        }
    };

    // ---- multiplying waves ----
    f32x4 acc[TM][4];
    auto clear_acc = [&]() {
#pragma unroll
        for (int t = 0; t < TM; ++t)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[t][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    clear_acc();
    // lane's 8 channels x 4 pixels of a step: channel 8 kg + j at byte j * RB, pixels of
    // group n16 of sub-tile ps, in the patch of the wave's list group
    const int glw = G > 1 ? m_loc0 / (MT / GG) : 0;
    const int b_lane = glw * PB1 + 8 * kg * RB + (ps * kGroups + n16) * 4 * 2 * MODE;
    // weights of step j of a stage (m-tile t at + t * a_mstr)
    const int a_mstr = res ? S * 1024 : 1024;
    auto read_step = [&](const unsigned char *pb, const unsigned char *w, typename GT::Raw &r, uint4 (&ar)[TM]) {
        const unsigned char *p = pb + b_lane;
#pragma unroll
        for (int j = 0; j < 8; ++j) __builtin_memcpy(&r.v[j], p + j * RB, sizeof(r.v[j]));
#pragma unroll
        for (int t = 0; t < TM; ++t) ar[t] = *(const uint4 *)(w + t * a_mstr);
    };
    auto mul_step = [&](const typename GT::Raw &r, const uint4 (&ar)[TM]) {
        typename GT::Frag f;
        GT::finish(r, f);
#pragma unroll
        for (int t = 0; t < TM; ++t) GT::mma(ar[t], f, acc[t]);
    };
    auto compute = [&](int st, int b) {
        const int nst = min(SPS, S - st * SPS);
        const unsigned char *buf = bufs + b * stage_b;
        // weights of the stage's first step for this wave's first m-tile and lane; step j: + j * a_step
        const unsigned char *w0 = res ? lds_w + ((m_loc0 * S + st * SPS) * 1024 + lane * 16)
                                      : buf + SPS * PB + m_loc0 * 1024 + lane * 16;
        const int a_step = res ? 1024 : MT * 1024;
        typename GT::Raw r0, r1;
        uint4 a0[TM], a1[TM];
        read_step(buf, w0, r0, a0);
        int j = 0;
        for (; j + 1 < nst; j += 2) {
            read_step(buf + (j + 1) * PB, w0 + (j + 1) * a_step, r1, a1);
            mul_step(r0, a0);
            if (j + 2 < nst) read_step(buf + (j + 2) * PB, w0 + (j + 2) * a_step, r0, a0);
            mul_step(r1, a1);
        }
        if (j < nst) mul_step(r0, a0);
    };

    // bias + ReLU + rounding; each lane stores its group's 4 pixels of its 4 rows per
    // m-tile (8 contiguous bytes, 16 for fp32 outputs; 16 lanes cover 64 pixels),
    // masked by ballots
    auto epilogue = [&](int t) {
        const int64_t grp = (int64_t)t * (kGroups * NSUB) + ps * kGroups + n16;
        const bool pix_ok = grp < a.n_groups_total;
        const int64_t gq = pix_ok ? grp : 0;
        const int row = (int)fdiv((uint32_t)gq, a.div_GPR);
        const int gi = (int)gq - row * a.GPR;
        const int img = (int)fdiv((uint32_t)row, a.div_Ho);
        const int oh = row - img * a.Ho;
        const int p0 = oh * a.Wo + 4 * gi;
        const int nvalid = pix_ok ? max(0, min(4, a.Wo - 4 * gi)) : 0;
        const float qnan = __builtin_nanf("");
        // lane masks of the tile: whole 4-pixel groups, and element e of partial groups
        const uint64_t full_px = ballot(nvalid == 4);
        const uint64_t part_px = ballot(nvalid > 0 && nvalid < 4);
        uint64_t part_e[3];
#pragma unroll
        for (int e = 0; e < 3; ++e) part_e[e] = part_px & ballot(e < nvalid);
        const int64_t ybase = (int64_t)img * a.y_is + p0;   // output row 0 at the lane's pixels
#pragma unroll
        for (int t2 = 0; t2 < TM; ++t2) {
            const int r0 = (m_loc0 + t2) * kMT + 4 * kg;     // the lane's first row in the m-block
            // its computed row: m-tiles of the identity list follow each other; a list
            // group's m-tiles hold its group_rows rows (rig: row inside the group)
            int crow0, rig0 = 0;
            bool all_rows;
            if constexpr (G == 0) {
                crow0 = mt_first * kMT + r0;
                all_rows = uni((mt_first + m_loc0 + t2 + 1) * kMT <= a.R ? 1 : 0) != 0;   // wave-uniform
            } else {
                const int gm = mt_first + m_loc0 + t2;
                const int gidx = gm / a.mt_per_group, mt_in = gm - gidx * a.mt_per_group;
                rig0 = mt_in * kMT + 4 * kg;
                crow0 = gidx * a.group_rows + rig0;
                all_rows = uni((mt_in + 1) * kMT <= a.group_rows && gidx * a.group_rows + (mt_in + 1) * kMT <= a.R
                                   ? 1 : 0) != 0;
            }
            // bias, ReLU and the header check on the accumulators, each only when it applies
            // (uniform branches: most layers need one of them or none)
            if (!ok) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt) acc[t2][nt][i] = qnan;
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
            int64_t yrow = ybase + (int64_t)(rig0 < a.group_rows && crow0 < a.R ? crow0 : 0) * a.y_cs;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int crow = crow0 + i;
                const bool row_ok = (G == 0 || rig0 + i < a.group_rows) && crow < a.R;
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
                    if (full) st_mask_b64(y, u32x2{w01, w23}, full);
                    if (part_px) {
#pragma unroll
                        for (int e = 0; e < 3; ++e) {
                            const uint64_t me = part_e[e] & rmask;
                            if (me) st_mask_b16(y + e, h[e], me);
                        }
                    }
                } else {
                    float *y = (float *)a.y + (a.ks > 1 ? kp * a.part_stride : 0) + yo;   // K part kp: its partial sums
                    if (full)
                        st_mask_b128(y, u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                                              __float_as_uint(o[3])}, full);
                    if (part_px) {
#pragma unroll
                        for (int e = 0; e < 3; ++e) {
                            const uint64_t me = part_e[e] & rmask;
                            if (me) st_mask_b32(y + e, __float_as_uint(o[e]), me);
                        }
                    }
                }
            }
        }
    };

    // bias and row map of the m-block (multiplying waves; read before the first barrier)
    if (!prod && (a.bias || MAP)) {
        for (int r = tid; r < MT * kMT; r += kThreads) {
            int crow = mt_first * kMT + r;
            if constexpr (G > 0) {
                const int gm = mt_first + r / kMT;
                const int gidx = gm / a.mt_per_group;
                crow = gidx * a.group_rows + (gm - gidx * a.mt_per_group) * kMT + r % kMT;
            }
            // tiles of another plan (!ok): no map is read; output rows stay in range
            const int out = MAP ? (crow < a.R && ok ? min(max(a.rowmap[crow], 0), a.Rout - 1) : min(crow, a.Rout - 1))
                                : crow;
            if constexpr (MAP) s_orow[r] = out;
            if (a.bias) s_bias[r] = crow < a.R ? a.bias[out] : 0.f;
        }
    }
    // every producer wave issues NCP copies per item (tile, stage), so when an item is
    // awaited the copies of the NB - 2 items issued after it may still be in flight.
    // Items are walked with cursors (tile, stage, buffer); nothing is divided in the loop.
    const int NCP = SPS * (PCOPY + wcopy);
    int ft = t_begin, fs = 0, fb = 0;   // next item to copy
    int wt = t_begin, ws = 0, wb = 0;   // next item to await
    auto adv = [&](int &t, int &st, int &b) {
        if (++st == NS) { st = 0; ++t; }
        if (++b == NB) b = 0;
    };
    if constexpr (G > 0) {
        // the m-block's lists (groups g_first .. g_first + GG - 1, consecutive in
        // dev_tiles), before any copy is issued; not read from tiles of another plan
        if (ok) {
            const int g_first = mt_first / a.mt_per_group;
            const uint32_t *src = (const uint32_t *)(a.tiles + a.off_desc16 + (size_t)g_first * a.LP * 2);
            uint32_t *dst = (uint32_t *)lds;
            const int nw = GG * a.LP / 2;
            for (int i = tid; i < nw; i += kPlThreads) dst[i] = src[i];
        }
        __syncthreads();
    }
    if (prod && ok) {
        if (res) {   // the m-block's weights: MT * S blocks of 1 KB, contiguous in dev_tiles
            if (a.ks == 1) {
                const unsigned char *src = A_g + (size_t)mt_first * S * 1024 + lane * 16;
                const int nblk = MT * S;
                for (int b0 = rw * 4; b0 < nblk; b0 += 16) {
                    const unsigned char *sb = src + (size_t)b0 * 1024;
                    dma_b4(sb, sb + 1024, sb + 2048, sb + 3072, ldsw0 + (uint32_t)b0 * 1024, min(4, nblk - b0));
                }
            } else {   // the part's steps of each m-tile: runs of S blocks, S_tot apart
                for (int b0 = rw; b0 < MT * S; b0 += kWaves) {
                    const int m = b0 / S, j = b0 - m * S;
                    dma_b4(A_g + ((size_t)(mt_first + m) * S_tot + s0 + j) * 1024 + lane * 16, nullptr, nullptr,
                           nullptr, ldsw0 + (uint32_t)b0 * 1024, 1);
                }
            }
        }
        for (int i = 0; i < NB - 1 && i < n_items; ++i) {
            fill(ft, fs, fb);
            adv(ft, fs, fb);
        }
        wait_vm(min(NB - 2, n_items - 1) * NCP);
        tail(wt, ws, wb);
        adv(wt, ws, wb);
    }
    __syncthreads();
    int ct = t_begin, cs = 0, cb = 0;   // item computed now
    const int nsx = ok ? NS : 1;
    for (int i = 0; i < n_items; ++i) {
        if (prod) {
            if (ok) {
                const bool more = i + NB - 1 < n_items;   // item i + NB - 1 goes out now
                if (more) {
                    fill(ft, fs, fb);
                    adv(ft, fs, fb);
                }
                if (i + 1 < n_items) {
                    // item i + 1 landed: the copies of items i + 2 .. min(i + NB - 1, last) may be pending
                    wait_vm(more ? (NB - 2) * NCP : max(0, n_items - 2 - i) * NCP);
                    tail(wt, ws, wb);
                    adv(wt, ws, wb);
                }
            }
        } else if (ok) {
            compute(cs, cb);
        }
        __syncthreads();
        // output of a finished tile: its stores overlap the next items
        if (!prod && cs == nsx - 1) {
            epilogue(ct);
            clear_acc();
        }
        if (++cs == nsx) { cs = 0; ++ct; }
        if (++cb == NB) cb = 0;
    }
}

typedef void (*pl_fn)(PwArgs);

// Instantiation choice: the m-block must hold a multiple of 4 m-tiles (one weight
// tile per copying wave and step), so with two sub-tiles a wave has 2 or 4 m-tiles.
template <int MODE>
pl_fn pl_pick(int NSUB, int TM, bool map) {
    if (NSUB == 1) {
        switch (TM) {
            case 1: return map ? k_pl<MODE, 1, 1, true> : k_pl<MODE, 1, 1, false>;
            case 2: return map ? k_pl<MODE, 1, 2, true> : k_pl<MODE, 1, 2, false>;
            case 4: return map ? k_pl<MODE, 1, 4, true> : k_pl<MODE, 1, 4, false>;
            default: return nullptr;
        }
    }
    if (NSUB == 2) {
        switch (TM) {
            case 2: return map ? k_pl<MODE, 2, 2, true> : k_pl<MODE, 2, 2, false>;
            case 4: return map ? k_pl<MODE, 2, 4, true> : k_pl<MODE, 2, 4, false>;
            default: return nullptr;
        }
    }
    return nullptr;
}

// Gathered lists at stride 1: G list groups per m-block; a wave's m-tiles must lie in
// one group, so groups of one m-tile take one m-tile per wave.
inline pl_fn pl_pick_g(int NSUB, int TM, int G) {
    if (G == 1) {
        if (NSUB == 1) return TM == 1 ? k_pl<1, 1, 1, false, 1> : TM == 2 ? k_pl<1, 1, 2, false, 1>
                                      : TM == 4 ? k_pl<1, 1, 4, false, 1> : nullptr;
        if (NSUB == 2) return TM == 2 ? k_pl<1, 2, 2, false, 1> : TM == 4 ? k_pl<1, 2, 4, false, 1> : nullptr;
    }
    if (G == 2) {
        if (NSUB == 1) return TM == 1 ? k_pl<1, 1, 1, false, 2> : TM == 2 ? k_pl<1, 1, 2, false, 2> : nullptr;
        if (NSUB == 2) return TM == 2 ? k_pl<1, 2, 2, false, 2> : nullptr;
    }
    if (G == 4 && NSUB == 1) return TM == 1 ? k_pl<1, 1, 1, false, 4> : TM == 2 ? k_pl<1, 1, 2, false, 4> : nullptr;
    return nullptr;
}

}  // namespace pl
}  // namespace bsp
