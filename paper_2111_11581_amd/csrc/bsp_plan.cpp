// Host planner: resolves a pruning scheme and a layer geometry into the list
// structure, the pixel tiling, the LDS layout of the forward, the work split and the
// dev_tiles layout.  Everything here is a pure function of its arguments (the batch
// size of a conv does not enter; the batch of a linear layer only picks its vector
// width).
#include <climits>
#include <cstring>

#include "bsp_common.h"

namespace bsp {

static int gcd_int(int a, int b) {
    while (b) { int t = a % b; a = b; b = t; }
    return a;
}

static int pow2_ceil(int v) {
    int p = 1;
    while (p < v) p *= 2;
    return p;
}

static int64_t align256(int64_t v) { return (v + 255) & ~(int64_t)255; }

static uint64_t fnv1a(const int *v, int n) {
    uint64_t h = 1469598103934665603ull;
    for (int i = 0; i < n; ++i) {
        uint32_t u = (uint32_t)v[i];
        for (int b = 0; b < 4; ++b) {
            h ^= (u >> (8 * b)) & 0xffu;
            h *= 1099511628211ull;
        }
    }
    return h;
}

// Worst case number of staged input rows over every phase of a row tiling.
static int max_slots(int rows, int Ho, int KH, int SH, int PH) {
    const int period = Ho / gcd_int(Ho, rows);
    int mx = 0;
    for (int t = 0; t < period; ++t) {
        const int v = slot_layout(t * rows, rows, Ho, INT_MAX, KH, SH, PH, nullptr, nullptr, nullptr);
        if (v > mx) mx = v;
    }
    return mx;
}

namespace {

struct MBlock {
    int split, T, G, msets, mb_tiles, mb_groups, mpg_blocks, n_mb;
};

// m-block candidates for m-sets of msets waves
int mblock_candidates(const Plan &p, int msets, MBlock *out) {
    int n = 0;
    // accumulator tiles per wave: fp32 and stride-2 gathers hold more registers
    const int max_tg = (p.esize == 4 || p.gather == 2) ? 2 : 4;
    if (p.n_groups == 1 || p.mt_per_group > 2) {
        for (int T = max_tg; T >= 1; T >>= 1) {
            MBlock m;
            m.split = 1; m.T = T; m.G = 1; m.msets = msets;
            m.mb_tiles = msets * T;
            if (m.mb_tiles > 2 * pow2_ceil(p.mt_per_group) && T > 1) continue;  // mostly idle waves
            m.mb_groups = 1;
            m.mpg_blocks = div_up(p.mt_per_group, m.mb_tiles);
            m.n_mb = p.n_groups * m.mpg_blocks;
            out[n++] = m;
        }
    } else {
        // per-group lists: at most two accumulator tiles per wave (more spill registers)
        const int T = pow2_ceil(p.mt_per_group);
        for (int G = 2 / T; G >= 1; G >>= 1) {
            MBlock m;
            m.split = 0; m.T = T; m.G = G; m.msets = msets;
            m.mb_groups = msets * G;
            if (m.mb_groups > 2 * pow2_ceil(p.n_groups) && G > 1) continue;
            m.mb_tiles = m.mb_groups * p.mt_per_group;
            m.mpg_blocks = 1;
            m.n_mb = div_up(p.n_groups, m.mb_groups);
            out[n++] = m;
        }
    }
    return n;
}

}  // namespace

bsp_status make_plan(const bsp_scheme *s, const bsp_conv_shape *conv, bsp_dtype wdt,
                     int batch_for_linear, Plan *p) {
    if (!s || !p) return BSP_EINVAL;
    std::memset(p, 0, sizeof(*p));
    if (s->rows <= 0 || s->cols <= 0 || s->bh < 0 || s->bw < 0 || s->rate < 1) return BSP_EINVAL;
    if (s->regularity < BSP_ROW || s->regularity > BSP_DENSE) return BSP_EINVAL;
    if (wdt != BSP_F32 && wdt != BSP_BF16) return BSP_EINVAL;
    p->R = s->rows;
    p->C = s->cols;
    p->bh = s->bh;
    p->bw = s->bw;
    p->reg = s->regularity;
    p->rate = s->rate;
    p->dt = wdt;
    p->esize = wdt == BSP_F32 ? 4 : 2;
    p->bh_eff = (s->bh == 0 || s->bh > p->R) ? p->R : s->bh;
    p->bw_eff = (s->bw == 0 || s->bw > p->C) ? p->C : s->bw;
    p->nbr = div_up(p->R, p->bh_eff);
    p->nbc = div_up(p->C, p->bw_eff);

    // canonical sizes and list structure
    if (p->reg == BSP_COL) {
        const int last_w = p->C - (p->nbc - 1) * p->bw_eff;
        p->L = (p->nbc - 1) * kept_count(p->bw_eff, p->rate) + kept_count(last_w, p->rate);
        p->n_indices = (int64_t)p->nbr * p->L;
        p->n_values = (int64_t)p->R * p->L;
        p->n_rowptr = p->nbr + 1;
        p->shared = 0;
        p->n_groups = p->nbr;
        p->group_rows = p->bh_eff;
    } else {
        if (p->reg == BSP_ROW) {
            const int last_h = p->R - (p->nbr - 1) * p->bh_eff;
            const int64_t kf = kept_count(p->bh_eff, p->rate), kl = kept_count(last_h, p->rate);
            p->n_indices = ((p->nbr - 1) * kf + kl) * p->nbc;
            p->n_values = ((p->nbr - 1) * kf + kl) * p->C;
            p->n_rowptr = (int64_t)p->nbr * p->nbc + 1;
        } else {
            p->n_indices = 0;
            p->n_values = (int64_t)p->R * p->C;
            p->n_rowptr = 0;
        }
        p->L = p->C;
        p->shared = 1;
        p->n_groups = 1;
        p->group_rows = p->R;
    }
    p->mt_per_group = div_up(p->group_rows, kMT);
    p->LP = div_up(p->L, kKS) * kKS;
    p->S = p->LP / kKS;
    if (!conv && batch_for_linear < 0) return BSP_OK;   // list structure only (prune, unpack)

    // geometry
    const int vmax = wdt == BSP_F32 ? 4 : 8;  // elements per 16-byte vector
    if (conv) {
        const bsp_conv_shape &c = *conv;
        if (c.cin <= 0 || c.h <= 0 || c.w <= 0 || c.kh <= 0 || c.kw <= 0 || c.stride_h <= 0 ||
            c.stride_w <= 0 || c.pad_h < 0 || c.pad_w < 0)
            return BSP_EINVAL;
        if ((int64_t)c.cin * c.kh * c.kw != p->C) return BSP_EINVAL;
        p->is_linear = 0;
        p->Cin = c.cin; p->H = c.h; p->W = c.w; p->KH = c.kh; p->KW = c.kw;
        p->SH = c.stride_h; p->SW = c.stride_w; p->PH = c.pad_h; p->PW = c.pad_w;
        p->Ho = (c.h + 2 * c.pad_h - c.kh) / c.stride_h + 1;
        p->Wo = (c.w + 2 * c.pad_w - c.kw) / c.stride_w + 1;
        if (c.h + 2 * c.pad_h < c.kh || c.w + 2 * c.pad_w < c.kw || p->Ho <= 0 || p->Wo <= 0)
            return BSP_EINVAL;
        p->gather = p->SW == 1 ? 1 : ((p->SW == 2 && wdt == BSP_BF16) ? 2 : 0);
    } else {
        p->is_linear = 1;
        p->Cin = p->C; p->H = 1; p->W = batch_for_linear > 0 ? batch_for_linear : 64;
        p->KH = p->KW = p->SH = p->SW = 1;
        p->PH = p->PW = 0;
        p->Ho = 1;
        p->Wo = p->W;
        p->gather = 1;
    }
    int vw = 1;
    while (vw < vmax && p->W % (2 * vw) == 0) vw *= 2;

    // Channels one 32-wide step of a kept list can span: the LDS window of a chunk
    // must hold at least that many.  Identity lists: 32 consecutive columns.  Column
    // blocks keep the same count in every block, so a step covers a known number of
    // blocks; whole-width blocks are data dependent (twice the mean spacing is used).
    int span_req;
    {
        const int khw = p->KH * p->KW;
        int64_t cols;
        if (p->shared) cols = kKS;
        else if (p->nbc > 1) cols = (int64_t)(div_up(kKS, kept_count(p->bw_eff, p->rate)) + 1) * p->bw_eff;
        else cols = (int64_t)2 * kKS * p->rate;
        span_req = (int)std::min<int64_t>(p->Cin, cols / khw + 2);
    }

    // search: sub-tile width x sub-tiles per workgroup x m-block x weight residency
    const int a_step = 64 * 8 * p->esize;   // one m-tile, one step
    const int64_t a_total = (int64_t)p->n_groups * p->mt_per_group * p->S * a_step;
    double best = 1e300;
    Plan bestp = *p;
    for (int tw = 4; tw <= 64; tw *= 2) {
        if (p->is_linear && tw != 64) continue;
        if (!p->is_linear && tw > 4 && div_up(p->Wo, 4) * 4 <= tw / 2) break;   // wider than needed
        const int wop = div_up(p->Wo, tw) * tw;
        // alignment unit of staged rows: the widest vector whose left pad stays <= 1
        int vec = 1;
        for (int v = vw; v >= 1; v >>= 1) {
            if (!p->is_linear && v > tw * p->SW) continue;
            const int left = (v - p->PW % v) % v;
            if (left <= 1 || p->PW % v == 0) { vec = v; break; }
        }
        const int left = (vec - p->PW % vec) % vec;
        const int need = left + (tw - 1) * p->SW + p->KW + (p->gather == 2 ? 1 : 0);
        // linear layers keep RL = 64 for every batch (their vector width varies)
        const int rl = p->is_linear ? 64 : div_up(need, vec) * vec;
        const int trw = kNPIX / tw;
        for (int nsub = 1; nsub <= 4; nsub *= 2) {
            if (trw * nsub > kMaxTileRows || (p->is_linear && nsub > 1)) continue;
            const int nslot = max_slots(trw * nsub, p->Ho, p->KH, p->SH, p->PH);
            if (nslot > kMaxSlots) continue;
            const int chs = nslot * rl;
            const int64_t pch = (int64_t)chs * p->esize;   // patch bytes per channel
            MBlock cand[8];
            const int nc = mblock_candidates(*p, 4 / nsub, cand);
            for (int ci = 0; ci < nc; ++ci) {
                const MBlock &m = cand[ci];
                const int64_t lds_a = (int64_t)m.mb_tiles * p->S * a_step;
                const int64_t lds_d = (int64_t)m.mb_groups * p->LP * 2;
                // residency x LDS budget (two or one workgroups per CU) x steps per item
                for (int opt = 0; opt < 8; ++opt) {
                    const int resident = opt < 2;
                    const int64_t budget = (opt & 1) ? kLdsOneWG : kLdsPerWG;
                    const int smax = resident ? 0 : std::min(p->S, 4 >> ((opt - 2) >> 1));
                    if (!resident && opt >= 4 && smax == std::min(p->S, 4 >> ((opt - 4) >> 1))) continue;
                    int64_t cc, lds_patch, lds_buf, total;
                    const int64_t item = resident ? 0
                        : (int64_t)m.mb_tiles * smax * a_step + (int64_t)m.mb_groups * smax * 64;
                    if (resident) {
                        const int64_t free_b = budget - align256(lds_a) - align256(lds_d);
                        if (free_b <= 0) continue;
                        cc = free_b / (2 * pch);
                    } else {
                        const int64_t free_b = budget / 2 - item - 256;
                        if (free_b <= 0) continue;
                        cc = free_b / pch;
                    }
                    if (cc > p->Cin) cc = p->Cin;
                    if (cc < span_req) continue;
                    lds_patch = (int64_t)cc * pch;
                    lds_patch = (lds_patch + 15) & ~(int64_t)15;
                    if (resident) {
                        lds_buf = lds_patch;
                        total = align256(lds_a) + align256(lds_d) + 2 * lds_patch;
                    } else {
                        lds_buf = align256(lds_patch + item);
                        total = 2 * lds_buf;
                    }
                    if (total > budget) continue;
                    // cost per output pixel (bytes moved into LDS, weighted)
                    const double px = (double)kNPIX * nsub;
                    const int chunks = (int)div_up64(p->Cin, cc);
                    // short contiguous runs per staged row cost extra load instructions
                    const double run = (double)rl * p->esize;
                    const double patch = (double)m.n_mb * p->Cin * pch / px * (1.0 + 32.0 / std::min(run, 128.0));
                    const double wts = resident ? (double)lds_a * m.n_mb / (px * 16.0) : (double)a_total / px;
                    const double gathers = (m.split ? (double)p->mt_per_group * p->n_groups / m.T
                                                    : (double)p->n_groups) * p->S * 64.0;
                    double cost = ((double)wop / p->Wo) * (patch + wts + 0.3 * gathers);
                    cost *= 1.0 + 0.05 * (chunks - 1);
                    if (!resident) cost *= 1.0 + 0.1 * (4 / std::max(smax, 1) - 1);   // items per step
                    if (budget > kLdsPerWG) cost *= 1.6;                              // one workgroup per CU
                    if (cost < best * (1 - 1e-9)) {
                        best = cost;
                        Plan q = *p;
                        q.TW = tw; q.TRW = trw; q.Wop = p->is_linear ? div_up(p->Wo, 64) * 64 : wop;
                        q.NSUB = nsub; q.VEC = p->is_linear ? vw : vec; q.LEFT = left; q.RL = rl;
                        q.NSLOT = nslot; q.CH_STRIDE = chs; q.CC = (int)cc;
                        q.split = m.split; q.T = m.T; q.G = m.G; q.msets = m.msets;
                        q.mb_tiles = m.mb_tiles; q.mb_groups = m.mb_groups; q.mpg_blocks = m.mpg_blocks;
                        q.n_mb = m.n_mb; q.resident = resident; q.SMAX = smax;
                        q.lds_a = resident ? (int)align256(lds_a) : 0;
                        q.lds_d = resident ? (int)align256(lds_d) : 0;
                        q.lds_patch = (int)lds_patch;
                        q.lds_buf = (int)lds_buf;
                        q.lds_total = (int)total;
                        bestp = q;
                    }
                }
            }
        }
    }
    if (best >= 1e300) return BSP_EUNSUPPORTED;
    *p = bestp;
    {
        const int vb = p->VEC * p->esize;
        p->gran = vb >= 16 ? 16 : (vb >= 4 ? 4 : 0);
    }

    // dev_tiles layout
    p->off_chunks = kHeaderBytes;
    p->off_desc = align256(p->off_chunks + (int64_t)16 * p->S);
    p->off_desc16 = align256(p->off_desc + (int64_t)4 * p->n_groups * p->LP);
    p->off_a = align256(p->off_desc16 + (int64_t)2 * p->n_groups * p->LP);
    p->tile_bytes = p->off_a + (int64_t)p->n_groups * p->mt_per_group * p->S * a_step;

    const int fpv[] = {p->R, p->C, p->bh_eff, p->bw_eff, p->reg, p->rate, p->dt, p->n_groups,
                       p->mt_per_group, p->LP, p->S, p->CH_STRIDE, p->RL, p->LEFT, p->NSLOT,
                       p->CC, p->KH, p->KW, p->is_linear, p->is_linear ? 0 : p->SW,
                       p->is_linear ? 0 : p->TW, p->NSUB, p->SMAX, p->resident, p->split, p->T,
                       p->G, p->msets};
    p->fingerprint = fnv1a(fpv, (int)(sizeof(fpv) / sizeof(fpv[0])));
    return BSP_OK;
}

}  // namespace bsp
