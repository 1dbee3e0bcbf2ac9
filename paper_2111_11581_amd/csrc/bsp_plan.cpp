// Host planner: resolves a pruning scheme and a layer geometry into the list
// structure, the pixel tiling, the LDS patch layout and the dev_tiles layout.
// Everything here is a pure function of its arguments.
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
        // pick the tile width: padded-pixel waste against LDS patch overhead
        int vw = 1;
        while (vw < vmax && p->W % (2 * vw) == 0) vw *= 2;
        double best = 1e30;
        for (int tw = 4; tw <= 64; tw *= 2) {
            const int wop = div_up(p->Wo, tw) * tw;
            if (tw > 4 && div_up(p->Wo, 4) * 4 <= tw / 2) break;   // wider than needed
            // alignment unit of the staged rows: the widest vector whose left pad stays <= 1
            int vec = 1;
            for (int v = vw; v >= 1; v >>= 1) {
                if (v > tw * p->SW) continue;
                const int left = (v - p->PW % v) % v;
                if (left <= 1 || p->PW % v == 0) { vec = v; break; }
            }
            const int left = (vec - p->PW % vec) % vec;
            const int need = left + (tw - 1) * p->SW + p->KW + (p->gather == 2 ? 1 : 0);
            const int rl = div_up(need, vec) * vec;
            const int trw = kNPIX / tw;
            const int period = p->Ho / gcd_int(p->Ho, trw);
            int nsl = 0;
            for (int t = 0; t < period; ++t) {
                const int v = slot_layout(t * trw, trw, p->Ho, INT_MAX, p->KH, p->SH, p->PH,
                                          nullptr, nullptr, nullptr);
                if (v > nsl) nsl = v;
            }
            if (nsl > kMaxSlots) continue;
            const double cost = (double)wop / p->Wo * (1.0 + 0.25 * rl * nsl / (double)kNPIX);
            if (cost < best - 1e-9) {
                best = cost;
                p->TW = tw; p->Wop = wop; p->VEC = vec; p->LEFT = left; p->RL = rl; p->NSLOT = nsl;
            }
        }
        if (best >= 1e30) return BSP_EUNSUPPORTED;
    } else {
        p->is_linear = 1;
        p->Cin = p->C; p->H = 1; p->W = batch_for_linear > 0 ? batch_for_linear : 64;
        p->KH = p->KW = p->SH = p->SW = 1;
        p->PH = p->PW = 0;
        p->Ho = 1;
        p->Wo = p->W;
        p->gather = 1;
        p->TW = 64;
        p->Wop = div_up(p->Wo, 64) * 64;
        int vw = 1;
        while (vw < vmax && p->W % (2 * vw) == 0) vw *= 2;
        // the layout constants below do not depend on the batch size
        p->VEC = vw;
        p->LEFT = 0;
        p->RL = 64;
        p->NSLOT = 1;
    }
    p->TRW = kNPIX / p->TW;
    // patch fill: direct-to-LDS granules of 16 or 4 bytes, else per-element register loads
    {
        const int vb = p->VEC * p->esize;
        p->gran = vb >= 16 ? 16 : (vb >= 4 ? 4 : 0);
    }
    p->CH_STRIDE = p->NSLOT * p->RL;
    {
        int64_t cc = kLdsBudget / ((int64_t)p->CH_STRIDE * p->esize);
        if (cc < 1) return BSP_EUNSUPPORTED;
        p->CC = (int)(cc < p->Cin ? cc : p->Cin);
    }

    choose_split(p, kTargetWGs);

    // dev_tiles layout
    p->off_chunks = kHeaderBytes;
    p->off_desc = align256(p->off_chunks + (int64_t)16 * p->S);
    p->off_desc16 = align256(p->off_desc + (int64_t)4 * p->n_groups * p->LP);
    p->off_a = align256(p->off_desc16 + (int64_t)2 * p->n_groups * p->LP);
    p->tile_bytes = p->off_a + (int64_t)p->n_groups * p->mt_per_group * p->S * 64 * 8 * p->esize;

    const int fpv[] = {p->R, p->C, p->bh_eff, p->bw_eff, p->reg, p->rate, p->dt, p->n_groups,
                       p->mt_per_group, p->LP, p->S, p->CH_STRIDE, p->RL, p->LEFT, p->NSLOT,
                       p->CC, p->KH, p->KW, p->is_linear, p->is_linear ? 0 : p->SW,
                       p->is_linear ? 0 : p->TW};
    p->fingerprint = fnv1a(fpv, (int)(sizeof(fpv) / sizeof(fpv[0])));
    return BSP_OK;
}

void choose_split(Plan *p, int64_t n_pt) {
    if (n_pt < 1) n_pt = 1;
    if (p->n_groups >= kWaves && p->mt_per_group <= 4) {
        p->T = pow2_ceil(p->mt_per_group);
        p->split = 0;
        p->mpg_blocks = 1;
        int g = 4;
        while (g > 1 && (g * p->T > 4 || n_pt * div_up(p->n_groups, kWaves * g) < kTargetWGs)) g >>= 1;
        p->G = g;
        p->n_mb = div_up(p->n_groups, kWaves * p->G);
    } else {
        p->G = 1;
        p->split = 1;
        int t = pow2_ceil(div_up(p->mt_per_group, kWaves));
        if (t > 4) t = 4;
        while (t > 1 && n_pt * p->n_groups * div_up(p->mt_per_group, kWaves * t) < kTargetWGs) t >>= 1;
        p->T = t;
        p->mpg_blocks = div_up(p->mt_per_group, kWaves * p->T);
        p->n_mb = p->n_groups * p->mpg_blocks;
    }
}

}  // namespace bsp
