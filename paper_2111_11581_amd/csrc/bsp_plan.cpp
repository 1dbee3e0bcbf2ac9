// Host planner: resolves a pruning scheme and a layer geometry into the list
// structure, the pixel tiling, the LDS layout of the forward, the wave work split
// and the dev_tiles layout.  Everything here is a pure function of its arguments:
// the batch (conv->n, the batch of a linear layer) does not enter, so tiles packed
// once serve every batch size.  Tiling choices are scored for a nominal batch.
#include <climits>
#include <cmath>
#include <cstring>
#include <vector>

#include "bsp_common.h"

namespace bsp {

static int gcd_int(int a, int b) {
    while (b) { int t = a % b; a = b; b = t; }
    return a;
}

static int64_t align256(int64_t v) { return (v + 255) & ~(int64_t)255; }
static int round_up(int v, int m) { return (v + m - 1) / m * m; }

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

// Output rows spanned by a tile of TG groups, worst case over its start phase.
static int rows_spanned(int TG, int GPR) {
    const int g = gcd_int(TG, GPR);
    return (GPR - g + TG - 1) / GPR + 1;
}

// Staged input rows of the worst tile, over every phase of the tiling inside an
// image (tiles may cross image boundaries).
static int max_slots(int TG, int GPR, int Ho, int KH, int SH, int PH) {
    const int64_t img_groups = (int64_t)Ho * GPR;
    const int64_t period = img_groups / gcd_int((int)(img_groups % INT_MAX), TG);
    int mx = 0;
    for (int64_t t = 0; t < period; ++t) {
        const int64_t G0 = t * TG;
        const int g0 = (int)(G0 / GPR), g1 = (int)((G0 + TG - 1) / GPR);
        const int v = slot_layout(g0, g1 - g0 + 1, Ho, INT_MAX, KH, SH, PH, nullptr, nullptr, nullptr);
        if (v > mx) mx = v;
    }
    return mx;
}

// Padding of the m-tile range, dev_tiles layout and the fingerprint the kernels
// check against the packed header.
static void finish_layout(Plan *p, int n_mt, int astep) {
    p->n_mt_pad = p->n_mb * p->MBT;
    p->n_g_pad = p->shared ? 1 : std::max(p->n_groups, p->n_mb * p->MBG);
    if (p->shared) p->n_mt_pad = std::max(p->n_mt_pad, n_mt);

    p->off_chunks = kHeaderBytes;
    p->off_desc = align256(p->off_chunks + (int64_t)16 * p->S);
    p->off_desc16 = align256(p->off_desc + (int64_t)4 * p->n_groups * p->LP);
    p->off_a = align256(p->off_desc16 + (int64_t)2 * p->n_g_pad * p->LP);
    p->off_rowmap = align256(p->off_a + (int64_t)p->n_mt_pad * p->S * astep);
    p->off_pruned = p->off_rowmap + (int64_t)4 * (p->rowmap ? p->n_mt_pad * kMT : 0);
    p->off_counts = align256(p->off_pruned + (int64_t)4 * (p->rowmap ? p->R - p->RK : 0));
    p->tile_bytes = p->off_counts + (p->counts ? count_tables_bytes(p->nbr, p->nbc, p->L) : 0);

    const int fpv[] = {p->R, p->C, p->bh_eff, p->bw_eff, p->reg, p->rate, p->dt, p->n_groups,
                       p->mt_per_group, p->LP, p->S, p->CH_STRIDE, p->RS, p->LEFT, p->NSLOT,
                       p->CC, p->KH, p->KW, p->is_linear, p->SW, p->NSUB, p->SMAX, p->resident,
                       p->MBT, p->MBG, p->n_mt_pad, p->n_g_pad, p->GE, p->NB, p->pw, p->NGR, p->VS, p->V,
                       p->rowmap, p->RK, p->khw, (int)p->counts_hash, p->counts != nullptr, p->pl, 13};
    p->fingerprint = fnv1a(fpv, (int)(sizeof(fpv) / sizeof(fpv[0])));
}

// Tiling of a pointwise layer for the pointwise kernel.  The patch row of a channel
// is the tile's granules (NGR of them, no padding), so a tiling is NSUB, the wave
// split, the m-block, the weight staging and the channels per chunk.  Scored for the
// nominal batch with a model of the chip: HBM, L2-to-LDS copies, LDS reads of the
// gathers, MFMA issue, and the copy latency of each chunk, hidden by the other
// workgroups of a CU.  Returns false when nothing fits.
static bool plan_pointwise(Plan *p, int span_req, int n_mt, int mpg, int astep) {
    const int GE = 16 / p->esize;
    const int gpg = p->SW == 1 ? GE / 4 : 1;
    int64_t groups_nom;   // groups of the nominal batch
    double hbm_bytes;
    if (p->is_linear) {
        groups_nom = round_up(div_up(kNominalVectors, 4), gpg);
        hbm_bytes = ((double)p->Cin + p->RK) * kNominalVectors * p->esize;
    } else if (p->SW == 1) {
        groups_nom = (int64_t)kNominalImages * round_up(div_up(p->H * p->W, 4), gpg);
        hbm_bytes = ((double)p->Cin + p->RK) * kNominalImages * p->H * p->W * p->esize;
    } else {
        groups_nom = (int64_t)kNominalImages * p->Ho * div_up(p->Wo, 4);
        hbm_bytes = ((double)p->Cin * p->H * p->W / 2 + (double)p->RK * p->Ho * p->Wo) * kNominalImages * p->esize;
    }
    hbm_bytes += (double)n_mt * p->S * astep;
    const double t_hbm = hbm_bytes / 5.5e12 * 2.4e9;
    const double mfma_cyc = p->esize == 4 ? 32.0 : 16.0;   // one step of one m-tile and n-tile

    double best = 1e300;
    Plan bestp = *p;
    for (int nsub = 1; nsub <= 4; nsub *= 2) {
        const int TG = kGroups * nsub;
        const int ngr = TG / gpg;
        const int rb = ngr * 16;               // patch bytes per channel
        const int chs = ngr * GE;              // patch elements per channel
        const int Q = kWaves / nsub;
        const double n_pt = std::ceil((double)groups_nom / TG);
        for (int qmode = 0; qmode <= 1; ++qmode) {
            if (qmode == 1 && Q == 1) continue;
            const int KS = qmode ? Q : 1;
            for (int TM = 1; TM <= 4; TM *= 2) {
                if (p->esize == 4 && TM > 2) continue;
                int TPG, MBT, MBG, n_mb;
                MBT = TM * (qmode == 0 ? Q : 1);
                if (MBT > 1 && MBT >= 2 * n_mt) continue;   // mostly idle waves
                if (p->shared) {
                    TPG = TM;
                    MBG = 1;
                } else {
                    TPG = std::min(TM, mpg);
                    if (TM % TPG) continue;
                    if (MBT % mpg != 0 && mpg % MBT != 0) continue;
                    MBG = std::max(1, MBT / mpg);
                }
                n_mb = div_up(n_mt, MBT);
                const int64_t d_res = align256((int64_t)MBG * p->LP * 2);
                const int64_t a_all = (int64_t)MBT * p->S * astep;
                const int occ_v = pw_occ(p->esize, p->SW == 2 ? 2 : 1, TM);   // register limit of the kernel
                for (int opt = 0; opt < 5; ++opt) {
                    const int resident = opt == 0;
                    const int smax = resident ? 0 : (1 << (opt - 1));   // 1, 2, 4, 8
                    if (!resident && smax > p->S) continue;
                    const int64_t astage = resident ? 0 : (int64_t)MBT * smax * astep;
                    const int64_t fixed = d_res + (resident ? align256(a_all) : 0);
                    for (int nb = 2; nb <= 3; ++nb) {
                        for (int occ = 1; occ <= occ_v; ++occ) {
                            // minus static LDS (bias, and the row map of row-mapped layers)
                            const int64_t budget = (160 * 1024) / occ - 1280 - (p->rowmap ? 1024 : 0);
                            const int64_t free_b = budget - fixed - nb * align256(astage) - nb * 256;
                            if (free_b <= 0) continue;
                            // patches are whole 1 KB copy slots of four waves (256 granules)
                            int64_t cc = free_b / (nb * 4096) * kThreads / ngr;
                            cc = std::min<int64_t>(cc, std::min(p->Cin, kMaxCC));
                            cc = std::min<int64_t>(cc, 65535 / chs);
                            if (p->shared && cc < p->Cin) cc = cc / kKS * kKS;
                            if (cc < span_req || cc < 1) continue;
                            // whole 1 KB copy slots of four waves
                            const int64_t lds_patch = div_up64(cc * ngr, kThreads) * 4096;
                            const int64_t lds_buf = lds_patch + align256(astage);
                            int64_t total = fixed + nb * lds_buf;
                            if (KS > 1) total = std::max<int64_t>(total, (int64_t)2 * TM * 4096);
                            if (total > budget) continue;
                            double nch = std::ceil((double)p->Cin / cc);
                            if (!resident) nch = std::max(nch, std::ceil((double)p->S / smax));
                            // persistent workgroups, as the launcher splits them
                            double wpm = std::max(1.0, std::ceil(256.0 * occ / n_mb));
                            if (KS > 1 || wpm > n_pt) wpm = n_pt;
                            const double tpw = std::ceil(n_pt / wpm);
                            const double n_wg = std::ceil(n_pt / tpw) * n_mb;
                            const double tiles = n_pt * n_mb;
                            // L2 -> LDS copies: patches per tile, weights per workgroup when
                            // resident (else per tile), offsets per workgroup
                            const double l2 = tiles * (double)p->Cin * rb + (resident ? n_wg : tiles) * (double)a_all +
                                              n_wg * MBG * p->LP * 2.0;
                            const double t_l2 = l2 / (256.0 * 64.0);
                            const int GW = TM / TPG;
                            const double stages = (double)p->S / KS * GW * kWaves;   // per tile, all waves
                            const double t_lds = tiles * stages * (8.0 * 64 * (p->SW == 2 ? 16 : 8) + TPG * 1024.0 + 1024.0) /
                                                 (256.0 * 128.0);
                            const double t_mfma = tiles * MBT * nsub * (double)p->S * 4 * mfma_cyc / (4.0 * 256 * 0.75);
                            // latency chain of one workgroup: nb - 1 chunks in flight, each item at
                            // least its own multiply; workgroups beyond occ per CU run in rounds
                            const double rounds = std::ceil(n_wg / (256.0 * occ));
                            const double item_mfma = TM * std::ceil((double)p->S / nch / KS) * 4 * mfma_cyc;
                            const double item = std::max(3000.0 / (nb - 1), item_mfma * std::min(occ, 4) / 4.0 + 400.0);
                            const double t_lat = rounds * (tpw * nch * item + 6000.0);
                            // Measured on gfx950 over the ResNet-50 pointwise layers (plan sweeps):
                            // two workgroups per CU (store phases and copy waits of one overlap
                            // the other's work), 128-pixel tiles, four m-tiles per wave and two
                            // buffers win where the model alone cannot tell; these enter as
                            // factors on the modelled time.
                            const double prior = (occ == 2 ? 1.0 : 1.3) * (nsub == 2 ? 1.0 : 1.15) *
                                                 (TM == 4 || p->esize == 4 || p->SW == 2 ? 1.0 : 1.15) *
                                                 (nb == 2 ? 1.0 : (p->SW == 2 ? 2.0 : 1.3));
                            const double cyc = (std::max(std::max(t_hbm, t_l2), std::max(std::max(t_lds, t_mfma), t_lat)) +
                                                (KS > 1 ? 1500.0 : 0.0)) * prior;
                            if (cyc < best * (1 - 1e-9)) {
                                best = cyc;
                                Plan q = *p;
                                q.pw = 1; q.NGR = ngr; q.gpg = gpg; q.occ = occ;
                                q.NSUB = nsub; q.CH_STRIDE = chs; q.CC = (int)cc;
                                q.FR = (int)div_up64(cc * ngr, kThreads);
                                q.qmode = qmode; q.KS = KS; q.TM = TM; q.TPG = TPG;
                                q.MBT = MBT; q.MBG = MBG; q.n_mb = n_mb;
                                q.resident = resident; q.SMAX = smax; q.NB = nb;
                                q.lds_d = (int)d_res;
                                q.lds_a = resident ? (int)align256(a_all) : 0;
                                q.lds_patch = (int)lds_patch;
                                q.lds_astage = (int)align256(astage);
                                q.lds_buf = (int)lds_buf;
                                q.lds_total = (int)total;
                                bestp = q;
                            }
                        }
                    }
                }
            }
        }
    }
    if (best >= 1e300) return false;
    *p = bestp;
    return true;
}

// Tiling of a bf16 pointwise layer with one identity list for its own kernel
// (k_pl): one workgroup of 8 waves per CU, 4 multiplying and 4 copying, an m-block of
// MT = TM * 4 / NSUB m-tiles (a multiple of 4) and tiles of 64 NSUB pixels; stages of
// SPS steps in NB LDS buffers.  Scored for the nominal batch with a serial model of a
// stage: the copying waves' issue time (about 90 cycles per 1 KB copy per wave, 2.2
// times that from input rows off 16-byte boundaries), the multiplying waves' steps
// (4 MFMAs of 16 cycles per m-tile and about 100 cycles of gathers and LDS latency),
// at least the copy latency spread over the stages ahead, plus a fixed cost per
// stage (barrier, waits, loop); per tile the epilogue's stores (10 bytes per cycle);
// never below the HBM time.  The fixed and latency costs were fitted to a GPU sweep
// of every tiling of the ResNet-50 pointwise layers (the model's choice is within 1%
// of the fastest tiling there), which found large stages (4 steps) with two or three
// buffers best.
// Per-block-row lists (column and block-punched blocks, stride 1) run with gathered
// lists: an m-block holds G whole list groups (or lies inside one group), each step
// stages G patches, and the m-block's lists (16-bit channels) stay in LDS; each patch
// copy costs a list read and a multiply-add more.  Returns false when nothing fits.
static bool pl_g_ok(int nsub, int tm, int g) {   // instantiated (NSUB, TM, G) of the gathered kernel
    if (g == 1) return nsub == 1 ? (tm == 1 || tm == 2 || tm == 4) : (tm == 2 || tm == 4);
    if (g == 2) return nsub == 1 ? (tm == 1 || tm == 2) : tm == 2;
    if (g == 4) return nsub == 1 && (tm == 1 || tm == 2);
    return false;
}

static bool plan_pl(Plan *p, int n_mt, int astep) {
    const bool lists = !p->shared;
    if (lists && (p->SW != 1 || p->counts || p->Cin > 0xffff)) return false;
    const int mpg = p->mt_per_group;
    const int gpg = p->SW == 1 ? 2 : 1;
    int64_t groups_nom;   // groups of the nominal batch
    double hbm_bytes;
    bool mis;             // granule sources off 16-byte boundaries
    if (p->is_linear) {
        groups_nom = round_up(div_up(kNominalVectors, 4), gpg);
        hbm_bytes = ((double)p->Cin + p->RK) * kNominalVectors * 2;
        mis = false;
    } else if (p->SW == 1) {
        groups_nom = (int64_t)kNominalImages * round_up(div_up(p->H * p->W, 4), gpg);
        hbm_bytes = ((double)p->Cin + p->RK) * kNominalImages * p->H * p->W * 2;
        mis = ((int64_t)p->H * p->W * 2) % 16 != 0 && !p->im2col;   // im2col planes: padded
    } else {
        groups_nom = (int64_t)kNominalImages * p->Ho * div_up(p->Wo, 4);
        hbm_bytes = ((double)p->Cin * p->H * p->W / 2 + (double)p->RK * p->Ho * p->Wo) * kNominalImages * 2;
        mis = ((int64_t)p->W * 2) % 16 != 0;
    }
    hbm_bytes += (double)n_mt * p->S * astep;
    const double t_hbm = hbm_bytes / 5.5e12 * 2.4e9;
    const int64_t budget = 160 * 1024 - 2048 - 512;   // minus static LDS (bias, row map) and slack
    const int mode = p->SW;

    double best = 1e300;
    Plan bestp = *p;
    for (int nsub = 1; nsub <= 2; ++nsub) {
        const int np = 64 * nsub;
        const int rb = np * 2 * mode;                 // patch bytes per channel
        const int pcopy = 32 * (rb / 16) / kThreads;  // patch copies per copying wave and step
        const double n_pt = std::ceil((double)groups_nom / (kGroups * nsub));
        for (int TM = 1; TM <= 4; TM *= 2) {
            const int MT = TM * (kWaves / nsub);
            if (MT % kWaves != 0) continue;
            if (MT > 4 && MT >= 2 * n_mt) continue;   // mostly idle waves
            int G = 0;   // list groups of an m-block (0: identity list)
            if (lists) {
                if (mpg <= MT && MT % mpg == 0) G = MT / mpg;
                else if (mpg % MT == 0) G = 1;
                else continue;
                if ((MT / G) % TM != 0 || !pl_g_ok(nsub, TM, G)) continue;
            }
            const int GG = std::max(G, 1);
            const int pc = GG * pcopy;   // patch copies per copying wave and step
            const int64_t lds_list = lists ? align256((int64_t)GG * p->LP * 2) : 0;
            const int n_mb = div_up(n_mt, MT);
            for (int resident = 0; resident <= 1; ++resident)
            for (int sps = 1; sps <= 4 && sps <= p->S; sps *= 2) {
                const int wcopy = resident ? 0 : MT / kWaves;
                const int64_t a_res = resident ? (int64_t)MT * p->S * 1024 : 0;
                const int64_t step_b = (int64_t)GG * 32 * rb + (resident ? 0 : (int64_t)MT * 1024);
                for (int nb = 2; nb <= 8; ++nb) {
                    const int64_t total = lds_list + a_res + nb * sps * step_b;
                    if (total > budget) continue;
                    const int ncp = sps * (pc + wcopy);
                    const double ns = std::ceil((double)p->S / sps);
                    double wpm = std::max(1.0, std::ceil(256.0 / n_mb));
                    if (wpm > n_pt) wpm = n_pt;
                    const double tpw = std::ceil(n_pt / wpm);
                    const double n_wg = std::ceil(n_pt / tpw) * n_mb;
                    const double rounds = std::ceil(n_wg / 256.0);
                    const double prod =
                        sps * (pc * ((mis ? 200.0 : 90.0) + (lists ? 10.0 : 0.0)) + wcopy * 90.0) + 100.0;
                    const double comp = sps * (TM * 64.0 + 100.0) + 150.0;
                    const double stage = std::max(std::max(prod, comp), 1000.0 / (nb - 1)) + 1500.0;
                    const double out_bytes = (double)MT * kMT * np * 2;
                    const double epi = TM * 4 * 60.0 + out_bytes / 10.0;
                    double cyc = rounds * (tpw * (ns * stage + epi) + a_res / 1024.0 * 25.0) + 5000.0;
                    if ((nb - 1) * ncp > 63) cyc *= 1.05;   // more copies in flight than a wave can count
                    // at equal cost three buffers measure best (two stages in flight, one barrier
                    // per stage), more than three slightly worse
                    cyc *= 1.0 + 0.01 * std::abs(nb - 3);
                    // gathered lists: 64-pixel tiles measured 15% faster than 128-pixel ones on
                    // the 4096x4096 FC stack at equal modelled cost
                    if (lists && nsub == 2) cyc *= 1.2;
                    cyc = std::max(cyc, t_hbm);
                    if (cyc < best * (1 - 1e-9)) {
                        best = cyc;
                        Plan q = *p;
                        q.pw = 1; q.pl = 1; q.gpg = gpg; q.occ = 1;
                        q.NSUB = nsub; q.NGR = rb / 16;
                        // gathered lists hold channel numbers (the lists' own; stride 1)
                        q.CH_STRIDE = lists ? 1 : np * mode; q.CC = 32 * sps; q.SMAX = sps;
                        q.FR = pc;
                        q.qmode = 0; q.KS = 1; q.TM = TM; q.TPG = TM;
                        q.MBT = MT; q.MBG = GG; q.n_mb = n_mb;
                        q.resident = resident; q.NB = nb;
                        q.lds_d = (int)lds_list; q.lds_a = (int)a_res;
                        q.lds_patch = GG * 32 * rb * sps;
                        q.lds_astage = resident ? 0 : MT * 1024 * sps;
                        q.lds_buf = (int)(sps * step_b);
                        q.lds_total = (int)total;
                        bestp = q;
                    }
                }
            }
        }
    }
    if (best >= 1e300) return false;
    *p = bestp;
    return true;
}

// Groups of block (bi, bj): columns (COL), rows (ROW) or kernel locations (PUNCHED).
static int block_groups(const Plan &p, int bi, int bj) {
    if (p.reg == BSP_PUNCHED) return p.khw;
    if (p.reg == BSP_COL || p.reg == BSP_ROWCOL) return std::min(p.C, (bj + 1) * p.bw_eff) - bj * p.bw_eff;
    return std::min(p.R, (bi + 1) * p.bh_eff) - bi * p.bh_eff;
}

int block_count(const Plan &p, int b) {
    if (p.counts) return p.counts[b];
    return kept_count(block_groups(p, b / p.nbc, b % p.nbc), p.rate);
}

int block_cols(const Plan &p, int i, int j) {
    const int k = block_count(p, i * p.nbc + j);
    if (p.reg != BSP_PUNCHED) return k;
    const int cin = p.C / p.khw;
    return k * (std::min(cin, (j + 1) * p.bw_eff) - j * p.bw_eff);
}

// Kept GEMM columns of block-row i (COL, PUNCHED).
static int64_t row_list_len(const Plan &p, int i) {
    int64_t L = 0;
    for (int j = 0; j < p.nbc; ++j) L += block_cols(p, i, j);
    return L;
}

void count_slots(const Plan &p, int32_t *P) {
    int64_t off = 0;
    for (int j = 0; j < p.nbc; ++j) {
        P[j] = (int32_t)off;
        int kmax = 0;
        for (int i = 0; i < p.nbr; ++i) kmax = std::max(kmax, block_cols(p, i, j));
        off += kmax;
    }
    P[p.nbc] = (int32_t)off;
}

void plan_rowptr(const Plan &p, int32_t *rowptr) {
    int64_t off = 0;
    if (p.reg == BSP_ROW) {
        for (int b = 0; b < p.nbr * p.nbc; ++b) {
            rowptr[b] = (int32_t)off;
            off += block_count(p, b);
        }
        rowptr[p.nbr * p.nbc] = (int32_t)off;
        return;
    }
    for (int i = 0; i < p.nbr; ++i) {
        rowptr[i] = (int32_t)off;
        off += row_list_len(p, i);
    }
    rowptr[p.nbr] = (int32_t)off;
}

// Widest span, in GEMM columns, of 32 consecutive kept columns of one list, from the
// per-block counts.  Units are column blocks, or the channels of punched blocks.  A
// window whose first kept column lies in unit u may take a single column of u, so it
// runs on through the following units until they hold 31 more (or the list ends).
static int64_t max_step_span_cols(const Plan &p) {
    // the forward lists give block column j the same slot run in every block-row
    // (count_slots), so the units are the block columns with their run lengths
    const int cin = p.C / p.khw;
    int64_t worst = 0;
    std::vector<int32_t> P(p.nbc + 1);
    count_slots(p, P.data());
    std::vector<int> cnt, width;
    {
        for (int j = 0; j < p.nbc; ++j) {
            cnt.push_back(P[j + 1] - P[j]);
            width.push_back(p.reg == BSP_PUNCHED ? (std::min(cin, (j + 1) * p.bw_eff) - j * p.bw_eff) * p.khw
                                                 : std::min(p.C, (j + 1) * p.bw_eff) - j * p.bw_eff);
        }
        const int n = (int)cnt.size();
        int e = 0;
        int64_t have = 0, span = 0;   // units (u, e) after the start unit: kept columns, width
        for (int u = 0; u < n; ++u) {
            if (e < u + 1) { e = u + 1; have = 0; span = 0; }
            while (e < n && have < kKS - 1) { have += cnt[e]; span += width[e]; ++e; }
            if (cnt[u] > 0) worst = std::max(worst, width[u] + span);
            if (e > u + 1) { have -= cnt[u + 1]; span -= width[u + 1]; }
        }
    }
    return worst;
}

// Channels one 32-wide step of a forward list can span (a chunk's channel window must
// hold at least that many) and the mean channels a step advances.  Identity lists: 32
// consecutive columns.  Column blocks keep the same count in every block, so a step
// covers a known number of blocks; whole-width blocks are data dependent (twice the
// mean spacing is used).
// Block-punched lists keep the same number of locations of every channel.
static void list_spans(const Plan &p, int *span_req, double *step_ch) {
    {
        const int khw = p.KH * p.KW;
        int64_t cols;
        if (p.shared) cols = kKS;
        else if (p.counts && p.nbc > 1) cols = max_step_span_cols(p);
        else if (p.counts)   // one block column: lists stretched over L slots, twice the mean spacing
            cols = std::min<int64_t>(p.C, 2 * (int64_t)kKS * p.C / p.L + 1);
        else if (p.reg == BSP_PUNCHED)   // a step may start at the last kept location of a channel
            cols = (int64_t)(div_up(kKS, kept_count(p.khw, p.rate)) + 1) * p.khw;
        else if (p.nbc > 1) cols = (int64_t)(div_up(kKS, kept_count(p.bw_eff, p.rate)) + 1) * p.bw_eff;
        else cols = (int64_t)2 * kKS * p.rate;
        *span_req = (int)std::min<int64_t>(p.Cin, cols / khw + 2);
    }
    // mean channels one step advances (for the chunk count of a channel window)
    {
        const int khw = p.KH * p.KW;
        if (p.shared) *step_ch = (double)kKS / khw;
        else if (p.counts) *step_ch = (double)kKS * p.nbr * p.C / std::max<int64_t>(p.n_indices, 1) / khw;
        else if (p.reg == BSP_PUNCHED) *step_ch = (double)kKS / kept_count(p.khw, p.rate);
        else if (p.nbc > 1) *step_ch = (double)kKS * p.bw_eff / kept_count(p.bw_eff, p.rate) / khw;
        else *step_ch = (double)kKS * p.rate / khw;
    }
}

// Tiling of the general forward kernel for the plan's list layout, scored for the
// nominal batch (CU cycles).  Sets *p to the best tiling and returns its score, or
// 1e300 (p unchanged) when nothing fits.
static double search_tiling(Plan *p, int span_req, double step_ch, int n_mt, int mpg, int astep,
                            int nominal_rows) {
    const double total_groups = (double)nominal_rows * p->GPR;
    // LDS budgets per workgroup: 1, 2, 3 or 4 workgroups per CU (160 KB, minus static tables)
    const int budgets[4] = {160 * 1024 - kLdsStatic, 80 * 1024 - kLdsStatic, 53 * 1024 - kLdsStatic,
                            40 * 1024 - kLdsStatic};

    double best = 1e300;
    Plan bestp = *p;
    // a second pass admits m-blocks much larger than the layer when nothing else fits
    for (int relax = 0; relax < 2 && best >= 1e300; ++relax)
    for (int nsub = 1; nsub <= 4; nsub *= 2) {
        const int TG = kGroups * nsub;
        const int trw = rows_spanned(TG, p->GPR);
        if (trw > kMaxTileRows) continue;
        const int nslot = max_slots(TG, p->GPR, p->Ho, p->KH, p->SH, p->PH);
        if (nslot > kMaxSlots) continue;
        const int chs = p->V * nslot * p->RS;             // patch elements per channel
        if (p->V * nslot * p->RG > 512) continue;         // granules per channel: per-tile lookup table
        const int Q = kWaves / nsub;
        const double n_pt = std::ceil(total_groups / TG);
        for (int qmode = 0; qmode <= 1; ++qmode) {
            if (qmode == 1 && Q == 1) continue;
            const int KS = qmode ? Q : 1;
            for (int TM = 1; TM <= 4; TM *= 2) {
                // instantiated kernels: fp32 and per-element gathers at most 2 m-tiles per
                // wave and no step split; 16-byte stride-2 gathers at most 4 m-tiles
                const bool narrow = p->esize == 4 || p->gather == 0;
                if (narrow && (TM > 2 || qmode == 1)) continue;
                if (p->gather == 2 && TM > 4) continue;
                int TPG, MBT, MBG, n_mb;
                MBT = TM * (qmode == 0 ? Q : 1);
                if (p->shared) {
                    TPG = TM;
                    if (!relax && MBT > 1 && MBT >= 2 * n_mt) continue;     // mostly idle waves
                    MBG = 1;
                    n_mb = div_up(n_mt, MBT);
                } else {
                    TPG = std::min(TM, mpg);
                    if (TM % TPG) continue;
                    if (MBT % mpg != 0 && mpg % MBT != 0) continue;
                    if (!relax && MBT > 1 && MBT >= 2 * n_mt) continue;
                    MBG = std::max(1, MBT / mpg);
                    n_mb = div_up(n_mt, MBT);
                }
                const int64_t d_res = align256((int64_t)MBG * p->LP * 2);
                const int64_t a_all = (int64_t)MBT * p->S * astep;
                for (int bi = 0; bi < (relax ? 4 : 1); ++bi) {   // measured: one workgroup per CU with large chunks is best
                    const int64_t budget = budgets[bi];
                    for (int opt = 0; opt < 10; ++opt) {
                        const int nb = opt < 5 ? 3 : 2;   // buffers (two when three do not fit)
                        const int resident = opt % 5 == 0;
                        const int smax = resident ? 0 : (1 << (opt % 5 - 1));   // 1, 2, 4, 8
                        if (!resident && smax > p->S) continue;
                        const int64_t astage = resident ? 0 : (int64_t)MBT * smax * astep;
                        const int64_t fixed = d_res + (resident ? align256(a_all) : 0) + 256;
                        const int64_t free_b = budget - fixed - nb * align256(astage) - nb * 512;
                        if (free_b <= 0) continue;
                        // patches are whole 1 KB copy slots of four waves (256 granules)
                        int64_t cc = free_b / (nb * 4096) * kThreads / ((int64_t)p->V * nslot * p->RG);
                        cc = std::min<int64_t>(cc, std::min(p->Cin, kMaxCC));
                        cc = std::min<int64_t>(cc, 65536 / chs);                       // 16-bit offsets
                        if (cc < span_req || cc < 1) continue;
                        int fr = (int)div_up64(cc * p->V * nslot * p->RG, kThreads);
                        if (fr > 32) {   // copies per wave and chunk: one bit each in the fixup mask
                            cc = 32 * kThreads / ((int64_t)p->V * nslot * p->RG);
                            if (cc < span_req || cc < 1) continue;
                            fr = (int)div_up64(cc * p->V * nslot * p->RG, kThreads);
                        }
                        const int64_t lds_patch = (int64_t)fr * 4096;   // whole 1 KB copy slots of four waves
                        const int64_t lds_buf = lds_patch + align256(astage);
                        int64_t total = fixed + nb * lds_buf + (p->gather == 3 ? 256 : 0);   // MODE 3 reads run past the patch
                        if (qmode == 1) total = std::max<int64_t>(total, (int64_t)2 * TM * 4096);   // partial sums
                        if (total > budget) continue;

                        // ---- score (nominal batch), in CU cycles ----
                        // persistent workgroups: occ per CU, each walking tpw pixel tiles
                        const int occ = std::min(fwd_occ(p->gather, TM, TPG), (160 * 1024) / (int)(total + kLdsStatic));
                        if (occ < 1) continue;
                        double wpm = std::max(1.0, std::ceil(256.0 * occ / n_mb));
                        if (KS > 1 || wpm > n_pt) wpm = n_pt;
                        const double tpw = std::ceil(n_pt / wpm);
                        const double n_wg = std::ceil(n_pt / tpw) * n_mb;
                        const double rounds = std::ceil(n_wg / (256.0 * occ));
                        // steps per chunk: consecutive steps advance step_ch channels each
                        // (staged weights: at most SMAX); the real count depends on the lists.
                        // Block-punched steps cover whole channels from a channel boundary,
                        // so a chunk holds a whole number of them.
                        double spc = p->reg == BSP_PUNCHED && !p->counts
                                         ? std::floor((double)cc / step_ch + 1e-9)
                                         : (cc - 1) / step_ch;
                        spc = std::max(1.0, spc);
                        if (!resident) spc = std::min<double>(spc, smax);
                        const double nch = std::max(1.0, p->S / spc);
                        // Serial time of one wave per chunk, fitted to measured plans on gfx950
                        // (ResNet-50 3x3 layers, 4x column pruning): a fixed cost (copy table
                        // reads, fixups, barrier, pipeline refill), each stage (8 kept columns
                        // gathered and 4 MFMAs per m-tile list; stride-2 gathers read 4 dwords
                        // per column), each 1 KB copy (twice when input rows start off 16-byte
                        // boundaries); three buffers make chunks smaller and cost more per chunk.
                        const double stages = std::ceil(spc / KS) * (TM / TPG);
                        const double copies = fr + (resident ? 0.0 : (double)astage / 4096.0);
                        const bool mis = ((int64_t)p->W * p->esize) % 16 != 0;
                        double per_chunk = 3000.0 + stages * (p->SW == 2 ? 900.0 : 500.0) + copies * (mis ? 100.0 : 50.0);
                        if (nb == 3) per_chunk *= 1.2;
                        if (occ > 1) per_chunk *= 0.8 * occ;                               // workgroups sharing a CU
                        // per tile: epilogue; per workgroup: header, tables, first fill
                        double cyc = rounds * (tpw * nch * per_chunk + tpw * 8000.0 + 8000.0);
                        const double hbm = ((double)nominal_rows / p->Ho * p->Cin * p->H * p->W * p->esize +
                                            total_groups * 4 * p->RK * 2.0) / 5.5e12 * 2.4e9;
                        // L2-to-LDS copies of the whole job (every m-block copies the patch of
                        // every tile it computes) at about 8 bytes per CU cycle
                        const double copy_bytes = n_mb * n_pt * nch * ((double)fr * 4096 + (resident ? 0.0 : (double)astage));
                        cyc = std::max(std::max(cyc, hbm), copy_bytes / (256.0 * 8.0));
                        if (qmode == 1) cyc = cyc * 1.5 + 1500.0;                           // partial-sum reduction
                        if (cyc < best * (1 - 1e-9)) {
                            best = cyc;
                            Plan q = *p;
                            q.NSUB = nsub; q.TRWMAX = trw; q.NSLOT = nslot; q.CH_STRIDE = chs; q.VS = nslot * p->RS;
                            q.CC = (int)cc; q.FR = fr;
                            q.qmode = qmode; q.KS = KS; q.TM = TM; q.TPG = TPG;
                            q.MBT = MBT; q.MBG = MBG; q.n_mb = n_mb;
                            q.resident = resident; q.SMAX = smax; q.NB = nb;
                            q.lds_d = (int)d_res;
                            q.lds_a = resident ? (int)align256(a_all) : 0;
                            q.lds_patch = (int)lds_patch;
                            q.lds_astage = (int)align256(astage);
                            q.lds_buf = (int)lds_buf;
                            q.lds_total = (int)total;
                            bestp = q;
                        }
                    }
                }
            }
        }
    }
    if (best < 1e300) *p = bestp;
    return best;
}

static bsp_status make_plan_impl(const bsp_scheme *s, const bsp_conv_shape *conv, bsp_dtype wdt,
                                 int batch_for_linear, Plan *p, bool im2col_inner);

// Output planes of at most this many pixels: the general kernel stages whole input rows
// per output row, which for 2x2 and 4x4 planes copies mostly padding, so such layers run
// as a 1x1 layer over their im2col input (its columns are the GEMM form's columns).
constexpr int kIm2colMaxPixels = 16;
// bf16 convs with per-block-row lists and output planes of at most this many pixels
// also run over their im2col input, with the pipelined gathered-list kernel: each kept
// column is then one contiguous input row, copied whole, where the general kernel
// re-gathers and pads every staged row of a small image.  At stride 1 the expanded
// input of the nominal batch must stay small: measured on gfx950, the 8x8 VGG-16
// layers (expanded input up to 19 MB) ran 25% faster this way, the 16x16 ones and
// ResNet-50's stride-1 7x7 and 14x14 layers (33-59 MB, beyond the L2 caches) slower.
// Strided layers with such planes gain regardless (ResNet-50's 512-channel stride-2
// layer, 14x14 -> 7x7: 110 -> 86 us), the general kernel's strided gathers being slower.
constexpr int kIm2colListPixels = 64;
constexpr int64_t kIm2colListBytes = 24ll << 20;

// 1x1 stride-2 bf16 convs without padding over one identity list (row-pruned and dense
// downsampling layers) with output planes of at most this many pixels run as a stride-1
// 1x1 layer over their subsampled input (the im2col input of a 1x1 conv): the strided
// pointwise kernel copies every other input column for nothing.  Measured on gfx950 at
// batch 64 (cold cache): ResNet-50's 512 -> 1024 layer at 28x28 -> 14x14 69 -> 61 us and
// 1024 -> 2048 at 14x14 -> 7x7 61 -> 49 us; the 256 -> 512 one at 56x56 -> 28x28 gains
// nothing (its subsampling reads 103 MB), so larger planes stay strided.
constexpr int kSubsampleMaxPixels = 196;

bsp_status make_plan(const bsp_scheme *s, const bsp_conv_shape *conv, bsp_dtype wdt,
                     int batch_for_linear, Plan *p) {
    const bool sub = s && conv && conv->kh == 1 && conv->kw == 1 && conv->stride_h == 2 && conv->stride_w == 2 &&
                     conv->pad_h == 0 && conv->pad_w == 0 && conv->cin > 0 && conv->h > 0 && conv->w > 0 &&
                     wdt == BSP_BF16 && !s->counts &&
                     (s->regularity == BSP_ROW || s->regularity == BSP_DENSE) &&
                     (int64_t)((conv->h - 1) / 2 + 1) * ((conv->w - 1) / 2 + 1) <= kSubsampleMaxPixels;
    if (s && conv && conv->kh > 0 && conv->kw > 0 && (conv->kh > 1 || conv->kw > 1 || sub) && conv->stride_h > 0 &&
        conv->stride_w > 0 && conv->pad_h >= 0 && conv->pad_w >= 0 && conv->cin > 0 &&
        conv->h + 2 * conv->pad_h >= conv->kh && conv->w + 2 * conv->pad_w >= conv->kw) {
        const int ho = (conv->h + 2 * conv->pad_h - conv->kh) / conv->stride_h + 1;
        const int wo = (conv->w + 2 * conv->pad_w - conv->kw) / conv->stride_w + 1;
        const bool lists = (s->regularity == BSP_COL || s->regularity == BSP_PUNCHED ||
                            s->regularity == BSP_ROWCOL) && !s->counts;
        const int64_t plane = (int64_t)ho * wo;
        const int64_t kcols = (int64_t)conv->cin * conv->kh * conv->kw;
        if (sub || plane <= kIm2colMaxPixels ||
            (wdt == BSP_BF16 && lists && plane <= kIm2colListPixels && kcols <= 0xffff &&
             (conv->stride_h > 1 || conv->stride_w > 1 ||
              (int64_t)kNominalImages * kcols * round_up((int)plane, 8) * 2 <= kIm2colListBytes))) {
            if ((int64_t)conv->cin * conv->kh * conv->kw != s->cols) return BSP_EINVAL;
            if (s->regularity == BSP_PUNCHED && conv->kh * conv->kw != s->khw) return BSP_EINVAL;
            const bsp_conv_shape c2 = {conv->n, conv->cin * conv->kh * conv->kw, ho, wo, 1, 1, 1, 1, 0, 0};
            const bsp_status st = make_plan_impl(s, &c2, wdt, batch_for_linear, p, true);
            // the pipelined kernel reads the im2col planes padded to whole granules
            if (st == BSP_OK && p->pl) p->xplane = (int)round_up((int)plane, p->GE);
            return st;
        }
    }
    return make_plan_impl(s, conv, wdt, batch_for_linear, p, false);
}

static bsp_status make_plan_impl(const bsp_scheme *s, const bsp_conv_shape *conv, bsp_dtype wdt,
                                 int batch_for_linear, Plan *p, bool im2col_inner) {
    if (!s || !p) return BSP_EINVAL;
    std::memset(p, 0, sizeof(*p));
    p->im2col = im2col_inner ? 1 : 0;
    if (s->rows <= 0 || s->cols <= 0 || s->bh < 0 || s->bw < 0 || s->rate < 1) return BSP_EINVAL;
    if (s->regularity < BSP_ROW || s->regularity > BSP_PATTERN) return BSP_EINVAL;
    if (s->regularity == BSP_PATTERN && (s->khw != 9 || s->cols % 9 != 0 || s->bh > 126 || s->counts))
        return BSP_EINVAL;
    if (s->regularity == BSP_ROWCOL && s->counts) return BSP_EUNSUPPORTED;
    if (wdt != BSP_F32 && wdt != BSP_BF16) return BSP_EINVAL;
    const int khw = s->regularity == BSP_PUNCHED ? std::max(s->khw, 1) : 1;
    if (s->regularity == BSP_PUNCHED && (s->khw < 0 || s->cols % khw != 0)) return BSP_EINVAL;
    p->R = s->rows;
    p->C = s->cols;
    p->bh = s->bh;
    p->bw = s->bw;
    p->reg = s->regularity;
    p->rate = s->rate;
    p->dt = wdt;
    p->esize = wdt == BSP_F32 ? 4 : 2;
    p->khw = khw;
    p->bh_eff = (s->bh == 0 || s->bh > p->R) ? p->R : s->bh;
    if (p->reg == BSP_PUNCHED) {   // blocks of bh_eff filters x bw_eff input channels
        const int cin = p->C / khw;
        p->bw_eff = (s->bw == 0 || s->bw > cin) ? cin : s->bw;
        p->nbc = div_up(cin, p->bw_eff);
    } else {
        p->bw_eff = (s->bw == 0 || s->bw > p->C) ? p->C : s->bw;
        p->nbc = div_up(p->C, p->bw_eff);
    }
    p->nbr = div_up(p->R, p->bh_eff);
    if (p->reg == BSP_PATTERN) {   // no blocks; bh is the library size
        p->khw = 9;
        p->bh_eff = s->bh ? s->bh : 8;
        p->bw_eff = p->C;
        p->nbr = p->nbc = 1;
    }
    if (s->counts && (p->reg == BSP_ROW || p->reg == BSP_COL || p->reg == BSP_PUNCHED)) {
        if ((int64_t)p->nbr * p->nbc > (1 << 24)) return BSP_EUNSUPPORTED;
        uint32_t h = 2166136261u;
        for (int b = 0; b < p->nbr * p->nbc; ++b) {
            const int k = s->counts[b];
            if (k < 0 || k > block_groups(*p, b / p->nbc, b % p->nbc)) return BSP_EINVAL;
            h = (h ^ (uint32_t)k) * 16777619u;
        }
        p->counts = s->counts;
        p->counts_hash = h;
    }

    // canonical sizes and list structure
    if (p->counts && p->reg != BSP_ROW) {
        // per-block counts: lists of different lengths, padded to the longest
        int64_t Lmax = 0, nv = 0, ni = 0;
        for (int i = 0; i < p->nbr; ++i) {
            const int64_t Li = row_list_len(*p, i);
            Lmax = std::max(Lmax, Li);
            ni += Li;
            nv += Li * (std::min(p->R, (i + 1) * p->bh_eff) - i * p->bh_eff);
        }
        (void)Lmax;
        std::vector<int32_t> P(p->nbc + 1);
        count_slots(*p, P.data());
        p->L = std::max(P[p->nbc], 1);   // forward lists: the slot runs of all block columns
        p->n_indices = ni;
        p->n_values = nv;
        p->n_rowptr = p->nbr + 1;
        p->shared = 0;
        p->n_groups = p->nbr;
        p->group_rows = p->bh_eff;
    } else if (p->reg == BSP_PUNCHED) {
        // a block-row keeps ceil(khw / rate) locations of every input channel
        p->L = (p->C / khw) * kept_count(khw, p->rate);
        p->n_indices = (int64_t)p->nbr * p->L;
        p->n_values = (int64_t)p->R * p->L;
        p->n_rowptr = p->nbr + 1;
        p->shared = 0;
        p->n_groups = p->nbr;
        p->group_rows = p->bh_eff;
    } else if (p->reg == BSP_COL || p->reg == BSP_ROWCOL) {
        const int last_w = p->C - (p->nbc - 1) * p->bw_eff;
        p->L = (p->nbc - 1) * kept_count(p->bw_eff, p->rate) + kept_count(last_w, p->rate);
        p->n_indices = (int64_t)p->nbr * p->L;
        p->n_values = (int64_t)p->R * p->L;
        p->n_rowptr = p->nbr + 1;
        p->shared = 0;
        p->n_groups = p->nbr;
        p->group_rows = p->bh_eff;
    } else {
        if (p->reg == BSP_ROW && p->counts) {
            int64_t ni = 0, nv = 0;
            for (int b = 0; b < p->nbr * p->nbc; ++b) {
                const int j = b % p->nbc;
                ni += p->counts[b];
                nv += (int64_t)p->counts[b] * (std::min(p->C, (j + 1) * p->bw_eff) - j * p->bw_eff);
            }
            p->n_indices = ni;
            p->n_values = nv;
            p->n_rowptr = (int64_t)p->nbr * p->nbc + 1;
        } else if (p->reg == BSP_ROW) {
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
        // whole-width row blocks keep the same filters for every column: compute only
        // those (a row map sends them to their output rows)
        if (p->reg == BSP_ROW && p->nbc == 1 && p->n_indices < p->R) {
            p->rowmap = 1;
            p->group_rows = (int)p->n_indices;
        }
    }
    p->RK = p->shared ? p->group_rows : p->R;
    p->mt_per_group = div_up(p->group_rows, kMT);
    p->LP = div_up(p->L, kKS) * kKS;
    p->S = p->LP / kKS;
    if (!conv && batch_for_linear < 0) return BSP_OK;   // list structure only (prune, unpack)

    // geometry
    int nominal_rows;   // output rows of the nominal batch, for scoring only
    if (conv) {
        const bsp_conv_shape &c = *conv;
        if (c.cin <= 0 || c.h <= 0 || c.w <= 0 || c.kh <= 0 || c.kw <= 0 || c.stride_h <= 0 ||
            c.stride_w <= 0 || c.pad_h < 0 || c.pad_w < 0)
            return BSP_EINVAL;
        if ((int64_t)c.cin * c.kh * c.kw != p->C) return BSP_EINVAL;
        if (p->reg == BSP_PUNCHED && c.kh * c.kw != p->khw && !im2col_inner) return BSP_EINVAL;
        p->is_linear = 0;
        p->Cin = c.cin; p->H = c.h; p->W = c.w; p->KH = c.kh; p->KW = c.kw;
        p->SH = c.stride_h; p->SW = c.stride_w; p->PH = c.pad_h; p->PW = c.pad_w;
        p->Ho = (c.h + 2 * c.pad_h - c.kh) / c.stride_h + 1;
        p->Wo = (c.w + 2 * c.pad_w - c.kw) / c.stride_w + 1;
        if (c.h + 2 * c.pad_h < c.kh || c.w + 2 * c.pad_w < c.kw || p->Ho <= 0 || p->Wo <= 0)
            return BSP_EINVAL;
        if (p->PW > 64) return BSP_EUNSUPPORTED;
        // gather mode (stride 1 may become 3 below, when the rows are staged once)
        p->gather = p->SW == 1 ? 1 : ((p->SW == 2 && wdt == BSP_BF16) ? 2 : 0);
        nominal_rows = kNominalImages * p->Ho;
    } else {
        // a linear layer is a 1x1 conv over rows of 64 batch vectors (feature-major x)
        p->is_linear = 1;
        p->Cin = p->C; p->H = 1; p->W = kLinRow;
        p->KH = p->KW = p->SH = p->SW = 1;
        p->PH = p->PW = 0;
        p->Ho = 1;
        p->Wo = kLinRow;
        p->gather = 1;
        nominal_rows = kNominalVectors / kLinRow;
    }
    p->GE = 16 / p->esize;
    p->Wop = round_up(p->Wo, 4);
    p->GPR = p->Wop / 4;
    // patch rows.  Stride 1: V = min(KW, 4) copies of each staged input row, copy m
    // starting at input column m - PW; filter column s reads copy s % V at offset
    // V * (s / V), so every 4-pixel read starts at a multiple of 4 elements.  Other
    // strides: one copy, LEFT zeros before input column 0.
    // Copies cost patch space and copy issue, misaligned reads cost gather time: the
    // copies are taken when their rows are at most 1.6 times the single copy's (measured
    // on gfx950: narrow images gain, wide ones lose).
    {
        const int left1 = round_up(p->PW, p->GE);
        const int maxpos = left1 - p->PW + (p->Wo - 1) * p->SW + p->KW;   // one past the last used
        const int rs1 = round_up(std::max(maxpos, left1 + div_up(p->W, p->GE) * p->GE), p->GE);
        const int vc = std::min(p->KW, 4);
        const int rsv = round_up(p->Wop + vc * ((p->KW - 1) / vc), p->GE);
        if (p->gather == 1 && vc > 1 && 10 * vc * rsv <= 16 * rs1) {
            p->V = vc;
            p->LEFT = 0;
            p->POFF = 0;
            p->RS = rsv;
        } else {
            p->V = 1;
            p->LEFT = left1;
            p->POFF = left1 - p->PW;
            p->RS = rs1;
            // bf16 reads at any element: aligned words joined by a shift (the pointwise
            // kernel, planned below, reads aligned groups and ignores the mode)
            if (p->gather == 1 && p->esize == 2) p->gather = 3;
        }
    }
    p->RG = p->RS / p->GE;

    int span_req;
    double step_ch;
    list_spans(*p, &span_req, &step_ch);

    const int astep = 64 * 8 * p->esize;   // weight bytes of one m-tile and step
    const int n_mt = p->n_groups * p->mt_per_group;
    const int mpg = p->mt_per_group;

    // pointwise layers (1x1 without padding, stride 1 or 2; linear): own kernel
    if (p->KH == 1 && p->KW == 1 && p->PH == 0 && p->PW == 0 && p->SH == p->SW &&
        (p->SW == 1 || (p->SW == 2 && p->esize == 2))) {
        // the pipelined kernel for per-block-row lists, linear layers and 1x1 convs with
        // more than 64 input channels; with 64 or fewer (weights resident, two workgroups
        // per CU) the general pointwise kernel was faster in the measured sweep.  Measured
        // on bf16 FC layers (4096x4096 at batch 64 to 2048, 2048->1000 at batch 64), the
        // pipelined kernel with its split K loop took 0.2-0.7 of the general one's time.
        if ((p->esize == 2 && (!p->shared || p->is_linear || p->Cin > 64) && plan_pl(p, n_mt, astep)) ||
            plan_pointwise(p, span_req, n_mt, mpg, astep)) {
            finish_layout(p, n_mt, astep);
            return BSP_OK;
        }
    }
    // The forward layout.  Per-block-row lists (column, block-punched and row-and-column
    // blocks without per-block counts) against the zero-expanded layout (one identity
    // list shared by every m-tile, pruned weights zero in the tiles).  Block-rows shorter
    // than a 16-row MFMA tile each take a tile of their own, so their lists execute
    // (16 / bh) x the kept fraction of the dense work, with a gather per tile.  Measured
    // on the block-size sweep layer (3x3 256->256 56x56), such lists were slower than the
    // zero-expanded layout whenever that product was 1/5 or more, and the model's score
    // of them was low by about 1.34 times more than its score of the zero-expanded
    // layout; so with that product at 1/5 or more the zero-expanded layout is taken when
    // its score is under 1.34 of the lists'.  Other lists give way to it when its score
    // is under 0.7 of theirs (lists whose channel windows are very wide).
    auto search = [&](Plan *q) {
        int sr;
        double sc;
        list_spans(*q, &sr, &sc);
        return search_tiling(q, sr, sc, q->n_groups * q->mt_per_group, q->mt_per_group, astep, nominal_rows);
    };
    Plan lists = *p;
    const bool alt = !p->shared && !p->counts && !p->is_linear;
    const bool padded_dense = alt && p->bh_eff < kMT &&
                              (double)kMT / p->bh_eff * ((double)p->L / p->C) >= 0.2;
    double best = search(&lists);
    if (alt) {
        Plan d = *p;
        d.shared = 1;
        d.L = p->C;
        d.n_groups = 1;
        d.group_rows = p->R;
        d.mt_per_group = div_up(p->R, kMT);
        d.LP = div_up(d.L, kKS) * kKS;
        d.S = d.LP / kKS;
        const double bd = search(&d);
        if (bd < (padded_dense ? 1.34 : 0.7) * best) {
            lists = d;
            best = bd;
        }
    }
    if (best >= 1e300) return BSP_EUNSUPPORTED;
    *p = lists;
    finish_layout(p, p->n_groups * p->mt_per_group, astep);
    return BSP_OK;
}

}  // namespace bsp
