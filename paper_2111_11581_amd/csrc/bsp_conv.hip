// Launcher of the forward kernel: argument set-up and instantiation choice.  The
// kernel template lives in bsp_fwd.h; its instantiations are compiled in
// bsp_fwd_*.hip (one translation unit per element type and gather mode).
#include "bsp_fwd.h"

namespace bsp {
namespace fwd {

// instantiation sets, one per translation unit (bsp_fwd_*.hip)
fwd_fn pick_b1_k1(int TM, int TPG, int KS);
fwd_fn pick_b1_k24(int TM, int TPG, int KS);
fwd_fn pick_b2(int TM, int TPG, int KS);
fwd_fn pick_b0(int TM, int TPG, int KS);
fwd_fn pick_f(int mode, int TM, int TPG, int KS);

static fwd_fn pick(int dt, int mode, int TM, int TPG, int KS) {
    if (dt == BSP_F32) return pick_f(mode == 2 ? 0 : mode, TM, TPG, KS);
    if (mode == 1) return KS == 1 ? pick_b1_k1(TM, TPG, KS) : pick_b1_k24(TM, TPG, KS);
    if (mode == 2) return pick_b2(TM, TPG, KS);
    return pick_b0(TM, TPG, KS);
}

}  // namespace fwd

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
    a.Cin = p.Cin; a.R = p.R;
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
    const int occ = std::max(1, std::min(p.TM == 1 ? 3 : 2, (160 * 1024) / (p.lds_total + kLdsStatic)));
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
    a.div_NSLOT = make_fastdiv((uint32_t)p.NSLOT);
    a.div_nmb = make_fastdiv((uint32_t)p.n_mb);
    fwd::fwd_fn fn = fwd::pick(p.dt, p.gather, p.TM, p.TPG, p.KS);
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
