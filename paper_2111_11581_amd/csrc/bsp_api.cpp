// C ABI entry points: argument validation, planning, dispatch.  No state is kept
// between calls; every device buffer belongs to the caller.
#include <climits>

#include <hip/hip_runtime.h>

#include "bsp_common.h"
#include "bsp_kernels.h"

using namespace bsp;

namespace {

constexpr int kMaxGroupsPerBlock = 8192;   // fp64 scores of one block held in LDS
constexpr int kMaxSteps = 8192;            // chunk builder stages the step spans in LDS

inline hipStream_t S(void *stream) { return (hipStream_t)stream; }

bsp_status check_scheme_for_prune(const Plan &p) {
    if ((int64_t)p.R * p.C > INT32_MAX) return BSP_EUNSUPPORTED;
    if (p.reg == BSP_COL && p.bw_eff > kMaxGroupsPerBlock) return BSP_EUNSUPPORTED;
    if (p.reg == BSP_ROW && p.bh_eff > kMaxGroupsPerBlock) return BSP_EUNSUPPORTED;
    if (p.reg == BSP_PUNCHED && p.khw > kMaxGroupsPerBlock) return BSP_EUNSUPPORTED;
    if (p.reg == BSP_ROWCOL && p.bh_eff + p.bw_eff > kMaxGroupsPerBlock) return BSP_EUNSUPPORTED;
    return BSP_OK;
}

}  // namespace

extern "C" {

const char *bsp_status_string(bsp_status s) {
    switch (s) {
        case BSP_OK: return "ok";
        case BSP_EINVAL: return "invalid argument";
        case BSP_EUNSUPPORTED: return "unsupported configuration";
        case BSP_EDEVICE: return "device error";
        case BSP_EMASK: return "mask does not have the block structure of the scheme";
        case BSP_ETOOLARGE: return "input larger than the fixed scratch of the allocation-free entry point";
        default: return "unknown status";
    }
}

int32_t bsp_version(void) { return 100; }

bsp_status bsp_packed_sizes(const bsp_scheme *scheme, const bsp_conv_shape *conv, bsp_dtype wdt,
                            int64_t *n_values, int64_t *n_indices, int64_t *n_rowptr,
                            int64_t *dev_tile_bytes) {
    if (!scheme || !n_values || !n_indices || !n_rowptr || !dev_tile_bytes) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, conv, wdt, 0, &p);
    if (st != BSP_OK) return st;
    *n_values = p.n_values;
    *n_indices = p.n_indices;
    *n_rowptr = p.n_rowptr;
    *dev_tile_bytes = p.tile_bytes;
    return BSP_OK;
}

bsp_status bsp_prune(const bsp_scheme *scheme, bsp_dtype wdt, const void *w, uint8_t *mask,
                     void *stream) {
    if (!scheme || !w || !mask) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, nullptr, wdt, -1, &p);
    if (st != BSP_OK) return st;
    if ((st = check_scheme_for_prune(p)) != BSP_OK) return st;
    return launch_prune(p, w, mask, S(stream)) == hipSuccess ? BSP_OK : BSP_EDEVICE;
}

bsp_status bsp_prune_noalloc(const bsp_scheme *scheme, bsp_dtype wdt, const void *w, uint8_t *mask,
                             void *stream) {
    if (!scheme || !w || !mask) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, nullptr, wdt, -1, &p);
    if (st != BSP_OK) return st;
    if ((st = check_scheme_for_prune(p)) != BSP_OK) return st;
    if (p.reg == BSP_PATTERN || p.counts) return BSP_EUNSUPPORTED;
    if (p.reg == BSP_UNSTRUCTURED && (uint64_t)p.R * (uint64_t)p.C > kNoAllocMaxWeights) return BSP_ETOOLARGE;
    return launch_prune_noalloc(p, w, mask, S(stream)) == hipSuccess ? BSP_OK : BSP_EDEVICE;
}

bsp_status bsp_pack(const bsp_scheme *scheme, bsp_dtype wdt, const void *w, const uint8_t *mask,
                    void *values, int32_t *indices, int32_t *rowptr, void *dev_tiles,
                    const bsp_conv_shape *conv, void *stream) {
    if (!scheme || !w || !mask || !values || !dev_tiles) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, conv, wdt, 0, &p);
    if (st != BSP_OK) return st;
    if ((st = check_scheme_for_prune(p)) != BSP_OK) return st;
    if (p.reg != BSP_DENSE && p.reg != BSP_UNSTRUCTURED && p.reg != BSP_PATTERN && (!indices || !rowptr)) return BSP_EINVAL;
    if (p.S > kMaxSteps) return BSP_EUNSUPPORTED;
    return run_pack(p, w, mask, values, indices, rowptr, (uint8_t *)dev_tiles, S(stream));
}

bsp_status bsp_unpack(const bsp_scheme *scheme, bsp_dtype wdt, const void *values,
                      const int32_t *indices, const int32_t *rowptr, void *w_out, void *stream) {
    if (!scheme || !values || !w_out) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, nullptr, wdt, -1, &p);
    if (st != BSP_OK) return st;
    if (p.reg != BSP_DENSE && p.reg != BSP_UNSTRUCTURED && p.reg != BSP_PATTERN && (!indices || !rowptr)) return BSP_EINVAL;
    return launch_unpack(p, values, indices, rowptr, w_out, S(stream)) == hipSuccess ? BSP_OK
                                                                                      : BSP_EDEVICE;
}

bsp_status bsp_to_bcs(const bsp_scheme *scheme, const int32_t *indices, const int32_t *rowptr,
                      int32_t *occurrence, int32_t *compact_cols, int32_t *col_stride, int32_t *row_offset,
                      int32_t *n_runs, void *stream) {
    if (!scheme || !indices || !rowptr || !occurrence || !compact_cols || !col_stride || !row_offset || !n_runs)
        return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, nullptr, BSP_BF16, -1, &p);
    if (st != BSP_OK) return st;
    if (p.reg != BSP_COL && p.reg != BSP_PUNCHED) return BSP_EUNSUPPORTED;
    if ((int64_t)p.R * p.C > INT32_MAX) return BSP_EUNSUPPORTED;
    return launch_bcs(p, indices, rowptr, occurrence, compact_cols, col_stride, row_offset, n_runs, S(stream)) ==
                   hipSuccess
               ? BSP_OK
               : BSP_EDEVICE;
}

bsp_status bsp_conv2d(const bsp_scheme *scheme, const bsp_conv_shape *shape, bsp_dtype in_dt,
                      bsp_dtype out_dt, const void *x, const void *dev_tiles, const float *bias,
                      int32_t relu, void *y, void *stream) {
    if (!scheme || !shape || !x || !dev_tiles || !y) return BSP_EINVAL;
    if (out_dt != BSP_F32 && out_dt != BSP_BF16) return BSP_EINVAL;
    if (shape->n < 0) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, shape, in_dt, 0, &p);
    if (st != BSP_OK) return st;
    if ((int64_t)shape->n * shape->cin * shape->h * shape->w > INT32_MAX ||
        (int64_t)shape->n * p.R * p.Ho * p.Wo > INT32_MAX || (int64_t)shape->n * p.Ho > INT32_MAX / 2)
        return BSP_EUNSUPPORTED;
    if (shape->n == 0) return BSP_OK;
    if (p.im2col) {
        if ((int64_t)shape->n * p.Cin * (p.xplane ? p.xplane : (int64_t)p.H * p.W) > INT32_MAX)
            return BSP_EUNSUPPORTED;
        return launch_conv_im2col(p, *shape, x, (const uint8_t *)dev_tiles, bias, relu ? 1 : 0,
                                  out_dt == BSP_BF16, y, S(stream)) == hipSuccess
                   ? BSP_OK
                   : BSP_EDEVICE;
    }
    return launch_conv(p, shape->n, x, (const uint8_t *)dev_tiles, bias, relu ? 1 : 0,
                       out_dt == BSP_BF16, y, S(stream)) == hipSuccess
               ? BSP_OK
               : BSP_EDEVICE;
}

bsp_status bsp_linear(const bsp_scheme *scheme, int32_t batch, bsp_dtype in_dt, bsp_dtype out_dt,
                      const void *x, const void *dev_tiles, const float *bias, int32_t relu,
                      void *y, void *stream) {
    if (!scheme || !x || !dev_tiles || !y || batch < 0) return BSP_EINVAL;
    if (out_dt != BSP_F32 && out_dt != BSP_BF16) return BSP_EINVAL;
    Plan p;
    bsp_status st = make_plan(scheme, nullptr, in_dt, batch > 0 ? batch : 64, &p);
    if (st != BSP_OK) return st;
    if ((int64_t)scheme->cols * batch > INT32_MAX || (int64_t)scheme->rows * batch > INT32_MAX)
        return BSP_EUNSUPPORTED;
    if (batch == 0) return BSP_OK;
    return launch_conv(p, batch, x, (const uint8_t *)dev_tiles, bias, relu ? 1 : 0, out_dt == BSP_BF16,
                       y, S(stream)) == hipSuccess
               ? BSP_OK
               : BSP_EDEVICE;
}

bsp_status bsp_maxpool2x2(bsp_dtype dt, int32_t n, int32_t c, int32_t h, int32_t w, const void *x,
                          void *y, void *stream) {
    if (!x || !y || n < 0 || c < 0 || h < 0 || w < 0) return BSP_EINVAL;
    if (dt != BSP_F32 && dt != BSP_BF16) return BSP_EINVAL;
    if ((int64_t)n * c * h * w > INT32_MAX) return BSP_EUNSUPPORTED;
    return launch_maxpool2x2(dt, n, c, h, w, x, y, S(stream)) == hipSuccess ? BSP_OK : BSP_EDEVICE;
}

}  // extern "C"
