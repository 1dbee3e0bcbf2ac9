// Launchers of the device kernels (host side).  All take a validated plan.
#pragma once

#include <hip/hip_runtime.h>

#include "bsp_common.h"

namespace bsp {

hipError_t launch_prune(const Plan &p, const void *w, uint8_t *mask, hipStream_t st);

// Weights the allocation-free prune handles (its fixed per-device scratch holds the
// radix select of this many).
constexpr size_t kNoAllocMaxWeights = (size_t)1 << 28;

// As launch_prune, allocating nothing: UNSTRUCTURED uses the library's fixed
// per-device scratch (R * C <= kNoAllocMaxWeights), the block kinds need none;
// PATTERN and per-block counts are not handled (hipErrorInvalidValue).
hipError_t launch_prune_noalloc(const Plan &p, const void *w, uint8_t *mask, hipStream_t st);

// Synchronous: returns BSP_OK, BSP_EMASK, BSP_EUNSUPPORTED or BSP_EDEVICE.
bsp_status run_pack(const Plan &p, const void *w, const uint8_t *mask, void *values,
                    int32_t *indices, int32_t *rowptr, uint8_t *tiles, hipStream_t st);

hipError_t launch_bcs(const Plan &p, const int32_t *indices, const int32_t *rowptr, int32_t *occurrence,
                      int32_t *compact, int32_t *col_stride, int32_t *row_offset, int32_t *n_runs, hipStream_t st);
hipError_t launch_unpack(const Plan &p, const void *values, const int32_t *indices,
                         const int32_t *rowptr, void *w_out, hipStream_t st);

// n: images of a conv; batch vectors of a linear layer.  part: device memory for the
// partial sums of a K loop split over workgroups (pw_part_bytes(p, n) bytes), or null
// to take them from the library's per-device workspace.
hipError_t launch_conv(const Plan &p, int n, const void *x, const uint8_t *tiles,
                       const float *bias, int relu, int out_bf16, void *y, hipStream_t st,
                       void *part = nullptr);

// Stem convolutions (stride 2, filters at most 8 wide, at most 32 (channel, filter
// row) pairs, at most 64 filters, identity list, bf16, 16-byte aligned x) run on their
// own kernel; launch_conv takes that route by itself when stem_ok holds.
bool stem_ok(const Plan &p, const void *x);
hipError_t launch_stem(const Plan &p, int n, const void *x, const uint8_t *tiles, const float *bias, int relu,
                       int out_bf16, void *y, hipStream_t st);

// Bytes of partial sums the pointwise kernel needs for n images (vectors), 0 when its
// K loop is not split.
size_t pw_part_bytes(const Plan &p, int n);

hipError_t launch_maxpool2x2(int dt, int n, int c, int h, int w, const void *x, void *y,
                             hipStream_t st);

// A conv whose plan is a 1x1 layer over its im2col input (Plan::im2col): the input is
// expanded into the library's per-device workspace, then the pointwise kernel runs.
hipError_t launch_conv_im2col(const Plan &p, const bsp_conv_shape &c, const void *x, const uint8_t *tiles,
                              const float *bias, int relu, int out_bf16, void *y, hipStream_t st);

}  // namespace bsp
