// Glue between VGG-16 stages: 2x2 max pooling, stride 2, NCHW.  Not part of the
// pruning method; the VGG stack workload needs it between its convs.
#include <hip/hip_runtime.h>

#include "bsp_kernels.h"

namespace bsp {

namespace {

__device__ __forceinline__ float ld(const float *p) { return *p; }
__device__ __forceinline__ float ld(const uint16_t *p) { return __uint_as_float((uint32_t)*p << 16); }

template <typename E>
__global__ void k_maxpool2x2(const E *__restrict__ x, E *__restrict__ y, int nc, int h, int w) {
    const int ho = h / 2, wo = w / 2;
    const size_t n = (size_t)nc * ho * wo;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        const size_t plane = i / ((size_t)ho * wo);
        const int r = (int)(i - plane * ho * wo);
        const int oh = r / wo, ow = r - oh * wo;
        const E *p = x + (plane * h + 2 * oh) * w + 2 * ow;
        // max of the four values, the winner copied bit-exactly; a NaN wins over
        // every number and the first NaN in window order is kept (NaN propagates)
        E best = p[0];
        float bv = ld(&p[0]);
        const E *cand[3] = {p + 1, p + w, p + w + 1};
        for (int k = 0; k < 3; ++k) {
            const float v = ld(cand[k]);
            if (bv == bv && !(v <= bv)) {
                bv = v;
                best = *cand[k];
            }
        }
        y[i] = best;
    }
}

}  // namespace

hipError_t launch_maxpool2x2(int dt, int n, int c, int h, int w, const void *x, void *y,
                             hipStream_t st) {
    const size_t total = (size_t)n * c * (h / 2) * (w / 2);
    if (total == 0) return hipSuccess;
    const int blocks = (int)std::min<size_t>(8192, (total + 255) / 256);
    if (dt == BSP_F32)
        k_maxpool2x2<float><<<blocks, 256, 0, st>>>((const float *)x, (float *)y, n * c, h, w);
    else
        k_maxpool2x2<uint16_t><<<blocks, 256, 0, st>>>((const uint16_t *)x, (uint16_t *)y, n * c, h, w);
    return hipGetLastError();
}

}  // namespace bsp
