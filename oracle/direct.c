/*
 * Oracle: direct convolution and matrix product in fp64 on masked dense
 * weights.  TEST INFRASTRUCTURE ONLY - never linked into the product library.
 *
 * A pruned layer computes exactly what the dense layer computes with the
 * pruned weights set to zero (layer i of Sec. 4.2: weights W_i, bias b_i);
 * pruning only removes work.  So the oracle is the plain definition:
 *
 *   conv:   y[n,o,oh,ow] = b[o] + sum_{c,r,s} W[o,c,r,s] * x[n,c,oh*sh-ph+r, ow*sw-pw+s]
 *           (input positions outside the image read as 0),
 *           Ho = (H + 2*ph - kh)/sh + 1, Wo likewise;
 *   linear: y[o,b] = b[o] + sum_k W[o,k] * x[k,b]   (feature-major x and y);
 *
 * optionally followed by ReLU.  Every MAC is done, zeros included, in fp64,
 * summing over c, then r, then s in ascending order.  OpenMP only splits the
 * independent outputs over threads.
 *
 * Pins: tests/test_oracle_direct.py (pure-Python brute force, torch conv2d /
 * numpy matmul in fp64 at rate 1, linearity, zero input, border-free shift
 * equivariance, whole-matrix row pruning leaves only the bias).
 */
#include <stddef.h>
#include <stdint.h>

int oracle_conv2d_f64(const double *x, const double *w, const double *bias, double *y,
                      int N, int C, int H, int W, int O, int KH, int KW,
                      int SH, int SW, int PH, int PW, int relu, int nthreads)
{
    if (N < 0 || C <= 0 || H <= 0 || W <= 0 || O <= 0 || KH <= 0 || KW <= 0 || SH <= 0 || SW <= 0)
        return -1;
    const int HO = (H + 2 * PH - KH) / SH + 1;
    const int WO = (W + 2 * PW - KW) / SW + 1;
    if (HO <= 0 || WO <= 0) return -1;
    const long long NO = (long long)N * O;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (long long no = 0; no < NO; ++no) {
        const int n = (int)(no / O), o = (int)(no % O);
        for (int oh = 0; oh < HO; ++oh) {
            for (int ow = 0; ow < WO; ++ow) {
                double acc = bias ? bias[o] : 0.0;
                for (int c = 0; c < C; ++c) {
                    for (int r = 0; r < KH; ++r) {
                        const int ih = oh * SH - PH + r;
                        if (ih < 0 || ih >= H) continue;
                        for (int s = 0; s < KW; ++s) {
                            const int iw = ow * SW - PW + s;
                            if (iw < 0 || iw >= W) continue;
                            acc += w[(((size_t)o * C + c) * KH + r) * KW + s] *
                                   x[(((size_t)n * C + c) * H + ih) * W + iw];
                        }
                    }
                }
                if (relu && acc < 0.0) acc = 0.0;
                y[(((size_t)n * O + o) * HO + oh) * WO + ow] = acc;
            }
        }
    }
    return 0;
}

int oracle_linear_f64(const double *x, const double *w, const double *bias, double *y,
                      int K, int B, int O, int relu, int nthreads)
{
    if (K <= 0 || B < 0 || O <= 0) return -1;
#pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads)
    for (int o = 0; o < O; ++o) {
        for (int b = 0; b < B; ++b) {
            double acc = bias ? bias[o] : 0.0;
            for (int k = 0; k < K; ++k)
                acc += w[(size_t)o * K + k] * x[(size_t)k * B + b];
            if (relu && acc < 0.0) acc = 0.0;
            y[(size_t)o * B + b] = acc;
        }
    }
    return 0;
}
