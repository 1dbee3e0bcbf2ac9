// Pruning masks on the device.
//
// Block row / column pruning (Sec. 4.1.1): one workgroup per block computes the
// squared Frobenius norm of each of the block's columns (Eq. 3) or rows (Eq. 2) in
// fp64, summed in ascending index order (the squares of fp32 / bf16 values are exact
// in fp64, so fma(v, v, s) rounds exactly like s + v*v), then keeps the
// ceil(extent / rate) largest (one-shot magnitude selection, Sec. 5.1) by counting,
// for each group, the groups that beat it (larger score, or equal score and lower
// index).  Unstructured pruning (Sec. 2.1.1) keeps the ceil(R*C/rate) largest |w| of
// the layer: a most-significant-digit radix select over the bit patterns of |w|
// (order preserving for non-negative floats) finds the threshold, and entries equal
// to it are admitted in flat-index order.  Block-punched pruning (Sec. 4.1.2, Eq. 4):
// one workgroup per block of filters x input channels scores each kernel location
// over the block's kernels, in ascending (filter, channel) order, keeps the best
// ceil(khw / rate) by the same rank count and writes them into every kernel of the
// block.
#include <hip/hip_runtime.h>

#include <hipcub/hipcub.hpp>

#include <mutex>

#include "bsp_kernels.h"

namespace bsp {

__device__ __forceinline__ double ld_f64(const float *w, size_t i) { return (double)w[i]; }
__device__ __forceinline__ double ld_f64(const uint16_t *w, size_t i) {
    return (double)__uint_as_float((uint32_t)w[i] << 16);
}
__device__ __forceinline__ uint32_t abs_key(const float *w, size_t i) {
    return __float_as_uint(w[i]) & 0x7fffffffu;
}
__device__ __forceinline__ uint32_t abs_key(const uint16_t *w, size_t i) {
    return ((uint32_t)w[i] & 0x7fffu) << 16;
}

template <typename E>
__global__ void k_prune_blocks(const E *__restrict__ w, uint8_t *__restrict__ mask, int R, int C,
                               int bh, int bw, int nbc, int col, int rate, const int32_t *__restrict__ counts) {
    extern __shared__ double sc[];
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw, c1 = min(C, c0 + bw);
    const int ng = col ? c1 - c0 : r1 - r0;
    const int k = counts ? counts[b] : (ng + rate - 1) / rate;
    for (int g = threadIdx.x; g < ng; g += blockDim.x) {
        double s = 0.0;
        if (col) {
            for (int p = r0; p < r1; ++p) {
                const double v = ld_f64(w, (size_t)p * C + c0 + g);
                s = fma(v, v, s);
            }
        } else {
            const size_t row = (size_t)(r0 + g) * C;
            for (int q = c0; q < c1; ++q) {
                const double v = ld_f64(w, row + q);
                s = fma(v, v, s);
            }
        }
        sc[g] = s;
    }
    __syncthreads();
    for (int g = threadIdx.x; g < ng; g += blockDim.x) {
        const double s = sc[g];
        int rank = 0;
        for (int h = 0; h < ng; ++h) {
            const double t = sc[h];
            rank += (t > s) || (t == s && h < g);
        }
        const uint8_t keep = rank < k ? 1 : 0;
        if (col) {
            for (int p = r0; p < r1; ++p) mask[(size_t)p * C + c0 + g] = keep;
        } else {
            uint8_t *mr = mask + (size_t)(r0 + g) * C;
            for (int q = c0; q < c1; ++q) mr[q] = keep;
        }
    }
}

template <typename E>
__global__ void k_prune_punched(const E *__restrict__ w, uint8_t *__restrict__ mask, int R, int C, int khw,
                                int bh, int bw, int nbc, int rate, const int32_t *__restrict__ counts) {
    extern __shared__ double sc[];   // khw scores, then khw keep flags
    uint8_t *keep = (uint8_t *)(sc + khw);
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int cin = C / khw;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw, c1 = min(cin, c0 + bw);
    const int k = counts ? counts[b] : (khw + rate - 1) / rate;
    for (int l = threadIdx.x; l < khw; l += blockDim.x) {
        double s = 0.0;
        for (int o = r0; o < r1; ++o) {
            const size_t base = (size_t)o * C + l;
            for (int c = c0; c < c1; ++c) {
                const double v = ld_f64(w, base + (size_t)c * khw);
                s = fma(v, v, s);
            }
        }
        sc[l] = s;
    }
    __syncthreads();
    for (int l = threadIdx.x; l < khw; l += blockDim.x) {
        const double s = sc[l];
        int rank = 0;
        for (int h = 0; h < khw; ++h) {
            const double t = sc[h];
            rank += (t > s) || (t == s && h < l);
        }
        keep[l] = rank < k ? 1 : 0;
    }
    __syncthreads();
    const int nc = c1 - c0;
    const int n = (r1 - r0) * nc * khw;
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
        const int kr = e / khw, l = e - kr * khw;
        const int o = r0 + kr / nc, c = c0 + kr % nc;
        mask[(size_t)o * C + (size_t)c * khw + l] = keep[l];
    }
}

// Simultaneous row and column pruning: the block's row scores (Eq. 2) and column
// scores (Eq. 3), each summed in ascending order, ranked separately; the block keeps
// the product of the kept rows and the kept columns.
template <typename E>
__global__ void k_prune_rowcol(const E *__restrict__ w, uint8_t *__restrict__ mask, int R, int C, int bh, int bw,
                               int nbc, int rate) {
    extern __shared__ double sc[];   // row scores [bh], column scores [bw], then keep flags
    const int b = blockIdx.x;
    const int bi = b / nbc, bj = b - bi * nbc;
    const int r0 = bi * bh, r1 = min(R, r0 + bh), c0 = bj * bw, c1 = min(C, c0 + bw);
    const int nr = r1 - r0, nc = c1 - c0;
    double *rs = sc, *cs = sc + bh;
    uint8_t *kr = (uint8_t *)(sc + bh + bw), *kc = kr + bh;
    for (int g = threadIdx.x; g < nr + nc; g += blockDim.x) {
        double s = 0.0;
        if (g < nr) {
            const size_t row = (size_t)(r0 + g) * C;
            for (int q = c0; q < c1; ++q) {
                const double v = ld_f64(w, row + q);
                s = fma(v, v, s);
            }
            rs[g] = s;
        } else {
            for (int p = r0; p < r1; ++p) {
                const double v = ld_f64(w, (size_t)p * C + c0 + (g - nr));
                s = fma(v, v, s);
            }
            cs[g - nr] = s;
        }
    }
    __syncthreads();
    const int kr_n = (nr + rate - 1) / rate, kc_n = (nc + rate - 1) / rate;
    for (int g = threadIdx.x; g < nr + nc; g += blockDim.x) {
        const bool isr = g < nr;
        const double *sv = isr ? rs : cs;
        const int n = isr ? nr : nc, x = isr ? g : g - nr;
        const double s = sv[x];
        int rank = 0;
        for (int h = 0; h < n; ++h) rank += (sv[h] > s) || (sv[h] == s && h < x);
        if (isr) kr[x] = rank < kr_n;
        else kc[x] = rank < kc_n;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < nr * nc; e += blockDim.x) {
        const int p = e / nc, q = e - p * nc;
        mask[(size_t)(r0 + p) * C + c0 + q] = kr[p] & kc[q];
    }
}

__global__ void k_fill_u8(uint8_t *p, size_t n, uint8_t v);

// ---- pattern-based pruning of 3x3 kernels (Sec. 2.1, Sec. 5.2.3) ------------------
// A kernel k = o * Cin + c holds w[o][c * khw + l].  Each kernel's own top-4 location
// set (squares, ties to the lower location) is counted in a histogram of bit masks;
// the library is the n_lib most frequent masks (ties to the smaller mask); every
// kernel takes the library pattern with the largest kept squared norm, summed in
// ascending location order (ties to the earlier pattern); connectivity keeps the
// kernels with the largest such norm (a stable descending sort: ties to the lower
// kernel index).
template <typename E>
__global__ void k_pattern_own(const E *__restrict__ w, int n_kernels, int khw, unsigned int *__restrict__ hist) {
    for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n_kernels; k += gridDim.x * blockDim.x) {
        double sq[9];
        for (int l = 0; l < 9; ++l) {
            const double v = ld_f64(w, (size_t)k * khw + l);
            sq[l] = v * v;
        }
        int code = 0;
        for (int l = 0; l < 9; ++l) {
            int rank = 0;
            for (int h = 0; h < 9; ++h) rank += (sq[h] > sq[l]) || (sq[h] == sq[l] && h < l);
            if (rank < 4) code |= 1 << l;
        }
        atomicAdd(&hist[code], 1u);
    }
}

__global__ void k_pattern_library(const unsigned int *__restrict__ hist, int n_lib, int *__restrict__ lib) {
    __shared__ unsigned int h[512];
    const int c = threadIdx.x;   // 512 threads, one per 9-bit mask
    h[c] = hist[c];
    if (c < n_lib) lib[c] = -1;
    __syncthreads();
    const unsigned int n = h[c];
    if (n == 0) return;
    int rank = 0;
    for (int d = 0; d < 512; ++d) rank += (h[d] > n) || (h[d] == n && d < c);
    if (rank < n_lib) lib[rank] = c;
}

template <typename E>
__global__ void k_pattern_assign(const E *__restrict__ w, int n_kernels, int khw, const int *__restrict__ lib,
                                 int n_lib, double *__restrict__ score, int *__restrict__ idx,
                                 int *__restrict__ pat) {
    for (int k = blockIdx.x * blockDim.x + threadIdx.x; k < n_kernels; k += gridDim.x * blockDim.x) {
        double sq[9];
        for (int l = 0; l < 9; ++l) {
            const double v = ld_f64(w, (size_t)k * khw + l);
            sq[l] = v * v;
        }
        double best = -1.0;
        int bp = 0;
        for (int j = 0; j < n_lib; ++j) {
            const int code = lib[j];
            if (code < 0) break;   // fewer distinct masks than library entries
            double s = 0.0;
            for (int l = 0; l < 9; ++l)
                if ((code >> l) & 1) s += sq[l];
            if (s > best) {
                best = s;
                bp = j;
            }
        }
        score[k] = best;
        idx[k] = k;
        pat[k] = bp;
    }
}

__global__ void k_pattern_mask(const int *__restrict__ order, int n_keep, int n_kernels, const int *__restrict__ lib,
                               const int *__restrict__ pat, int khw, uint8_t *__restrict__ mask) {
    // order[0 .. n_keep) are the kept kernels; each thread writes one kept kernel's row
    // of 9 bytes, the mask having been cleared before
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n_keep; i += gridDim.x * blockDim.x) {
        const int k = order[i];
        const int code = lib[pat[k]];
        for (int l = 0; l < 9; ++l) mask[(size_t)k * khw + l] = (code >> l) & 1;
    }
    (void)n_kernels;
}

template <typename E>
static hipError_t prune_pattern(const Plan &p, const E *w, uint8_t *mask, hipStream_t st) {
    const int n = p.R * (p.C / p.khw);
    const int n_lib = p.bh_eff;   // library size (planner: bh, 0 -> 8)
    const int n_keep = pattern_kept(n, p.rate);
    size_t cub_bytes = 0;
    hipError_t e = hipcub::DeviceRadixSort::SortPairsDescending(nullptr, cub_bytes, (const uint64_t *)nullptr,
                                                                (uint64_t *)nullptr, (const int *)nullptr,
                                                                (int *)nullptr, n, 0, 64, st);
    if (e != hipSuccess) return e;
    // scratch: histogram, library, scores, sorted keys, indices, sorted indices, patterns, sort temp
    const size_t off_lib = 512 * 4, off_sc = 4096, off_keys = off_sc + 8 * (size_t)n,
                 off_idx = off_keys + 8 * (size_t)n, off_idx2 = off_idx + 4 * (size_t)n,
                 off_pat = off_idx2 + 4 * (size_t)n, off_tmp = (off_pat + 4 * (size_t)n + 255) / 256 * 256;
    char *scr = nullptr;
    e = hipMallocAsync((void **)&scr, off_tmp + cub_bytes, st);
    if (e != hipSuccess) return e;
    unsigned int *hist = (unsigned int *)scr;
    int *lib = (int *)(scr + off_lib);
    double *score = (double *)(scr + off_sc);
    uint64_t *keys2 = (uint64_t *)(scr + off_keys);
    int *idx = (int *)(scr + off_idx), *idx2 = (int *)(scr + off_idx2), *pat = (int *)(scr + off_pat);
    const int blocks = (int)std::min<int64_t>(4096, (n + 255) / 256);
    k_fill_u8<<<4, 256, 0, st>>>((uint8_t *)hist, 512 * 4, 0);
    k_fill_u8<<<(int)std::min<size_t>(8192, ((size_t)p.R * p.C + 255) / 256), 256, 0, st>>>(mask, (size_t)p.R * p.C, 0);
    k_pattern_own<E><<<blocks, 256, 0, st>>>(w, n, p.khw, hist);
    k_pattern_library<<<1, 512, 0, st>>>(hist, n_lib, lib);
    k_pattern_assign<E><<<blocks, 256, 0, st>>>(w, n, p.khw, lib, n_lib, score, idx, pat);
    // non-negative doubles sort like their bit patterns; the sort is stable
    e = hipcub::DeviceRadixSort::SortPairsDescending(scr + off_tmp, cub_bytes, (const uint64_t *)score, keys2, idx,
                                                      idx2, n, 0, 64, st);
    if (e == hipSuccess) {
        k_pattern_mask<<<blocks, 256, 0, st>>>(idx2, n_keep, n, lib, pat, p.khw, mask);
        e = hipGetLastError();
    }
    const hipError_t e2 = hipFreeAsync(scr, st);
    return e != hipSuccess ? e : e2;
}

__global__ void k_fill_u8(uint8_t *p, size_t n, uint8_t v) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// ---- unstructured: radix select ---------------------------------------------------
struct SelState {
    uint32_t prefix, pmask;
    uint32_t remaining;   // how many keys still to take at or below the current prefix
    uint32_t pad;
    uint32_t hist[256];
};

__global__ void k_sel_init(SelState *st, uint32_t k) {
    const int t = threadIdx.x;
    st->hist[t] = 0;
    if (t == 0) {
        st->prefix = 0;
        st->pmask = 0;
        st->remaining = k;
    }
}

template <typename E>
__global__ void k_sel_hist(const E *__restrict__ w, size_t n, SelState *st, int shift) {
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const uint32_t prefix = st->prefix, pmask = st->pmask;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        const uint32_t key = abs_key(w, i);
        if ((key & pmask) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (h[threadIdx.x]) atomicAdd(&st->hist[threadIdx.x], h[threadIdx.x]);
}

__global__ void k_sel_pick(SelState *st, int shift) {
    // single thread: walk the digits from the largest down
    uint32_t above = 0, rem = st->remaining;
    int chosen = 0;
    for (int b = 255; b >= 0; --b) {
        const uint32_t c = st->hist[b];
        if (above + c >= rem) {
            chosen = b;
            break;
        }
        above += c;
    }
    st->remaining = rem - above;
    st->prefix |= (uint32_t)chosen << shift;
    st->pmask |= 255u << shift;
    for (int b = 0; b < 256; ++b) st->hist[b] = 0;
}

constexpr int kSelChunk = 4096;  // elements per workgroup in the final pass

template <typename E>
__global__ void k_sel_count_eq(const E *__restrict__ w, size_t n, const SelState *st,
                               uint32_t *chunk_cnt) {
    __shared__ uint32_t cnt;
    if (threadIdx.x == 0) cnt = 0;
    __syncthreads();
    const uint32_t thr = st->prefix;
    const size_t base = (size_t)blockIdx.x * kSelChunk;
    uint32_t c = 0;
    for (int j = threadIdx.x; j < kSelChunk; j += blockDim.x) {
        const size_t i = base + j;
        if (i < n && abs_key(w, i) == thr) ++c;
    }
    if (c) atomicAdd(&cnt, c);
    __syncthreads();
    if (threadIdx.x == 0) chunk_cnt[blockIdx.x] = cnt;
}

__global__ void k_sel_scan(uint32_t *chunk_cnt, int nchunks) {
    uint32_t acc = 0;
    for (int i = 0; i < nchunks; ++i) {
        const uint32_t c = chunk_cnt[i];
        chunk_cnt[i] = acc;
        acc += c;
    }
}

template <typename E>
__global__ void k_sel_write(const E *__restrict__ w, size_t n, const SelState *st,
                            const uint32_t *chunk_off, uint8_t *__restrict__ mask) {
    // 256 threads x 16 consecutive elements each = one chunk
    __shared__ uint32_t pre[256];
    const uint32_t thr = st->prefix, need = st->remaining;
    const size_t base = (size_t)blockIdx.x * kSelChunk + (size_t)threadIdx.x * 16;
    uint32_t c = 0;
    for (int j = 0; j < 16; ++j) {
        const size_t i = base + j;
        if (i < n && abs_key(w, i) == thr) ++c;
    }
    pre[threadIdx.x] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t acc = 0;
        for (int t = 0; t < 256; ++t) {
            const uint32_t v = pre[t];
            pre[t] = acc;
            acc += v;
        }
    }
    __syncthreads();
    uint32_t rank = chunk_off[blockIdx.x] + pre[threadIdx.x];
    for (int j = 0; j < 16; ++j) {
        const size_t i = base + j;
        if (i >= n) break;
        const uint32_t key = abs_key(w, i);
        uint8_t keep = 0;
        if (key > thr) keep = 1;
        else if (key == thr) keep = (rank++ < need) ? 1 : 0;
        mask[i] = keep;
    }
}

// scratch of the radix select: the state, then one count per chunk of kSelChunk weights
inline size_t sel_scratch_bytes(size_t n) {
    return sizeof(SelState) + sizeof(uint32_t) * ((n + kSelChunk - 1) / kSelChunk);
}

// fixed: a caller's scratch of at least sel_scratch_bytes(n) bytes (nothing allocated),
// or null (a stream-ordered allocation, freed before returning).  Every part of the
// scratch that is read is first written by a kernel of this call.
template <typename E>
static hipError_t prune_unstructured(const Plan &p, const E *w, uint8_t *mask, hipStream_t st,
                                     void *fixed = nullptr) {
    const size_t n = (size_t)p.R * p.C;
    const uint32_t k = (uint32_t)((n + p.rate - 1) / p.rate);
    const int nchunks = (int)((n + kSelChunk - 1) / kSelChunk);
    void *scr = fixed;
    hipError_t e = hipSuccess;
    if (!fixed) {
        e = hipMallocAsync(&scr, sel_scratch_bytes(n), st);
        if (e != hipSuccess) return e;
    }
    SelState *s = (SelState *)scr;
    uint32_t *cc = (uint32_t *)((char *)scr + sizeof(SelState));
    const int hblocks = (int)std::min<size_t>(2048, (n + 255) / 256);
    k_sel_init<<<1, 256, 0, st>>>(s, k);
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        k_sel_hist<E><<<hblocks, 256, 0, st>>>(w, n, s, shift);
        k_sel_pick<<<1, 1, 0, st>>>(s, shift);
    }
    k_sel_count_eq<E><<<nchunks, 256, 0, st>>>(w, n, s, cc);
    k_sel_scan<<<1, 1, 0, st>>>(cc, nchunks);
    k_sel_write<E><<<nchunks, 256, 0, st>>>(w, n, s, cc, mask);
    e = hipGetLastError();
    if (fixed) return e;
    hipError_t e2 = hipFreeAsync(scr, st);
    return e != hipSuccess ? e : e2;
}

// ---- scratch of the allocation-free entry point -------------------------------------
// One fixed array per GPU (the module's device copy), sized for the radix select of
// up to kNoAllocMaxWeights weights.  Host code never uses the array's name as an
// address: the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[sizeof(SelState) +
                                                       sizeof(uint32_t) * (kNoAllocMaxWeights / kSelChunk)];
static_assert(kNoAllocMaxWeights % kSelChunk == 0, "whole chunks");

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once known
}  // namespace

// Device address of the current device's scratch (looked up on its first use there).
static hipError_t scratch_address(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!ptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_prune_noalloc(const Plan &p, const void *w, uint8_t *mask, hipStream_t st) {
    if (p.reg == BSP_UNSTRUCTURED) {
        if ((size_t)p.R * p.C > kNoAllocMaxWeights) return hipErrorInvalidValue;
        void *scr = nullptr;
        hipError_t e = scratch_address(&scr);
        if (e != hipSuccess) return e;
        return p.dt == BSP_F32 ? prune_unstructured(p, (const float *)w, mask, st, scr)
                               : prune_unstructured(p, (const uint16_t *)w, mask, st, scr);
    }
    if (p.reg == BSP_PATTERN || p.counts) return hipErrorInvalidValue;
    return launch_prune(p, w, mask, st);   // block kinds: no scratch
}

hipError_t launch_prune(const Plan &p, const void *w, uint8_t *mask, hipStream_t st) {
    const size_t n = (size_t)p.R * p.C;
    if (p.reg == BSP_DENSE) {
        const int blocks = (int)std::min<size_t>(4096, (n + 255) / 256);
        k_fill_u8<<<blocks, 256, 0, st>>>(mask, n, 1);
        return hipGetLastError();
    }
    if (p.reg == BSP_UNSTRUCTURED) {
        return p.dt == BSP_F32 ? prune_unstructured(p, (const float *)w, mask, st)
                               : prune_unstructured(p, (const uint16_t *)w, mask, st);
    }
    if (p.reg == BSP_PATTERN) {
        return p.dt == BSP_F32 ? prune_pattern(p, (const float *)w, mask, st)
                               : prune_pattern(p, (const uint16_t *)w, mask, st);
    }
    // per-block counts: a stream-ordered device copy, freed after the launch; the call
    // then waits for its stream, so the caller's host array may go once it returns
    int32_t *counts = nullptr;
    const size_t cbytes = sizeof(int32_t) * (size_t)p.nbr * p.nbc;
    if (p.counts) {
        hipError_t e = hipMallocAsync((void **)&counts, cbytes, st);
        if (e != hipSuccess) return e;
        e = hipMemcpyAsync(counts, p.counts, cbytes, hipMemcpyHostToDevice, st);
        if (e != hipSuccess) return e;
    }
    const int blocks = p.nbr * p.nbc;
    if (p.reg == BSP_ROWCOL) {
        const size_t lds = (sizeof(double) + 1) * (size_t)(p.bh_eff + p.bw_eff);
        if (p.dt == BSP_F32)
            k_prune_rowcol<float><<<blocks, 256, lds, st>>>((const float *)w, mask, p.R, p.C, p.bh_eff, p.bw_eff,
                                                            p.nbc, p.rate);
        else
            k_prune_rowcol<uint16_t><<<blocks, 256, lds, st>>>((const uint16_t *)w, mask, p.R, p.C, p.bh_eff,
                                                               p.bw_eff, p.nbc, p.rate);
    } else if (p.reg == BSP_PUNCHED) {
        const size_t lds = (sizeof(double) + 1) * (size_t)p.khw;
        if (p.dt == BSP_F32)
            k_prune_punched<float><<<blocks, 256, lds, st>>>((const float *)w, mask, p.R, p.C, p.khw, p.bh_eff,
                                                             p.bw_eff, p.nbc, p.rate, counts);
        else
            k_prune_punched<uint16_t><<<blocks, 256, lds, st>>>((const uint16_t *)w, mask, p.R, p.C, p.khw,
                                                                p.bh_eff, p.bw_eff, p.nbc, p.rate, counts);
    } else {
        const int col = p.reg == BSP_COL;
        const int ng_max = col ? p.bw_eff : p.bh_eff;
        const int threads = std::min(256, ((ng_max + 63) / 64) * 64);
        const size_t lds = sizeof(double) * (size_t)ng_max;
        if (p.dt == BSP_F32)
            k_prune_blocks<float><<<blocks, threads, lds, st>>>((const float *)w, mask, p.R, p.C,
                                                                p.bh_eff, p.bw_eff, p.nbc, col, p.rate, counts);
        else
            k_prune_blocks<uint16_t><<<blocks, threads, lds, st>>>((const uint16_t *)w, mask, p.R, p.C,
                                                                   p.bh_eff, p.bw_eff, p.nbc, col, p.rate,
                                                                   counts);
    }
    hipError_t e = hipGetLastError();
    if (counts) {
        const hipError_t e2 = hipFreeAsync(counts, st);
        const hipError_t e3 = hipStreamSynchronize(st);
        if (e == hipSuccess) e = e2 != hipSuccess ? e2 : e3;
    }
    return e;
}

}  // namespace bsp
