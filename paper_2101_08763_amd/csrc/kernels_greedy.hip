// kernels_greedy.hip -- the small kernels of the on-device Greedy optimizer
// (Algorithm 1): state initialisation and the deterministic argmax that picks
// each round's element without a round trip to the host.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace exemcl {

namespace {

constexpr int kThreads = 256;
constexpr int64_t kMaxBlocks = 1024;
constexpr int64_t kItemsPerBlock = 16 * kThreads;

// (v, i) beats (bv, bi) when larger, or equal with a lower index: the
// lowest candidate position wins ties.
__device__ inline void take(float &bv, int32_t &bi, float v, int32_t i) {
    if (v > bv || (v == bv && i < bi)) {
        bv = v;
        bi = i;
    }
}

// Block-wide best pair; the result is valid in thread 0.
__device__ inline void block_best(float &bv, int32_t &bi) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int32_t oi = __shfl_xor(bi, off);
        take(bv, bi, ov, oi);
    }
    __shared__ float sv[kThreads / 64];
    __shared__ int32_t si[kThreads / 64];
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        sv[w] = bv;
        si[w] = bi;
    }
    __syncthreads();
    if (threadIdx.x == 0)
        for (int q = 1; q < kThreads / 64; ++q) take(bv, bi, sv[q], si[q]);
}

__global__ __launch_bounds__(kThreads) void greedy_init_kernel(int32_t *__restrict__ cands,
                                                               uint8_t *__restrict__ taken,
                                                               float *__restrict__ g, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= n) return;
    cands[i] = (int32_t)i;
    taken[i] = 0;
    g[i] = 0.0f;  // S empty: only e0, whose h is 0 everywhere
}

// Stage 1: the best untaken candidate of each block's grid-stride share.  A
// NaN score ranks below every number.
__global__ __launch_bounds__(kThreads) void argmax_blocks_kernel(const float *__restrict__ scores,
                                                                 const uint8_t *__restrict__ taken, int64_t n,
                                                                 float *__restrict__ pval,
                                                                 int32_t *__restrict__ pidx) {
    float bv = -INFINITY;
    int32_t bi = INT32_MAX;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        if (taken[i]) continue;
        float v = scores[i];
        if (isnan(v)) v = -INFINITY;
        take(bv, bi, v, (int32_t)i);
    }
    block_best(bv, bi);
    if (threadIdx.x == 0) {
        pval[blockIdx.x] = bv;
        pidx[blockIdx.x] = bi;
    }
}

// Stage 2 (one block): the overall best; record it as this round's element,
// its score as f of the grown set, and mark it taken.
__global__ __launch_bounds__(kThreads) void argmax_final_kernel(const float *__restrict__ pval,
                                                                const int32_t *__restrict__ pidx, int64_t nb,
                                                                const float *__restrict__ scores,
                                                                uint8_t *__restrict__ taken, int64_t n,
                                                                int32_t *__restrict__ S_slot,
                                                                float *__restrict__ f_slot) {
    float bv = -INFINITY;
    int32_t bi = INT32_MAX;
    for (int64_t b = threadIdx.x; b < nb; b += kThreads) take(bv, bi, pval[b], pidx[b]);
    block_best(bv, bi);
    if (threadIdx.x == 0) {
        if (bi >= 0 && bi < n) {
            *S_slot = bi;
            *f_slot = scores[bi];
            taken[bi] = 1;
        } else {  // nothing left to take (the host never asks for that)
            *S_slot = kEmptySlot;
            *f_slot = __builtin_nanf("");
        }
    }
}

}  // namespace

int64_t argmax_blocks(int64_t n) {
    int64_t b = (n + kItemsPerBlock - 1) / kItemsPerBlock;
    return b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b);
}

hipError_t launch_greedy_init(int32_t *cands, uint8_t *taken, float *g, int64_t n, hipStream_t st) {
    hipLaunchKernelGGL(greedy_init_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, st,
                       cands, taken, g, n);
    return hipGetLastError();
}

hipError_t launch_argmax(const float *scores, uint8_t *taken, int64_t n, float *pval, int32_t *pidx,
                         int32_t *S_slot, float *f_slot, hipStream_t st) {
    const int64_t nb = argmax_blocks(n);
    hipLaunchKernelGGL(argmax_blocks_kernel, dim3((unsigned)nb), dim3(kThreads), 0, st, scores, taken, n, pval, pidx);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(argmax_final_kernel, dim3(1), dim3(kThreads), 0, st, pval, pidx, nb, scores, taken, n, S_slot,
                       f_slot);
    return hipGetLastError();
}

}  // namespace exemcl
