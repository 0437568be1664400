// kernels_sqnorm.hip -- squared norms of the ground points (A1), one
// HBM-bound pass over V.
#include <stdint.h>
#include <stdlib.h>

#include <algorithm>

#include "device.hpp"
#include "internal.h"

namespace exemcl {

// ---------------------------------------------------------------------------
// q[i] = ||v_i||^2 in fp32 (A1).  HBM-bound: L consecutive lanes share a row
// (L a power of two, enough for one pass over the row where d allows), lane
// j takes the groups of G coordinates j, j + L, j + 2L, ... (G = 16 bytes'
// worth when d allows, else 1), so a wavefront reads whole contiguous rows;
// the L lane sums are added by a fixed xor tree.  Each lane group works on U
// rows at once, so U independent loads are in flight per lane.  The order
// of additions of a row depends on d and the storage type only; VLOAD
// (16-byte aligned rows) and U only change how the groups are loaded.
// ---------------------------------------------------------------------------
#ifndef EXEMCL_SQ_UNROLL
#define EXEMCL_SQ_UNROLL 4
#endif
// Non-temporal 16-byte loads: V is read once, so its lines need not stay in
// the caches (large1m: 7.2 TB/s instead of 6.2).
#ifndef EXEMCL_SQ_NT
#define EXEMCL_SQ_NT 1
#endif
#ifndef EXEMCL_SQ_MAX_BLOCKS
#define EXEMCL_SQ_MAX_BLOCKS 65536
#endif

template <typename T, int G, bool VLOAD, int U>
__global__ __launch_bounds__(256) void sqnorm_kernel(const T *__restrict__ V, int64_t n, int d, int L,
                                                      float *__restrict__ q) {
    typedef T vec_t __attribute__((ext_vector_type(G)));
    const int rpb = 256 / L;  // rows per workgroup and unrolled slot
    const int j = threadIdx.x % L;
    const int r = threadIdx.x / L;
    // every thread of the workgroup runs the same passes, so the whole
    // wavefront takes part in each shuffle
    for (int64_t base = (int64_t)blockIdx.x * rpb * U; base < n; base += (int64_t)gridDim.x * rpb * U) {
        const T *row[U];
        float s[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            // rows past n read the last row (in bounds) and are not stored
            const int64_t i = base + (int64_t)u * rpb + r;
            row[u] = V + (i < n ? i : n - 1) * (int64_t)d;
            s[u] = 0.0f;
        }
        for (int64_t t0 = (int64_t)j * G; t0 < d; t0 += (int64_t)L * G) {  // 64-bit: d may be near INT32_MAX
            vec_t v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if constexpr (VLOAD) {
#if EXEMCL_SQ_NT
                    v[u] = __builtin_nontemporal_load(reinterpret_cast<const vec_t *>(row[u] + t0));
#else
                    v[u] = *reinterpret_cast<const vec_t *>(row[u] + t0);
#endif
                } else {
#pragma unroll
                    for (int e = 0; e < G; ++e) v[u][e] = row[u][t0 + e];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int e = 0; e < G; ++e) {
                    const float x = to_f32((T)v[u][e]);
                    s[u] = fmaf(x, x, s[u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            for (int off = L / 2; off >= 1; off >>= 1) s[u] += __shfl_xor(s[u], off);
            const int64_t i = base + (int64_t)u * rpb + r;
            if (i < n && j == 0) q[i] = s[u];
        }
    }
}

// Workgroups per launch at most; larger inputs take several passes.
// EXEMCL_SQNORM_MAX_BLOCKS=<b> lowers the cap (tests: several passes at a
// small n); results do not depend on it.
constexpr int64_t kSqnormMaxBlocks = EXEMCL_SQ_MAX_BLOCKS;

static int64_t sqnorm_block_cap() {
    const char *s = getenv("EXEMCL_SQNORM_MAX_BLOCKS");
    const long long b = s ? atoll(s) : 0;
    return b >= 1 && b < kSqnormMaxBlocks ? (int64_t)b : kSqnormMaxBlocks;
}

template <typename T>
hipError_t sqnorm_t(const void *V, int64_t n, int d, float *q, hipStream_t st) {
    constexpr int VEC = 16 / (int)sizeof(T);
    constexpr int U = EXEMCL_SQ_UNROLL;
    const bool grouped = d % VEC == 0;
    const int G = grouped ? VEC : 1;
    int L = 1;
    while (L < 64 && (int64_t)L * G < d) L <<= 1;
    const int64_t rows_per_block = (int64_t)(256 / L) * U;
    const int64_t blocks = std::min<int64_t>((n + rows_per_block - 1) / rows_per_block, sqnorm_block_cap());
    const T *Vt = (const T *)V;
    if (grouped && (uintptr_t)V % 16 == 0)
        hipLaunchKernelGGL((sqnorm_kernel<T, VEC, true, U>), dim3((unsigned)blocks), dim3(256), 0, st, Vt, n, d, L, q);
    else if (grouped)
        hipLaunchKernelGGL((sqnorm_kernel<T, VEC, false, U>), dim3((unsigned)blocks), dim3(256), 0, st, Vt, n, d, L,
                           q);
    else
        hipLaunchKernelGGL((sqnorm_kernel<T, 1, false, U>), dim3((unsigned)blocks), dim3(256), 0, st, Vt, n, d, L, q);
    return hipGetLastError();
}

hipError_t launch_sqnorm(int prec, const void *V, int64_t n, int d, float *q, hipStream_t st) {
    switch (prec) {
    case P_FP32: return sqnorm_t<float>(V, n, d, q, st);
    case P_FP16: return sqnorm_t<_Float16>(V, n, d, q, st);
    case P_BF16: return sqnorm_t<__bf16>(V, n, d, q, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
