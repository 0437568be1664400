// kernels_aux.hip -- vector-ALU evaluation for small d, the fixed-order
// reduction of partial sums, row padding and the out-of-core accumulation.
#include <float.h>
#include <math.h>

#include "device.hpp"
#include "internal.h"

namespace exemcl {

// ---------------------------------------------------------------------------
// VALU evaluation (small d).
//
// Each thread keeps RPT ground points in registers (fp32, zero-padded to DP
// coordinates).  The exemplars of a chunk of sets are gathered once per
// workgroup into LDS as records [bias, s_0 .. s_{DP-1}] (bias = -||s||^2/2),
// and every wavefront reads them with uniform addresses (broadcast).  Per
// (point, set): m = max(m0, max_p (b_p + <v, s_p>)), the clamp form of
// min(||v||^2, min_p ||v - s_p||^2).  The per-thread sum over its points is
// reduced across the wavefront with a fixed xor tree and across the 4
// wavefronts in fixed order into partials[rb][j].
// ---------------------------------------------------------------------------
template <typename T, int DP, int RPT>
__global__ __launch_bounds__(256) void eval_valu_kernel(const T *__restrict__ V, int64_t n, int d,
                                                         const int32_t *__restrict__ sets, int64_t l, int64_t k,
                                                         int sets_per_chunk, float *__restrict__ partials,
                                                         int64_t lpad) {
    constexpr int REC = ((DP + 1) + 3) / 4 * 4;
    extern __shared__ __align__(16) float ex[];
    float *red = ex + (int64_t)sets_per_chunk * k * REC;  // [4][sets_per_chunk]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t rb = blockIdx.x;
    const int64_t j0 = (int64_t)blockIdx.y * sets_per_chunk;
    const int nsets = (int)min((int64_t)sets_per_chunk, l - j0);

    // Stage the chunk's exemplars: one record per (set, member).
    for (int64_t e = tid; e < (int64_t)nsets * k; e += 256) {
        const int64_t jj = e / k, p = e - (e / k) * k;
        const int64_t idx = sets[(j0 + jj) * k + p];
        float *rec = ex + e * REC;
        if (idx >= 0 && idx < n) {
            const T *row = V + idx * (int64_t)d;
            float q = 0.0f;
            for (int t = 0; t < DP; ++t) {
                const float x = t < d ? to_f32(row[t]) : 0.0f;
                rec[1 + t] = x;
                q = fmaf(x, x, q);
            }
            rec[0] = -0.5f * q;
        } else {
            for (int t = 0; t < DP; ++t) rec[1 + t] = 0.0f;
            rec[0] = -FLT_MAX;
        }
    }

    float v[RPT][DP];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int64_t i = rb * (256 * RPT) + r * 256 + tid;
#pragma unroll
        for (int t = 0; t < DP; ++t) v[r][t] = (i < n && t < d) ? to_f32(V[i * (int64_t)d + t]) : 0.0f;
    }
    __syncthreads();

    for (int jj = 0; jj < nsets; ++jj) {
        float m[RPT];
#pragma unroll
        for (int r = 0; r < RPT; ++r) m[r] = 0.0f;
        const float *recs = ex + (int64_t)jj * k * REC;
        for (int64_t p = 0; p < k; ++p) {
            const float *rec = recs + p * REC;
            float s[REC];
#pragma unroll
            for (int q = 0; q < REC; q += 4) {
                const float4 w = *reinterpret_cast<const float4 *>(rec + q);
                s[q] = w.x;
                s[q + 1] = w.y;
                s[q + 2] = w.z;
                s[q + 3] = w.w;
            }
#pragma unroll
            for (int r = 0; r < RPT; ++r) {
                float h = s[0];
#pragma unroll
                for (int t = 0; t < DP; ++t) h = fmaf(v[r][t], s[1 + t], h);
                m[r] = fmaxf(m[r], h);
            }
        }
        float sum = m[0];
#pragma unroll
        for (int r = 1; r < RPT; ++r) sum += m[r];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
        if (lane == 0) red[wave * sets_per_chunk + jj] = sum;
    }
    __syncthreads();
    for (int jj = tid; jj < nsets; jj += 256) {
        const float tot = ((red[jj] + red[sets_per_chunk + jj]) + red[2 * sets_per_chunk + jj]) +
                          red[3 * sets_per_chunk + jj];
        partials[rb * lpad + j0 + jj] = tot;
    }
}

bool valu_plan(int prec, int64_t d, int64_t k, ValuPlan *p) {
    (void)prec;
    if (d < 1 || d > 16 || k < 1) return false;
    ValuPlan q{};
    q.dp = d <= 1 ? 1 : d <= 2 ? 2 : d <= 4 ? 4 : d <= 8 ? 8 : 16;
    q.rpt = 4;
    q.rows = 256 * q.rpt;
    q.rec = ((q.dp + 1) + 3) / 4 * 4;
    const int64_t budget = 48 * 1024;
    const int64_t per_set = k * q.rec * (int64_t)sizeof(float) + 4 * sizeof(float);
    int64_t spc = budget / per_set;
    if (spc < 1) return false;
    if (spc > 64) spc = 64;
    q.sets_per_chunk = (int)spc;
    *p = q;
    return true;
}

template <typename T, int DP>
static hipError_t valu_t(const ValuPlan &pl, const void *V, int64_t n, int d, const int32_t *sets, int64_t l,
                         int64_t k, float *partials, int64_t lpad, hipStream_t st) {
    constexpr int RPT = 4;
    const int64_t G = (n + pl.rows - 1) / pl.rows;
    const int64_t chunks = (l + pl.sets_per_chunk - 1) / pl.sets_per_chunk;
    const size_t lds = ((size_t)pl.sets_per_chunk * k * pl.rec + 4 * (size_t)pl.sets_per_chunk) * sizeof(float);
    hipLaunchKernelGGL((eval_valu_kernel<T, DP, RPT>), dim3((unsigned)G, (unsigned)chunks), dim3(256), lds, st,
                       (const T *)V, n, d, sets, l, k, pl.sets_per_chunk, partials, lpad);
    return hipGetLastError();
}

template <typename T>
static hipError_t valu_dispatch(const ValuPlan &pl, const void *V, int64_t n, int d, const int32_t *sets, int64_t l,
                                int64_t k, float *partials, int64_t lpad, hipStream_t st) {
    switch (pl.dp) {
    case 1: return valu_t<T, 1>(pl, V, n, d, sets, l, k, partials, lpad, st);
    case 2: return valu_t<T, 2>(pl, V, n, d, sets, l, k, partials, lpad, st);
    case 4: return valu_t<T, 4>(pl, V, n, d, sets, l, k, partials, lpad, st);
    case 8: return valu_t<T, 8>(pl, V, n, d, sets, l, k, partials, lpad, st);
    case 16: return valu_t<T, 16>(pl, V, n, d, sets, l, k, partials, lpad, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_valu(int prec, const ValuPlan &pl, const void *V, int64_t n, int d, const int32_t *sets,
                       int64_t l, int64_t k, float *partials, int64_t lpad, hipStream_t st) {
    switch (prec) {
    case P_FP32: return valu_dispatch<float>(pl, V, n, d, sets, l, k, partials, lpad, st);
    case P_FP16: return valu_dispatch<_Float16>(pl, V, n, d, sets, l, k, partials, lpad, st);
    case P_BF16: return valu_dispatch<__bf16>(pl, V, n, d, sets, l, k, partials, lpad, st);
    }
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Second pass: out[j] = (2/n) * sum_g partials[g][j], fp64, one launch.
//
// A workgroup owns RJ sets and all G partial rows; its threads are RQ row
// lanes x RJ sets (consecutive threads read consecutive sets of one row).
// Row lane q adds rows q, q + RQ, q + 2 RQ, ... in order; the RQ lane sums
// are then added by a fixed pairwise tree.  The order depends on G only, so
// the result of a set does not depend on the batch it is in.  The index
// check turns a set with an index outside [0, n) other than the empty slot
// into NaN: row lane q checks members q, q + RQ, ... and a failed check makes
// its lane sum NaN, which the tree carries to the result.
// ---------------------------------------------------------------------------
#ifndef EXEMCL_RED_RJ
#define EXEMCL_RED_RJ 16
#endif
#ifndef EXEMCL_RED_RQ
#define EXEMCL_RED_RQ 64
#endif
constexpr int RJ = EXEMCL_RED_RJ;
constexpr int RQ = EXEMCL_RED_RQ;
static_assert((RQ & (RQ - 1)) == 0 && RJ * RQ <= 1024, "RQ a power of two, at most 1024 threads");

__device__ inline bool bad_index(int64_t idx, int64_t n) { return idx != kEmptySlot && (idx < 0 || idx >= n); }

__global__ __launch_bounds__(RJ * RQ) void reduce_sets_kernel(const float *__restrict__ partials, int64_t G,
                                                              int64_t lpad, int64_t l, int64_t n,
                                                              const int32_t *__restrict__ sets, int64_t kset,
                                                              const int32_t *__restrict__ common, int64_t kcommon,
                                                              float *__restrict__ out) {
    __shared__ double part[RQ][RJ];
    const int tid = threadIdx.x;
    const int jl = tid % RJ, q = tid / RJ;
    const int64_t j = (int64_t)blockIdx.x * RJ + jl;

    // The first member of each row lane's share is loaded before the
    // partial sums (from an address clamped into the arrays, without a
    // branch) and checked after them, so the loads overlap.  kset >= 1 and
    // l >= 1 whenever this kernel runs; when common is empty, sets[0] is read
    // in its place and ignored.
    const int32_t i0 = sets[(j < l ? j : l - 1) * kset + (q < kset ? q : kset - 1)];
    const int32_t c0 = *(kcommon > 0 ? common + (q < kcommon ? q : kcommon - 1) : sets);

    // Loads are issued UNR at a time (rows past G re-read row G-1 and are
    // then replaced by +0.0, which changes no sum), so the additions still
    // run in row order.
    constexpr int UNR = 16;
    double acc = 0.0;
    if (j < l) {
        for (int64_t g = q; g < G; g += RQ * UNR) {
            float x[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) x[u] = partials[min(g + u * RQ, G - 1) * lpad + j];
#pragma unroll
            for (int u = 0; u < UNR; ++u)
                if (g + u * RQ >= G) x[u] = 0.0f;
#pragma unroll
            for (int u = 0; u < UNR; ++u) acc += (double)x[u];
        }
    }
    bool bad = false;
    if (j < l) {
        bad = (q < kset && bad_index(i0, n)) || (q < kcommon && bad_index(c0, n));
        for (int64_t p = q + RQ; p < kset; p += RQ) bad |= bad_index(sets[j * kset + p], n);
        for (int64_t p = q + RQ; p < kcommon; p += RQ) bad |= bad_index(common[p], n);
    }
    part[q][jl] = bad ? __builtin_nan("") : acc;
    __syncthreads();
#pragma unroll
    for (int w = RQ / 2; w >= 1; w >>= 1) {
        if (q < w) part[q][jl] += part[q + w][jl];
        __syncthreads();
    }
    if (q != 0 || j >= l) return;
    out[j] = (float)(2.0 * part[0][jl] / (double)n);
}

hipError_t launch_reduce(const float *partials, int64_t G, int64_t lpad, int64_t l, int64_t n,
                         const int32_t *sets, int64_t kset, const int32_t *common, int64_t kcommon, float *out,
                         hipStream_t st) {
    if (l == 0) return hipSuccess;
    hipLaunchKernelGGL(reduce_sets_kernel, dim3((unsigned)((l + RJ - 1) / RJ)), dim3(RJ * RQ), 0, st, partials, G,
                       lpad, l, n, sets, kset, common, kcommon, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Rows padded for the MFMA kernels: one thread per 16-byte output vector.
// ---------------------------------------------------------------------------
int64_t mfma_row_stride(int prec, int64_t d) {
    const int64_t vec = prec == P_FP32 ? 4 : 8;
    return (d + vec - 1) / vec * vec;
}

// Rows of d elements that the MFMA kernels (and the exemplar staging) can
// read in place, with row stride d: every lane vector of a row lies wholly
// inside the row or wholly past its end (those read as zeros), which holds
// when d is a whole number of lane vectors -- or, for fp16/bf16 plans whose
// last k-block is a half one (8-byte lane vectors of 4 coordinates after
// whole 32-coordinate blocks), when d is a multiple of 4 (d = 100: 3 x 32
// coordinates, then 4 of the half block).  fp32 rows must start 16-byte
// aligned, fp16/bf16 rows 8-byte aligned (a 16-byte lane vector then sits
// at an 8-byte aligned address; the loads need 4-byte alignment).
bool mfma_rows_in_place(int prec, int64_t d) {
    MfmaPlan pl;
    if (!mfma_plan(prec, d, &pl)) return false;
    if (prec == P_FP32) return d % 4 == 0;
    return d % 8 == 0 || (pl.half && d % 4 == 0);
}

bool mfma_rows_ready(int prec, const void *V, int64_t d) {
    const uintptr_t align = prec == P_FP32 ? 16 : 8;
    return mfma_rows_in_place(prec, d) && (uintptr_t)V % align == 0;
}

template <typename T>
__global__ __launch_bounds__(256) void pad_rows_kernel(const T *__restrict__ V, int64_t n, int d, T *__restrict__ Vp,
                                                       int ld) {
    constexpr int VEC = 16 / sizeof(T);
    const int64_t vpr = ld / VEC;
    const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (q >= n * vpr) return;
    const int64_t i = q / vpr;
    const int t0 = (int)(q - i * vpr) * VEC;
    T *dst = Vp + i * (int64_t)ld + t0;
#pragma unroll
    for (int e = 0; e < VEC; ++e) dst[e] = t0 + e < d ? V[i * (int64_t)d + t0 + e] : (T)0.0f;
}

hipError_t launch_pad(int prec, const void *V, int64_t n, int d, void *Vp, int ld, hipStream_t st) {
    const int64_t vec = prec == P_FP32 ? 4 : 8;
    const int64_t blocks = (n * (ld / vec) + 255) / 256;
    switch (prec) {
    case P_FP32:
        hipLaunchKernelGGL(pad_rows_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, st, (const float *)V, n, d,
                           (float *)Vp, ld);
        break;
    case P_FP16:
        hipLaunchKernelGGL(pad_rows_kernel<_Float16>, dim3((unsigned)blocks), dim3(256), 0, st, (const _Float16 *)V, n,
                           d, (_Float16 *)Vp, ld);
        break;
    case P_BF16:
        hipLaunchKernelGGL(pad_rows_kernel<__bf16>, dim3((unsigned)blocks), dim3(256), 0, st, (const __bf16 *)V, n, d,
                           (__bf16 *)Vp, ld);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// f of empty sets (k = 0): out[j] = 0, e0 alone.
__global__ __launch_bounds__(256) void zero_kernel(float *__restrict__ out, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < count) out[i] = 0.0f;
}

hipError_t launch_zero(float *out, int64_t count, hipStream_t st) {
    if (count == 0) return hipSuccess;
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, out, count);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Out-of-core evaluation: the per-set sums of one block of ground points are
// added to an fp64 accumulator (acc[j] = sum over blocks in order, each block
// summed over its partial rows in the fixed order of the second pass: row
// lanes q, q + RQ, ... then a pairwise tree), and the accumulator is turned
// into f(S_j) = (2/n) * acc[j] at the end (NaN for a set with an invalid
// index).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(RJ * RQ) void accum_sets_kernel(const float *__restrict__ partials, int64_t G,
                                                             int64_t lpad, int64_t l, int first,
                                                             double *__restrict__ acc) {
    __shared__ double part[RQ][RJ];
    const int tid = threadIdx.x;
    const int jl = tid % RJ, q = tid / RJ;
    const int64_t j = (int64_t)blockIdx.x * RJ + jl;
    constexpr int UNR = 16;
    double s = 0.0;
    if (j < l) {
        for (int64_t g = q; g < G; g += RQ * UNR) {
            float x[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) x[u] = partials[min(g + u * RQ, G - 1) * lpad + j];
#pragma unroll
            for (int u = 0; u < UNR; ++u)
                if (g + u * RQ >= G) x[u] = 0.0f;
#pragma unroll
            for (int u = 0; u < UNR; ++u) s += (double)x[u];
        }
    }
    part[q][jl] = s;
    __syncthreads();
#pragma unroll
    for (int w = RQ / 2; w >= 1; w >>= 1) {
        if (q < w) part[q][jl] += part[q + w][jl];
        __syncthreads();
    }
    if (q != 0 || j >= l) return;
    acc[j] = first ? part[0][jl] : acc[j] + part[0][jl];
}

hipError_t launch_accum(const float *partials, int64_t G, int64_t lpad, int64_t l, bool first, double *acc,
                        hipStream_t st) {
    if (l == 0) return hipSuccess;
    hipLaunchKernelGGL(accum_sets_kernel, dim3((unsigned)((l + RJ - 1) / RJ)), dim3(RJ * RQ), 0, st, partials, G,
                       lpad, l, first ? 1 : 0, acc);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void finish_sets_kernel(const double *__restrict__ acc,
                                                           const uint8_t *__restrict__ bad, int64_t l, double scale,
                                                           float *__restrict__ out) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j >= l) return;
    out[j] = bad[j] ? __builtin_nanf("") : (float)(scale * acc[j]);
}

hipError_t launch_finish(const double *acc, const uint8_t *bad, int64_t l, int64_t n, float *out, hipStream_t st) {
    if (l == 0) return hipSuccess;
    hipLaunchKernelGGL(finish_sets_kernel, dim3((unsigned)((l + 255) / 256)), dim3(256), 0, st, acc, bad, l,
                       2.0 / (double)n, out);
    return hipGetLastError();
}

}  // namespace exemcl
