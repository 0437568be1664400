// bigd_kernels.hpp -- the evaluation kernel for dimensions above 512.
//
// The main kernel (mfma_kernels.hpp) keeps a wavefront's ground points in
// registers over all d coordinates, which bounds d.  Here the coordinates
// are split instead: the 8 wavefronts of a workgroup share one block of 32
// points, and wavefront w holds, in registers, the points' k-blocks
// (r*KW + j)*8 + w, j < KW, of round r (one round when 8*KW*KB_DIMS >= d;
// more rounds reload the registers per tile batch, so d has no upper
// bound; blocks past d are skipped).  For each staged exemplar tile every wavefront
// forms the dot products of its k-blocks (MFMA, fp32 accumulate); the eight
// partial products are added in LDS in wavefront order, the column's bias
// -||s||^2/2 is added, and the clamp-form epilogue follows as in the main
// kernel: a running max over the set's members (and e0's 0, or the cached
// value when scoring S u {c}) per (point, set), summed over the points when
// the set group ends.  The distance matrix is never written.
//
// Work split after the LDS sum: wavefront w owns row tile w / 4 and
// accumulator element w % 4 of the 16x16 MFMA output layout, i.e. points
// 16*(w/4) + 4*g + w%4 (g = lane / 16) of the block, column lane % 16.  Its
// partial sum per set covers those four points: partials[(rb*8 + w)*lpad +
// j], in the same layout as the main kernel's (one row per wavefront).
//
// Exemplar fragments are read straight from the staged tiles in global
// memory (every workgroup walks the same tiles, which stay in L2) through
// a ring of PF fragments in flight per wavefront.
#pragma once

#include <float.h>

#include <hip/hip_ext.h>

#include "device.hpp"
#include "internal.h"

namespace exemcl {

constexpr int kBigdWaves = 8;
constexpr int kBigdRT = 2;     // row tiles of 16 points per block
constexpr int kBigdBatch = 4;  // tiles per LDS reduction

template <typename T, int KW, int MODE, bool HAS_M0>
__global__ __launch_bounds__(kBigdWaves * 64, 1) void eval_bigd_kernel(
    const T *__restrict__ V, int64_t n, int ld, int nkb, int rounds, const unsigned char *__restrict__ tiles,
    int64_t kt, int64_t ngroups, int64_t gpc, const float *__restrict__ m0, float *__restrict__ partials,
    int64_t lpad, float *__restrict__ rowmax) {
    using M = Mfma<T, 16>;
    using vec_t = typename M::vec_t;
    using acc_t = typename M::acc_t;
    constexpr int TM = 16, NB = M::NB, RT = kBigdRT, W = kBigdWaves, TBATCH = kBigdBatch;
    constexpr int HDR = (TM * NB * 4 + 127) / 128 * 128;
    constexpr int U = TBATCH * KW * NB;  // fragments a wavefront uses per tile batch and round
    constexpr int PF = U < 16 ? U : 16;  // fragments in flight
    static_assert(M::ACC == 4, "16x16 output: four accumulators per lane");

    extern __shared__ __align__(16) unsigned char smem[];
    float *red = reinterpret_cast<float *>(smem);  // [TBATCH][W][RT][NB][4][64]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane % TM, grp = lane / TM;
    const int64_t tbytes = HDR + (int64_t)nkb * NB * 1024;
    const int64_t rb = blockIdx.x;
    const int64_t row0 = rb * (RT * TM);
    const int64_t wrows = min((int64_t)(RT * TM), n - row0);
    const auto vwin = window_rsrc(V + row0 * (int64_t)ld, (uint32_t)(wrows * ld * (int64_t)sizeof(T)));

    // This wavefront's k-blocks of round r, in A-operand order; blocks past
    // the data (kb >= nkb, or a vector past ld) are zero.
    vec_t a[RT][KW];
    auto load_a = [&](int r) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int j = 0; j < KW; ++j) {
                const int kb = (r * KW + j) * W + wave;
                const int d0 = M::dim(kb, grp, 0);
                const bool live = kb < nkb && d0 < ld;
                a[rt][j] = window_load16<vec_t>(vwin, live ? (uint32_t)(((rt * TM + lr) * ld + d0) * (int)sizeof(T))
                                                           : kDeadOffset);
            }
    };
    if (rounds == 1) load_a(0);

    // The (point, set) this lane owns after the LDS sum.
    const int rto = wave >> 2, io = wave & 3;
    const int64_t orow = row0 + rto * TM + 4 * grp + io;
    const float minit = HAS_M0 ? (orow < n ? m0[orow] : 0.0f) : 0.0f;
    float m = minit;

    const int64_t g0 = (int64_t)blockIdx.y * gpc, g1 = min(ngroups, g0 + gpc);
    float *wpart = partials + (rb * W + wave) * lpad;
    for (int64_t g = g0; g < g1; ++g) {
        for (int64_t q0 = 0; q0 < kt; q0 += TBATCH) {
            const int nt = (int)min((int64_t)TBATCH, kt - q0);
            // tile t of the batch (a batch past the group's last tile re-reads it)
            auto tile_of = [&](int t) { return tiles + (g * kt + q0 + (t < nt ? t : nt - 1)) * tbytes; };
            acc_t acc[TBATCH][RT][NB];
#pragma unroll
            for (int t = 0; t < TBATCH; ++t)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int h = 0; h < NB; ++h)
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[t][rt][h][i] = 0.0f;
            for (int r = 0; r < rounds; ++r) {
                if (rounds > 1) load_a(r);
                // fragment u = (t*KW + j)*NB + h: block kb = (r*KW + j)*W + wave
                // of tile t, member h (blocks past the data read the last one
                // and are not used)
                auto frag = [&](int u) -> vec_t {
                    const int t = u / (KW * NB), j = (u / NB) % KW, h = u % NB;
                    int kb = (r * KW + j) * W + wave;
                    kb = kb < nkb ? kb : nkb - 1;
                    return reinterpret_cast<const vec_t *>(tile_of(t) + HDR)[(kb * NB + h) * 64 + lane];
                };
                vec_t bq[PF];
#pragma unroll
                for (int u = 0; u < PF; ++u) bq[u] = frag(u);
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const vec_t b = bq[u % PF];
                    if (u + PF < U) bq[u % PF] = frag(u + PF);
                    const int t = u / (KW * NB), j = (u / NB) % KW, h = u % NB;
                    __builtin_amdgcn_sched_barrier(0);
                    if ((r * KW + j) * W + wave < nkb) {  // uniform: the wavefront's block exists
#pragma unroll
                        for (int e = 0; e < M::KS_PER_KB; ++e)
#pragma unroll
                            for (int rt = 0; rt < RT; ++rt) acc[t][rt][h] = M::mma(a[rt][j], b, e, acc[t][rt][h]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            // Sum the wavefronts' partial products in LDS (wavefront order),
            // add the bias, fold into the running max.
#pragma unroll
            for (int t = 0; t < TBATCH; ++t)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int h = 0; h < NB; ++h)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            red[((((t * W + wave) * RT + rt) * NB + h) * 4 + i) * 64 + lane] = acc[t][rt][h][i];
            __syncthreads();
            for (int t = 0; t < nt; ++t) {
                const float *hb = reinterpret_cast<const float *>(tile_of(t));
#pragma unroll
                for (int h = 0; h < NB; ++h) {
                    float s = 0.0f;
#pragma unroll
                    for (int w = 0; w < W; ++w) s += red[((((t * W + w) * RT + rto) * NB + h) * 4 + io) * 64 + lane];
                    m = fmaxf(m, s + hb[h * TM + lr]);
                }
            }
            __syncthreads();
        }
        if constexpr (MODE == MODE_SUM) {
            // the set group ends: the wavefront's four points per set
            float sum = m;
#pragma unroll
            for (int off = TM; off < 64; off <<= 1) sum += __shfl_xor(sum, off);
            if (grp == 0) wpart[g * TM + lr] = sum;
            m = minit;
        }
    }
    if constexpr (MODE == MODE_ROWMAX) {
        // the point's maximum over every staged column, clamped at e0's 0
        float x = fmaxf(m, 0.0f);
#pragma unroll
        for (int off = 1; off < TM; off <<= 1) x = fmaxf(x, __shfl_xor(x, off));
        if (lr == 0 && orow < n) rowmax[orow] = x;
    }
}

template <typename T, int KW, int MODE, bool HAS_M0>
hipError_t bigd_launch_t(const MfmaPlan &pl, const MfmaArgs &x, hipStream_t st) {
    constexpr int NB = Mfma<T, 16>::NB;
    auto kern = eval_bigd_kernel<T, KW, MODE, HAS_M0>;
    const size_t lds = (size_t)kBigdBatch * kBigdWaves * kBigdRT * NB * 4 * 64 * sizeof(float);
    if (lds > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    const int64_t rows = (int64_t)kBigdRT * 16;
    const int64_t G = (x.n + rows - 1) / rows;
    const int64_t chunks = (x.ngroups + x.gpc - 1) / x.gpc;
    hipExtLaunchKernelGGL(kern, dim3((unsigned)G, (unsigned)chunks), dim3(kBigdWaves * 64), lds, st, x.ev_start,
                          x.ev_stop, 0, (const T *)x.V, x.n, x.ld, pl.nkb, pl.rounds, (const unsigned char *)x.tiles,
                          x.kt, x.ngroups, x.gpc, x.m0, x.partials, x.lpad, x.rowmax);
    return hipGetLastError();
}

template <typename T, int MODE, bool HAS_M0>
hipError_t bigd_dispatch_kw(const MfmaPlan &pl, const MfmaArgs &x, hipStream_t st) {
    switch (pl.kw) {
    case 2: return bigd_launch_t<T, 2, MODE, HAS_M0>(pl, x, st);
    case 4: return bigd_launch_t<T, 4, MODE, HAS_M0>(pl, x, st);
    case 8: return bigd_launch_t<T, 8, MODE, HAS_M0>(pl, x, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
