// kernels_mfma.hip -- exemplar staging and the matrix-core evaluation kernel.
//
// The paper's GPU algorithm (Algorithm 3) assigns one thread to each cell
// W[j][i] = min_{s in S_j} d(v_i, s) / n of the work matrix (Eq. (7)), loops
// over the set members and writes W to global memory before a row sum
// (Section IV-B).  Here the same quantity is computed as a dense contraction
// on the MFMA units with a fused epilogue, and W is never materialised:
//
//   min(||v||^2, min_s ||v - s||^2) = ||v||^2 - 2 max(0, max_s h_s(v)),
//   h_s(v) = <v, s> - ||s||^2 / 2,
//
// so f(S) = L({e0}) - L(S u {e0}) = (2/n) sum_v max(0, max_s h_s(v)).  The 0
// is e0's contribution (Eq. (4)).  For every (row block, set) pair a
// workgroup produces one partial sum; a second pass adds the partials in a
// fixed order.
//
// Data layout.  A workgroup owns `rows` consecutive ground points and keeps
// them in registers in MFMA A-operand order for its whole life.  Exemplars
// are streamed: for every (group of TM sets, slot p) a "tile" holds the p-th
// member of each of the TM sets, already in B-operand order (k-block-major,
// 64 lanes x 16 bytes per k-block), plus one fp32 bias -||s||^2/2 per column.
// Tiles are double-buffered through LDS.  Each lane's output column is one
// set, so the minimum over a set's members is a per-register running max
// across successive tiles -- no cross-lane traffic until the set group ends.
#include <float.h>

#include "device.hpp"
#include "internal.h"

namespace exemcl {

// ---------------------------------------------------------------------------
// Staging: gather exemplar rows by index into tiles, with their norms.
// One wavefront per tile.  Tile t = g*k + p holds column c = set g*TM + c,
// member p.  Padding columns (set >= l) and invalid indices become zero
// vectors with bias -FLT_MAX, which never wins the running max.
// ---------------------------------------------------------------------------
template <typename T, int TILE>
__global__ __launch_bounds__(64) void pack_tiles_kernel(const T *__restrict__ V, int64_t n, int d,
                                                        const int32_t *__restrict__ sets, int64_t l,
                                                        int64_t k, int nkb, typename Mfma<T, TILE>::vec_t *tiles,
                                                        float *__restrict__ bias, bool vec_ok) {
    using M = Mfma<T, TILE>;
    const int64_t t = blockIdx.x;
    const int64_t g = t / k, p = t - (t / k) * k;
    const int lane = threadIdx.x;
    const int col = lane % M::TM, grp = lane / M::TM;
    const int64_t j = g * M::TM + col;
    int64_t idx = -1;
    if (j < l) idx = sets[j * k + p];
    const bool valid = idx >= 0 && idx < n;
    typename M::vec_t *dst = tiles + t * (int64_t)nkb * 64;
    for (int kb = 0; kb < nkb; ++kb) {
        dst[kb * 64 + lane] = load_lanevec<M>(V, n, d, valid ? idx : n, kb, grp, vec_ok);
    }
    if (grp == 0) {
        float q = 0.0f;
        if (valid) {
            const T *row = V + idx * (int64_t)d;
            for (int e = 0; e < d; ++e) {
                const float x = to_f32(row[e]);
                q = fmaf(x, x, q);
            }
        }
        bias[t * M::TM + col] = valid ? -0.5f * q : -FLT_MAX;
    }
}

// ---------------------------------------------------------------------------
// Evaluation kernel.
//
// grid.x = row blocks (rows consecutive points each), grid.y = chunks of set
// groups.  Block = WAVES wavefronts; wavefront w owns RT row tiles of TM rows.
// Dynamic LDS: two tile buffers of nkb KiB, then the cross-wave reduction
// buffer red[2][WAVES][TM].
// ---------------------------------------------------------------------------
template <typename T, int TILE, int KBMAX, int RT, int WAVES, int MODE>
__global__ __launch_bounds__(WAVES * 64) void eval_mfma_kernel(
    const T *__restrict__ V, int64_t n, int d, int nks, int nkb, const typename Mfma<T, TILE>::vec_t *__restrict__ tiles,
    const float *__restrict__ bias, int64_t k, int64_t ngroups, int64_t groups_per_chunk,
    const float *__restrict__ m0, float *__restrict__ partials, int64_t lpad, float *__restrict__ rowmax,
    bool vec_ok) {
    using M = Mfma<T, TILE>;
    using vec_t = typename M::vec_t;
    using acc_t = typename M::acc_t;
    constexpr int TM = M::TM;
    constexpr int NT = WAVES * 64;
    constexpr int RMAX = (KBMAX * 64 + NT - 1) / NT;

    extern __shared__ __align__(16) unsigned char smem[];
    vec_t *buf0 = reinterpret_cast<vec_t *>(smem);
    vec_t *buf1 = buf0 + nkb * 64;
    float *red = reinterpret_cast<float *>(buf1 + nkb * 64);  // [2][WAVES][TM]

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int lr = lane % TM, grp = lane / TM;
    const int64_t rb = blockIdx.x;
    const int64_t g0 = (int64_t)blockIdx.y * groups_per_chunk;
    const int64_t g1 = min(ngroups, g0 + groups_per_chunk);
    const int64_t row0 = rb * (int64_t)(WAVES * RT * TM) + (int64_t)wave * RT * TM;

    // Ground points of this wavefront, in A-operand order, resident for the
    // whole kernel.
    vec_t a[RT][KBMAX];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int kb = 0; kb < KBMAX; ++kb)
            if (kb < nkb) a[rt][kb] = load_lanevec<M>(V, n, d, row0 + rt * TM + lr, kb, grp, vec_ok);

    // Initial value of the running max for each output element: e0's 0, or
    // the per-point cached value when scoring S u {c}.
    float minit[RT][M::ACC];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < M::ACC; ++i) {
            const int64_t r = row0 + rt * TM + out_row<TM>(i, grp);
            minit[rt][i] = (m0 != nullptr && r < n) ? m0[r] : 0.0f;
        }

    const int64_t ntiles = (g1 - g0) * k;
    const int64_t tile_vecs = (int64_t)nkb * 64;
    const vec_t *src0 = tiles + g0 * k * tile_vecs;
    const float *bias0 = bias + g0 * k * TM;

    vec_t pre[RMAX];
    float bnext = 0.0f;
    auto gload = [&](int64_t t) {
        const vec_t *src = src0 + t * tile_vecs;
#pragma unroll
        for (int r = 0; r < RMAX; ++r) {
            const int idx = tid + r * NT;
            if (idx < tile_vecs) pre[r] = src[idx];
        }
        bnext = bias0[t * TM + lr];
    };
    auto lstore = [&](vec_t *dst) {
#pragma unroll
        for (int r = 0; r < RMAX; ++r) {
            const int idx = tid + r * NT;
            if (idx < tile_vecs) dst[idx] = pre[r];
        }
    };

    float m[RT][M::ACC];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < M::ACC; ++i) m[rt][i] = minit[rt][i];

    if (ntiles > 0) {
        gload(0);
        lstore(buf0);
    }
    __syncthreads();

    int64_t g = g0;
    int64_t p = 0;
    for (int64_t t = 0; t < ntiles; ++t) {
        const float b = bnext;
        if (t + 1 < ntiles) gload(t + 1);
        const vec_t *B = (t & 1) ? buf1 : buf0;

        acc_t acc[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i) acc[rt][i] = b;

#pragma unroll
        for (int kb = 0; kb < KBMAX; ++kb) {
            if (kb < nkb) {
                const vec_t bv = B[kb * 64 + lane];
#pragma unroll
                for (int e = 0; e < M::KS_PER_KB; ++e) {
                    if (kb * M::KS_PER_KB + e < nks) {
#pragma unroll
                        for (int rt = 0; rt < RT; ++rt) acc[rt] = M::mma(a[rt][kb], bv, e, acc[rt]);
                    }
                }
            }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i) m[rt][i] = fmaxf(m[rt][i], acc[rt][i]);

        const bool group_end = (MODE == MODE_SUM) && (p == k - 1);
        if (group_end) {
            // Sum this lane's rows for its column, then the K-groups holding
            // the other rows of the same column, in a fixed order.
            float s = 0.0f;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < M::ACC; ++i) s += m[rt][i];
#pragma unroll
            for (int off = TM; off < 64; off <<= 1) s += __shfl_xor(s, off);
            if (grp == 0) red[((g & 1) * WAVES + wave) * TM + lr] = s;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < M::ACC; ++i) m[rt][i] = minit[rt][i];
        }
        if (t + 1 < ntiles) lstore((t & 1) ? buf0 : buf1);
        __syncthreads();
        if (group_end && wave == 0 && lane < TM) {
            const float *rr = red + (g & 1) * WAVES * TM;
            float tot = rr[lane];
#pragma unroll
            for (int w = 1; w < WAVES; ++w) tot += rr[w * TM + lane];
            partials[rb * lpad + g * TM + lane] = tot;
        }
        if (++p == k) {
            p = 0;
            ++g;
        }
    }

    if constexpr (MODE == MODE_ROWMAX) {
        // Maximum over all staged columns (the members of S) for every row,
        // clamped at e0's 0: the per-point cache g(v).
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i) {
                float x = fmaxf(m[rt][i], 0.0f);
#pragma unroll
                for (int off = 1; off < TM; off <<= 1) x = fmaxf(x, __shfl_xor(x, off));
                m[rt][i] = x;
            }
        if (lr == 0) {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < M::ACC; ++i) {
                    const int64_t r = row0 + rt * TM + out_row<TM>(i, grp);
                    if (r < n) rowmax[r] = m[rt][i];
                }
        }
    }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
static int next_pow2(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

bool mfma_plan(int prec, int64_t d, MfmaPlan *p) {
    if (d < 1 || d > 512) return false;
    MfmaPlan q{};
    q.waves = 4;
    if (prec == P_FP32) {
        if (d <= 256) {
            q.tile = 32;
            q.kb_dims = 8;
            q.nks = (int)((d + 1) / 2);
        } else {
            q.tile = 16;
            q.kb_dims = 16;
            q.nks = (int)((d + 3) / 4);
        }
    } else {
        q.tile = 32;
        q.kb_dims = 16;
        q.nks = (int)((d + 15) / 16);
    }
    q.nkb = (int)((d + q.kb_dims - 1) / q.kb_dims);
    q.kbmax = next_pow2(q.nkb);
    q.rt = q.kbmax <= 16 ? 2 : 1;
    q.rows = q.waves * q.rt * q.tile;
    *p = q;
    return true;
}

template <typename T, int TILE>
static hipError_t pack_t(const MfmaPlan &pl, const void *V, int64_t n, int d, const int32_t *sets, int64_t l,
                         int64_t k, void *tiles, float *bias, hipStream_t st) {
    using M = Mfma<T, TILE>;
    const int64_t ngroups = (l + TILE - 1) / TILE;
    const bool vec_ok = ((uintptr_t)V % 16 == 0) && ((d * (int64_t)sizeof(T)) % 16 == 0);
    hipLaunchKernelGGL((pack_tiles_kernel<T, TILE>), dim3((unsigned)(ngroups * k)), dim3(64), 0, st,
                       (const T *)V, n, d, sets, l, k, pl.nkb, (typename M::vec_t *)tiles, bias, vec_ok);
    return hipGetLastError();
}

hipError_t launch_pack(int prec, const MfmaPlan &pl, const void *V, int64_t n, int d, const int32_t *sets,
                       int64_t l, int64_t k, void *tiles, float *bias, hipStream_t st) {
    switch (prec) {
    case P_FP32:
        return pl.tile == 32 ? pack_t<float, 32>(pl, V, n, d, sets, l, k, tiles, bias, st)
                             : pack_t<float, 16>(pl, V, n, d, sets, l, k, tiles, bias, st);
    case P_FP16: return pack_t<_Float16, 32>(pl, V, n, d, sets, l, k, tiles, bias, st);
    case P_BF16: return pack_t<__bf16, 32>(pl, V, n, d, sets, l, k, tiles, bias, st);
    }
    return hipErrorInvalidValue;
}

template <typename T, int TILE, int KBMAX, int RT, int MODE>
static hipError_t mfma_t(const MfmaPlan &pl, const void *V, int64_t n, int d, const void *tiles, const float *bias,
                         int64_t k, int64_t ngroups, int64_t gpc, const float *m0, float *partials, int64_t lpad,
                         float *rowmax, hipStream_t st) {
    using M = Mfma<T, TILE>;
    constexpr int WAVES = 4;
    auto kern = eval_mfma_kernel<T, TILE, KBMAX, RT, WAVES, MODE>;
    const size_t lds = 2 * (size_t)pl.nkb * 64 * 16 + 2 * WAVES * TILE * sizeof(float);
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    const int64_t G = (n + pl.rows - 1) / pl.rows;
    const int64_t chunks = (ngroups + gpc - 1) / gpc;
    const bool vec_ok = ((uintptr_t)V % 16 == 0) && ((d * (int64_t)sizeof(T)) % 16 == 0);
    hipLaunchKernelGGL(kern, dim3((unsigned)G, (unsigned)chunks), dim3(WAVES * 64), lds, st, (const T *)V, n, d,
                       pl.nks, pl.nkb, (const typename M::vec_t *)tiles, bias, k, ngroups, gpc, m0, partials, lpad,
                       rowmax, vec_ok);
    return hipGetLastError();
}

template <typename T, int TILE, int MODE>
static hipError_t mfma_dispatch_kb(const MfmaPlan &pl, const void *V, int64_t n, int d, const void *tiles,
                                   const float *bias, int64_t k, int64_t ngroups, int64_t gpc, const float *m0,
                                   float *partials, int64_t lpad, float *rowmax, hipStream_t st) {
#define EXEMCL_KB(KB, RT)                                                                                         \
    case KB:                                                                                                      \
        return mfma_t<T, TILE, KB, RT, MODE>(pl, V, n, d, tiles, bias, k, ngroups, gpc, m0, partials, lpad, rowmax, \
                                             st);
    if constexpr (TILE == 16) {
        switch (pl.kbmax) { EXEMCL_KB(32, 1) }
    } else {
        switch (pl.kbmax) {
            EXEMCL_KB(1, 2)
            EXEMCL_KB(2, 2)
            EXEMCL_KB(4, 2)
            EXEMCL_KB(8, 2)
            EXEMCL_KB(16, 2)
            EXEMCL_KB(32, 1)
        }
    }
#undef EXEMCL_KB
    return hipErrorInvalidValue;
}

hipError_t launch_mfma(int prec, int mode, const MfmaPlan &pl, const void *V, int64_t n, int d, const void *tiles,
                       const float *bias, int64_t k, int64_t ngroups, int64_t gpc, const float *m0, float *partials,
                       int64_t lpad, float *rowmax, hipStream_t st) {
    if (mode == MODE_ROWMAX) {
        if (prec != P_FP32) return hipErrorInvalidValue;
        return pl.tile == 32 ? mfma_dispatch_kb<float, 32, MODE_ROWMAX>(pl, V, n, d, tiles, bias, k, ngroups, gpc,
                                                                         m0, partials, lpad, rowmax, st)
                             : mfma_dispatch_kb<float, 16, MODE_ROWMAX>(pl, V, n, d, tiles, bias, k, ngroups, gpc,
                                                                         m0, partials, lpad, rowmax, st);
    }
    switch (prec) {
    case P_FP32:
        return pl.tile == 32 ? mfma_dispatch_kb<float, 32, MODE_SUM>(pl, V, n, d, tiles, bias, k, ngroups, gpc, m0,
                                                                      partials, lpad, rowmax, st)
                             : mfma_dispatch_kb<float, 16, MODE_SUM>(pl, V, n, d, tiles, bias, k, ngroups, gpc, m0,
                                                                      partials, lpad, rowmax, st);
    case P_FP16:
        return mfma_dispatch_kb<_Float16, 32, MODE_SUM>(pl, V, n, d, tiles, bias, k, ngroups, gpc, m0, partials, lpad,
                                                        rowmax, st);
    case P_BF16:
        return mfma_dispatch_kb<__bf16, 32, MODE_SUM>(pl, V, n, d, tiles, bias, k, ngroups, gpc, m0, partials, lpad,
                                                      rowmax, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
