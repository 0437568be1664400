// mfma_kernels.hpp -- exemplar staging and the matrix-core evaluation kernel
// (templates; instantiated per storage type in kernels_mfma_*.hip).
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
// is e0's contribution (Eq. (4)).  For every (row block, wavefront, set) a
// partial sum is written; a second pass adds the partials in a fixed order.
//
// Data layout.  A workgroup owns WAVES*RT*TM consecutive ground points and
// keeps them in registers in MFMA A-operand order for its whole life.
// Exemplars are streamed: for every (group of TM sets, member p) a "tile"
// holds the p-th member of each of the TM sets, already in B-operand order,
// plus one fp32 bias -||s||^2/2 per column.  Tiles stream through a ring of
// LDS stage buffers.  Each lane's output column is one set, so the minimum
// over a set's members is a per-register running max across successive tiles
// -- no cross-lane traffic until the set group ends.
//
// The number of k-blocks NKB is a compile-time bucket (d is zero-padded up to
// it), so every MFMA chain is straight-line code: a runtime bound on the
// k-loop would split the chain into basic blocks, and the accumulators would
// be copied out of and back into the matrix-core registers at every split.
#pragma once

#include <atomic>
#include <float.h>
#include <stdlib.h>

#include <hip/hip_ext.h>

#include "device.hpp"
#include "internal.h"

namespace exemcl {

// 32-column tiles (fp32 32x32x2, fp16/bf16 32x32x16) of at most
// EXEMCL_SPLAT_MAX_NKB k-blocks seed their accumulators with the bias by one
// bf16 MFMA (see eval_mfma_kernel); their header holds each column's bias as
// three bf16 parts.
#ifndef EXEMCL_SPLAT_MFMA
#define EXEMCL_SPLAT_MFMA 1
#endif
#ifndef EXEMCL_SPLAT_MAX_NKB
#define EXEMCL_SPLAT_MAX_NKB 4
#endif
#ifndef EXEMCL_SPLAT_F32
#define EXEMCL_SPLAT_F32 1
#endif
constexpr bool splat_bias(int elem_bytes, int tile, int nkb) {
    return EXEMCL_SPLAT_MFMA && (elem_bytes == 2 || EXEMCL_SPLAT_F32) && tile == 32 && nkb <= EXEMCL_SPLAT_MAX_NKB;
}

// fp32 32x32x2 tiles whose last k-block holds r <= 4 coordinates pair them
// per instruction: in that k-block element e of lane group g holds
// coordinate 2e + g, so instruction e covers coordinates 2e and 2e + 1 and
// ceil(r / 2) instructions cover it (the contiguous layout, e and 4 + e per
// instruction, needs all 4 once r > 2).  With a single k-block (d <= 8)
// every row is read one coordinate at a time, so V needs no 16-byte
// alignment or padding.  A kernel uses the paired last block when it has
// one k-block or fewer than 4 instructions in the last one.
#ifndef EXEMCL_IL
#define EXEMCL_IL 1
#endif
constexpr bool il_layout(int elem_bytes, int tile, int nkb, int nks_last) {
    return EXEMCL_IL && elem_bytes == 4 && tile == 32 && (nkb == 1 || nks_last < 4);
}
__device__ __forceinline__ int il_dim(int grp, int e) { return 2 * e + grp; }

// Largest finite bf16 (0x7F7F).
constexpr float kBf16Max = 3.38953139e38f;

// Tile header: the TM * NB fp32 biases of a tile's columns, padded to a
// multiple of 128 bytes; with `splat` (NB = 1), column c's bias as bf16
// (hi, mid, lo, 0) at byte 8c, 256 bytes.
constexpr int hdr_bytes(int tm, int nb, bool splat = false) {
    return splat ? (tm * 8 + 127) / 128 * 128 : (tm * nb * 4 + 127) / 128 * 128;
}

// Bytes of a staged tile: header, NFF whole fragments of 1 KiB and, when the
// last k-block is a half one, NB half fragments of 512 bytes.
constexpr int tile_bytes_of(int hdr, int nff, int nhalf) { return hdr + nff * 1024 + nhalf * 512; }

// ---------------------------------------------------------------------------
// Staging: gather exemplar rows by index into tiles, with their norms.
//
// A set group (TM consecutive sets) spans kt = ceil(k / NB) tiles; tile
// t = g*kt + q holds members q*NB .. q*NB+NB-1 of the sets g*TM .. g*TM+TM-1,
// member q*NB + h in column group h.  Byte layout of one tile
// (HDR + nkb * NB * 1024 bytes):
//   [0, HDR)                         TM*NB fp32 biases -||s||^2/2, column
//                                    c of group h at index h*TM + c (with
//                                    `splat`: column c's bias as bf16
//                                    hi, mid, lo, 0 at byte 8c, where
//                                    hi + mid + lo equals the fp32 bias)
//   [HDR + (kb*NB + h)*1024 + 16*L)  lane L's 16-byte B-operand vector for
//                                    k-block kb of column group h
// Padding columns (set >= l), members past k, empty slots and invalid
// indices become zero vectors with bias -FLT_MAX, which never wins the
// running max.  Rows are ld elements, zero past the data's d.  One wavefront
// per tile; ||s||^2 is summed from the lane vectors (fp32, k-blocks then
// elements in order, then the K-groups of the column with a fixed xor tree).
// ---------------------------------------------------------------------------
template <typename T, int TILE>
__global__ __launch_bounds__(64) void pack_tiles_kernel(const T *__restrict__ V, int64_t n, int ld,
                                                        const int32_t *__restrict__ sets, int64_t l,
                                                        int64_t k, int nkb, int half, int splat, int il,
                                                        unsigned char *__restrict__ tiles) {
    using M = Mfma<T, TILE>;
    constexpr int NB = M::NB;
    const int64_t kt = (k + NB - 1) / NB;
    const int64_t t = blockIdx.x;
    const int64_t g = t / kt, q = t - (t / kt) * kt;
    const int lane = threadIdx.x;
    const int col = lane % M::TM, grp = lane / M::TM;
    const int64_t j = g * M::TM + col;
    const int HDR = hdr_bytes(M::TM, NB, splat != 0);
    const int nfull = nkb - half;  // whole k-blocks; a half one follows when half = 1
    unsigned char *tile = tiles + t * (int64_t)tile_bytes_of(HDR, nfull * NB, half * NB);
    typename M::vec_t *dst = reinterpret_cast<typename M::vec_t *>(tile + HDR);
    // Member indices of every column group first, from addresses clamped
    // into the set matrix (l, k >= 1 whenever this kernel runs), so their
    // loads overlap.
    int32_t raw[NB];
#pragma unroll
    for (int h = 0; h < NB; ++h) {
        const int64_t p = q * NB + h;
        raw[h] = sets[(j < l ? j : l - 1) * k + (p < k ? p : k - 1)];
    }
#pragma unroll
    for (int h = 0; h < NB; ++h) {
        const int64_t p = q * NB + h;
        const int64_t idx = (j < l && p < k) ? (int64_t)raw[h] : -1;
        const bool valid = idx >= 0 && idx < n;
        const int64_t r = valid ? idx : n;  // row n reads as zeros
        float sq = 0.0f;
        // Up to KBATCH k-blocks are loaded before any is stored, so the loads
        // overlap (indices past the last block re-read it and are not
        // stored); ||s||^2 still runs over k-blocks and elements in order.
        // A paired last k-block (fp32) follows the others.
        const bool paired = sizeof(T) == 4 && il;
        const int nreg = paired ? nfull - 1 : nfull;
        constexpr int KBATCH = 8;
        for (int kb0 = 0; kb0 < nreg; kb0 += KBATCH) {
            typename M::vec_t vb[KBATCH];
#pragma unroll
            for (int u = 0; u < KBATCH; ++u) {
                const int kb = kb0 + u < nreg ? kb0 + u : nreg - 1;
                vb[u] = lanevec_raw<M>(V, n, ld, r, kb, grp);
            }
#pragma unroll
            for (int u = 0; u < KBATCH; ++u) {
                const int kb = kb0 + u;
                if (kb < nreg) {
                    const typename M::vec_t v = lanevec_keep<M>(vb[u], lanevec_live<M>(n, ld, r, kb, grp));
                    dst[(kb * NB + h) * 64 + lane] = v;
#pragma unroll
                    for (int e = 0; e < M::VEC; ++e) {
                        const float x = to_f32(v[e]);
                        sq = fmaf(x, x, sq);
                    }
                }
            }
        }
        if (paired) {
            // last k-block: coordinate kb*8 + 2e + grp, read one at a time
            // (single-block rows may be unpadded)
            const int kb = nfull - 1;
            typename M::vec_t v;
#pragma unroll
            for (int e = 0; e < M::VEC; ++e) {
                const int c = kb * M::KB_DIMS + il_dim(grp, e);
                v[e] = (r < n && c < ld) ? V[r * (int64_t)ld + c] : (typename M::elem_t)0.0f;
            }
            dst[(kb * NB + h) * 64 + lane] = v;
#pragma unroll
            for (int e = 0; e < M::VEC; ++e) {
                const float x = to_f32(v[e]);
                sq = fmaf(x, x, sq);
            }
        }
        if constexpr (M::HAS_HALF) {
            if (half) {
                // Half fragment h: lane L's 8 bytes = coordinates
                // nfull*32 + (L/TM)*4 + {0..3}, after all whole fragments.
                using hvec_t = typename M::hvec_t;
                const int d0 = M::hdim(nfull, grp, 0);
                const bool live = r < n && d0 < ld;  // ld and d0 are multiples of 4: all 4 in the row
                hvec_t v = *reinterpret_cast<const hvec_t *>(V + (live ? r : 0) * (int64_t)ld + (live ? d0 : 0));
#pragma unroll
                for (int e = 0; e < M::HVEC; ++e) v[e] = live ? v[e] : (typename M::elem_t)0.0f;
                reinterpret_cast<hvec_t *>(tile + HDR + nfull * NB * 1024)[h * 64 + lane] = v;
#pragma unroll
                for (int e = 0; e < M::HVEC; ++e) {
                    const float x = to_f32(v[e]);
                    sq = fmaf(x, x, sq);
                }
            }
        }
#pragma unroll
        for (int off = M::TM; off < 64; off <<= 1) sq += __shfl_xor(sq, off);
        const float b = valid ? -0.5f * sq : -FLT_MAX;
        if (grp == 0) {
            if (splat) {
                // Exact three-way split: hi is b rounded to bf16, mid the
                // rest rounded again, lo what is left (8 bits at most), so
                // hi + mid + lo == b.  Clamped to a finite value first, so a
                // zero operand times any part is 0.
                const float bc = fmaxf(b, -kBf16Max);
                const __bf16 hi = (__bf16)bc;
                const float r1 = bc - (float)hi;
                const __bf16 mid = (__bf16)r1;
                const __bf16 lo = (__bf16)(r1 - (float)mid);
                bf16x4 hv;
                hv[0] = hi;
                hv[1] = mid;
                hv[2] = lo;
                hv[3] = (__bf16)0.0f;
                reinterpret_cast<bf16x4 *>(tile)[col] = hv;
            } else {
                reinterpret_cast<float *>(tile)[h * M::TM + col] = b;
            }
        }
    }
}

// Stage geometry, fixed at compile time per k-block bucket.  Workgroups of
// EXEMCL_SMALL_WAVES wavefronts serve tiles of at most EXEMCL_BIG_NKB
// k-blocks, EXEMCL_BIG_WAVES above.  Small tiles are batched into stages of
// at least EXEMCL_STAGE_MIN bytes; large tiles go EXEMCL_TPS_BIG per stage.
// A stage is rounded up to one 16-byte load per thread, at most two stages
// share the 160 KiB of LDS, and the ring has up to EXEMCL_RING_SMALL /
// EXEMCL_RING_BIG buffers.  Fewer, larger stages mean fewer barriers.  Inside
// a tile, up to EXEMCL_PF B fragments are read from LDS ahead of their use.
#ifndef EXEMCL_PF
#define EXEMCL_PF 3
#endif
#ifndef EXEMCL_PF_SCHED
#define EXEMCL_PF_SCHED 4
#endif
#ifndef EXEMCL_PF_BIG3
#define EXEMCL_PF_BIG3 2
#endif
#ifndef EXEMCL_PERSIST_DEFAULT
#define EXEMCL_PERSIST_DEFAULT 1
#endif
#ifndef EXEMCL_SCHED_MIN_NF
#define EXEMCL_SCHED_MIN_NF 16
#endif
#ifndef EXEMCL_SCHED16
#define EXEMCL_SCHED16 1
#endif
// Tiles of at least EXEMCL_FENCE_MIN_NF fragments (and fewer than
// EXEMCL_SCHED_MIN_NF) keep their in-tile reads ahead of use with the same
// scheduling fences, without reads across tiles.
#ifndef EXEMCL_FENCE_MIN_NF
#define EXEMCL_FENCE_MIN_NF 4
#endif
#ifndef EXEMCL_SCHED32
#define EXEMCL_SCHED32 0
#endif
#ifndef EXEMCL_PAIR
#define EXEMCL_PAIR 1
#endif
#ifndef EXEMCL_RT1_NKB32
#define EXEMCL_RT1_NKB32 0
#endif
#ifndef EXEMCL_PAIR_NKB32
#define EXEMCL_PAIR_NKB32 8
#endif
#ifndef EXEMCL_PAIR_NKB16
#define EXEMCL_PAIR_NKB16 4
#endif
#ifndef EXEMCL_SMALL_WAVES
#define EXEMCL_SMALL_WAVES 4
#endif
#ifndef EXEMCL_BIG_WAVES
#define EXEMCL_BIG_WAVES 8
#endif
// fp16/bf16 32x32x16 tiles (d <= 16): every tile's bias splat is one MFMA
// shared by the wavefront's row tiles, a third of the matrix-core time with
// 2 row tiles and a fifth with 4 (about 240 VGPRs: two wavefronts per SIMD).
#ifndef EXEMCL_RT16_SMALL
#define EXEMCL_RT16_SMALL 4
#endif
#ifndef EXEMCL_RT16_MID
#define EXEMCL_RT16_MID 2
#endif
#ifndef EXEMCL_RT16_BIG
#define EXEMCL_RT16_BIG 1
#endif
#ifndef EXEMCL_RT16X16_NKB
#define EXEMCL_RT16X16_NKB 8
#endif
#ifndef EXEMCL_RT16X16_SMALL
#define EXEMCL_RT16X16_SMALL 4
#endif
#ifndef EXEMCL_RT16X16_BIG
#define EXEMCL_RT16X16_BIG 2
#endif
#ifndef EXEMCL_WAVES16_BIG
#define EXEMCL_WAVES16_BIG EXEMCL_BIG_WAVES
#endif
#ifndef EXEMCL_BIG_NKB
#define EXEMCL_BIG_NKB 8
#endif
#ifndef EXEMCL_STAGE_MIN
#define EXEMCL_STAGE_MIN 24576
#endif
#ifndef EXEMCL_TPS_BIG
#define EXEMCL_TPS_BIG 4
#endif
#ifndef EXEMCL_RING_SMALL
#define EXEMCL_RING_SMALL 2
#endif
#ifndef EXEMCL_RING_BIG
#define EXEMCL_RING_BIG 3
#endif
#ifndef EXEMCL_TPS_FILL_MAX
#define EXEMCL_TPS_FILL_MAX 8
#endif
// fp16/bf16 two-member tiles of at least EXEMCL_WIDE16_MIN_NKB k-blocks run
// as one 8-wavefront workgroup per CU (their registers allow two wavefronts
// per SIMD either way): the CU's eight wavefronts share each staged tile and
// advance together, and the persistent launch gives every CU equal work.
#ifndef EXEMCL_WIDE16_MIN_NKB
#define EXEMCL_WIDE16_MIN_NKB 4
#endif
#ifndef EXEMCL_WIDE16_WAVES
#define EXEMCL_WIDE16_WAVES 8
#endif
// Up to 8 k-blocks these plans take as many row tiles per wavefront as fit
// EXEMCL_WIDE16_A_BLOCKS A fragments (4 VGPRs each: 160 of the 256), at most
// EXEMCL_RT_WIDE16_MAX: every B fragment read from LDS then feeds 5-6 MFMAs.
// Their cross-tile reads keep EXEMCL_PF_WIDE16 fragments in flight, which
// leaves the registers for the fifth row tile.
#ifndef EXEMCL_WIDE16_A_BLOCKS
#define EXEMCL_WIDE16_A_BLOCKS 40
#endif
#ifndef EXEMCL_RT_WIDE16_MAX
#define EXEMCL_RT_WIDE16_MAX 6
#endif
#ifndef EXEMCL_PF_WIDE16
#define EXEMCL_PF_WIDE16 2
#endif
// Shorter two-member tiles (EXEMCL_W12_MIN_NKB .. EXEMCL_WIDE16_MIN_NKB - 1
// k-blocks) fit three wavefronts per SIMD: one 12-wavefront workgroup per CU.
#ifndef EXEMCL_W12_MIN_NKB
#define EXEMCL_W12_MIN_NKB 2
#endif
// ... and tiles of at most EXEMCL_W16_MAX_NKB k-blocks four per SIMD: one
// 16-wavefront workgroup per CU.
#ifndef EXEMCL_W16_MAX_NKB
#define EXEMCL_W16_MAX_NKB 1
#endif

constexpr int kLdsBytes = 160 * 1024;

template <int NKB, int WAVES>
constexpr int round_stage(int bytes) {
    return (bytes + WAVES * 1024 - 1) / (WAVES * 1024) * (WAVES * 1024);
}

// LDS one workgroup's ring may use: workgroups of at most 4 wavefronts (one
// per SIMD) leave room for a second workgroup on the CU, so that each SIMD
// can interleave two wavefronts.
template <int WAVES>
constexpr int lds_budget() {
    return WAVES <= 4 ? kLdsBytes / 2 : kLdsBytes;
}

// One-workgroup-per-CU plans (8 or more wavefronts, two members per tile:
// FILL below) add their wavefronts' partial sums in LDS at each set group's
// end and store one partial-sum row per workgroup; the host sizes the
// partial sums with the same rule.  kWgSumLds bytes of LDS are kept for it.
constexpr bool wg_sum(int waves, int nb) { return waves >= 8 && nb == 2; }
constexpr int kWgSumLds = 4096;

// Stage geometry for tiles of TB bytes and NFRAG B fragments.  FILL (8
// wavefronts, two-member tiles: one workgroup per CU in lockstep) takes as
// many tiles per stage as two stages fit in the LDS, since the cost of a
// stage is its barrier, which every wavefront of the CU waits at.
// EVEN (fp16/bf16 tiles of one member, folded in pairs): an even number of
// tiles per stage, rounded up while two stages fit, so that a set group of
// even k never leaves a lone tile at a stage's end (fp32 d = 2 ran 5 %
// slower with it, fp16 d = 16 2.8 % faster).
template <int TB, int NFRAG, int WAVES, bool FILL = false, bool EVEN = false>
constexpr int tiles_per_stage() {
    int tps = FILL ? EXEMCL_TPS_FILL_MAX
                   : NFRAG <= EXEMCL_BIG_NKB ? (EXEMCL_STAGE_MIN / TB > 1 ? EXEMCL_STAGE_MIN / TB : 1) : EXEMCL_TPS_BIG;
    constexpr int budget = FILL ? kLdsBytes - kWgSumLds : lds_budget<WAVES>();
    if (EVEN && (tps & 1)) tps = 2 * round_stage<NFRAG, WAVES>((tps + 1) * TB) <= budget ? tps + 1 : tps > 1 ? tps - 1 : tps;
    while (tps > 1 && 2 * round_stage<NFRAG, WAVES>(tps * TB) > budget) tps -= (EVEN && tps > 2) ? 2 : 1;
    return tps;
}

template <int TB, int NFRAG, int WAVES, bool FILL = false, bool EVEN = false>
constexpr int stage_bytes() {
    return round_stage<NFRAG, WAVES>(tiles_per_stage<TB, NFRAG, WAVES, FILL, EVEN>() * TB);
}

template <int TB, int NFRAG, int WAVES, bool FILL = false, bool EVEN = false>
constexpr int ring_depth() {
    constexpr int want = FILL ? 2 : NFRAG <= EXEMCL_BIG_NKB ? EXEMCL_RING_SMALL : EXEMCL_RING_BIG;
    constexpr int sb = stage_bytes<TB, NFRAG, WAVES, FILL, EVEN>();
    constexpr int fit = (sb * 2 <= lds_budget<WAVES>() ? lds_budget<WAVES>() : kLdsBytes) / sb;
    return want < fit ? want : fit;
}

// Prefetch depth for reads that run across tiles: the largest divisor of
// nkb not above `want`; when that is 1, all nkb fragments of a short tile.
constexpr int prefetch_depth(int nkb, int want) {
    int best = 1;
    for (int p = 2; p <= want && p <= nkb; ++p)
        if (nkb % p == 0) best = p;
    return (best == 1 && nkb <= 2 * want + 1) ? nkb : best;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ---------------------------------------------------------------------------
// Evaluation kernel.
//
// grid.x = row blocks of WAVES*RT*TM consecutive points, grid.y = chunks of
// gpc set groups (or, PERSIST, one workgroup per resident slot walking
// several (row block, set group range) segments).  Wavefront w owns RT row
// tiles of TM points, held in registers for the whole segment.
//
// The chunk's tiles are one contiguous byte range in global memory, streamed
// into a ring of NBUF LDS stage buffers of SB bytes (TPS whole tiles each) by
// direct global->LDS loads (global_load_lds_dwordx4).  Every thread issues
// exactly CNT 16-byte loads per stage, so "stage s has landed while the next
// NBUF-2 stages are in flight" is vmcnt(CNT*(NBUF-2)).  One barrier per stage
// both publishes stage s and frees the buffer of stage s-1 for stage
// s+NBUF-1.
//
// NKS_LAST = MFMA instructions fed by the last k-block (fp32 packs KS_PER_KB
// instructions per k-block; tiny d uses fewer, see il_layout).
//
// Per tile: the accumulators start at the column's bias (a splat, or one
// bf16 MFMA for SPLAT tiles), the MFMA chain adds <v, s>, and the running max
// per (point, set) folds the tile in (pairs of tiles with one max3 where a
// tile holds one member).  At a set group's end the running max is summed
// and set back to its initial value.
//
// MODE_SUM: each wavefront writes its partial sum per set,
//   partials[(rb * WAVES + w) * lpad + j] = sum over its rows of
//   max(m0(v), max_p h_{s_jp}(v)),
// in a fixed order (its registers, then the K-groups of the MFMA layout).
// MODE_ROWMAX: rowmax[v] = max(m0(v), 0, max over all staged columns of
// h_s(v)) (m0 = 0 when null); rowmax must not alias m0.
// ---------------------------------------------------------------------------
template <typename T, int TILE, int NKB, int NKS_LAST, int RT, int WAVES, int MODE, bool HAS_M0, bool HALF,
          bool PERSIST>
__global__ __launch_bounds__(WAVES * 64, PERSIST ? 2 : 1) void eval_mfma_kernel(const T *__restrict__ V, int64_t n, int ld,
                                                                 const unsigned char *__restrict__ tiles, int64_t kt,
                                                                 int64_t ngroups, int64_t gpc, int64_t nrb,
                                                                 const float *__restrict__ m0,
                                                                 float *__restrict__ partials, int64_t lpad,
                                                                 float *__restrict__ rowmax) {
    using M = Mfma<T, TILE>;
    using vec_t = typename M::vec_t;
    using acc_t = typename M::acc_t;
    constexpr int TM = M::TM;
    constexpr int NB = M::NB;     // column groups (set members) per tile
    constexpr int NF = NKB * NB;  // B fragments per tile, fragment f = kb * NB + h
    // With HALF the last k-block holds 16 coordinates: its NB half fragments
    // (512 bytes each) follow the NFF whole ones and bypass the prefetch ring.
    constexpr int NFF = HALF ? (NKB - 1) * NB : NF;
    constexpr int NT = WAVES * 64;
    // On short 32-column tiles the 16-register bias splat that seeds each
    // tile's accumulators is a large share of the VALU work (fp16/bf16: the
    // busiest unit; fp32: its MFMA does not overlap VALU work).  There
    // (SPLAT) the header holds every column's bias as three bf16 parts and
    // one bf16 MFMA of a ones operand (coordinates 0-2 of the lanes of
    // K-group 0, zero elsewhere) against them builds the splat exactly on
    // the matrix cores, in the 32x32 accumulator layout all these shapes
    // share; the VALU only folds.
    constexpr bool SPLAT = splat_bias((int)sizeof(T), TILE, NKB);
    constexpr bool IL = il_layout((int)sizeof(T), TILE, NKB, NKS_LAST);
    constexpr int NBIAS = SPLAT ? 2 : NB;  // bias registers per tile (SPLAT: the 8 header bytes)
    constexpr int HDR = hdr_bytes(TM, NB, SPLAT);
    constexpr int TB = tile_bytes_of(HDR, NFF, HALF ? NB : 0);
    constexpr bool FILL = wg_sum(WAVES, NB);
    constexpr int SB = stage_bytes<TB, NF, WAVES, FILL, NB == 1 && sizeof(T) == 2>();
    constexpr int TPS = tiles_per_stage<TB, NF, WAVES, FILL, NB == 1 && sizeof(T) == 2>();
    constexpr int CNT = SB / (NT * 16);
    constexpr int NBUF = ring_depth<TB, NF, WAVES, FILL, NB == 1 && sizeof(T) == 2>();
    // Wavefront partial sums added in LDS per set group (wg_sum): two
    // buffers of WAVES x TM floats after the stage ring, by group parity.
    constexpr bool WGSUM = FILL && MODE == MODE_SUM;
    static_assert(!WGSUM || 2 * WAVES * TM * 4 <= kWgSumLds, "partial-sum buffers");
    static_assert(!FILL || NBUF * SB + kWgSumLds <= kLdsBytes, "LDS");
    static_assert(!HALF || (M::HAS_HALF && NKB >= 2), "half k-block needs the 16x16x16 instruction and a whole block");
    // Reads across tiles pay off for long tiles; short ones keep the registers
    // for a third wavefront per SIMD instead.
    constexpr bool SCHED = (sizeof(T) == 4 ? EXEMCL_SCHED32 : EXEMCL_SCHED16) && NF >= EXEMCL_SCHED_MIN_NF && !HALF;
    // B fragments in flight ahead of use.  When the reads run across tiles
    // (SCHED) the ring of PF slots must wrap exactly at a tile's end, so PF
    // divides NF; the next tile then finds fragment i in slot i.
    constexpr int PF = SCHED ? prefetch_depth(NF, FILL && NKB <= EXEMCL_RT16X16_NKB ? EXEMCL_PF_WIDE16
                                                  : FILL && RT >= 3                   ? EXEMCL_PF_BIG3
                                                                                      : EXEMCL_PF_SCHED)
                             : (NFF < EXEMCL_PF ? NFF : EXEMCL_PF);
    static_assert(!SCHED || NF % PF == 0, "cross-tile prefetch ring must wrap at the tile end");
    static_assert(!SPLAT || (!SCHED && NB == 1 && !HALF), "splat tiles");
    static_assert(MODE == MODE_SUM || NB == 1, "the row-max mode stages one member per tile");
    // Pairs of tiles per fold (not for HAS_M0: the scoring of S u {c} has
    // single-member sets, where every tile is a set group of its own).
    constexpr bool PAIR = EXEMCL_PAIR && NB == 1 && !HAS_M0 &&
                          NKB <= (sizeof(T) == 4 ? EXEMCL_PAIR_NKB32 : EXEMCL_PAIR_NKB16);
    static_assert(TPS >= 1 && TPS * TB <= SB && NBUF >= 2 && NBUF * SB <= kLdsBytes, "stage geometry");
    static_assert(CNT * (NBUF - 2) < 64, "vmcnt range");
    static_assert(NKS_LAST >= 1 && NKS_LAST <= M::KS_PER_KB, "k-steps of the last block");

    extern __shared__ __align__(16) unsigned char smem[];

    // Units of work are (row block, set group) pairs.  A workgroup takes
    // either one row block and one chunk of gpc groups (grid = row blocks x
    // chunks), or -- persistent launch (PERSIST), one workgroup per resident
    // slot, S of them -- first the whole row blocks w, w + S, w + 2S, ...
    // (q = nrb / S of them: all workgroups walk the set groups in step, so the
    // exemplar tiles stay hot in L2), then an equal contiguous share of the
    // units of the remaining nrb - q*S row blocks (row block major), walked as
    // segments of one row block each.
    // One segment: row block rb, set groups [g0, g1).
    auto segment = [&](const int64_t rb, const int64_t g0, const int64_t g1) {
    // Per-lane offsets do not change from one segment to the next; hiding
    // the thread index and ld per segment keeps the compiler from hoisting
    // them (RT*NKB load offsets among them) out of the persistent loop,
    // where they would hold registers through every MFMA chain.
    int tid = threadIdx.x, ldv = ld;
    if constexpr (PERSIST) asm volatile("" : "+v"(tid), "+s"(ldv));
    // The wavefront index is uniform: held in a scalar register, so the LDS
    // destination of every stage copy is scalar arithmetic (M0) too.
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane % TM, grp = lane / TM;
    const int64_t row0 = rb * (int64_t)(WAVES * RT * TM) + (int64_t)wave * RT * TM;

    const int64_t ntiles = (g1 - g0) * kt;
    const int64_t nstages = (ntiles + TPS - 1) / TPS;
    const unsigned char *chunk = tiles + g0 * kt * (int64_t)TB;
    const int64_t chunk_bytes = ntiles * (int64_t)TB;

    // Queue the direct-to-LDS copy of stage s (CNT 16-byte loads per thread).
    auto issue = [&](int64_t s) {
        unsigned char *buf = smem + (int)(s % NBUF) * SB;
        const int64_t base = s * (int64_t)(TPS * TB);
        // A window over this stage's bytes: loads past the chunk end read zeros.
        const auto win = window_rsrc(chunk + base, (uint32_t)min((int64_t)(TPS * TB), chunk_bytes - base));
#pragma unroll
        for (int r = 0; r < CNT; ++r)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                win, (__attribute__((address_space(3))) void *)(buf + (r * NT + wave * 64) * 16), 16,
                (r * NT + tid) * 16, 0, 0, 0);
    };

    if (nstages > 0) {
#pragma unroll
        for (int s = 0; s < NBUF - 1; ++s)
            if (s < nstages) issue(s);
    }

    // Ground points of this wavefront, in A-operand order, resident for the
    // whole kernel (zero past d and past n).
    constexpr int NKF = HALF ? NKB - 1 : NKB;  // whole k-blocks
    using hvec_t = typename M::hvec_t;
    vec_t a[RT][NKF];
    hvec_t ah[HALF ? RT : 1];  // the half k-block's 8-byte lane vectors
    // The workgroup's rows as one buffer window (at most 1 536 rows of at
    // most 1 024 elements, so 32-bit offsets): rows past n read as zeros, and
    // so do vectors past ld, without a branch.
    const int64_t wrow0 = rb * (int64_t)(WAVES * RT * TM);
    const int64_t wrows = min((int64_t)(WAVES * RT * TM), n - wrow0);
    const auto vwin = window_rsrc(V + wrow0 * (int64_t)ld, (uint32_t)(wrows * ld * (int64_t)sizeof(T)));
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int lrow = wave * RT * TM + rt * TM + lr;
#pragma unroll
        for (int kb = 0; kb < NKF; ++kb) {
            if (IL && kb == NKF - 1) {
#pragma unroll
                for (int e = 0; e < M::VEC; ++e) {
                    const int c = kb * M::KB_DIMS + il_dim(grp, e);
                    a[rt][kb][e] = window_load4(vwin, c < ldv ? (uint32_t)((lrow * ldv + c) * 4) : kDeadOffset);
                }
            } else {
                const int d0 = M::dim(kb, grp, 0);
                a[rt][kb] =
                    window_load16<vec_t>(vwin, d0 < ldv ? (uint32_t)((lrow * ldv + d0) * (int)sizeof(T)) : kDeadOffset);
            }
        }
        if constexpr (HALF) {
            const int d0 = M::hdim(NKF, grp, 0);  // ld and d0 are multiples of 4: the 4 elements are in the row
            ah[rt] = window_load8<hvec_t>(vwin, d0 < ldv ? (uint32_t)((lrow * ldv + d0) * (int)sizeof(T)) : kDeadOffset);
        }
    }

    // Initial value of the running max for each output element: e0's 0, or
    // (HAS_M0) the per-point cached value when scoring S u {c}.
    float minit[HAS_M0 ? RT : 1][HAS_M0 ? M::ACC : 1];
    if constexpr (HAS_M0) {
        const auto mwin = window_rsrc(m0 + wrow0, (uint32_t)(wrows * 4));
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i)
                minit[rt][i] = window_load4(mwin, (uint32_t)((wave * RT * TM + rt * TM + out_row<TM>(i, grp)) * 4));
    }
    auto m_init = [&](int rt, int i) -> float {
        if constexpr (HAS_M0) return minit[rt][i];
        else return 0.0f;
    };
    float m[RT][M::ACC];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int i = 0; i < M::ACC; ++i) m[rt][i] = m_init(rt, i);

    // One tile: each column group's bias enters as its accumulators' initial
    // value (fp32), then the branch-free MFMA chain over the NKB k-blocks.
    // B fragments are software-pipelined: bq holds the next PF fragments in
    // use order, and each use reads the fragment PF positions ahead -- past
    // the end of this tile that is the start of `tnext` (the following tile
    // of the same stage, or this tile again for the last one: a harmless
    // re-read), whose biases are read with its first fragment.  With SCHED
    // the compiler may not move instructions across k-block boundaries, so
    // the reads stay ahead of their use instead of being sunk next to it;
    // without it every tile starts its own reads (no reads across tiles).
    constexpr bool FENCE = SCHED || (NF >= EXEMCL_FENCE_MIN_NF && sizeof(T) == 2);
    auto fence = [&]() {
        if constexpr (FENCE) __builtin_amdgcn_sched_barrier(0);
    };
    auto head = [&](const unsigned char *tb, vec_t (&bq)[PF], float (&bias)[NBIAS]) {
        const vec_t *B = reinterpret_cast<const vec_t *>(tb + HDR);
#pragma unroll
        for (int i = 0; i < PF; ++i) bq[i] = B[i * 64 + lane];
        if constexpr (SPLAT) {
            // every lane reads its column's parts; K-group 1 multiplies them by 0
            bias[0] = reinterpret_cast<const float *>(tb)[2 * lr];
            bias[1] = reinterpret_cast<const float *>(tb)[2 * lr + 1];
        } else {
#pragma unroll
            for (int h = 0; h < NB; ++h) bias[h] = reinterpret_cast<const float *>(tb)[h * TM + lr];
        }
    };
    // The ones operand of the splat MFMA: bf16 1.0 in elements 0-2 of the
    // K-group 0 lanes.
    u32x4 ones_w = {0u, 0u, 0u, 0u};
    if (SPLAT && grp == 0) {
        ones_w[0] = 0x3F803F80u;
        ones_w[1] = 0x00003F80u;
    }
    const bf16x8 ones = __builtin_bit_cast(bf16x8, ones_w);
    auto chain = [&](const unsigned char *tb, const unsigned char *tnext, vec_t (&bq)[PF], float (&bias)[NBIAS],
                     acc_t (&acc)[RT][NB], bool read_head = true) {
        if (!SCHED && read_head) head(tb, bq, bias);
        const vec_t *B = reinterpret_cast<const vec_t *>(tb + HDR);
        const vec_t *Bn = reinterpret_cast<const vec_t *>(tnext + HDR);
        if constexpr (SPLAT) {
            u32x4 w = {__builtin_bit_cast(uint32_t, bias[0]), __builtin_bit_cast(uint32_t, bias[1]), 0u, 0u};
            const acc_t seed = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ones, __builtin_bit_cast(bf16x8, w), acc_t{},
                                                                       0, 0, 0);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc[rt][0] = seed;
        } else {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int h = 0; h < NB; ++h)
#pragma unroll
                    for (int i = 0; i < M::ACC; ++i) acc[rt][h][i] = bias[h];
        }
        float bias_next[NB];
#pragma unroll
        for (int h = 0; h < NB; ++h) bias_next[h] = 0.0f;
#pragma unroll
        for (int kb = 0; kb < NKF; ++kb) {
            vec_t bv[NB];
#pragma unroll
            for (int h = 0; h < NB; ++h) {
                const int f = kb * NB + h;
                bv[h] = bq[f % PF];
                const int ahead = f + PF;
                if (ahead < NFF) {
                    bq[f % PF] = B[ahead * 64 + lane];
                } else if constexpr (SCHED) {
                    bq[f % PF] = Bn[(ahead - NF) * 64 + lane];
                    if (ahead == NF) {
#pragma unroll
                        for (int hh = 0; hh < NB; ++hh)
                            bias_next[hh] = reinterpret_cast<const float *>(tnext)[hh * TM + lr];
                    }
                }
            }
            fence();
#pragma unroll
            for (int e = 0; e < M::KS_PER_KB; ++e) {
                if (kb < NKB - 1 || e < NKS_LAST) {
#pragma unroll
                    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                        for (int h = 0; h < NB; ++h) acc[rt][h] = M::mma(a[rt][kb], bv[h], e, acc[rt][h]);
                }
            }
            fence();
        }
        if constexpr (HALF) {
            const hvec_t *Bh = reinterpret_cast<const hvec_t *>(tb + HDR + NFF * 1024);
            hvec_t bh[NB];
#pragma unroll
            for (int h = 0; h < NB; ++h) bh[h] = Bh[h * 64 + lane];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int h = 0; h < NB; ++h) acc[rt][h] = M::mma_half(ah[rt], bh[h], acc[rt][h]);
        }
        if constexpr (SCHED) {
#pragma unroll
            for (int h = 0; h < NB; ++h) bias[h] = bias_next[h];
        }
    };
    // m = max(m, every column group of x), in place: with NB = 2 one max3
    // per element.  After each set group's sum the running max goes back to
    // its initial value (MODE_SUM; MODE_ROWMAX keeps one running max over
    // everything staged).
    auto fold = [&](const acc_t (&x)[RT][NB]) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i) {
                float v = m[rt][i];
#pragma unroll
                for (int h = 0; h < NB; ++h) v = fmaxf(v, x[rt][h][i]);
                m[rt][i] = v;
            }
    };
    // Two single-member tiles of the same set group (NB = 1): one max3.
    auto fold2 = [&](const acc_t (&x)[RT][NB], const acc_t (&y)[RT][NB]) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i) m[rt][i] = fmaxf(fmaxf(m[rt][i], x[rt][0][i]), y[rt][0][i]);
    };
    // Sum of this lane's running maxima in a fixed pairwise order: each level
    // adds the upper ceil(n/2) values to the lower ones (for a power of two,
    // halves).
    auto lane_sum = [&]() {
        constexpr int NV = RT * M::ACC;
        float v[NV];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < M::ACC; ++i) v[rt * M::ACC + i] = m[rt][i];
#pragma unroll
        for (int n = NV; n > 1; n = (n + 1) / 2) {
            const int h = (n + 1) / 2;
#pragma unroll
            for (int i = 0; i + h < n; ++i) v[i] += v[i + h];
        }
        return v[0];
    };

    // Set-group and member counters fit 32 bits (ngroups * TM <= lpad, a
    // partial-sum row of fp32 values); keeping them 32-bit keeps them in
    // scalar registers.
    const int ktile = (int)kt;
    float *wpart = partials + (WGSUM ? rb : rb * WAVES + wave) * lpad;
    int g = (int)g0;
    int p = 0;
    const int nst = (int)nstages;
    // Close set group g after its last tile has been folded: sum this lane's
    // rows for its column, then the K-groups holding the other rows of the
    // same column; store, and start group g + 1.
    auto group_end = [&]() {
        if constexpr (MODE == MODE_SUM) {
            float sum = lane_sum();
#pragma unroll
            for (int off = TM; off < 64; off <<= 1) sum += __shfl_xor(sum, off);
            if constexpr (WGSUM) {
                // every wavefront of the workgroup ends group g here: add
                // their sums in wavefront order and store one row (the next
                // group's barrier separates reuse of a parity's buffer)
                float *red = reinterpret_cast<float *>(smem + NBUF * SB) + (g & 1) * (WAVES * TM);
                if (grp == 0) red[wave * TM + lr] = sum;
                __syncthreads();
                if (wave == 0 && grp == 0) {
                    float t = red[lr];
#pragma unroll
                    for (int w = 1; w < WAVES; ++w) t += red[w * TM + lr];
                    wpart[(int64_t)g * TM + lr] = t;
                }
            } else {
                if (grp == 0) wpart[(int64_t)g * TM + lr] = sum;
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < M::ACC; ++i) m[rt][i] = m_init(rt, i);
        }
        ++g;
    };
    for (int s = 0; s < nst; ++s) {
        if (s + NBUF - 2 < nst) wait_vmcnt<CNT * (NBUF - 2)>();
        else wait_vmcnt<0>();
        __syncthreads();

        const unsigned char *buf = smem + (s % NBUF) * SB;
        const int tn = (int)min((int64_t)TPS, ntiles - (int64_t)s * TPS);
        auto tile_at = [&](int i) { return buf + (i < tn ? i : tn - 1) * TB; };
        vec_t bq[PF];
        float bias[NBIAS];
#pragma unroll
        for (int h = 0; h < NBIAS; ++h) bias[h] = 0.0f;
        // The stage's first fragments are read before the next stage's copy
        // is queued, so their LDS latency overlaps the copy's issue.
        if constexpr (SCHED) head(buf, bq, bias);
        if (s + NBUF - 1 < nst) issue(s + NBUF - 1);
        if constexpr (PAIR && NKB == 1) {
            // Tiles of one k-block hold a few MFMAs each: the operands of the
            // next pair are read from LDS while this pair is folded (a
            // scheduling barrier keeps the reads there), instead of right
            // before their use.  Otherwise as below.
            vec_t bqa[PF], bqb[PF];
            float ba[NBIAS], bbb[NBIAS];
            int tt = 0;
            head(tile_at(0), bqa, ba);
            head(tile_at(1), bqb, bbb);
            while (tt < tn) {
                while (tt + 1 < tn && p + 1 < ktile) {
                    acc_t x[RT][NB], y[RT][NB];
                    chain(tile_at(tt), tile_at(tt + 1), bqa, ba, x, false);
                    chain(tile_at(tt + 1), tile_at(tt + 2), bqb, bbb, y, false);
                    head(tile_at(tt + 2), bqa, ba);
                    head(tile_at(tt + 3), bqb, bbb);
                    __builtin_amdgcn_sched_barrier(0);
                    fold2(x, y);
                    tt += 2;
                    p += 2;
                    if (p == ktile) {
                        group_end();
                        p = 0;
                    }
                }
                if (tt < tn) {
                    acc_t x[RT][NB];
                    chain(tile_at(tt), tile_at(tt + 1), bqa, ba, x, false);
                    fold(x);
                    tt += 1;
                    if (++p == ktile) {
                        group_end();
                        p = 0;
                    }
                    head(tile_at(tt), bqa, ba);
                    head(tile_at(tt + 1), bqb, bbb);
                }
            }
        } else if constexpr (PAIR) {
            // Pairs of members of the same set group in an inner loop with
            // one fold site, so the running max stays in one set of
            // registers (with a pair site and a single site in one loop the
            // compiler copies it back every iteration); a lone member (odd k,
            // stage end) is folded outside that loop.
            int tt = 0;
            while (tt < tn) {
                while (tt + 1 < tn && p + 1 < ktile) {
                    acc_t x[RT][NB], y[RT][NB];
                    chain(tile_at(tt), tile_at(tt + 1), bq, bias, x);
                    chain(tile_at(tt + 1), tile_at(tt + 2), bq, bias, y);
                    fold2(x, y);
                    tt += 2;
                    p += 2;
                    if (p == ktile) {
                        group_end();
                        p = 0;
                    }
                }
                if (tt < tn) {
                    acc_t x[RT][NB];
                    chain(tile_at(tt), tile_at(tt + 1), bq, bias, x);
                    fold(x);
                    tt += 1;
                    if (++p == ktile) {
                        group_end();
                        p = 0;
                    }
                }
            }
        } else {
            for (int tt = 0; tt < tn; ++tt) {
                acc_t x[RT][NB];
                chain(tile_at(tt), tile_at(tt + 1), bq, bias, x);
                fold(x);
                if (++p == ktile) {
                    group_end();
                    p = 0;
                }
            }
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
    };

    if constexpr (!PERSIST) {
        const int64_t g0 = (int64_t)blockIdx.y * gpc;
        segment((int64_t)blockIdx.x, g0, min(ngroups, g0 + gpc));
    } else {
        const int64_t S = gridDim.x;
        const int64_t q = nrb / S;
        const int64_t U2 = (nrb - q * S) * ngroups;
        int64_t v = (int64_t)blockIdx.x * U2 / S;
        const int64_t v1 = ((int64_t)blockIdx.x + 1) * U2 / S;
        for (int64_t seg = 0;; ++seg) {
            int64_t rb, g0, g1;
            if (seg < q) {
                rb = seg * S + (int64_t)blockIdx.x;
                g0 = 0;
                g1 = ngroups;
            } else {
                if (v >= v1) break;
                rb = q * S + v / ngroups;
                g0 = v - (v / ngroups) * ngroups;
                g1 = min(ngroups, g0 + (v1 - v));
                v += g1 - g0;
            }
            // The previous segment's last stage may still be read by other waves.
            if (seg > 0) __syncthreads();
            segment(rb, g0, g1);
        }
    }
}

// ---------------------------------------------------------------------------
// Host-side launch helpers.
// ---------------------------------------------------------------------------
// Launch-mode switch, read on every launch so that tests can flip it:
// EXEMCL_PERSIST=0 never launches persistently, 2 always does (whenever the
// mode allows it, however few units there are), anything else (default) uses
// the rule in eval_launch_t.  0 and 2 exist for A/B runs and for tests that
// compare both launches bit for bit.
enum { kPersistOff = 0, kPersistAuto = 1, kPersistForce = 2 };
inline int persistent_mode() {
    const char *s = getenv("EXEMCL_PERSIST");
    if (s && s[0] == '0' && s[1] == '\0') return kPersistOff;
    if (s && s[0] == '2' && s[1] == '\0') return kPersistForce;
    return EXEMCL_PERSIST_DEFAULT ? kPersistAuto : kPersistOff;
}

// Compute units of the current device (cached per device index).
inline int64_t device_cu_count() {
    static std::atomic<int> cus[64];  // 0 = not queried yet
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int c = cus[dev].load(std::memory_order_relaxed);
    if (c == 0) {
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cus[dev].store(c, std::memory_order_relaxed);
    }
    return c;
}
template <typename T, int TILE>
hipError_t pack_launch(const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets, int64_t l,
                       int64_t k, void *tiles, hipStream_t st) {
    if (pl.half && !Mfma<T, TILE>::HAS_HALF) return hipErrorInvalidValue;
    if ((pl.splat != 0) != splat_bias((int)sizeof(T), TILE, pl.nkb)) return hipErrorInvalidValue;
    if ((pl.il != 0) != il_layout((int)sizeof(T), TILE, pl.nkb, pl.nks_last)) return hipErrorInvalidValue;
    if (l < 1 || k < 1) return hipErrorInvalidValue;  // the kernel reads sets[0] at least
    const int64_t ngroups = (l + TILE - 1) / TILE;
    const int64_t kt = (k + Mfma<T, TILE>::NB - 1) / Mfma<T, TILE>::NB;
    hipLaunchKernelGGL((pack_tiles_kernel<T, TILE>), dim3((unsigned)(ngroups * kt)), dim3(64), 0, st,
                       (const T *)V, n, ld, sets, l, k, pl.nkb, pl.half, pl.splat, pl.il, (unsigned char *)tiles);
    return hipGetLastError();
}

template <typename T, int TILE, int NKB, int NKS_LAST, int RT, int WAVES, int MODE, bool HAS_M0, bool HALF>
hipError_t eval_launch_t(const MfmaArgs &x, hipStream_t st) {
    constexpr int NB = Mfma<T, TILE>::NB;
    constexpr int NF = NKB * NB;
    constexpr int TB = tile_bytes_of(hdr_bytes(TILE, NB, splat_bias((int)sizeof(T), TILE, NKB)),
                                     HALF ? (NKB - 1) * NB : NF, HALF ? NB : 0);
    constexpr bool FILL = wg_sum(WAVES, NB);
    constexpr int SB = stage_bytes<TB, NF, WAVES, FILL, NB == 1 && sizeof(T) == 2>();
    constexpr int NBUF = ring_depth<TB, NF, WAVES, FILL, NB == 1 && sizeof(T) == 2>();
    auto kern = eval_mfma_kernel<T, TILE, NKB, NKS_LAST, RT, WAVES, MODE, HAS_M0, HALF, false>;
    auto kernp = eval_mfma_kernel<T, TILE, NKB, NKS_LAST, RT, WAVES, MODE, HAS_M0, HALF, MODE == MODE_SUM>;
    const size_t lds = (size_t)NBUF * SB + (FILL && MODE == MODE_SUM ? kWgSumLds : 0);
    if (lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e == hipSuccess && MODE == MODE_SUM)
            e = hipFuncSetAttribute((const void *)kernp, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    const int64_t rows = (int64_t)WAVES * RT * TILE;
    const int64_t G = (x.n + rows - 1) / rows;
    const int64_t chunks = (x.ngroups + x.gpc - 1) / x.gpc;
    // Persistent launch: as many workgroups as are resident at once, each
    // with an equal share of the units (whole row blocks in step first), so
    // no partly filled last round.  Not for the row-max mode, whose
    // workgroup must see every group of its row block.  The rule: at least 8
    // units per slot (fewer cannot be balanced better than the grid does),
    // and one workgroup per CU for both variants -- with one workgroup per
    // CU a CU whose workgroup ends early in the plain grid's last round
    // idles, while with two a single remaining 4-wavefront workgroup still
    // keeps every SIMD's matrix core nearly busy, and the plain grid then
    // measures as fast or faster.
    int64_t slots = 0;
    bool use_persist = false;
    const int pmode = MODE == MODE_SUM ? persistent_mode() : kPersistOff;
    if (pmode != kPersistOff) {
        // Per instantiation: blocks per CU of the persistent and the plain
        // variant; -1 = not queried yet.  The occupancy does not change.
        static std::atomic<int> occ_p{-1}, occ_q{-1};
        int np = occ_p.load(std::memory_order_relaxed), nq = occ_q.load(std::memory_order_relaxed);
        if (np < 0 || nq < 0) {
            if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&np, (const void *)kernp, WAVES * 64, lds) != hipSuccess ||
                hipOccupancyMaxActiveBlocksPerMultiprocessor(&nq, (const void *)kern, WAVES * 64, lds) != hipSuccess) {
                (void)hipGetLastError();
                np = nq = 0;
            }
            occ_p.store(np, std::memory_order_relaxed);
            occ_q.store(nq, std::memory_order_relaxed);
        }
        slots = (int64_t)np * device_cu_count();
        if (pmode == kPersistForce) use_persist = slots > 0;
        else use_persist = slots > 0 && np == 1 && nq == 1 && G * x.ngroups >= 8 * slots;
    }
    if (use_persist) {
        hipExtLaunchKernelGGL(kernp, dim3((unsigned)slots, 1), dim3(WAVES * 64), lds, st, x.ev_start, x.ev_stop, 0,
                              (const T *)x.V, x.n, x.ld, (const unsigned char *)x.tiles, x.kt, x.ngroups, x.gpc, G,
                              x.m0, x.partials, x.lpad, x.rowmax);
    } else {
        hipExtLaunchKernelGGL(kern, dim3((unsigned)G, (unsigned)chunks), dim3(WAVES * 64), lds, st, x.ev_start,
                              x.ev_stop, 0, (const T *)x.V, x.n, x.ld, (const unsigned char *)x.tiles, x.kt,
                              x.ngroups, x.gpc, G, x.m0, x.partials, x.lpad, x.rowmax);
    }
    return hipGetLastError();
}

template <typename T, int TILE, int NKB, int NKS_LAST, int RT, int WAVES, int MODE, bool HALF = false>
hipError_t eval_launch(const MfmaArgs &x, hipStream_t st) {
    if constexpr (sizeof(T) == 4) {
        if (x.m0) return eval_launch_t<T, TILE, NKB, NKS_LAST, RT, WAVES, MODE, true, HALF>(x, st);
    }
    return eval_launch_t<T, TILE, NKB, NKS_LAST, RT, WAVES, MODE, false, HALF>(x, st);
}

constexpr int wide16_rt(int nkb) {
    return EXEMCL_WIDE16_A_BLOCKS / nkb < EXEMCL_RT_WIDE16_MAX ? EXEMCL_WIDE16_A_BLOCKS / nkb : EXEMCL_RT_WIDE16_MAX;
}

// The 12-wavefront plans (168 VGPRs) take EXEMCL_W12_A_BLOCKS A fragments,
// at least EXEMCL_RT16X16_SMALL and at most EXEMCL_RT_W12_MAX row tiles; the
// 16-wavefront one (128 VGPRs) EXEMCL_RT16X16_W16; above 256 coordinates up
// to EXEMCL_RT16X16_BIG3_NKB k-blocks take 3 row tiles (with EXEMCL_PF_BIG3
// fragments in flight, which leaves the registers for them), the rest 2.
#ifndef EXEMCL_W12_A_BLOCKS
#define EXEMCL_W12_A_BLOCKS 16
#endif
#ifndef EXEMCL_RT_W12_MAX
#define EXEMCL_RT_W12_MAX 6
#endif
#ifndef EXEMCL_RT16X16_W16
#define EXEMCL_RT16X16_W16 6
#endif
#ifndef EXEMCL_RT16X16_BIG3_NKB
#define EXEMCL_RT16X16_BIG3_NKB 14
#endif
constexpr int w12_rt(int nkb) {
    const int r = EXEMCL_W12_A_BLOCKS / nkb < EXEMCL_RT_W12_MAX ? EXEMCL_W12_A_BLOCKS / nkb : EXEMCL_RT_W12_MAX;
    return r > EXEMCL_RT16X16_SMALL ? r : EXEMCL_RT16X16_SMALL;
}

// Row tiles per wavefront and wavefronts per workgroup for a k-block bucket,
// as functions of (element bytes, tile, k-blocks) so that the host-side plan
// (mfma_plan) and the compiled instantiations follow one rule.
constexpr int plan_rt(int elem_bytes, int tile, int nkb) {
    if (tile == 16)
        return elem_bytes == 4            ? 1
               : (nkb >= EXEMCL_WIDE16_MIN_NKB && nkb <= EXEMCL_RT16X16_NKB) ? wide16_rt(nkb)
               : nkb <= EXEMCL_W16_MAX_NKB ? EXEMCL_RT16X16_W16
               : nkb <= EXEMCL_RT16X16_NKB ? w12_rt(nkb)
               : nkb <= EXEMCL_RT16X16_BIG3_NKB ? 3
               : nkb <= 16                 ? EXEMCL_RT16X16_BIG
                                           : 1;  // 512 < d <= 1024: one row tile of 32 k-blocks
    if (elem_bytes == 4) return nkb <= EXEMCL_RT1_NKB32 ? 1 : nkb <= 16 ? 2 : 1;
    return nkb <= EXEMCL_BIG_NKB ? EXEMCL_RT16_SMALL : nkb <= 16 ? EXEMCL_RT16_MID : EXEMCL_RT16_BIG;
}

constexpr int plan_waves(int elem_bytes, int tile, int nkb) {
    if (elem_bytes == 2 && tile == 16 && nkb >= EXEMCL_WIDE16_MIN_NKB && nkb <= EXEMCL_RT16X16_NKB) return EXEMCL_WIDE16_WAVES;
    if (elem_bytes == 2 && tile == 16 && nkb >= EXEMCL_WIDE16_MIN_NKB) return EXEMCL_BIG_WAVES;
    if (elem_bytes == 2 && tile == 16 && nkb >= EXEMCL_W12_MIN_NKB) return 12;
    if (elem_bytes == 2 && tile == 16 && nkb <= EXEMCL_W16_MAX_NKB) return 16;
    if (nkb <= EXEMCL_BIG_NKB) return EXEMCL_SMALL_WAVES;
    return (elem_bytes == 2 && tile == 32 && nkb > 16) ? EXEMCL_WAVES16_BIG : EXEMCL_BIG_WAVES;
}

template <typename T, int TILE, int NKB>
constexpr int rt_of() {
    return plan_rt((int)sizeof(T), TILE, NKB);
}

template <typename T, int TILE, int NKB>
constexpr int waves_of() {
    return plan_waves((int)sizeof(T), TILE, NKB);
}

// One storage type: pick the instantiation for the plan's k-block bucket.
// fp32 32x32x2 with more than one k-block and a paired last block of
// KSL (1 or 2) instructions.
template <typename T, int TILE, int MODE, int KSL>
hipError_t eval_dispatch_last(const MfmaPlan &pl, const MfmaArgs &x, hipStream_t st) {
    switch (pl.nkb) {
    case 2: return eval_launch<T, TILE, 2, KSL, rt_of<T, TILE, 2>(), waves_of<T, TILE, 2>(), MODE>(x, st);
    case 3: return eval_launch<T, TILE, 3, KSL, rt_of<T, TILE, 3>(), waves_of<T, TILE, 3>(), MODE>(x, st);
    case 4: return eval_launch<T, TILE, 4, KSL, rt_of<T, TILE, 4>(), waves_of<T, TILE, 4>(), MODE>(x, st);
    case 5: return eval_launch<T, TILE, 5, KSL, rt_of<T, TILE, 5>(), waves_of<T, TILE, 5>(), MODE>(x, st);
    case 6: return eval_launch<T, TILE, 6, KSL, rt_of<T, TILE, 6>(), waves_of<T, TILE, 6>(), MODE>(x, st);
    case 7: return eval_launch<T, TILE, 7, KSL, rt_of<T, TILE, 7>(), waves_of<T, TILE, 7>(), MODE>(x, st);
    case 8: return eval_launch<T, TILE, 8, KSL, rt_of<T, TILE, 8>(), waves_of<T, TILE, 8>(), MODE>(x, st);
    case 10: return eval_launch<T, TILE, 10, KSL, rt_of<T, TILE, 10>(), waves_of<T, TILE, 10>(), MODE>(x, st);
    case 12: return eval_launch<T, TILE, 12, KSL, rt_of<T, TILE, 12>(), waves_of<T, TILE, 12>(), MODE>(x, st);
    case 13: return eval_launch<T, TILE, 13, KSL, rt_of<T, TILE, 13>(), waves_of<T, TILE, 13>(), MODE>(x, st);
    case 14: return eval_launch<T, TILE, 14, KSL, rt_of<T, TILE, 14>(), waves_of<T, TILE, 14>(), MODE>(x, st);
    case 16: return eval_launch<T, TILE, 16, KSL, rt_of<T, TILE, 16>(), waves_of<T, TILE, 16>(), MODE>(x, st);
    case 20: return eval_launch<T, TILE, 20, KSL, rt_of<T, TILE, 20>(), waves_of<T, TILE, 20>(), MODE>(x, st);
    case 24: return eval_launch<T, TILE, 24, KSL, rt_of<T, TILE, 24>(), waves_of<T, TILE, 24>(), MODE>(x, st);
    case 28: return eval_launch<T, TILE, 28, KSL, rt_of<T, TILE, 28>(), waves_of<T, TILE, 28>(), MODE>(x, st);
    case 32: return eval_launch<T, TILE, 32, KSL, rt_of<T, TILE, 32>(), waves_of<T, TILE, 32>(), MODE>(x, st);
    }
    return hipErrorInvalidValue;
}

template <typename T, int TILE, int MODE>
hipError_t eval_dispatch(const MfmaPlan &pl, const MfmaArgs &x, hipStream_t st) {
    if constexpr (TILE == 16 && sizeof(T) == 4) {
        switch (pl.nkb) {
        case 20: return eval_launch<T, TILE, 20, 4, rt_of<T, TILE, 20>(), waves_of<T, TILE, 20>(), MODE>(x, st);
        case 24: return eval_launch<T, TILE, 24, 4, rt_of<T, TILE, 24>(), waves_of<T, TILE, 24>(), MODE>(x, st);
        case 28: return eval_launch<T, TILE, 28, 4, rt_of<T, TILE, 28>(), waves_of<T, TILE, 28>(), MODE>(x, st);
        case 32: return eval_launch<T, TILE, 32, 4, rt_of<T, TILE, 32>(), waves_of<T, TILE, 32>(), MODE>(x, st);
        }
    } else {
        constexpr int KL = Mfma<T, TILE>::KS_PER_KB;
        if constexpr (Mfma<T, TILE>::HAS_HALF) {
            if (pl.half) {
                // d mod 32 in (0, 16] up to the plan's limit: 2 .. 6 k-blocks.
                switch (pl.nkb) {
                case 2: return eval_launch<T, TILE, 2, KL, rt_of<T, TILE, 2>(), waves_of<T, TILE, 2>(), MODE, true>(x, st);
                case 3: return eval_launch<T, TILE, 3, KL, rt_of<T, TILE, 3>(), waves_of<T, TILE, 3>(), MODE, true>(x, st);
                case 4: return eval_launch<T, TILE, 4, KL, rt_of<T, TILE, 4>(), waves_of<T, TILE, 4>(), MODE, true>(x, st);
                case 5: return eval_launch<T, TILE, 5, KL, rt_of<T, TILE, 5>(), waves_of<T, TILE, 5>(), MODE, true>(x, st);
                case 6: return eval_launch<T, TILE, 6, KL, rt_of<T, TILE, 6>(), waves_of<T, TILE, 6>(), MODE, true>(x, st);
                }
                return hipErrorInvalidValue;
            }
        }
        if (pl.half) return hipErrorInvalidValue;
        if (pl.nkb == 1) {
            if constexpr (KL == 4) {
                switch (pl.nks_last) {
                case 1: return eval_launch<T, TILE, 1, 1, rt_of<T, TILE, 1>(), waves_of<T, TILE, 1>(), MODE>(x, st);
                case 2: return eval_launch<T, TILE, 1, 2, rt_of<T, TILE, 1>(), waves_of<T, TILE, 1>(), MODE>(x, st);
                case 3: return eval_launch<T, TILE, 1, 3, rt_of<T, TILE, 1>(), waves_of<T, TILE, 1>(), MODE>(x, st);
                case 4: return eval_launch<T, TILE, 1, 4, rt_of<T, TILE, 1>(), waves_of<T, TILE, 1>(), MODE>(x, st);
                }
                return hipErrorInvalidValue;
            } else {
                return eval_launch<T, TILE, 1, KL, rt_of<T, TILE, 1>(), waves_of<T, TILE, 1>(), MODE>(x, st);
            }
        }
        if constexpr (KL == 4 && TILE == 32) {
            // a last k-block of at most 4 coordinates, paired per instruction
            if (pl.nks_last == 1) return eval_dispatch_last<T, TILE, MODE, 1>(pl, x, st);
            if (pl.nks_last == 2) return eval_dispatch_last<T, TILE, MODE, 2>(pl, x, st);
        }
        if (pl.nks_last != KL) return hipErrorInvalidValue;
        switch (pl.nkb) {
        case 2: return eval_launch<T, TILE, 2, KL, rt_of<T, TILE, 2>(), waves_of<T, TILE, 2>(), MODE>(x, st);
        case 3: return eval_launch<T, TILE, 3, KL, rt_of<T, TILE, 3>(), waves_of<T, TILE, 3>(), MODE>(x, st);
        case 4: return eval_launch<T, TILE, 4, KL, rt_of<T, TILE, 4>(), waves_of<T, TILE, 4>(), MODE>(x, st);
        case 5: return eval_launch<T, TILE, 5, KL, rt_of<T, TILE, 5>(), waves_of<T, TILE, 5>(), MODE>(x, st);
        case 6: return eval_launch<T, TILE, 6, KL, rt_of<T, TILE, 6>(), waves_of<T, TILE, 6>(), MODE>(x, st);
        case 7: return eval_launch<T, TILE, 7, KL, rt_of<T, TILE, 7>(), waves_of<T, TILE, 7>(), MODE>(x, st);
        case 8: return eval_launch<T, TILE, 8, KL, rt_of<T, TILE, 8>(), waves_of<T, TILE, 8>(), MODE>(x, st);
        case 10: return eval_launch<T, TILE, 10, KL, rt_of<T, TILE, 10>(), waves_of<T, TILE, 10>(), MODE>(x, st);
        case 12: return eval_launch<T, TILE, 12, KL, rt_of<T, TILE, 12>(), waves_of<T, TILE, 12>(), MODE>(x, st);
        case 13: return eval_launch<T, TILE, 13, KL, rt_of<T, TILE, 13>(), waves_of<T, TILE, 13>(), MODE>(x, st);
        case 14: return eval_launch<T, TILE, 14, KL, rt_of<T, TILE, 14>(), waves_of<T, TILE, 14>(), MODE>(x, st);
        case 16: return eval_launch<T, TILE, 16, KL, rt_of<T, TILE, 16>(), waves_of<T, TILE, 16>(), MODE>(x, st);
        }
        // The 16x16x32 shape reaches d = 1024 with 32 k-blocks (one row
        // tile per wavefront); the 16- and 8-coordinate shapes reach 512.
        {
            switch (pl.nkb) {
            case 20: return eval_launch<T, TILE, 20, KL, rt_of<T, TILE, 20>(), waves_of<T, TILE, 20>(), MODE>(x, st);
            case 24: return eval_launch<T, TILE, 24, KL, rt_of<T, TILE, 24>(), waves_of<T, TILE, 24>(), MODE>(x, st);
            case 28: return eval_launch<T, TILE, 28, KL, rt_of<T, TILE, 28>(), waves_of<T, TILE, 28>(), MODE>(x, st);
            case 32: return eval_launch<T, TILE, 32, KL, rt_of<T, TILE, 32>(), waves_of<T, TILE, 32>(), MODE>(x, st);
            }
        }
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
