// device.hpp -- gfx950 building blocks shared by the library's kernels.
//
// The evaluation is a contraction of the ground points (rows) against the
// exemplar vectors (columns): acc(v, s) = <v, s> over the d coordinates.
// On CDNA4 that contraction runs on the matrix cores (MFMA).  Everything here
// describes how one 64-lane wavefront holds operands and results of one MFMA
// instruction, and how V rows are loaded into that layout.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace exemcl {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Element conversion to fp32 (exact for all three storage types).
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(_Float16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }

// Set members per staged tile for the 16x16x32 shape (see Mfma<_Float16, 16>).
#ifndef EXEMCL_NB16
#define EXEMCL_NB16 2
#endif

// One MFMA shape, seen from one lane.
//
//   TM      output tile is TM x TM (rows = ground points, columns = exemplars)
//   GROUPS  64 / TM lane groups; lane L holds A row / output column L % TM and
//           belongs to K-group L / TM
//   VEC     storage elements per 16-byte lane vector
//   KS_PER_KB  instructions fed by one 16-byte lane vector (a "k-block")
//   KB_DIMS    coordinates covered by one k-block across the wavefront
//   ACC     fp32 accumulators per lane
//   NB      set members per staged tile: NB groups of TM exemplar columns
//           (member q*NB + h of the same TM sets in column group h), so the
//           minimum over a set's members is also taken across the groups
//
// Coordinate of lane-vector element e, for a lane in K-group `grp`, inside
// k-block kb: dim(kb, grp, e) = kb*KB_DIMS + grp*VEC + e, so every lane
// vector is VEC consecutive coordinates of one row (one 16-byte load).  A
// (rows) and B (exemplars) use the same map, so each instruction pairs
// matching coordinates; which K slot of the instruction a coordinate lands
// in only changes the summation order.
template <typename T, int TILE>
struct Mfma;

// fp32: v_mfma_f32_32x32x2_f32.  Element e of the lane vector feeds
// instruction e of the k-block, which covers coordinates kb*8 + {e, 4 + e}.
template <>
struct Mfma<float, 32> {
    static constexpr int TM = 32, GROUPS = 2, VEC = 4;
    static constexpr int KS_PER_KB = 4, KB_DIMS = 8, ACC = 16, NB = 1;
    using acc_t = f32x16;
    using vec_t = f32x4;
    using elem_t = float;
    static constexpr bool HAS_HALF = false;  // no half k-block
    using hvec_t = vec_t;
    __device__ __forceinline__ static int dim(int kb, int grp, int e) { return kb * KB_DIMS + grp * VEC + e; }
    __device__ __forceinline__ static acc_t mma(vec_t a, vec_t b, int e, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], c, 0, 0, 0);
    }
};

// fp32: v_mfma_f32_16x16x4_f32 (16 rows per tile: half the A registers of the
// 32x32 shape per row, used for large d).  Instruction e covers coordinates
// kb*16 + {e, 4 + e, 8 + e, 12 + e}.
template <>
struct Mfma<float, 16> {
    static constexpr int TM = 16, GROUPS = 4, VEC = 4;
    static constexpr int KS_PER_KB = 4, KB_DIMS = 16, ACC = 4, NB = 1;
    using acc_t = f32x4;
    using vec_t = f32x4;
    using elem_t = float;
    static constexpr bool HAS_HALF = false;  // no half k-block
    using hvec_t = vec_t;
    __device__ __forceinline__ static int dim(int kb, int grp, int e) { return kb * KB_DIMS + grp * VEC + e; }
    __device__ __forceinline__ static acc_t mma(vec_t a, vec_t b, int e, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
    }
};

// fp16: v_mfma_f32_32x32x16_f16 (gfx950).  One lane vector = the 8 K
// elements of one instruction.
template <>
struct Mfma<_Float16, 32> {
    static constexpr int TM = 32, GROUPS = 2, VEC = 8;
    static constexpr int KS_PER_KB = 1, KB_DIMS = 16, ACC = 16, NB = 1;
    using acc_t = f32x16;
    using vec_t = f16x8;
    using elem_t = _Float16;
    static constexpr bool HAS_HALF = false;  // no half k-block
    using hvec_t = vec_t;
    __device__ __forceinline__ static int dim(int kb, int grp, int e) { return kb * KB_DIMS + grp * VEC + e; }
    __device__ __forceinline__ static acc_t mma(vec_t a, vec_t b, int, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
};

// bf16: v_mfma_f32_32x32x16_bf16 (gfx950), same layout as fp16.
template <>
struct Mfma<__bf16, 32> {
    static constexpr int TM = 32, GROUPS = 2, VEC = 8;
    static constexpr int KS_PER_KB = 1, KB_DIMS = 16, ACC = 16, NB = 1;
    using acc_t = f32x16;
    using vec_t = bf16x8;
    using elem_t = __bf16;
    static constexpr bool HAS_HALF = false;  // no half k-block
    using hvec_t = vec_t;
    __device__ __forceinline__ static int dim(int kb, int grp, int e) { return kb * KB_DIMS + grp * VEC + e; }
    __device__ __forceinline__ static acc_t mma(vec_t a, vec_t b, int, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

// fp16: v_mfma_f32_16x16x32_f16 (gfx950), 16 rows per tile, 32 coordinates
// per instruction: lane L holds row / column L % 16 and coordinates
// kb*32 + (L/16)*8 + {0..7}.  On random data this shape sustains a markedly
// higher rate than the 32x32x16 one (the matrix cores draw less power per
// flop, so the clock stays higher), so it serves every d above one 16-wide
// k-block.  A staged tile holds two members of 16 sets (NB = 2): each A
// fragment feeds two instructions, and a tile carries twice the work of a
// single-member one for the same per-tile bookkeeping.
template <>
struct Mfma<_Float16, 16> {
    static constexpr int TM = 16, GROUPS = 4, VEC = 8;
    static constexpr int KS_PER_KB = 1, KB_DIMS = 32, ACC = 4, NB = EXEMCL_NB16;
    using acc_t = f32x4;
    using vec_t = f16x8;
    using elem_t = _Float16;
    __device__ __forceinline__ static int dim(int kb, int grp, int e) { return kb * KB_DIMS + grp * VEC + e; }
    __device__ __forceinline__ static acc_t mma(vec_t a, vec_t b, int, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    // Half k-block (16 coordinates, v_mfma_f32_16x16x16_f16): lane L holds
    // coordinates kb*32 + (L/16)*4 + {0..3} as an 8-byte vector.
    static constexpr bool HAS_HALF = true;
    static constexpr int HVEC = 4;
    using hvec_t = f16x4;
    __device__ __forceinline__ static int hdim(int kb, int grp, int e) { return kb * KB_DIMS + grp * HVEC + e; }
    __device__ __forceinline__ static acc_t mma_half(hvec_t a, hvec_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
    }
};

// bf16: v_mfma_f32_16x16x32_bf16 (gfx950), same layout as fp16.
template <>
struct Mfma<__bf16, 16> {
    static constexpr int TM = 16, GROUPS = 4, VEC = 8;
    static constexpr int KS_PER_KB = 1, KB_DIMS = 32, ACC = 4, NB = EXEMCL_NB16;
    using acc_t = f32x4;
    using vec_t = bf16x8;
    using elem_t = __bf16;
    __device__ __forceinline__ static int dim(int kb, int grp, int e) { return kb * KB_DIMS + grp * VEC + e; }
    __device__ __forceinline__ static acc_t mma(vec_t a, vec_t b, int, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    // Half k-block (v_mfma_f32_16x16x16_bf16), same layout as fp16.
    static constexpr bool HAS_HALF = true;
    static constexpr int HVEC = 4;
    using hvec_t = bf16x4;
    __device__ __forceinline__ static int hdim(int kb, int grp, int e) { return kb * KB_DIMS + grp * HVEC + e; }
    __device__ __forceinline__ static acc_t mma_half(hvec_t a, hvec_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a), __builtin_bit_cast(i16x4, b), c, 0,
                                                         0, 0);
    }
};

// Output layout of the TM x TM fp32 result: accumulator i of a lane in
// K-group grp holds row (i/4)*4*GROUPS + 4*grp + i%4 of the tile, column
// lane % TM.
template <int TM>
__device__ __forceinline__ int out_row(int i, int grp) {
    constexpr int GROUPS = 64 / TM;
    return (i >> 2) * (4 * GROUPS) + 4 * grp + (i & 3);
}

// Lane vector of row `r` for k-block kb in MFMA operand order, for rows of
// `ld` elements that are whole 16-byte lane vectors (16-byte aligned, ld a
// multiple of VEC, zero past the data's own d).  Rows >= n and vectors past
// ld read as zero: lanevec_raw loads from a clamped, always in-bounds
// address and lanevec_keep applies lanevec_live, so there is no divergent
// branch.
template <typename M, typename T>
__device__ __forceinline__ typename M::vec_t lanevec_raw(const T *__restrict__ V, int64_t n, int ld, int64_t r,
                                                         int kb, int grp) {
    const int d0 = M::dim(kb, grp, 0);
    const bool live = r < n && d0 < ld;
    return *reinterpret_cast<const typename M::vec_t *>(V + (live ? r : 0) * (int64_t)ld + (live ? d0 : 0));
}

template <typename M>
__device__ __forceinline__ bool lanevec_live(int64_t n, int ld, int64_t r, int kb, int grp) {
    return r < n && M::dim(kb, grp, 0) < ld;
}

template <typename M>
__device__ __forceinline__ typename M::vec_t lanevec_keep(typename M::vec_t v, bool live) {
    typename M::vec_t z;
    for (int e = 0; e < M::VEC; ++e) z[e] = live ? v[e] : (typename M::elem_t)0.0f;
    return z;
}

// Buffer resource over `bytes` bytes at `base`: raw buffer loads through it
// return zero past the end instead of touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t window_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// 16-byte load at byte offset `off` of a window; an offset at or past the
// window's end (kDeadOffset) reads as zeros.
constexpr uint32_t kDeadOffset = 0x80000000u;
template <typename vec_t>
__device__ __forceinline__ vec_t window_load16(__amdgpu_buffer_rsrc_t rsrc, uint32_t off) {
    return __builtin_bit_cast(vec_t, __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)off, 0, 0));
}

template <typename hvec_t>
__device__ __forceinline__ hvec_t window_load8(__amdgpu_buffer_rsrc_t rsrc, uint32_t off) {
    return __builtin_bit_cast(hvec_t, __builtin_amdgcn_raw_buffer_load_b64(rsrc, (int)off, 0, 0));
}

__device__ __forceinline__ float window_load4(__amdgpu_buffer_rsrc_t rsrc, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, (int)off, 0, 0));
}

}  // namespace exemcl
