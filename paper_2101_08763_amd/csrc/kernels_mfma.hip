// kernels_mfma.hip -- MFMA path planning and dispatch by storage type.  The
// kernels themselves are in mfma_kernels.hpp, instantiated per storage type
// in kernels_mfma_{f32,f16,bf16}.hip.
#include <stdlib.h>

#include "internal.h"
#include "mfma_kernels.hpp"

// fp16/bf16 rows of at least EXEMCL_F16_WIDE_D coordinates use the 16x16x32
// shape, unless padding d to 32-coordinate k-blocks costs more than
// EXEMCL_F16_WIDE_PAD percent over 16-coordinate ones (d = 100 pads to 128
// instead of 112: the 32x32x16 shape is faster there).
#ifndef EXEMCL_F16_WIDE_D
#define EXEMCL_F16_WIDE_D 17
#endif
#ifndef EXEMCL_F16_WIDE_PAD
#define EXEMCL_F16_WIDE_PAD 8
#endif

namespace exemcl {

// k-block counts with a compiled kernel; d is zero-padded up to the next one.
static const int kBuckets[] = {1, 2, 3, 4, 5, 6, 7, 8, 10, 12, 13, 14, 16, 20, 24, 28, 32};

static int bucket(int nkb) {
    for (int b : kBuckets)
        if (b >= nkb) return b;
    return -1;
}

bool mfma_plan(int prec, int64_t d, MfmaPlan *p) {
    if (d < 1 || d > 512) return false;
    MfmaPlan q{};
    q.waves = 4;
    q.nb = 1;
    if (prec == P_FP32 && d <= 256) {
        // v_mfma_f32_32x32x2_f32, 8 coordinates per k-block
        q.tile = 32;
        q.kb_dims = 8;
        q.nkb = bucket((int)((d + 7) / 8));
        q.nks_last = q.nkb == 1 ? (int)(d < 4 ? d : 4) : 4;  // instruction e covers dims e and 4 + e
    } else if (prec == P_FP32) {
        // v_mfma_f32_16x16x4_f32, 16 coordinates per k-block
        q.tile = 16;
        q.kb_dims = 16;
        q.nkb = bucket((int)((d + 15) / 16));
        q.nks_last = 4;
    } else if (d >= EXEMCL_F16_WIDE_D && (d + 31) / 32 * 32 * 100 <= (d + 15) / 16 * 16 * (100 + EXEMCL_F16_WIDE_PAD)) {
        // v_mfma_f32_16x16x32_{f16,bf16}, 32 coordinates per k-block, two
        // set members per tile
        q.tile = 16;
        q.kb_dims = 32;
        q.nkb = bucket((int)((d + 31) / 32));
        q.nks_last = 1;
        q.nb = EXEMCL_NB16;
    } else {
        // v_mfma_f32_32x32x16_{f16,bf16}, 16 coordinates per k-block (one
        // k-block for d <= 16, where 32-coordinate blocks would be half padding)
        q.tile = 32;
        q.kb_dims = 16;
        q.nkb = bucket((int)((d + 15) / 16));
        q.nks_last = 1;
    }
    if (q.nkb < 1) return false;
    const int eb = prec == P_FP32 ? 4 : 2;
    q.rt = plan_rt(eb, q.tile, q.nkb);
    q.waves = plan_waves(eb, q.tile, q.nkb);
    q.rows = q.waves * q.rt * q.tile;
    *p = q;
    return true;
}

int64_t mfma_tile_bytes(const MfmaPlan &pl) { return hdr_bytes(pl.tile, pl.nb) + (int64_t)pl.nkb * pl.nb * 1024; }

int64_t mfma_tiles_per_group(const MfmaPlan &pl, int64_t k) { return (k + pl.nb - 1) / pl.nb; }

hipError_t launch_pack(int prec, const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets,
                       int64_t l, int64_t k, void *tiles, hipStream_t st) {
    switch (prec) {
    case P_FP32: return pack_run_f32(pl, V, n, ld, sets, l, k, tiles, st);
    case P_FP16: return pack_run_f16(pl, V, n, ld, sets, l, k, tiles, st);
    case P_BF16: return pack_run_bf16(pl, V, n, ld, sets, l, k, tiles, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_mfma(int prec, int mode, const MfmaPlan &pl, const void *V, int64_t n, int ld, const void *tiles,
                       int64_t kt, int64_t ngroups, int64_t gpc, const float *m0, float *partials, int64_t lpad,
                       float *rowmax, hipStream_t st) {
    const MfmaArgs x{V, n, ld, tiles, kt, ngroups, gpc, m0, partials, lpad, rowmax};
    switch (prec) {
    case P_FP32: return eval_run_f32(pl, mode, x, st);
    case P_FP16: return mode == MODE_SUM ? eval_run_f16(pl, mode, x, st) : hipErrorInvalidValue;
    case P_BF16: return mode == MODE_SUM ? eval_run_bf16(pl, mode, x, st) : hipErrorInvalidValue;
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
