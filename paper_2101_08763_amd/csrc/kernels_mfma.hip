// kernels_mfma.hip -- MFMA path planning and dispatch by storage type.  The
// kernels themselves are in mfma_kernels.hpp, instantiated per storage type
// in kernels_mfma_{f32,f16,bf16}.hip.
#include <stdlib.h>

#include "internal.h"
#include "mfma_kernels.hpp"

// fp16/bf16 rows of at least EXEMCL_F16_WIDE_D coordinates use the 16x16x32
// shape.  Up to EXEMCL_HALF_MAX_D coordinates a last k-block of 16 covers
// d mod 32 in (0, 16] (d = 100: 3 x 32 + 16 = 112 instead of 128); above it
// d pads to whole 32-coordinate blocks (at most 8 % more work) and long tiles
// keep their cross-tile prefetch, which a half block does not take part in.
#ifndef EXEMCL_F16_WIDE_D
#define EXEMCL_F16_WIDE_D 17
#endif
#ifndef EXEMCL_HALF_MAX_D
#define EXEMCL_HALF_MAX_D 192
#endif
#ifndef EXEMCL_MAIN_MAX_D16
#define EXEMCL_MAIN_MAX_D16 1024
#endif
#if EXEMCL_HALF_MAX_D > 192
#error "half k-blocks are compiled for 2 to 6 k-blocks (d <= 192)"
#endif

namespace exemcl {

// k-block counts with a compiled kernel; d is zero-padded up to the next one.
static const int kBuckets[] = {1, 2, 3, 4, 5, 6, 7, 8, 10, 12, 13, 14, 16, 20, 24, 28, 32};

static int bucket(int nkb) {
    for (int b : kBuckets)
        if (b >= nkb) return b;
    return -1;
}

// Largest d: the kernels address a block of rows through 32-bit byte
// offsets (32 rows of at most 2^24 fp32 coordinates).
constexpr int64_t kMaxD = int64_t(1) << 24;

bool mfma_plan(int prec, int64_t d, MfmaPlan *p) {
    if (d < 1 || d > kMaxD) return false;
    MfmaPlan q{};
    // fp16/bf16 up to d = 1024 stay on the register-resident kernel (one row
    // tile of 16 points and 32 k-blocks per wavefront); above that, and fp32
    // above 512, the coordinates are split over the wavefronts.
    const int64_t dmax_main = (prec == P_FP32) ? 512 : EXEMCL_MAIN_MAX_D16;
    if (d > dmax_main) {
        // Coordinates split over the 8 wavefronts of a workgroup sharing 32
        // points: 16x16x4 (fp32, 16 coordinates per k-block) or 16x16x32
        // (fp16/bf16, 32 per k-block, two members per tile); each wavefront
        // holds kw k-blocks per round, and d needs `rounds` rounds.
        q.bigd = 1;
        q.tile = 16;
        q.nb = prec == P_FP32 ? 1 : EXEMCL_NB16;
        q.kb_dims = prec == P_FP32 ? 16 : 32;
        q.nkb = (int)((d + q.kb_dims - 1) / q.kb_dims);
        q.nks_last = prec == P_FP32 ? 4 : 1;
        const int per = (q.nkb + 7) / 8;
        q.kw = per <= 2 ? 2 : per <= 4 ? 4 : 8;
        q.rounds = (q.nkb + 8 * q.kw - 1) / (8 * q.kw);
        q.rt = 2;
        q.waves = 8;
        q.rows = 32;
        *p = q;
        return true;
    }
    q.waves = 4;
    q.nb = 1;
    q.half = 0;
    q.splat = 0;
    q.il = 0;
    if (prec == P_FP32 && d <= 256) {
        // v_mfma_f32_32x32x2_f32, 8 coordinates per k-block
        q.tile = 32;
        q.kb_dims = 8;
        q.nkb = bucket((int)((d + 7) / 8));
        // instruction e covers dims e and 4 + e, or 2e and 2e + 1 in a
        // paired last k-block (il): one k-block, or an exact bucket whose
        // last block holds r <= 4 coordinates
        const int r = (int)(d - 8 * ((d + 7) / 8 - 1));  // coordinates in the last block, 1..8
        if (q.nkb == 1)
            q.nks_last = EXEMCL_IL ? (int)((d + 1) / 2) : (int)(d < 4 ? d : 4);
        else if (q.nkb == (d + 7) / 8 && r <= 4)
            q.nks_last = EXEMCL_IL ? (r + 1) / 2 : 4;
        else
            q.nks_last = 4;
        q.il = il_layout(4, 32, q.nkb, q.nks_last) ? 1 : 0;
    } else if (prec == P_FP32) {
        // v_mfma_f32_16x16x4_f32, 16 coordinates per k-block
        q.tile = 16;
        q.kb_dims = 16;
        q.nkb = bucket((int)((d + 15) / 16));
        q.nks_last = 4;
    } else if (d >= EXEMCL_F16_WIDE_D) {
        // v_mfma_f32_16x16x32_{f16,bf16}, 32 coordinates per k-block, two
        // set members per tile; when d mod 32 is in (0, 16] the last k-block
        // holds 16 coordinates (v_mfma_f32_16x16x16) instead of padding to 32
        q.tile = 16;
        q.kb_dims = 32;
        q.nkb = bucket((int)((d + 31) / 32));
        q.nks_last = 1;
        q.nb = EXEMCL_NB16;
        q.half = (d % 32 != 0 && d % 32 <= 16 && d <= EXEMCL_HALF_MAX_D && q.nkb == (d + 31) / 32) ? 1 : 0;
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
    q.splat = splat_bias(eb, q.tile, q.nkb) ? 1 : 0;
    q.wgsum = wg_sum(q.waves, q.nb) ? 1 : 0;
    *p = q;
    return true;
}

int64_t mfma_tile_bytes(const MfmaPlan &pl) {
    return hdr_bytes(pl.tile, pl.nb, pl.splat != 0) + (int64_t)(pl.nkb - pl.half) * pl.nb * 1024 +
           (int64_t)pl.half * pl.nb * 512;
}

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
                       float *rowmax, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
    const MfmaArgs x{V, n, ld, tiles, kt, ngroups, gpc, m0, partials, lpad, rowmax, ev_start, ev_stop};
    if (pl.bigd) return bigd_run(prec, mode, pl, x, st);
    switch (prec) {
    case P_FP32: return eval_run_f32(pl, mode, x, st);
    case P_FP16: return mode == MODE_SUM ? eval_run_f16(pl, mode, x, st) : hipErrorInvalidValue;
    case P_BF16: return mode == MODE_SUM ? eval_run_bf16(pl, mode, x, st) : hipErrorInvalidValue;
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
