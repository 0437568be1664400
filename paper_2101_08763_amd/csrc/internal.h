// internal.h -- host-side launch interface between the ABI layer and the
// kernel translation units.  Not installed; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace exemcl {

enum Prec { P_FP32 = 0, P_FP16 = 1, P_BF16 = 2 };

// Index of an empty slot: pads sets shorter than the batch's k.
constexpr int32_t kEmptySlot = -1;

// Geometry of one MFMA evaluation launch; a pure function of (d, precision),
// never of n or l, so that the partial-sum layout seen by one set does not
// depend on the batch it arrives in.
struct MfmaPlan {
    int tile;       // TM: sets per column tile (32 or 16)
    int nkb;        // k-blocks per tile: ceil(d / kb_dims) rounded up to a compiled bucket
    int nks_last;   // MFMA instructions fed by the last k-block
    int rt;         // row tiles per wavefront
    int waves;      // wavefronts per workgroup
    int rows;       // rows per workgroup = waves * rt * tile
    int kb_dims;    // coordinates per k-block
    int nb;         // set members per staged tile (a set group spans ceil(k / nb) tiles)
    int half;       // 1: the last k-block holds 16 coordinates (16x16x16 instruction)
    int splat;      // 1: tile headers hold bf16 bias parts for the splat MFMA (32-column tiles, few k-blocks)
    int il;         // 1: fp32 single k-block with coordinates 2e + g (ceil(d/2) instructions; rows need no padding)
    int wgsum;      // 1: the kernel adds its wavefronts' partial sums: one partial-sum row per row block
    int bigd;       // 1: d > 512, the coordinates split over the wavefronts (bigd_kernels.hpp)
    int kw;         // bigd: k-blocks per wavefront and round (a compiled bucket: 2, 4, 8)
    int rounds;     // bigd: rounds of 8 * kw k-blocks that cover d
};

bool mfma_plan(int prec, int64_t d, MfmaPlan *p);

// Arguments of one launch of the MFMA evaluation kernel.
struct MfmaArgs {
    const void *V;
    int64_t n;
    int ld;  // row stride in elements: rows are whole 16-byte lane vectors
    const void *tiles;
    int64_t kt, ngroups, gpc;  // staged tiles per set group, set groups, groups per chunk
    const float *m0;
    float *partials;
    int64_t lpad;
    float *rowmax;
    // Optional: events the kernel's dispatch itself records at its start and
    // end (hipExtLaunchKernel), so their interval is the kernel's run time.
    hipEvent_t ev_start = nullptr, ev_stop = nullptr;
};

// Per-storage-type instantiations (kernels_mfma_{f32,f16,bf16}.hip).
hipError_t pack_run_f32(const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets, int64_t l,
                        int64_t k, void *tiles, hipStream_t st);
hipError_t pack_run_f16(const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets, int64_t l,
                        int64_t k, void *tiles, hipStream_t st);
hipError_t pack_run_bf16(const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets, int64_t l,
                         int64_t k, void *tiles, hipStream_t st);
hipError_t eval_run_f32(const MfmaPlan &pl, int mode, const MfmaArgs &x, hipStream_t st);
hipError_t eval_run_f16(const MfmaPlan &pl, int mode, const MfmaArgs &x, hipStream_t st);
hipError_t eval_run_bf16(const MfmaPlan &pl, int mode, const MfmaArgs &x, hipStream_t st);
// The d > 512 kernel (kernels_mfma_bigd.hip), every storage type.
hipError_t bigd_run(int prec, int mode, const MfmaPlan &pl, const MfmaArgs &x, hipStream_t st);

// Geometry of one VALU evaluation launch.
struct ValuPlan {
    int dp;         // padded dimension held in registers (1, 2, 4, 8, 16)
    int rpt;        // rows per thread
    int rows;       // rows per workgroup = 256 * rpt
    int rec;        // floats per staged exemplar record (bias + dp coords, padded to 4)
    int sets_per_chunk;
};

bool valu_plan(int prec, int64_t d, int64_t k, ValuPlan *p);

// The MFMA kernels read V as rows of `ld` elements whose lane vectors are
// wholly inside a row or wholly past its data (zero there).  V can be read in
// place (ld = d) when mfma_rows_in_place(prec, d) and V is aligned as
// mfma_rows_ready checks; otherwise a zero-padded copy with row stride
// mfma_row_stride (whole 16-byte vectors) is made (launch_pad).
int64_t mfma_row_stride(int prec, int64_t d);
bool mfma_rows_in_place(int prec, int64_t d);
bool mfma_rows_ready(int prec, const void *V, int64_t d);

// Vp[i][t] = V[i][t] for t < d, 0 for d <= t < ld (n rows).
hipError_t launch_pad(int prec, const void *V, int64_t n, int d, void *Vp, int ld, hipStream_t st);

// Stage the exemplar tiles of `l` sets of `k` indices: for every set group,
// ceil(k / nb) tiles, each holding members q*nb .. q*nb+nb-1 of the group's
// TM sets as nb column groups: TM*nb biases -||s||^2/2 (-FLT_MAX for padding
// columns, members past k and invalid indices) and the B lane vectors.
hipError_t launch_pack(int prec, const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets,
                       int64_t l, int64_t k, void *tiles, hipStream_t st);

// Bytes of one staged tile (bias header + B lane vectors), and staged tiles
// per set group of k members.
int64_t mfma_tile_bytes(const MfmaPlan &pl);
int64_t mfma_tiles_per_group(const MfmaPlan &pl, int64_t k);

// Mode of the MFMA kernel's epilogue.
enum Mode { MODE_SUM = 0, MODE_ROWMAX = 1 };

// `kt` = staged tiles per set group (mfma_tiles_per_group).
// partials[(rb * waves + w) * lpad + j] = sum over the rows of wavefront w
// of row block rb of max(m0(v), max_p (<v, s_jp> - ||s_jp||^2 / 2)); m0 = 0
// when null (fp32 only otherwise).  MODE_ROWMAX (fp32, groups_per_chunk =
// ngroups) instead writes rowmax[v] = max(m0(v), 0, max over all staged
// columns); rowmax must not alias m0.
hipError_t launch_mfma(int prec, int mode, const MfmaPlan &pl, const void *V, int64_t n, int ld,
                       const void *tiles, int64_t kt, int64_t ngroups, int64_t groups_per_chunk,
                       const float *m0, float *partials, int64_t lpad, float *rowmax, hipStream_t st,
                       hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

hipError_t launch_valu(int prec, const ValuPlan &pl, const void *V, int64_t n, int d, const int32_t *sets,
                       int64_t l, int64_t k, float *partials, int64_t lpad, hipStream_t st);

// out[j] = (2/n) * sum_g partials[g * lpad + j] (fp64, fixed order), or NaN
// when an index of set j (or of the common list) is outside [0, n) and not
// the empty slot.
hipError_t launch_reduce(const float *partials, int64_t G, int64_t lpad, int64_t l, int64_t n,
                         const int32_t *sets, int64_t kset, const int32_t *common, int64_t kcommon, float *out,
                         hipStream_t st);

// Out-of-core evaluation: acc[j] (+)= sum_{g < G} partials[g * lpad + j]
// (fp64, g in order; `first` overwrites), and out[j] = (2/n) * acc[j], or NaN
// where bad[j] != 0.
hipError_t launch_accum(const float *partials, int64_t G, int64_t lpad, int64_t l, bool first, double *acc,
                        hipStream_t st);
hipError_t launch_finish(const double *acc, const uint8_t *bad, int64_t l, int64_t n, float *out, hipStream_t st);

hipError_t launch_sqnorm(int prec, const void *V, int64_t n, int d, float *q, hipStream_t st);

// out[i] = 0 for i < count (f of empty sets).
hipError_t launch_zero(float *out, int64_t count, hipStream_t st);

// Greedy optimizer state (kernels_greedy.hip): cands[i] = i, taken[i] = 0,
// g[i] = 0 for i < n.
hipError_t launch_greedy_init(int32_t *cands, uint8_t *taken, float *g, int64_t n, hipStream_t st);

// Partial-result slots the argmax needs (pval and pidx hold this many).
int64_t argmax_blocks(int64_t n);

// Best untaken scores[i] (largest, lowest i on ties, NaN last): writes its
// index to *S_slot and its score to *f_slot, and sets taken[i] = 1.
hipError_t launch_argmax(const float *scores, uint8_t *taken, int64_t n, float *pval, int32_t *pidx,
                         int32_t *S_slot, float *f_slot, hipStream_t st);

}  // namespace exemcl
