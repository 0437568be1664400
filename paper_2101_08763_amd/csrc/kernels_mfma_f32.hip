// kernels_mfma_f32.hip -- fp32 instantiations of the MFMA kernels
// (32x32x2 tiles for d <= 256, 16x16x4 tiles above).
#include "mfma_kernels.hpp"

namespace exemcl {

hipError_t pack_run_f32(const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets, int64_t l,
                        int64_t k, void *tiles, hipStream_t st) {
    return pl.tile == 32 ? pack_launch<float, 32>(pl, V, n, ld, sets, l, k, tiles, st)
                         : pack_launch<float, 16>(pl, V, n, ld, sets, l, k, tiles, st);
}

hipError_t eval_run_f32(const MfmaPlan &pl, int mode, const MfmaArgs &x, hipStream_t st) {
    if (mode == MODE_ROWMAX)
        return pl.tile == 32 ? eval_dispatch<float, 32, MODE_ROWMAX>(pl, x, st)
                             : eval_dispatch<float, 16, MODE_ROWMAX>(pl, x, st);
    return pl.tile == 32 ? eval_dispatch<float, 32, MODE_SUM>(pl, x, st)
                         : eval_dispatch<float, 16, MODE_SUM>(pl, x, st);
}

}  // namespace exemcl
