// kernels_mfma_bf16.hip -- bf16 instantiations of the MFMA kernels
// (v_mfma_f32_32x32x16_bf16, fp32 accumulate).
#include "mfma_kernels.hpp"

namespace exemcl {

hipError_t pack_run_bf16(const MfmaPlan &pl, const void *V, int64_t n, int ld, const int32_t *sets, int64_t l,
                         int64_t k, void *tiles, hipStream_t st) {
    return pl.tile == 32 ? pack_launch<__bf16, 32>(pl, V, n, ld, sets, l, k, tiles, st)
                         : pack_launch<__bf16, 16>(pl, V, n, ld, sets, l, k, tiles, st);
}

hipError_t eval_run_bf16(const MfmaPlan &pl, int mode, const MfmaArgs &x, hipStream_t st) {
    (void)mode;
    return pl.tile == 32 ? eval_dispatch<__bf16, 32, MODE_SUM>(pl, x, st)
                         : eval_dispatch<__bf16, 16, MODE_SUM>(pl, x, st);
}

}  // namespace exemcl
