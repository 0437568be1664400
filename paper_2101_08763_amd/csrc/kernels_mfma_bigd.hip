// kernels_mfma_bigd.hip -- instantiations of the evaluation kernel for
// d > 512 (bigd_kernels.hpp), per storage type, epilogue mode and k-blocks
// per wavefront.
#include "bigd_kernels.hpp"

namespace exemcl {

hipError_t bigd_run(int prec, int mode, const MfmaPlan &pl, const MfmaArgs &x, hipStream_t st) {
    switch (prec) {
    case P_FP32:
        if (mode == MODE_ROWMAX)
            return x.m0 ? bigd_dispatch_kw<float, MODE_ROWMAX, true>(pl, x, st)
                        : bigd_dispatch_kw<float, MODE_ROWMAX, false>(pl, x, st);
        return x.m0 ? bigd_dispatch_kw<float, MODE_SUM, true>(pl, x, st)
                    : bigd_dispatch_kw<float, MODE_SUM, false>(pl, x, st);
    case P_FP16:
        if (mode != MODE_SUM || x.m0) return hipErrorInvalidValue;
        return bigd_dispatch_kw<_Float16, MODE_SUM, false>(pl, x, st);
    case P_BF16:
        if (mode != MODE_SUM || x.m0) return hipErrorInvalidValue;
        return bigd_dispatch_kw<__bf16, MODE_SUM, false>(pl, x, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace exemcl
