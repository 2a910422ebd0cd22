// Stage 1 of the preconditioning: X^T = (Linv G)^T, plus the ||G||^2
// partials (implementation in precond_gemm_impl.h).
#define MKOR_GEMM_STAGE 1
#include "precond_gemm_impl.h"

namespace mkor {

hipError_t launch_gemm_xt(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream) {
    return launch_stage<1>(layers, tiles, ntiles, partials, stream);
}

}  // namespace mkor
