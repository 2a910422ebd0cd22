// Stage 2 of the preconditioning: dW_hat = X Rinv, plus one ||dW_hat||^2
// partial per tile (implementation in precond_gemm_impl.h).
#define MKOR_GEMM_STAGE 2
#include "precond_gemm_impl.h"

namespace mkor {

hipError_t launch_gemm_dw(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream) {
    return launch_stage<2>(layers, tiles, ntiles, partials, stream);
}

}  // namespace mkor
