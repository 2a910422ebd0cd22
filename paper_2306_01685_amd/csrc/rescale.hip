// Gradient rescaling and first-order pass-through (Algorithm 1, rescale line
// and else-branch; "Rescaling Gradients").
//
// dW already holds dW_hat (written by the second preconditioning GEMM).  Each
// workgroup of a second-order layer reduces that layer's ||G||^2 and
// ||dW_hat||^2 partials in a fixed order (so all of them agree), forms
// scale = ||G||_F / ||dW_hat||_F (0 when dW_hat is zero) and scales its
// chunk of dW in place.  First-order layers copy G into dW (bf16 upcast).
#include "gmem.h"
#include "mkor_internal.h"

#include <math.h>

namespace mkor {
namespace {

__device__ __forceinline__ void rescale_block(const RescaleLayer* __restrict__ layers,
                                              const RescaleBlock* __restrict__ blocks,
                                              const float* __restrict__ gpart,
                                              const float* __restrict__ dpart, int rescale, int bi,
                                              double* s_g, double* s_d, float* s_scale) {
    const RescaleBlock b = blocks[bi];
    const RescaleLayer L = layers[b.layer];
    const int t = threadIdx.x;
    const int64_t end = min(b.start + (int64_t)RS_ELEMS, L.numel);

    if (!L.second_order) {
        if (L.g_bf16) {
            const unsigned short* G = static_cast<const unsigned short*>(L.G);
            for (int64_t i = b.start + t; i < end; i += RS_THREADS)
                gst(L.dW + i, __uint_as_float(((unsigned)gld_u16(G + i)) << 16));
        } else {
            const float* G = static_cast<const float*>(L.G);
            if ((L.numel & 3) == 0) {
                for (int64_t i = (b.start >> 2) + t; i < (end >> 2); i += RS_THREADS)
                    gst4(L.dW + 4 * i, gld4(G + 4 * i));
            } else {
                for (int64_t i = b.start + t; i < end; i += RS_THREADS) gst(L.dW + i, gld(G + i));
            }
        }
        return;
    }

    double g2 = 0.0, d2 = 0.0;
    for (int i = t; i < L.ngpart; i += RS_THREADS) g2 += (double)gld(gpart + L.gpart0 + i);
    for (int i = t; i < L.ndpart; i += RS_THREADS) d2 += (double)gld(dpart + L.dpart0 + i);
    s_g[t] = g2; s_d[t] = d2;
    __syncthreads();
    for (int o = RS_THREADS / 2; o > 0; o >>= 1) {
        if (t < o) { s_g[t] += s_g[t + o]; s_d[t] += s_d[t + o]; }
        __syncthreads();
    }
    if (t == 0) {
        const double nG = sqrt(s_g[0]), nD = sqrt(s_d[0]);
        const double sc = rescale ? (nD > 0.0 ? nG / nD : 0.0) : 1.0;
        *s_scale = (float)sc;
        if (bi == L.first_blk && L.stats != nullptr) {
            L.stats->norm_G = (float)nG;
            L.stats->norm_dW_hat = (float)nD;
            L.stats->scale = (float)sc;
            L.stats->nonfinite_scale = (isfinite(nG) && isfinite(nD)) ? 0 : 1;
        }
    }
    __syncthreads();
    const float sc = *s_scale;
    __syncthreads();   // s_g, s_d and s_scale are reused by the next block
    if (!rescale) return;
    if ((L.numel & 3) == 0) {
        for (int64_t i = (b.start >> 2) + t; i < (end >> 2); i += RS_THREADS) {
            float4 v = gld4_nt(L.dW + 4 * i);
            v.x *= sc; v.y *= sc; v.z *= sc; v.w *= sc;
            gst4_nt(L.dW + 4 * i, v);
        }
    } else {
        for (int64_t i = b.start + t; i < end; i += RS_THREADS) gst(L.dW + i, gld(L.dW + i) * sc);
    }
}

// Grid-stride over the rescale blocks (long streams per workgroup).
__global__ __launch_bounds__(RS_THREADS) void rescale_kernel(
    const RescaleLayer* __restrict__ layers, const RescaleBlock* __restrict__ blocks, int nblocks,
    const float* __restrict__ gpart, const float* __restrict__ dpart, int rescale) {
    __shared__ double s_g[RS_THREADS], s_d[RS_THREADS];
    __shared__ float s_scale;
    for (int bi = blockIdx.x; bi < nblocks; bi += gridDim.x)
        rescale_block(layers, blocks, gpart, dpart, rescale, bi, s_g, s_d, &s_scale);
}

}  // namespace

hipError_t launch_rescale(const RescaleLayer* layers, const RescaleBlock* blocks, int32_t nblocks,
                          const float* gpart, const float* dpart, int32_t rescale,
                          hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    const int32_t grid = (RS_GRID > 0 && nblocks > RS_GRID) ? RS_GRID : nblocks;
    hipLaunchKernelGGL(rescale_kernel, dim3(grid), dim3(RS_THREADS), 0, stream, layers, blocks, nblocks,
                       gpart, dpart, rescale);
    return hipGetLastError();
}

}  // namespace mkor
