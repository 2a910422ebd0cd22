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

// scale = ||G||_F / ||dW_hat||_F of a second-order layer (0 when dW_hat is
// zero; 1 with the rescale off), from its partials in a fixed order, so every
// block of the layer computes the same value.  The layer's first block also
// records the norms.  Block-uniform; ends with a barrier.
__device__ __forceinline__ float layer_scale(const RescaleLayer& L, int bi, const float* __restrict__ gpart,
                                             const float* __restrict__ dpart, int rescale, double* s_g,
                                             double* s_d, float* s_scale) {
    const int t = threadIdx.x;
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
    return sc;
}

__device__ __forceinline__ void rescale_block(const RescaleLayer* __restrict__ layers,
                                              const RescaleBlock* __restrict__ blocks,
                                              const float* __restrict__ gpart,
                                              const float* __restrict__ dpart, int rescale, int bi,
                                              double* s_g, double* s_d, float* s_scale) {
    const RescaleBlock b = blocks[bi];
    const RescaleLayer L = layers[b.layer];
    const int t = threadIdx.x;
    const int64_t end = min(b.start + (int64_t)RS_ELEMS, L.numel);

    if (!L.second_order || !gld_i32(L.mode)) {   // planned or switched first-order: dW = G
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

    const float sc = layer_scale(L, bi, gpart, dpart, rescale, s_g, s_d, s_scale);
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

// ------------------------------------------------------------------ optimizer
// The backend optimizer step fused into the rescale (Algorithm 1, last line).
// Element i of a layer with weights: g = scale * dW_hat[i] (second-order) or
// G[i] (first-order), then
//   SGD:   d = g + wd W, m = mu m + d, W = W - lr m               (pass A)
//   LAMB:  m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2,
//          r = (m bc1) / (sqrt(v bc2) + eps) + wd W                 (pass A: m, v
//          stored, sum W^2 and sum r^2 per block), the layer's ratio from the
//          block sums (opt_trust_kernel), then W = W - lr ratio r with r formed
//          again from the stored m, v, W, bit for bit the same     (pass B).
// Layers without weights get dW = g.
__device__ __forceinline__ float lamb_r(float m, float v, float w, const OptArgs& o) {
    return __fmaf_rn(o.wd, w, __fdiv_rn(__fmul_rn(m, o.bc1), __fadd_rn(__fsqrt_rn(__fmul_rn(v, o.bc2)), o.eps)));
}

template <int KIND>
__device__ void opt_elem(const RescaleLayer& L, int64_t i, float g, const OptArgs& o, float& w2, float& r2) {
    if (L.W == nullptr || o.store_dw) gst(L.dW + i, g);
    if (L.W == nullptr) return;
    const float w = gld(L.W + i);
    if constexpr (KIND == MKOR_OPT_SGD) {
        const float d = __fmaf_rn(o.wd, w, g);
        const float m = __fmaf_rn(o.mom, gld(L.m + i), d);
        gst(L.m + i, m);
        gst(L.W + i, __fmaf_rn(-o.lr, m, w));
    } else {
        const float m = __fmaf_rn(o.b1, gld(L.m + i), __fmul_rn(1.f - o.b1, g));
        const float v = __fmaf_rn(o.b2, gld(L.v + i), __fmul_rn(1.f - o.b2, __fmul_rn(g, g)));
        gst(L.m + i, m);
        gst(L.v + i, v);
        const float r = lamb_r(m, v, w, o);
        w2 = fmaf(w, w, w2);
        r2 = fmaf(r, r, r2);
    }
}

// Four consecutive elements (i a multiple of 4), 16-byte accesses.
template <int KIND>
__device__ void opt_elem4(const RescaleLayer& L, int64_t i, const float (&g)[4], const OptArgs& o, float& w2,
                          float& r2) {
    if (L.W == nullptr || o.store_dw) gst4(L.dW + i, make_float4(g[0], g[1], g[2], g[3]));
    if (L.W == nullptr) return;
    const float4 w4 = gld4(L.W + i), m4 = gld4(L.m + i);
    const float w[4] = {w4.x, w4.y, w4.z, w4.w}, mo[4] = {m4.x, m4.y, m4.z, m4.w};
    float wn[4], mn[4];
    if constexpr (KIND == MKOR_OPT_SGD) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float d = __fmaf_rn(o.wd, w[c], g[c]);
            mn[c] = __fmaf_rn(o.mom, mo[c], d);
            wn[c] = __fmaf_rn(-o.lr, mn[c], w[c]);
        }
        gst4(L.m + i, make_float4(mn[0], mn[1], mn[2], mn[3]));
        gst4(L.W + i, make_float4(wn[0], wn[1], wn[2], wn[3]));
    } else {
        const float4 v4 = gld4(L.v + i);
        const float vo[4] = {v4.x, v4.y, v4.z, v4.w};
        float vn[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            mn[c] = __fmaf_rn(o.b1, mo[c], __fmul_rn(1.f - o.b1, g[c]));
            vn[c] = __fmaf_rn(o.b2, vo[c], __fmul_rn(1.f - o.b2, __fmul_rn(g[c], g[c])));
            const float r = lamb_r(mn[c], vn[c], w[c], o);
            w2 = fmaf(w[c], w[c], w2);
            r2 = fmaf(r, r, r2);
        }
        gst4(L.m + i, make_float4(mn[0], mn[1], mn[2], mn[3]));
        gst4(L.v + i, make_float4(vn[0], vn[1], vn[2], vn[3]));
    }
}

template <int KIND>
__global__ __launch_bounds__(RS_THREADS) void opt_pass_a_kernel(
    const RescaleLayer* __restrict__ layers, const RescaleBlock* __restrict__ blocks, int nblocks,
    const float* __restrict__ gpart, const float* __restrict__ dpart, int rescale, OptArgs o,
    float2* __restrict__ lpart) {
    __shared__ double s_g[RS_THREADS], s_d[RS_THREADS];
    __shared__ float s_scale;
    __shared__ float s_w[RS_THREADS / 64], s_r[RS_THREADS / 64];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    for (int bi = blockIdx.x; bi < nblocks; bi += gridDim.x) {
        const RescaleBlock b = blocks[bi];
        const RescaleLayer L = layers[b.layer];
        const int64_t end = min(b.start + (int64_t)RS_ELEMS, L.numel);
        const bool so = L.second_order && gld_i32(L.mode);   // block-uniform
        const float sc = so ? layer_scale(L, bi, gpart, dpart, rescale, s_g, s_d, &s_scale) : 1.f;
        float w2 = 0.f, r2 = 0.f;
        if ((L.numel & 3) == 0) {   // blocks start at multiples of RS_ELEMS: 16-byte groups
            for (int64_t i = b.start + 4 * t; i < end; i += 4 * RS_THREADS) {
                float g[4];
                if (so) {
                    const float4 d = gld4(L.dW + i);
                    g[0] = __fmul_rn(d.x, sc); g[1] = __fmul_rn(d.y, sc);
                    g[2] = __fmul_rn(d.z, sc); g[3] = __fmul_rn(d.w, sc);
                } else if (L.g_bf16) {
                    const uint2 h = gld_u2(static_cast<const unsigned short*>(L.G) + i);
                    g[0] = bf2f((unsigned short)(h.x & 0xffffu)); g[1] = bf2f((unsigned short)(h.x >> 16));
                    g[2] = bf2f((unsigned short)(h.y & 0xffffu)); g[3] = bf2f((unsigned short)(h.y >> 16));
                } else {
                    const float4 d = gld4(static_cast<const float*>(L.G) + i);
                    g[0] = d.x; g[1] = d.y; g[2] = d.z; g[3] = d.w;
                }
                opt_elem4<KIND>(L, i, g, o, w2, r2);
            }
        } else {
            for (int64_t i = b.start + t; i < end; i += RS_THREADS) {
                float g;
                if (so)              g = __fmul_rn(gld(L.dW + i), sc);
                else if (L.g_bf16)   g = __uint_as_float(((unsigned)gld_u16(static_cast<const unsigned short*>(L.G) + i)) << 16);
                else                 g = gld(static_cast<const float*>(L.G) + i);
                opt_elem<KIND>(L, i, g, o, w2, r2);
            }
        }
        if (KIND == MKOR_OPT_LAMB && L.W != nullptr) {   // block sums in a fixed order
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                w2 += __shfl_xor(w2, off, 64);
                r2 += __shfl_xor(r2, off, 64);
            }
            if (lane == 0) { s_w[wave] = w2; s_r[wave] = r2; }
            __syncthreads();
            if (t == 0) {
                float aw = 0.f, ar = 0.f;
                for (int x = 0; x < RS_THREADS / 64; ++x) { aw += s_w[x]; ar += s_r[x]; }
                lpart[bi] = make_float2(aw, ar);
            }
            __syncthreads();
        }
    }
}

// Per-layer LAMB ratio ||W|| / ||r|| from the block sums (fixed order).
__global__ __launch_bounds__(RS_THREADS) void opt_trust_kernel(const RescaleLayer* __restrict__ layers,
                                                              const float2* __restrict__ lpart,
                                                              float* __restrict__ trust) {
    const RescaleLayer L = layers[blockIdx.x];
    if (L.W == nullptr) return;
    __shared__ double s_w[RS_THREADS], s_r[RS_THREADS];
    const int t = threadIdx.x;
    double aw = 0.0, ar = 0.0;
    for (int k = t; k < L.nblk; k += RS_THREADS) {
        const float2 p = lpart[L.first_blk + k];
        aw += (double)p.x;
        ar += (double)p.y;
    }
    s_w[t] = aw; s_r[t] = ar;
    __syncthreads();
    for (int o = RS_THREADS / 2; o > 0; o >>= 1) {
        if (t < o) { s_w[t] += s_w[t + o]; s_r[t] += s_r[t + o]; }
        __syncthreads();
    }
    if (t == 0) {
        const double nw = sqrt(s_w[0]), nr = sqrt(s_r[0]);
        trust[blockIdx.x] = (nw > 0.0 && nr > 0.0) ? (float)(nw / nr) : 1.f;
    }
}

__global__ __launch_bounds__(RS_THREADS) void opt_pass_b_kernel(
    const RescaleLayer* __restrict__ layers, const RescaleBlock* __restrict__ blocks, int nblocks, OptArgs o,
    const float* __restrict__ trust) {
    for (int bi = blockIdx.x; bi < nblocks; bi += gridDim.x) {
        const RescaleBlock b = blocks[bi];
        const RescaleLayer L = layers[b.layer];
        if (L.W == nullptr) continue;
        const float step = __fmul_rn(o.lr, trust[b.layer]);
        const int64_t end = min(b.start + (int64_t)RS_ELEMS, L.numel);
        if ((L.numel & 3) == 0) {
            for (int64_t i = b.start + 4 * threadIdx.x; i < end; i += 4 * RS_THREADS) {
                const float4 w = gld4(L.W + i), m = gld4(L.m + i), v = gld4(L.v + i);
                gst4(L.W + i, make_float4(__fmaf_rn(-step, lamb_r(m.x, v.x, w.x, o), w.x),
                                          __fmaf_rn(-step, lamb_r(m.y, v.y, w.y, o), w.y),
                                          __fmaf_rn(-step, lamb_r(m.z, v.z, w.z, o), w.z),
                                          __fmaf_rn(-step, lamb_r(m.w, v.w, w.w, o), w.w)));
            }
        } else {
            for (int64_t i = b.start + threadIdx.x; i < end; i += RS_THREADS) {
                const float w = gld(L.W + i);
                gst(L.W + i, __fmaf_rn(-step, lamb_r(gld(L.m + i), gld(L.v + i), w, o), w));
            }
        }
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

hipError_t launch_rescale_opt(const RescaleLayer* layers, int32_t nlayers, const RescaleBlock* blocks,
                              int32_t nblocks, const float* gpart, const float* dpart, int32_t rescale,
                              const OptArgs& opt, float2* lpart, float* trust, hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    const int32_t grid = (RS_GRID > 0 && nblocks > RS_GRID) ? RS_GRID : nblocks;
    if (opt.kind == MKOR_OPT_SGD) {
        hipLaunchKernelGGL(opt_pass_a_kernel<MKOR_OPT_SGD>, dim3(grid), dim3(RS_THREADS), 0, stream, layers,
                           blocks, nblocks, gpart, dpart, rescale, opt, lpart);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(opt_pass_a_kernel<MKOR_OPT_LAMB>, dim3(grid), dim3(RS_THREADS), 0, stream, layers, blocks,
                       nblocks, gpart, dpart, rescale, opt, lpart);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(opt_trust_kernel, dim3(nlayers), dim3(RS_THREADS), 0, stream, layers, lpart, trust);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(opt_pass_b_kernel, dim3(grid), dim3(RS_THREADS), 0, stream, layers, blocks, nblocks, opt,
                       trust);
    return hipGetLastError();
}

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
