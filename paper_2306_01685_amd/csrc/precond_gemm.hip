// Grouped fp32 MFMA GEMMs of the preconditioning dW_hat = Linv G Rinv
// (Algorithm 1, precondition line; Eq. 2 in the stored orientation).
//
// Both stages are the same "TN" contraction  C[m][n] = sum_k At[k][m] B[k][n]
// with At (K x M) and B (K x N) row-major, so both operands are staged into
// LDS with plain row copies and no transpose:
//
//   stage 1:  At = Linv (symmetric, d_in x d_in), B = G (d_in x d_out, fp32 or
//             bf16 upcast in the load path), C = X^T stored transposed
//             (d_out x d_in) so that it is already k-major for stage 2.
//             Tiles of the first M row also sum G^2 over their column panel
//             (the ||G||_F partials of the rescale) as the panel streams by.
//   stage 2:  At = X^T, B = Rinv (symmetric, d_out x d_out), C = dW_hat
//             (d_in x d_out, row-major) written straight into dW, plus one
//             sum of dW_hat^2 per tile for the rescale.
//
// Each workgroup (4 waves, 2 x 2) computes a 128 x 128 tile; each wave owns
// 64 x 64 = 2 x 2 blocks of v_mfma_f32_32x32x2_f32.  K advances in 16-deep
// slabs, double-buffered in LDS; the next slab's global loads are issued
// before the current slab's MFMAs.  The grid is one grouped launch over a
// tile table that the host orders longest-K first.
#include "mkor_internal.h"

namespace mkor {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = GEMM_BM, BN = GEMM_BN, BK = GEMM_BK;
constexpr int NT = GEMM_THREADS;

__device__ __forceinline__ float bf16_to_f32(unsigned short h) {
    return __uint_as_float(((unsigned)h) << 16);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Sum of one float over the workgroup, fixed order; result valid in thread 0.
__device__ __forceinline__ float block_sum(float v, float* red) {
    v = wave_sum(v);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float s = 0.f;
    if (threadIdx.x == 0)
        for (int w = 0; w < NT / 64; ++w) s += red[w];
    return s;
}

// Register staging of one K slab of At and B for the vector paths.
struct SlabRegs {
    float4 a[2];
    float4 b[2];   // fp32 B: two float4; bf16 B: 8 values packed in b[0] and b[1]
};

template <bool BF16, bool VEC>
struct Loader {
    // Global -> registers (VEC) or global -> LDS directly (scalar path).
    __device__ static void load(SlabRegs& r, const GemmLayer& L, int m0, int n0, int k0,
                                float* As, float* Bs, float& gsq, bool want_gsq) {
        const int t = threadIdx.x;
        if constexpr (VEC) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int idx = t + i * NT;
                const int row = idx >> 5, c4 = idx & 31;
                const int k = k0 + row, m = m0 + 4 * c4;
                r.a[i] = (k < L.K && m < L.M)
                    ? *reinterpret_cast<const float4*>(L.At + (size_t)k * L.M + m)
                    : make_float4(0.f, 0.f, 0.f, 0.f);
            }
            if constexpr (!BF16) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int idx = t + i * NT;
                    const int row = idx >> 5, c4 = idx & 31;
                    const int k = k0 + row, n = n0 + 4 * c4;
                    r.b[i] = (k < L.K && n < L.N)
                        ? *reinterpret_cast<const float4*>(
                              static_cast<const float*>(L.B) + (size_t)k * L.N + n)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            } else {
                const int row = t >> 4, c8 = t & 15;
                const int k = k0 + row, n = n0 + 8 * c8;
                uint4 h = make_uint4(0u, 0u, 0u, 0u);
                if (k < L.K && n < L.N)
                    h = *reinterpret_cast<const uint4*>(
                        static_cast<const unsigned short*>(L.B) + (size_t)k * L.N + n);
                r.b[0] = make_float4(__uint_as_float(h.x << 16), __uint_as_float(h.x & 0xffff0000u),
                                     __uint_as_float(h.y << 16), __uint_as_float(h.y & 0xffff0000u));
                r.b[1] = make_float4(__uint_as_float(h.z << 16), __uint_as_float(h.z & 0xffff0000u),
                                     __uint_as_float(h.w << 16), __uint_as_float(h.w & 0xffff0000u));
            }
            if (want_gsq) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    gsq = fmaf(r.b[i].x, r.b[i].x, gsq);
                    gsq = fmaf(r.b[i].y, r.b[i].y, gsq);
                    gsq = fmaf(r.b[i].z, r.b[i].z, gsq);
                    gsq = fmaf(r.b[i].w, r.b[i].w, gsq);
                }
            }
        } else {
            // scalar path: ragged sizes, straight into LDS
#pragma unroll
            for (int i = 0; i < (BK * BM) / NT; ++i) {
                const int idx = t + i * NT;
                const int row = idx / BM, col = idx % BM;
                const int k = k0 + row, m = m0 + col;
                As[row * BM + col] = (k < L.K && m < L.M) ? L.At[(size_t)k * L.M + m] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < (BK * BN) / NT; ++i) {
                const int idx = t + i * NT;
                const int row = idx / BN, col = idx % BN;
                const int k = k0 + row, n = n0 + col;
                float v = 0.f;
                if (k < L.K && n < L.N) {
                    const size_t off = (size_t)k * L.N + n;
                    v = BF16 ? bf16_to_f32(static_cast<const unsigned short*>(L.B)[off])
                             : static_cast<const float*>(L.B)[off];
                }
                if (want_gsq) gsq = fmaf(v, v, gsq);
                Bs[row * BN + col] = v;
            }
        }
    }

    __device__ static void store(const SlabRegs& r, float* As, float* Bs) {
        if constexpr (VEC) {
            const int t = threadIdx.x;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int idx = t + i * NT;
                const int row = idx >> 5, c4 = idx & 31;
                *reinterpret_cast<float4*>(As + row * BM + 4 * c4) = r.a[i];
            }
            if constexpr (!BF16) {
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int idx = t + i * NT;
                    const int row = idx >> 5, c4 = idx & 31;
                    *reinterpret_cast<float4*>(Bs + row * BN + 4 * c4) = r.b[i];
                }
            } else {
                const int row = t >> 4, c8 = t & 15;
                *reinterpret_cast<float4*>(Bs + row * BN + 8 * c8) = r.b[0];
                *reinterpret_cast<float4*>(Bs + row * BN + 8 * c8 + 4) = r.b[1];
            }
        }
    }
};

template <bool BF16, bool VEC, int STAGE>
__device__ void gemm_tile(const GemmLayer& L, const GemmTile& tile, float* partials,
                          float* smem) {
    float* As0 = smem;
    float* Bs0 = smem + BK * BM;
    float* As1 = smem + BK * (BM + BN);
    float* Bs1 = As1 + BK * BM;
    float* red = smem + 2 * BK * (BM + BN);

    const int m0 = tile.tm * BM, n0 = tile.tn * BN;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wave & 1, wn = wave >> 1;
    const int li = lane & 31, lk = lane >> 5;
    const bool want_gsq = (STAGE == 1) && tile.tm == 0;

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    float gsq = 0.f;
    SlabRegs regs;
    const int nslab = (L.K + BK - 1) / BK;

    Loader<BF16, VEC>::load(regs, L, m0, n0, 0, As0, Bs0, gsq, want_gsq);
    Loader<BF16, VEC>::store(regs, As0, Bs0);
    __syncthreads();

    for (int s = 0; s < nslab; ++s) {
        float* As = (s & 1) ? As1 : As0;
        float* Bs = (s & 1) ? Bs1 : Bs0;
        float* An = (s & 1) ? As0 : As1;
        float* Bn = (s & 1) ? Bs0 : Bs1;
        const bool more = s + 1 < nslab;
        if (more && VEC) Loader<BF16, VEC>::load(regs, L, m0, n0, (s + 1) * BK, An, Bn, gsq, want_gsq);

#pragma unroll
        for (int kk = 0; kk < BK / 2; ++kk) {
            const int k = 2 * kk + lk;
            const float a0 = As[k * BM + wm * 64 + li];
            const float a1 = As[k * BM + wm * 64 + 32 + li];
            const float b0 = Bs[k * BN + wn * 64 + li];
            const float b1 = Bs[k * BN + wn * 64 + 32 + li];
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
        }

        if (more) {
            if constexpr (VEC) {
                Loader<BF16, VEC>::store(regs, An, Bn);
            } else {
                // scalar path loads straight into the other buffer, which no
                // wave reads during this slab
                Loader<BF16, VEC>::load(regs, L, m0, n0, (s + 1) * BK, An, Bn, gsq, want_gsq);
            }
        }
        __syncthreads();
    }

    // Epilogue.  Output element (i, j) of block (mi, ni) of this wave:
    //   i = 8 * (r / 4) + 4 * (lane / 32) + r % 4,  j = lane % 32.
    float csq = 0.f;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
            const int n = n0 + wn * 64 + ni * 32 + li;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int mb = m0 + wm * 64 + mi * 32 + 8 * g + 4 * lk;
                const float v0 = acc[mi][ni][4 * g + 0], v1 = acc[mi][ni][4 * g + 1];
                const float v2 = acc[mi][ni][4 * g + 2], v3 = acc[mi][ni][4 * g + 3];
                if constexpr (STAGE == 1) {
                    // C stored transposed: X^T[n][m], leading dimension M
                    if (n < L.N) {
                        float* dst = L.C + (size_t)n * L.M + mb;
                        if (VEC && mb + 3 < L.M) {
                            *reinterpret_cast<float4*>(dst) = make_float4(v0, v1, v2, v3);
                        } else {
                            if (mb + 0 < L.M) dst[0] = v0;
                            if (mb + 1 < L.M) dst[1] = v1;
                            if (mb + 2 < L.M) dst[2] = v2;
                            if (mb + 3 < L.M) dst[3] = v3;
                        }
                    }
                } else {
                    if (n < L.N) {
                        float* dst = L.C + (size_t)mb * L.N + n;
                        if (mb + 0 < L.M) { dst[0] = v0; csq = fmaf(v0, v0, csq); }
                        if (mb + 1 < L.M) { dst[(size_t)L.N] = v1; csq = fmaf(v1, v1, csq); }
                        if (mb + 2 < L.M) { dst[2 * (size_t)L.N] = v2; csq = fmaf(v2, v2, csq); }
                        if (mb + 3 < L.M) { dst[3 * (size_t)L.N] = v3; csq = fmaf(v3, v3, csq); }
                    }
                }
            }
        }
    }

    if constexpr (STAGE == 1) {
        if (want_gsq) {
            const float s = block_sum(gsq, red);
            if (threadIdx.x == 0) partials[L.part0 + tile.tn] = s;
        }
    } else {
        const float s = block_sum(csq, red);
        if (threadIdx.x == 0) partials[L.part0 + tile.tm * L.ntn + tile.tn] = s;
    }
}

constexpr int SMEM_FLOATS = 2 * BK * (BM + BN) + NT / 64;

template <int STAGE>
__global__ __launch_bounds__(NT, 2) void gemm_kernel(const GemmLayer* __restrict__ layers,
                                                     const GemmTile* __restrict__ tiles,
                                                     float* __restrict__ partials) {
    __shared__ __attribute__((aligned(16))) float smem[SMEM_FLOATS];
    const GemmTile tile = tiles[blockIdx.x];
    const GemmLayer L = layers[tile.layer];
    if (L.b_bf16) {
        if (L.vec) gemm_tile<true, true, STAGE>(L, tile, partials, smem);
        else       gemm_tile<true, false, STAGE>(L, tile, partials, smem);
    } else {
        if (L.vec) gemm_tile<false, true, STAGE>(L, tile, partials, smem);
        else       gemm_tile<false, false, STAGE>(L, tile, partials, smem);
    }
}

}  // namespace

hipError_t launch_gemm_xt(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream) {
    if (ntiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_kernel<1>, dim3(ntiles), dim3(NT), 0, stream, layers, tiles, partials);
    return hipGetLastError();
}

hipError_t launch_gemm_dw(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream) {
    if (ntiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_kernel<2>, dim3(ntiles), dim3(NT), 0, stream, layers, tiles, partials);
    return hipGetLastError();
}

}  // namespace mkor
