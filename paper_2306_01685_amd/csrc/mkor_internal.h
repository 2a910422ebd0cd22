// Internal device-side descriptors and kernel launchers of libmkor.
//
// The host (mkor_abi.cpp) lays these tables out in the caller's workspace at
// plan creation; every kernel is a single grouped launch over all layers that
// reads its work item from one of the tables below.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

#include "../../include/mkor.h"

namespace mkor {

// ---------------------------------------------------------------- SM update
// One inverse factor P (d x d) and its driving vector x.
struct FactorDesc {
    float*            P;
    const float*      x;
    float*            u;       // workspace, d floats: u_raw = P x (before blending)
    mkor_layer_stats* stats;   // may be null
    int32_t           d;
    int32_t           blk0;    // first row block of this factor in the row-block table
    int32_t           nblk;    // number of row blocks of this factor
    int32_t           side;    // 0 = Linv (driven by a), 1 = Rinv (driven by g)
};

// Rows handled by one workgroup of the SM kernels (4 waves x 4 rows).
constexpr int SM_THREADS = 256;
constexpr int SM_ROWS_PER_WAVE = 4;
constexpr int SM_ROWS = (SM_THREADS / 64) * SM_ROWS_PER_WAVE;

struct RowBlock {
    int32_t factor;
    int32_t row0;
};

// Scalars of one factor's update, decided on the device from the K1 partials.
struct SmScalars {
    float c1, c2, sgn, sqc;   // P <- c1 P + c2 I + sgn * w w^T,  w = sqc * u
    float zp, zq;             // u = zp * u_raw + zq * x
    int   stab, skip;
    float nu, s;
};

// ---------------------------------------------------------------- GEMMs
// C = At^T * B for one layer: At is K x M (row-major, M contiguous), B is
// K x N (row-major, N contiguous), C is M x N, stored row-major (ldc = N) or
// transposed (N x M, ldc = M).
struct GemmLayer {
    const float* At;
    const void*  B;
    float*       C;
    int32_t      M, N, K;
    int32_t      b_bf16;      // element type of B
    int32_t      vec;         // rows of At, B and C allow 16-byte vector access
    int32_t      part0;       // first partial-sum slot of this layer
    int32_t      ntn;         // number of N tiles
    int32_t      _pad;
};

struct GemmTile {
    int32_t layer;
    int32_t tm, tn;
    int32_t _pad;
};

constexpr int GEMM_BM = 128;
constexpr int GEMM_BN = 128;
constexpr int GEMM_BK = 16;
constexpr int GEMM_THREADS = 256;

// ---------------------------------------------------------------- rescale
struct RescaleLayer {
    const void*       G;
    float*            dW;
    mkor_layer_stats* stats;
    int64_t           numel;
    int32_t           second_order;
    int32_t           g_bf16;
    int32_t           gpart0, ngpart;   // ||G||^2 partials (written by GEMM 1)
    int32_t           dpart0, ndpart;   // ||dW_hat||^2 partials (written by GEMM 2)
    int32_t           first_blk;        // first rescale block of this layer
    int32_t           _pad;
};

constexpr int RS_THREADS = 256;
constexpr int RS_ELEMS = 8192;   // elements per rescale workgroup

struct RescaleBlock {
    int32_t layer;
    int32_t _pad;
    int64_t start;
};

// ---------------------------------------------------------------- launchers
// Each returns the hipError_t of its launch.
hipError_t launch_sm_matvec(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                            float4* partials, int32_t norm_kind, hipStream_t stream);

hipError_t launch_sm_update(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                            const float4* partials, const mkor_params& p, hipStream_t stream);

// GEMM 1: X^T = (Linv G)^T, plus ||G||^2 partials from the tiles of the first M row.
hipError_t launch_gemm_xt(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream);
// GEMM 2: dW_hat = X Rinv, plus one ||dW_hat||^2 partial per tile.
hipError_t launch_gemm_dw(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream);

hipError_t launch_rescale(const RescaleLayer* layers, const RescaleBlock* blocks, int32_t nblocks,
                          const float* gpart, const float* dpart, int32_t rescale,
                          hipStream_t stream);

}  // namespace mkor
