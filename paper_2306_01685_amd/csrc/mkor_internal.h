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

// ---------------------------------------------------------------- layer modes
// Every layer has a mode word in the workspace: 1 while it takes the
// second-order branch of Algorithm 1, 0 while it takes the first-order one
// (dW = G; its factors are neither read nor updated).  A layer planned
// first-order always has 0; mkor_set_second_order rewrites the words of the
// others on the stream.  Each descriptor below carries a pointer to its
// layer's word, and every kernel of a step skips the work of a layer whose
// word is 0, except the rescale, which then copies G into dW.

// ---------------------------------------------------------------- rank-1 means
// Column means of the rows x cols activation / output-gradient matrices.
constexpr int MEAN_COLS = 512;      // columns per chunk: 8 per lane of one wave
// Rows per block of the partial sums: a power of two between MEAN_ROWS_MIN
// and MEAN_ROWS_MAX, the largest that still gives the plan MEAN_MIN_BLOCKS
// blocks (longer blocks stream better; enough of them fill the chip).
constexpr int MEAN_ROWS_MIN = 512, MEAN_ROWS_MAX = 8192;
constexpr int64_t MEAN_MIN_BLOCKS = 1024;
constexpr int MEAN_THREADS = 256;   // 4 waves, each taking every 4th row of a block

struct MeanMat {
    const void* X;        // rows x cols, row-major
    float*      out;      // cols
    int32_t     rows, cols;
    int32_t     bf16;     // element type of X
    int32_t     vec;      // cols % 8 == 0: vector loads of 8 columns
    int32_t     nchunk;   // column chunks of MEAN_COLS
    int32_t     nrb;      // row blocks of rpb rows
    int32_t     rpb;      // rows per block (the plan's, see MEAN_ROWS_MIN)
    int32_t     _pad;
    int64_t     part0;    // first partial (double) of this matrix
    const int32_t* mode;  // the layer's mode word (see LayerMode)
};

struct MeanItem {
    int32_t mat, chunk, rb, _pad;
};

// ---------------------------------------------------------------- SM update
// The current value of an inverse factor is its caller buffer S with one
// pending rank-1 term applied:
//
//   P = c1 * S + c2 * I + sgn * w w^T      (has = 1)
//   P = S                                   (has = 0)
//
// Element (i, j) is evaluated as fadd(fma(c1, S_ij, sgn * fmul(w_i, w_j)), c2 * [i == j])
// with every rounding pinned, by every kernel that reads a factor, so the
// streaming pass that later writes P into S and the GEMM loads that apply it
// on the fly see bit-identical values.
//
// A factor marked lazy (FactorDesc.lazy) may carry two such terms, one
// after the other, so that the pass writes S only every other step:
//
//   P' = c1 * S + c2 * I + sgn * w w^T,
//   P  = c1b * P' + c2b * I + sgnb * w2 w2^T              (has = 2, w2 = w + d)
//
// each element evaluated in that order with the same roundings, so the values
// are those that writing P' back first would give, bit for bit.
struct Pending {
    float   c1, c2, sgn;
    int32_t has;
    float   c1b, c2b, sgnb;
    int32_t _pad;
};

// One inverse factor P (d x d) and its driving vector x.
struct FactorDesc {
    void*             P;       // caller buffer S (fp32, or bf16 when half = 1)
    const float*      x;
    float*            u;       // workspace, d floats: u_raw = P x (current P, before blending)
    float*            w;       // workspace, d floats: w of the pending term
    Pending*          pend;    // workspace
    mkor_layer_stats* stats;   // may be null
    int32_t           d;
    int32_t           blk0;    // first row block of this factor in the row-block table
    int32_t           nblk;    // number of row blocks of this factor
    int32_t           side;    // 0 = Linv (driven by a), 1 = Rinv (driven by g)
    int32_t           half;    // 1: S is stored in bf16 (d a multiple of 64)
    int32_t           rank;    // r vectors: x, u and w are d x r (vector l at + l * d)
    int32_t           lazy;    // rank 1, fp32: up to two pending terms (w holds 2 d floats)
    int32_t           _pad;
    const int32_t*    mode;    // the layer's mode word
};

// Rank-r factors (rank > 1): per row block, the Gram partials
// sum_rows x_l[i] (P x_m)[i] (MAXR x MAXR) and sum_rows x_l[i] x_m[i] (MAXR x MAXR).
constexpr int MAXR = MKOR_MAX_RANK;
constexpr int GRAM = 2 * MAXR * MAXR;

// Rows handled by one workgroup of the SM pass (4 waves x SM_ROWS_PER_WAVE;
// 8 rows per wave measured 4 % faster than 4 with lazy factors in the mix).
#ifndef MKOR_SM_RPW
#define MKOR_SM_RPW 8
#endif
#ifndef MKOR_SM_NT
#define MKOR_SM_NT 1
#endif
#ifndef MKOR_SM_GRID
#define MKOR_SM_GRID 512
#endif
constexpr int SM_GRID = MKOR_SM_GRID;   // workgroups of the SM pass (0: one per row block)
constexpr int SM_THREADS = 256;
constexpr int SM_ROWS_PER_WAVE = MKOR_SM_RPW;
constexpr int SM_ROWS = (SM_THREADS / 64) * SM_ROWS_PER_WAVE;
// bf16 factors: 8 rows per wave (16 bytes per lane and row), non-temporal
// loads and stores (same-box A/B at the BERT-Large set: 0.793 against 0.819
// ms per pass; 16 rows per wave no faster, 4 rows 0.97 ms)
#ifndef MKOR_SM_RPW_HALF
#define MKOR_SM_RPW_HALF 8
#endif
#ifndef MKOR_SM_NT_HALF
#define MKOR_SM_NT_HALF 1
#endif
constexpr int SM_ROWS_PER_WAVE_HALF = MKOR_SM_RPW_HALF;
constexpr int SM_ROWS_HALF = (SM_THREADS / 64) * SM_ROWS_PER_WAVE_HALF;

struct RowBlock {
    int32_t factor;
    int32_t row0;
};

// ---------------------------------------------------------------- GEMMs
// C = At^T * B for one layer: At is K x M (row-major, M contiguous), B is
// K x N (row-major, N contiguous), C is M x N, stored row-major (ldc = N) or
// transposed (N x M, ldc = M).
struct GemmLayer {
    const float*   At;
    const void*    B;
    float*         C;
    const Pending* pend;      // pending term of the factor operand (At in stage 1, B in stage 2)
    const float*   w;         // its w vector
    int32_t        M, N, K;
    int32_t        b_bf16;    // element type of B
    int32_t        vec;       // rows of At, B and C allow 16-byte vector access
    int32_t        part0;     // first partial-sum slot of this layer
    int32_t        ntn;       // number of N tiles
    int32_t        _pad;
    const int32_t* mode;      // the layer's mode word
};

struct GemmTile {
    int32_t layer;            // -1: padding, the workgroup exits
    int32_t tm, tn;
    int32_t _pad;
};

// Tile shapes of the preconditioning GEMMs, per stage (stage 1: X^T =
// (Linv G)^T, stage 2: dW_hat = X Rinv): a workgroup of wm x wn waves computes
// a bm x bn tile, K in bk-deep slabs, at least minb workgroups per CU.
#ifndef MKOR_GEMM1_SHAPE
#define MKOR_GEMM1_SHAPE 128, 256, 16, 2, 2, 2
#endif
#ifndef MKOR_GEMM2_SHAPE
#define MKOR_GEMM2_SHAPE 256, 128, 16, 2, 2, 2
#endif
struct GemmShape {
    int bm, bn, bk, wm, wn, minb;
    constexpr int threads() const { return wm * wn * 64; }
};
constexpr GemmShape GEMM_SHAPE[2] = {GemmShape{MKOR_GEMM1_SHAPE}, GemmShape{MKOR_GEMM2_SHAPE}};

// Tile scheduling: workgroup b of a launch runs on XCD b % GEMM_XCDS (the
// hardware's round-robin dispatch), and each XCD takes super-tiles of one
// layer covering up to GEMM_SUPER x GEMM_SUPER outputs, so the tiles that run
// together on an XCD share their operand panels in that XCD's L2.  2048: a
// 4096-row layer's first GEMM is two super-tiles of 32 tiles (one per CU of
// an XCD) rather than four of 16, which halves the re-reads of its Q panel by
// other XCDs (1024 and 4096 measured slower).
constexpr int GEMM_XCDS = 8;
#ifndef MKOR_GEMM_SUPER
#define MKOR_GEMM_SUPER 2048
#endif
constexpr int GEMM_SUPER = MKOR_GEMM_SUPER;

// ---------------------------------------------------------------- half factors
// bf16 MFMA GEMMs of layers with bf16 factors (see precond_hgemm.hip).  Both
// stages are  C = P_eff Q^T  with the factor as P (rows i of C) and a data
// matrix as Q (rows j of C), both contiguous along k:
//   stage 1:  Y^T = R G^T        P = S_R, Q = G (bf16), C = Y^T (bf16, d_out x d_in)
//   stage 2:  dW_hat = L Y       P = S_L, Q = Y^T,      C = dW_hat (fp32, d_in x d_out)
// where P_eff = c1 S + c2 I + sgn w w^T is the factor with its pending term.
#ifndef MKOR_HG_BI
#define MKOR_HG_BI 256
#endif
#ifndef MKOR_HG_BJ
#define MKOR_HG_BJ 256
#endif
#ifndef MKOR_HG_NS
#define MKOR_HG_NS 2
#endif
#ifndef MKOR_HG_BK
#define MKOR_HG_BK 64
#endif
// Each wave computes 128 x HG_TJ outputs: 128 (four waves, one per SIMD,
// 256 accumulators each) or 64 (eight waves, two per SIMD, 128 each).
#ifndef MKOR_HG_TJ
#define MKOR_HG_TJ 64
#endif
constexpr int HG_BI = MKOR_HG_BI, HG_BJ = MKOR_HG_BJ;   // tile of C (rows i x columns j)
constexpr int HG_TJ = MKOR_HG_TJ;
constexpr int HG_THREADS = 64 * (HG_BI / 128) * (HG_BJ / HG_TJ);
constexpr int HG_NS = MKOR_HG_NS;                       // stages of the LDS ring
constexpr int SG_BI = 256, SG_BJ = 256;                  // tile of C of the split GEMMs (sgemm)
constexpr int SG_BI1H = 128, SG_BJ1H = 512;              // ... of the first one when Q is bf16
// qdot_kernel blocks: Q rows in multiples of 32 (4 waves x 8 rows per pass),
// as many as make about QD_BYTES of Q, between 32 and QD_MAX_ROWS, so that a
// layer with long rows does not form the tail
#ifndef MKOR_QD_BYTES
#define MKOR_QD_BYTES (512 << 10)
#endif
constexpr int QD_MAX_ROWS = 256;
constexpr int64_t QD_BYTES = MKOR_QD_BYTES;
constexpr int32_t qd_rows(int32_t K, int32_t elem_bytes) {
    const int64_t r = QD_BYTES / ((int64_t)K * elem_bytes) / 32 * 32;
    return r < 32 ? 32 : (r > QD_MAX_ROWS ? QD_MAX_ROWS : (int32_t)r);
}
constexpr int HG_BK = MKOR_HG_BK;                       // k per stage

// Layer descriptor of the bf16-MFMA preconditioning stages (C = P_eff Q^T):
// bf16 factors (hgemm: P, Q bf16; C bf16 in stage 1) and fp32 factors on the
// three-way bf16 split (sgemm: P fp32, Q fp32 or bf16, C fp32).
struct HgLayer {
    const void*    P;      // factor S (I x K)
    const void*    Q;      // J x K
    void*          C;      // I x J
    const Pending* pend;   // pending term of the factor
    const float*   w;      // its w vector (K = I entries)
    int32_t        I, J, K;
    int32_t        part0;  // first partial slot of this layer
    int32_t        ntj;    // number of column tiles
    int32_t        qf32;   // sgemm: Q is fp32 (else bf16)
    int32_t        fq;     // sgemm: the factor is the Q operand, C = P Q_eff^T (else C = P_eff Q^T)
    int32_t        wide;   // sgemm stage 1, bf16 Q: SG_BI1H x SG_BJ1H tiles (else SG_BI x SG_BJ)
    float*         rq;     // sgemm stage 1: (Q w) per Q row, formed by qdot_kernel before the GEMM
    const int32_t* mode;   // the layer's mode word
};

// Rows of the stage-1 Q operand of the split GEMMs, one block of `rows` rows
// per workgroup (qd_rows of the layer): (Q w) for the pending term and the
// ||G||^2 partial
struct QdBlock {
    int32_t layer, rb;     // index into the stage-1 layer table, row block
    int32_t rows;          // rows per block of this layer (a multiple of 32)
};

// bf16 transposes (G^T for the split GEMMs that contract over d_in)
struct TrItem {
    const unsigned short* src;   // rows x cols
    unsigned short*       dst;   // cols x rows
    int32_t               rows, cols;   // multiples of 64
    const int32_t*        mode;         // the layer's mode word
};
struct TrBlock {
    int32_t item, r0, c0, _pad;  // 64 x 64 tile at (r0, c0) of src
};

// fp32 -> bf16 copy of fp32 gradients of bf16-factor layers (the stage-1 Q)
struct CvtItem {
    const float*    src;
    unsigned short* dst;
    int64_t         n;      // elements (a multiple of 8)
    const int32_t*  mode;   // the layer's mode word
};
struct CvtBlock {
    int32_t item, _pad;
    int64_t off;            // first element of this workgroup's range
};
constexpr int CVT_ELEMS = 1 << 16;   // elements per workgroup of the conversion

hipError_t launch_sgemm(int stage, const HgLayer* layers, const GemmTile* tiles, int32_t ntiles,
                        float* partials, hipStream_t stream);
hipError_t launch_qdot(const HgLayer* layers, const QdBlock* blocks, int32_t nblocks, float* partials,
                       hipStream_t stream);
hipError_t launch_transpose_bf16(const TrItem* items, const TrBlock* blocks, int32_t nblocks, hipStream_t stream);
hipError_t launch_hgemm(int stage, const HgLayer* layers, const GemmTile* tiles, int32_t ntiles,
                        float* partials, hipStream_t stream);
hipError_t launch_cvt_bf16(const CvtItem* items, const CvtBlock* blocks, int32_t nblocks, hipStream_t stream);

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
    int32_t           nblk;             // rescale blocks of this layer
    float*            W;                // backend optimizer state (null when unused)
    float*            m;
    float*            v;
    const int32_t*    mode;             // the layer's mode word
};

// Backend optimizer fused with the rescale (host-computed scalars).
struct OptArgs {
    int32_t kind;            // MKOR_OPT_SGD or MKOR_OPT_LAMB
    int32_t store_dw;
    float   lr, mom, b1, b2, eps, wd;
    float   bc1, bc2;        // 1 / (1 - b1^t), 1 / (1 - b2^t)
};

#ifndef MKOR_RS_GRID
#define MKOR_RS_GRID 1024
#endif
constexpr int RS_THREADS = 256;
constexpr int RS_GRID = MKOR_RS_GRID;   // workgroups of the rescale (0: one per block)
#ifndef MKOR_RS_ELEMS
#define MKOR_RS_ELEMS 8192
#endif
constexpr int RS_ELEMS = MKOR_RS_ELEMS;   // elements per rescale block

struct RescaleBlock {
    int32_t layer;
    int32_t _pad;
    int64_t start;
};

// ---------------------------------------------------------------- launchers
// Each returns the hipError_t of its launch.
// a = mean of the rows of A, g = mean of the rows of Gout (Algorithm 1, the
// rank-1 approximation lines): partial sums per (matrix, column chunk, row
// block), then one fixed-order combine per column.
hipError_t launch_colmean(const MeanMat* mats, const MeanItem* items, int32_t nitems,
                          const MeanItem* chunks, int32_t nchunks, double* part, hipStream_t stream);

// Streaming pass over every factor: applies the pending term in place (when
// there is one) and, with matvec = 1, forms u_raw = P x, the row norms and the
// per-row-block partials of the current P.
// ranked: the plan has rank-r factors (their blocks run in a kernel of their own)
hipError_t launch_sm_pass(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                          float4* partials, float* gram, int32_t norm_kind, int32_t matvec, int32_t ranked,
                          hipStream_t stream);
// writes the pending rank-r terms into the rank-r factors and clears them
hipError_t launch_sm_apply_rank(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                                int32_t nfactors, hipStream_t stream);

// One workgroup per factor: stabiliser decision and update coefficients from
// the pass partials, new pending term (coefficients and w), stats.
hipError_t launch_sm_finalize(const FactorDesc* factors, int32_t nfactors, const float4* partials,
                              const float* gram, const mkor_params& p, hipStream_t stream);

// Marks every pending term applied (after a materialising pass).
hipError_t launch_sm_reset(const FactorDesc* factors, int32_t nfactors, hipStream_t stream);

// Sets the mode words mode[first .. first + count) from bit i of `bits`
// (count <= MODE_CHUNK), stream-ordered.
constexpr int MODE_CHUNK = 1024;
hipError_t launch_set_modes(int32_t* mode, int32_t first, int32_t count, const uint32_t* bits,
                            hipStream_t stream);

// GEMM 1: X^T = (Linv G)^T, plus ||G||^2 partials from the tiles of the first M row.
hipError_t launch_gemm_xt(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream);
// GEMM 2: dW_hat = X Rinv, plus one ||dW_hat||^2 partial per tile.
hipError_t launch_gemm_dw(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                          float* partials, hipStream_t stream);

// Rescale fused with the optimizer: pass A (scale, moments, SGD step or LAMB
// norm partials), then for LAMB the per-layer ratio and pass B (weight step).
hipError_t launch_rescale_opt(const RescaleLayer* layers, int32_t nlayers, const RescaleBlock* blocks,
                              int32_t nblocks, const float* gpart, const float* dpart, int32_t rescale,
                              const OptArgs& opt, float2* lpart, float* trust, hipStream_t stream);
hipError_t launch_rescale(const RescaleLayer* layers, const RescaleBlock* blocks, int32_t nblocks,
                          const float* gpart, const float* dpart, int32_t rescale,
                          hipStream_t stream);

}  // namespace mkor
