// Rank-1 approximation vectors of Algorithm 1 (its first two lines, and the
// "Rank-1 Approximation" paragraph): a = mean of the layer's activation rows,
// g = mean of its output-gradient rows, i.e. the column means of the row-major
// rows x d matrices A and Gout.
//
// Two grouped launches over every such matrix of the plan:
//
//   colmean_partial_kernel  one workgroup per (matrix, MEAN_COLS-column
//                           chunk, block of rpb rows): each thread sums its
//                           MEAN_COLS / 64 contiguous columns over the block's
//                           rows (one row per wave and step: with 512 columns
//                           a wave reads 1 KB (bf16) or 2 KB (fp32) of a row
//                           at a time) in float64, the four waves are combined
//                           in a fixed order, and the block's partial sums are
//                           stored.
//   colmean_final_kernel    one thread per column: sums the row-block partials
//                           in a fixed order and stores sum / rows as fp32.
//
// The stream is read-only and HBM-bound, so the float64 accumulation costs no
// time; it makes the result the float64 mean rounded once to fp32, and the
// fixed orders make it deterministic.
#include "gmem.h"
#include "mkor_internal.h"

namespace mkor {
namespace {

constexpr int MT = MEAN_THREADS;
constexpr int MW = MT / 64;

__device__ __forceinline__ void acc_bf16x2(double& lo, double& hi, unsigned h) {
    lo += (double)__uint_as_float(h << 16);
    hi += (double)__uint_as_float(h & 0xffff0000u);
}

__global__ __launch_bounds__(MT) void colmean_partial_kernel(const MeanMat* __restrict__ mats,
                                                             const MeanItem* __restrict__ items,
                                                             double* __restrict__ part) {
    const MeanItem it = items[blockIdx.x];
    const MeanMat m = mats[it.mat];
    if (!gld_i32(m.mode)) return;   // first-order layer: no means (block-uniform)
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    constexpr int CPT = MEAN_COLS / 64;                // columns per thread
    static_assert(CPT % 8 == 0, "whole 16-byte bf16 loads per lane");
    const int c0 = it.chunk * MEAN_COLS + CPT * lane;  // this thread's columns
    const int r0 = it.rb * m.rpb;
    const int r1 = min(r0 + m.rpb, m.rows);
    double s[CPT];
#pragma unroll
    for (int e = 0; e < CPT; ++e) s[e] = 0.0;
    if (m.vec && c0 + CPT - 1 < m.cols) {
        // each row is read once: streaming (non-temporal) loads, 8 rows in
        // flight per wave
        if (m.bf16) {
            // 8 bf16 = 16 bytes per load: a wave reads MEAN_COLS * 2 bytes of a row at a time
            const unsigned short* X = static_cast<const unsigned short*>(m.X) + c0;
#pragma unroll 8
            for (int r = r0 + wave; r < r1; r += MW) {
#pragma unroll
                for (int l = 0; l < CPT / 8; ++l) {
                    const uint4 h = gld_u4_nt(X + (size_t)r * m.cols + 8 * l);
                    acc_bf16x2(s[8 * l + 0], s[8 * l + 1], h.x);
                    acc_bf16x2(s[8 * l + 2], s[8 * l + 3], h.y);
                    acc_bf16x2(s[8 * l + 4], s[8 * l + 5], h.z);
                    acc_bf16x2(s[8 * l + 6], s[8 * l + 7], h.w);
                }
            }
        } else {
            const float* X = static_cast<const float*>(m.X) + c0;
#pragma unroll 8
            for (int r = r0 + wave; r < r1; r += MW) {
#pragma unroll
                for (int l = 0; l < CPT / 4; ++l) {
                    const float4 v = gld4_nt(X + (size_t)r * m.cols + 4 * l);
                    s[4 * l + 0] += (double)v.x; s[4 * l + 1] += (double)v.y;
                    s[4 * l + 2] += (double)v.z; s[4 * l + 3] += (double)v.w;
                }
            }
        }
    } else {
        // ragged: any column count, element by element
        for (int r = r0 + wave; r < r1; r += MW) {
#pragma unroll
            for (int e = 0; e < CPT; ++e) {
                const int c = c0 + e;
                if (c < m.cols) {
                    const size_t off = (size_t)r * m.cols + c;
                    s[e] += m.bf16 ? (double)__uint_as_float(
                                         ((unsigned)gld_u16(static_cast<const unsigned short*>(m.X) + off)) << 16)
                                   : (double)gld(static_cast<const float*>(m.X) + off);
                }
            }
        }
    }
    __shared__ double red[MW][MEAN_COLS];
#pragma unroll
    for (int e = 0; e < CPT; ++e) red[wave][CPT * lane + e] = s[e];
    __syncthreads();
    // partial slot of this block: part0 + (rb * nchunk + chunk) * MEAN_COLS
    double* dst = part + m.part0 + ((size_t)it.rb * m.nchunk + it.chunk) * MEAN_COLS;
    for (int c = t; c < MEAN_COLS; c += MT) {
        double acc = red[0][c];
#pragma unroll
        for (int w = 1; w < MW; ++w) acc += red[w][c];
        dst[c] = acc;
    }
}

__global__ __launch_bounds__(MEAN_COLS) void colmean_final_kernel(const MeanMat* __restrict__ mats,
                                                                  const MeanItem* __restrict__ chunks,
                                                                  const double* __restrict__ part) {
    const MeanItem ch = chunks[blockIdx.x];
    const MeanMat m = mats[ch.mat];
    if (!gld_i32(m.mode)) return;
    const int c = ch.chunk * MEAN_COLS + threadIdx.x;
    if (c >= m.cols) return;
    const double* p = part + m.part0 + (size_t)ch.chunk * MEAN_COLS + threadIdx.x;
    double acc = 0.0;
    for (int rb = 0; rb < m.nrb; ++rb) acc += p[(size_t)rb * m.nchunk * MEAN_COLS];
    gst(m.out + c, (float)(acc / (double)m.rows));
}

}  // namespace

hipError_t launch_colmean(const MeanMat* mats, const MeanItem* items, int32_t nitems,
                          const MeanItem* chunks, int32_t nchunks, double* part, hipStream_t stream) {
    if (nitems <= 0) return hipSuccess;
    hipLaunchKernelGGL(colmean_partial_kernel, dim3(nitems), dim3(MT), 0, stream, mats, items, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(colmean_final_kernel, dim3(nchunks), dim3(MEAN_COLS), 0, stream, mats, chunks, part);
    return hipGetLastError();
}

}  // namespace mkor
