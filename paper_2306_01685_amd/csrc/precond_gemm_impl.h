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
// The factor operand (Linv in stage 1, Rinv in stage 2) is the caller buffer S
// plus the pending rank-1 term of the SM update (struct Pending).  The stores
// into LDS apply that term element by element with the same pinned roundings
// as the SM pass, so the GEMMs multiply with the current factor without it
// being written first; doing it on the store side keeps the arithmetic off
// the path between a global load and the MFMAs that overlap it.
//
// A workgroup of WM x WN waves computes a BM x BN tile (GEMM_SHAPE of the
// stage); each wave owns a (BM / WM) x (BN / WN) sub-tile of 32 x 32 blocks of
// v_mfma_f32_32x32x2_f32.  K advances in BK-deep slabs, double-buffered in
// LDS; the next slab's global loads are issued before the current slab's
// MFMAs and stored after them.  The grid is one grouped launch over a tile
// table that the host orders for the XCDs (see the plan code).
//
// This file is the implementation of one stage: it is included by
// precond_gemm_xt.hip (MKOR_GEMM_STAGE 1) and precond_gemm_dw.hip
// (MKOR_GEMM_STAGE 2), so each stage is compiled with its own tile shape.
#ifndef MKOR_GEMM_STAGE
#error "define MKOR_GEMM_STAGE (1 or 2) before including this file"
#endif
#include "gmem.h"
#include "mkor_internal.h"

namespace mkor {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int STAGE_OF_TU = MKOR_GEMM_STAGE;
constexpr GemmShape SHP = GEMM_SHAPE[STAGE_OF_TU - 1];
constexpr int BM = SHP.bm, BN = SHP.bn, BK = SHP.bk;
constexpr int WM = SHP.wm, WN = SHP.wn;
constexpr int NT = SHP.threads();
constexpr int TM = BM / WM, TN = BN / WN;   // wave sub-tile
constexpr int FM = TM / 32, FN = TN / 32;   // 32 x 32 MFMA blocks per wave
constexpr int AC4 = BM / 4, BC4 = BN / 4, BC8 = BN / 8;   // vectors per slab row
constexpr int A4 = BK * BM / 4 / NT;        // float4 of At per thread and slab
constexpr int B4 = BK * BN / 4 / NT;        // float4 of fp32 B per thread and slab
constexpr int B8 = BK * BN / 8 / NT;        // 2 x 4 bf16 of B per thread and slab
// ds_read2_b32 instructions per k-step: the FM (FN) operands of a wave are
// 32 floats apart, two per instruction
constexpr int DS_PER_K = (FM + 1) / 2 + (FN + 1) / 2;
static_assert(NT == WM * WN * 64, "one wave per sub-tile");
static_assert(TM % 32 == 0 && TN % 32 == 0 && BK % 2 == 0, "tile shape");
static_assert(A4 * NT * 4 == BK * BM && B4 * NT * 4 == BK * BN && B8 * NT * 8 == BK * BN,
              "slab divides evenly among the threads");
static_assert(NT % AC4 == 0 && NT % BC4 == 0 && NT % BC8 == 0,
              "a thread stages the same columns in every slab");

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

// Pending rank-1 term of the factor operand.  swc = sgn * w of the columns this
// thread stages (fixed for a tile in the vector paths); multiplying by sgn = +-1
// is exact, so sgn * (w_k * w_c) = w_k * (sgn * w_c) bit for bit.
struct Xform {
    float c1, c2, sgn;
    const float* w;
    float4 swc;
};

// Element (k, c) of the current factor from stored value v: see Pending.
// DIAG: the element may lie on the diagonal (k == c is checked).
template <bool DIAG>
__device__ __forceinline__ float xf1(const Xform& x, float v, float wk, float swc, int k, int c) {
    v = __fmaf_rn(x.c1, v, __fmul_rn(wk, swc));
    if (DIAG && k == c) v = __fadd_rn(v, x.c2);
    return v;
}

template <bool DIAG>
__device__ __forceinline__ float4 xf4(const Xform& x, float4 v, float wk, int k, int c) {
    v.x = xf1<DIAG>(x, v.x, wk, x.swc.x, k, c + 0);
    v.y = xf1<DIAG>(x, v.y, wk, x.swc.y, k, c + 1);
    v.z = xf1<DIAG>(x, v.z, wk, x.swc.z, k, c + 2);
    v.w = xf1<DIAG>(x, v.w, wk, x.swc.w, k, c + 3);
    return v;
}

__device__ __forceinline__ void sq4(float& acc, const float4& v) {
    acc = fmaf(v.x, v.x, acc);
    acc = fmaf(v.y, v.y, acc);
    acc = fmaf(v.z, v.z, acc);
    acc = fmaf(v.w, v.w, acc);
}

// Register staging of one K slab (vector paths).  wk holds w of the slab rows
// this thread stages when the pending term is applied.
template <bool BF16>
struct SlabRegs {
    float4 a[A4];
    float4 b[B4];
    float  wk[A4 > B4 ? A4 : B4];
};
template <>
struct SlabRegs<true> {
    float4 a[A4];
    uint2  h[2 * B8];   // 4 bf16 of the left half of the tile, 4 of the right half
    float  wk[A4];
};

// XF: 0 = plain operands, 1 = apply the pending term to At, 2 = to B (fp32).
// FULL: the tile lies inside the matrices and K is a multiple of BK, so the
// vector paths need no range checks.  Partial tiles load from a clamped (valid)
// address and zero the out-of-range values at store time, which keeps the
// loads unconditional and lets them all be in flight during the MFMAs.
template <bool BF16, bool VEC, bool FULL, int XF>
struct Loader {
    // Vector paths: global -> registers, issued before the slab's MFMAs.  In
    // interior tiles every address is a uniform slab base plus a per-thread
    // 32-bit offset that does not change from slab to slab.
    __device__ static void load(SlabRegs<BF16>& r, const GemmLayer& L, int m0, int n0, int k0) {
        if constexpr (VEC) {
            const int t = threadIdx.x;
            const int m = m0 + 4 * (t % AC4);
            if constexpr (FULL) {
                const float* Ab = L.At + (size_t)k0 * L.M + m0;
#pragma unroll
                for (int i = 0; i < A4; ++i) {
                    const unsigned row = (unsigned)((t + i * NT) / AC4);
                    r.a[i] = gld4_off(Ab, 4u * (row * (unsigned)L.M + 4u * (t % AC4)));
                    if constexpr (XF == 1) r.wk[i] = gld_off(L.w + k0, 4u * row);
                }
            } else {
#pragma unroll
                for (int i = 0; i < A4; ++i) {
                    const int k = k0 + (t + i * NT) / AC4;
                    const bool ok = k < L.K && m < L.M;
                    r.a[i] = gld4(L.At + (ok ? (size_t)k * L.M + m : 0));
                    if constexpr (XF == 1) r.wk[i] = gld(L.w + (ok ? k : 0));
                }
            }
            if constexpr (!BF16) {
                const int n = n0 + 4 * (t % BC4);
                const float* B = static_cast<const float*>(L.B);
                const float* Bb = B + (size_t)k0 * L.N + n0;
#pragma unroll
                for (int i = 0; i < B4; ++i) {
                    const int row = (t + i * NT) / BC4;
                    if constexpr (FULL) {
                        r.b[i] = gld4_off(Bb, 4u * ((unsigned)row * (unsigned)L.N + 4u * (t % BC4)));
                        if constexpr (XF == 2) r.wk[i] = gld_off(L.w + k0, 4u * (unsigned)row);
                    } else {
                        const int k = k0 + row;
                        const bool ok = k < L.K && n < L.N;
                        r.b[i] = gld4(B + (ok ? (size_t)k * L.N + n : 0));
                        if constexpr (XF == 2) r.wk[i] = gld(L.w + (ok ? k : 0));
                    }
                }
            } else {
                // columns n and n + BN / 2, so that the LDS stores of a wave
                // are contiguous (no bank conflicts)
                const int n = n0 + 4 * (t % BC8);
                const unsigned short* B = static_cast<const unsigned short*>(L.B);
                const unsigned short* Bb = B + (size_t)k0 * L.N + n0;
#pragma unroll
                for (int i = 0; i < B8; ++i) {
                    const int row = (t + i * NT) / BC8;
                    if constexpr (FULL) {
                        const unsigned off = 2u * ((unsigned)row * (unsigned)L.N + 4u * (t % BC8));
                        r.h[2 * i] = gld_u2_off(Bb, off);
                        r.h[2 * i + 1] = gld_u2_off(Bb, off + BN);
                    } else {
                        const int k = k0 + row;
                        const bool ok0 = k < L.K && n < L.N;
                        const bool ok1 = k < L.K && n + BN / 2 < L.N;
                        r.h[2 * i] = gld_u2(B + (ok0 ? (size_t)k * L.N + n : 0));
                        r.h[2 * i + 1] = gld_u2(B + (ok1 ? (size_t)k * L.N + n + BN / 2 : 0));
                    }
                }
            }
        }
    }

    // Registers -> LDS after the MFMAs (vector paths; range masking, the
    // pending term and the bf16 upcast are applied here), or global -> LDS
    // directly (scalar path for ragged sizes).  DIAG: the slab may hold
    // diagonal elements of the factor operand.
    template <bool DIAG>
    __device__ static void store(const SlabRegs<BF16>& r, const GemmLayer& L, const Xform& xf,
                                 int m0, int n0, int k0, float* As, float* Bs, double& gsq,
                                 bool want_gsq) {
        const int t = threadIdx.x;
        float part = 0.f;   // this slab's squares: a short fp32 chain, added to gsq in fp64
        const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
        if constexpr (VEC) {
            const int ca = 4 * (t % AC4);
#pragma unroll
            for (int i = 0; i < A4; ++i) {
                const int row = (t + i * NT) / AC4;
                const int k = k0 + row, m = m0 + ca;
                const bool ok = FULL || (k < L.K && m < L.M);
                float4 v = ok ? r.a[i] : zero;
                if constexpr (XF == 1) {
                    if (ok) v = xf4<DIAG>(xf, v, r.wk[i], k, m);
                }
                *reinterpret_cast<float4*>(As + row * BM + ca) = v;
            }
            if constexpr (!BF16) {
                const int cb = 4 * (t % BC4);
#pragma unroll
                for (int i = 0; i < B4; ++i) {
                    const int row = (t + i * NT) / BC4;
                    const int k = k0 + row, n = n0 + cb;
                    const bool ok = FULL || (k < L.K && n < L.N);
                    float4 v = ok ? r.b[i] : zero;
                    if constexpr (XF == 2) {
                        if (ok) v = xf4<DIAG>(xf, v, r.wk[i], k, n);
                    }
                    if (want_gsq) sq4(part, v);
                    *reinterpret_cast<float4*>(Bs + row * BN + cb) = v;
                }
            } else {
                const int cb = 4 * (t % BC8);
#pragma unroll
                for (int i = 0; i < B8; ++i) {
                    const int row = (t + i * NT) / BC8;
                    const int k = k0 + row, n = n0 + cb;
                    const bool ok0 = FULL || (k < L.K && n < L.N);
                    const bool ok1 = FULL || (k < L.K && n + BN / 2 < L.N);
                    const uint2 h0 = ok0 ? r.h[2 * i] : make_uint2(0u, 0u);
                    const uint2 h1 = ok1 ? r.h[2 * i + 1] : make_uint2(0u, 0u);
                    const float4 v0 = make_float4(
                        __uint_as_float(h0.x << 16), __uint_as_float(h0.x & 0xffff0000u),
                        __uint_as_float(h0.y << 16), __uint_as_float(h0.y & 0xffff0000u));
                    const float4 v1 = make_float4(
                        __uint_as_float(h1.x << 16), __uint_as_float(h1.x & 0xffff0000u),
                        __uint_as_float(h1.y << 16), __uint_as_float(h1.y & 0xffff0000u));
                    if (want_gsq) { sq4(part, v0); sq4(part, v1); }
                    *reinterpret_cast<float4*>(Bs + row * BN + cb) = v0;
                    *reinterpret_cast<float4*>(Bs + row * BN + cb + BN / 2) = v1;
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < (BK * BM) / NT; ++i) {
                const int idx = t + i * NT;
                const int row = idx / BM, col = idx % BM;
                const int k = k0 + row, m = m0 + col;
                float v = 0.f;
                if (k < L.K && m < L.M) {
                    v = gld(L.At + (size_t)k * L.M + m);
                    if constexpr (XF == 1) v = xf1<true>(xf, v, gld(xf.w + k), xf.sgn * gld(xf.w + m), k, m);
                }
                As[row * BM + col] = v;
            }
#pragma unroll
            for (int i = 0; i < (BK * BN) / NT; ++i) {
                const int idx = t + i * NT;
                const int row = idx / BN, col = idx % BN;
                const int k = k0 + row, n = n0 + col;
                float v = 0.f;
                if (k < L.K && n < L.N) {
                    const size_t off = (size_t)k * L.N + n;
                    v = BF16 ? bf16_to_f32(gld_u16(static_cast<const unsigned short*>(L.B) + off))
                             : gld(static_cast<const float*>(L.B) + off);
                    if constexpr (XF == 2) v = xf1<true>(xf, v, gld(xf.w + k), xf.sgn * gld(xf.w + n), k, n);
                }
                if (want_gsq) part = fmaf(v, v, part);
                Bs[row * BN + col] = v;
            }
        }
        if (want_gsq) gsq += (double)part;
    }
};

// MFMAs of one K slab held in LDS (As: BK x BM, Bs: BK x BN).  With OP_DB the
// operands of k-step kk + 1 are read before the MFMAs of k-step kk are issued,
// so the LDS latency overlaps those MFMAs (the caller pins that order with
// sched_barriers_slab in the same basic block); without it, each k-step reads
// its own operands (fewer live registers; enough when a k-step has many MFMAs).
#ifndef MKOR_GEMM_OPDB
#define MKOR_GEMM_OPDB (FM * FN < 8)
#endif
constexpr bool OP_DB = MKOR_GEMM_OPDB;

__device__ __forceinline__ void mma_slab(floatx16 (&acc)[FM][FN], const float* As, const float* Bs,
                                         int wm, int wn, int li, int lk) {
    const float* Aw = As + wm * TM + li + lk * BM;
    const float* Bw = Bs + wn * TN + li + lk * BN;
    if constexpr (OP_DB) {
        float a[2][FM], b[2][FN];
#pragma unroll
        for (int i = 0; i < FM; ++i) a[0][i] = Aw[i * 32];
#pragma unroll
        for (int j = 0; j < FN; ++j) b[0][j] = Bw[j * 32];
#pragma unroll
        for (int kk = 0; kk < BK / 2; ++kk) {
            const int cur = kk & 1, nxt = cur ^ 1;
            if (kk + 1 < BK / 2) {
#pragma unroll
                for (int i = 0; i < FM; ++i) a[nxt][i] = Aw[(2 * kk + 2) * BM + i * 32];
#pragma unroll
                for (int j = 0; j < FN; ++j) b[nxt][j] = Bw[(2 * kk + 2) * BN + j * 32];
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[cur][i], b[cur][j], acc[i][j], 0, 0, 0);
        }
    } else {
#pragma unroll
        for (int kk = 0; kk < BK / 2; ++kk) {
            float a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) a[i] = Aw[2 * kk * BM + i * 32];
#pragma unroll
            for (int j = 0; j < FN; ++j) b[j] = Bw[2 * kk * BN + j * 32];
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }
}

// Schedule of one slab's MFMA block.  OP_DB: reads of k-steps 0 and 1, MFMAs
// of 0, reads of 2, MFMAs of 1, ..., MFMAs of the last k-step; otherwise the
// reads of each k-step right before its MFMAs.
__device__ __forceinline__ void sched_barriers_slab() {
    constexpr int KS = BK / 2;
    if constexpr (OP_DB) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * DS_PER_K, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
#pragma unroll
        for (int kk = 1; kk + 1 < KS; ++kk) {
            __builtin_amdgcn_sched_group_barrier(0x100, DS_PER_K, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
    } else {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            __builtin_amdgcn_sched_group_barrier(0x100, DS_PER_K, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
        }
    }
}

// Stores the accumulators of one tile and its norm partials.  Output element
// (i, j) of block (mi, ni) of a wave: i = 8 * (r / 4) + 4 * (lane / 32) + r % 4,
// j = lane % 32.
template <bool VEC, int STAGE>
__device__ __forceinline__ void tile_epilogue(const GemmLayer& L, const GemmTile& tile,
                                              const floatx16 (&acc)[FM][FN], float gsq,
                                              bool want_gsq, float* partials, float* red) {
    const int m0 = tile.tm * BM, n0 = tile.tn * BN;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wave % WM, wn = wave / WM;
    const int li = lane & 31, lk = lane >> 5;
    float csq = 0.f;
#pragma unroll
    for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
            const int n = n0 + wn * TN + ni * 32 + li;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int mb = m0 + wm * TM + mi * 32 + 8 * g + 4 * lk;
                const float v0 = acc[mi][ni][4 * g + 0], v1 = acc[mi][ni][4 * g + 1];
                const float v2 = acc[mi][ni][4 * g + 2], v3 = acc[mi][ni][4 * g + 3];
                if constexpr (STAGE == 1) {
                    // C stored transposed: X^T[n][m], leading dimension M
                    if (n < L.N) {
                        float* dst = L.C + (size_t)n * L.M + mb;
                        if (VEC && mb + 3 < L.M) {
                            gst4(dst, make_float4(v0, v1, v2, v3));
                        } else {
                            if (mb + 0 < L.M) gst(dst + 0, v0);
                            if (mb + 1 < L.M) gst(dst + 1, v1);
                            if (mb + 2 < L.M) gst(dst + 2, v2);
                            if (mb + 3 < L.M) gst(dst + 3, v3);
                        }
                    }
                } else {
                    if (n < L.N) {
                        float* dst = L.C + (size_t)mb * L.N + n;
                        if (mb + 0 < L.M) { gst(dst, v0); csq = fmaf(v0, v0, csq); }
                        if (mb + 1 < L.M) { gst(dst + (size_t)L.N, v1); csq = fmaf(v1, v1, csq); }
                        if (mb + 2 < L.M) { gst(dst + 2 * (size_t)L.N, v2); csq = fmaf(v2, v2, csq); }
                        if (mb + 3 < L.M) { gst(dst + 3 * (size_t)L.N, v3); csq = fmaf(v3, v3, csq); }
                    }
                }
            }
        }
    }

    if constexpr (STAGE == 1) {
        if (want_gsq) {
            const float s = block_sum(gsq, red);
            if (threadIdx.x == 0) gst(partials + L.part0 + tile.tn, s);
        }
    } else {
        const float s = block_sum(csq, red);
        if (threadIdx.x == 0) gst(partials + L.part0 + tile.tm * L.ntn + tile.tn, s);
    }
}


template <bool BF16, bool VEC, bool FULL, int STAGE, int XF>
__device__ void gemm_tile(const GemmLayer& L, const GemmTile& tile, const Pending& q,
                          float* partials, float* smem) {
    using Ld = Loader<BF16, VEC, FULL, XF>;
    using Regs = SlabRegs<BF16>;
    float* As0 = smem;
    float* Bs0 = smem + BK * BM;
    float* As1 = smem + BK * (BM + BN);
    float* Bs1 = As1 + BK * BM;
    float* red = smem + 2 * BK * (BM + BN);

    const int m0 = tile.tm * BM, n0 = tile.tn * BN;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wave % WM, wn = wave / WM;
    const int li = lane & 31, lk = lane >> 5;
    const bool want_gsq = (STAGE == 1) && tile.tm == 0;

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    Xform xf{q.c1, q.c2, q.sgn, L.w, make_float4(0.f, 0.f, 0.f, 0.f)};
    if constexpr (XF != 0 && VEC) {
        // the columns this thread stages are fixed for the tile
        const int c = XF == 1 ? m0 + 4 * (threadIdx.x % AC4) : n0 + 4 * (threadIdx.x % BC4);
        if (c < (XF == 1 ? L.M : L.N)) {
            const float4 w = gld4(L.w + c);
            xf.swc = make_float4(q.sgn * w.x, q.sgn * w.y, q.sgn * w.z, q.sgn * w.w);
        }
    }
    // does slab [k0, k0 + BK) of the factor operand cross its diagonal?
    auto diag_of = [&](int k0) -> bool {
        if constexpr (XF == 0) return false;
        if constexpr (!FULL) return true;
        const int c0 = XF == 1 ? m0 : n0;
        const int cw = XF == 1 ? BM : BN;
        return k0 < c0 + cw && c0 < k0 + BK;
    };

    // ||G||^2 over this thread's share of the whole K range: per-slab fp32
    // sums accumulated in fp64 (one fp32 chain over thousands of positive
    // terms drifts low by several 1e-6 relative, a bias the rescale would
    // carry into every element of dW)
    double gsq = 0.0;
    const int nslab = (L.K + BK - 1) / BK;

    Regs regs;
    Ld::load(regs, L, m0, n0, 0);
    if (diag_of(0)) Ld::template store<true>(regs, L, xf, m0, n0, 0, As0, Bs0, gsq, want_gsq);
    else            Ld::template store<false>(regs, L, xf, m0, n0, 0, As0, Bs0, gsq, want_gsq);
    __syncthreads();
    for (int s = 0; s < nslab; ++s) {
        const float* As = (s & 1) ? As1 : As0;
        const float* Bs = (s & 1) ? Bs1 : Bs0;
        float* An = (s & 1) ? As0 : As1;
        float* Bn = (s & 1) ? Bs0 : Bs1;
        const bool more = s + 1 < nslab;
        if (more) Ld::load(regs, L, m0, n0, (s + 1) * BK);
        mma_slab(acc, As, Bs, wm, wn, li, lk);
        sched_barriers_slab();
        // the other buffer was last read in slab s - 1, before the barrier
        if (more) {
            if (diag_of((s + 1) * BK))
                Ld::template store<true>(regs, L, xf, m0, n0, (s + 1) * BK, An, Bn, gsq, want_gsq);
            else
                Ld::template store<false>(regs, L, xf, m0, n0, (s + 1) * BK, An, Bn, gsq, want_gsq);
        }
        __syncthreads();
    }

    tile_epilogue<VEC, STAGE>(L, tile, acc, (float)gsq, want_gsq, partials, red);
}

constexpr int SMEM_BYTES = 4 * (2 * BK * (BM + BN) + NT / 64);

template <bool BF16, int STAGE, int XF>
__device__ __forceinline__ void run_tile_dt(const GemmLayer& L, const GemmTile& tile,
                                            const Pending& q, float* partials, float* smem) {
    if (L.vec) {
        const bool full = (tile.tm + 1) * BM <= L.M && (tile.tn + 1) * BN <= L.N && L.K % BK == 0;
        if (full) gemm_tile<BF16, true, true, STAGE, XF>(L, tile, q, partials, smem);
        else      gemm_tile<BF16, true, false, STAGE, XF>(L, tile, q, partials, smem);
    } else {
        gemm_tile<BF16, false, false, STAGE, XF>(L, tile, q, partials, smem);
    }
}

// Stage 2's B operand is always fp32 (Rinv), so only stage 1 has bf16 variants.
template <int STAGE, int XF>
__device__ __forceinline__ void run_tile(const GemmLayer& L, const GemmTile& tile, const Pending& q,
                                         float* partials, float* smem) {
    if constexpr (STAGE == 1) {
        if (L.b_bf16) {
            run_tile_dt<true, STAGE, XF>(L, tile, q, partials, smem);
            return;
        }
    }
    run_tile_dt<false, STAGE, XF>(L, tile, q, partials, smem);
}

template <int STAGE>
__global__ __launch_bounds__(NT, SHP.minb) void gemm_kernel(
    const GemmLayer* __restrict__ layers, const GemmTile* __restrict__ tiles,
    float* __restrict__ partials) {
    __shared__ __attribute__((aligned(16))) float smem[SMEM_BYTES / 4];
    const GemmTile tile = tiles[blockIdx.x];
    if (tile.layer < 0) return;   // padding of the XCD interleave
    const GemmLayer L = layers[tile.layer];
    if (!gld_i32(L.mode)) return;   // first-order layer this step
    const Pending q = *L.pend;
    // the factor operand is At in stage 1 and B in stage 2
    if (q.has) run_tile<STAGE, STAGE>(L, tile, q, partials, smem);
    else       run_tile<STAGE, 0>(L, tile, q, partials, smem);
}

template <int STAGE>
hipError_t launch_stage(const GemmLayer* layers, const GemmTile* tiles, int32_t ntiles,
                        float* partials, hipStream_t stream) {
    static_assert(STAGE == STAGE_OF_TU, "each translation unit launches its own stage");
    if (ntiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(gemm_kernel<STAGE>, dim3(ntiles), dim3(NT), 0, stream, layers, tiles, partials);
    return hipGetLastError();
}

}  // namespace
}  // namespace mkor
