// Grouped momentum Sherman-Morrison update of all inverse factors
// (Algorithm 1: norm-based stabilisation, then SM-based factor inversion;
// Eq. 4-7, Eq. 9-11), as one streaming pass per step.
//
// The update P_t = c1 P_hat + ... needs u = P_hat x over the whole of P before
// any element of P_t can be written, so an update that writes P_t in the same
// step reads P twice.  Here each factor is carried as its buffer S plus one
// pending rank-1 term (struct Pending), and a step is:
//
//   sm_pass_kernel      one read + one write of S: applies the previous
//                       step's pending term (S <- P_{t-1}), and over those
//                       values forms u_raw = P_{t-1} x_t (row dot products,
//                       wave-shuffle reductions), the row absolute sums (or
//                       max |entry|) and per-row-block partials
//                       {norm max, sum x_i u_raw_i, sum x_i^2}.
//   sm_finalize_kernel  one workgroup per factor reduces the partials in a
//                       fixed order, takes the stabiliser decision, and stores
//                       the new pending term  P_t = c1 S + c2 I + sgn w w^T.
//
// The preconditioning GEMMs apply the pending term in their operand loads, so
// they multiply with P_t itself; the next step's pass writes the same values
// into S.  8 bytes of HBM traffic per factor element and step, the minimum
// for reading and rewriting a dense fp32 factor.
//
// The stabiliser blend P_hat = zeta P + (1 - zeta) I is never materialised: it
// is folded into u = zeta u_raw + (1 - zeta) x, s = zeta x^T u_raw +
// (1 - zeta) x^T x and the coefficients c1, c2.  The rank-1 term is written as
// sgn * w_i * w_j with w = sqrt(|c3|) u, so (i,j) and (j,i) round identically
// and a symmetric factor stays bitwise symmetric.
#include "gmem.h"
#include "mkor_internal.h"

#include <math.h>

namespace mkor {
namespace {

__device__ __forceinline__ float nanmax(float a, float b) {
    return (a != a || b != b) ? __builtin_nanf("") : fmaxf(a, b);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ float wave_nanmax(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = nanmax(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ float absacc(float acc, float v, int maxabs) {
    return maxabs ? nanmax(acc, fabsf(v)) : acc + fabsf(v);
}

// Off-diagonal part of one element of the current factor (see Pending).
__device__ __forceinline__ float apply(const Pending& q, float s, float wi, float wj) {
    return __fmaf_rn(q.c1, s, q.sgn * __fmul_rn(wi, wj));
}
// The second of two terms, applied to the value after the first (with its
// diagonal c2 added): the same operations as the pass that would have
// written the first term back.
__device__ __forceinline__ float apply_b(const Pending& q, float v, float wi, float wj) {
    return __fmaf_rn(q.c1b, v, q.sgnb * __fmul_rn(wi, wj));
}

// ------------------------------------------------------------------ pass
// Rows rbase .. rbase + nr - 1 of one fp32 factor, d a multiple of 4.  FULL: nr = R.
// ST: write the current values into S; T2: the pending term has two parts.
template <int RW, bool HAS, bool MV, bool FULL, bool ST = HAS, bool T2 = false>
__device__ __forceinline__ void pass_rows4(const FactorDesc& f, const Pending& q, int rbase, int nr,
                                           int lane, int maxabs, float (&dot)[RW], float (&nrm)[RW]) {
    const int d = f.d, d4 = d >> 2;
    float* __restrict__ P = static_cast<float*>(f.P) + (size_t)rbase * d;
    float wi[RW], wi2[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) {
        wi[r] = (HAS && (FULL || r < nr)) ? gld(f.w + rbase + r) : 0.f;
        wi2[r] = (T2 && (FULL || r < nr)) ? gld(f.w + d + rbase + r) : 0.f;
    }

    for (int j = lane; j < d4; j += 64) {
        float4 p[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (!FULL && r >= nr) continue;
            p[r] = MKOR_SM_NT ? gld4_nt(P + (size_t)r * d + 4 * j) : gld4(P + (size_t)r * d + 4 * j);
        }
        float4 xv = make_float4(0.f, 0.f, 0.f, 0.f), wv = xv, wv2 = xv;
        if constexpr (MV) xv = gld4(f.x + 4 * j);
        if constexpr (HAS) wv = gld4(f.w + 4 * j);
        if constexpr (T2) wv2 = gld4(f.w + d + 4 * j);
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (!FULL && r >= nr) break;
            if constexpr (HAS) {
                p[r].x = apply(q, p[r].x, wi[r], wv.x);
                p[r].y = apply(q, p[r].y, wi[r], wv.y);
                p[r].z = apply(q, p[r].z, wi[r], wv.z);
                p[r].w = apply(q, p[r].w, wi[r], wv.w);
                const int row = rbase + r;
                const bool diag = (row >> 2) == j;
                const int c = row & 3;
                if (diag) {
                    if (c == 0) p[r].x = __fadd_rn(p[r].x, q.c2);
                    else if (c == 1) p[r].y = __fadd_rn(p[r].y, q.c2);
                    else if (c == 2) p[r].z = __fadd_rn(p[r].z, q.c2);
                    else p[r].w = __fadd_rn(p[r].w, q.c2);
                }
                if constexpr (T2) {
                    p[r].x = apply_b(q, p[r].x, wi2[r], wv2.x);
                    p[r].y = apply_b(q, p[r].y, wi2[r], wv2.y);
                    p[r].z = apply_b(q, p[r].z, wi2[r], wv2.z);
                    p[r].w = apply_b(q, p[r].w, wi2[r], wv2.w);
                    if (diag) {
                        if (c == 0) p[r].x = __fadd_rn(p[r].x, q.c2b);
                        else if (c == 1) p[r].y = __fadd_rn(p[r].y, q.c2b);
                        else if (c == 2) p[r].z = __fadd_rn(p[r].z, q.c2b);
                        else p[r].w = __fadd_rn(p[r].w, q.c2b);
                    }
                }
                if constexpr (ST) {
                    if (MKOR_SM_NT) {
                        gst4_nt(P + (size_t)r * d + 4 * j, p[r]);
                    } else {
                        gst4(P + (size_t)r * d + 4 * j, p[r]);
                    }
                }
            }
            if constexpr (MV) {
                dot[r] = fmaf(p[r].x, xv.x, dot[r]);
                dot[r] = fmaf(p[r].y, xv.y, dot[r]);
                dot[r] = fmaf(p[r].z, xv.z, dot[r]);
                dot[r] = fmaf(p[r].w, xv.w, dot[r]);
                nrm[r] = absacc(nrm[r], p[r].x, maxabs);
                nrm[r] = absacc(nrm[r], p[r].y, maxabs);
                nrm[r] = absacc(nrm[r], p[r].z, maxabs);
                nrm[r] = absacc(nrm[r], p[r].w, maxabs);
            }
        }
    }
}

// bf16 factor, d a multiple of 64: 8 elements (16 bytes) per lane and row.
// The pending term is applied in fp32 and the result rounded to bf16 (nearest
// even); the norm and the matvec use those rounded values, which are the
// factor from then on.
__device__ __forceinline__ void unpack8(const uint4& h, float (&v)[8]) {
    const unsigned u[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf2f((unsigned short)(u[i] & 0xffffu));
        v[2 * i + 1] = bf2f((unsigned short)(u[i] >> 16));
    }
}

__device__ __forceinline__ uint4 pack8(const float (&v)[8]) {
    return make_uint4(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]), f2bf2(v[4], v[5]), f2bf2(v[6], v[7]));
}

template <int RW, bool HAS, bool MV, bool FULL>
__device__ __forceinline__ void pass_rows8h(const FactorDesc& f, const Pending& q, int rbase, int nr,
                                            int lane, int maxabs, float (&dot)[RW], float (&nrm)[RW]) {
    const int d = f.d, d8 = d >> 3;
    unsigned short* __restrict__ P16 = static_cast<unsigned short*>(f.P) + (size_t)rbase * d;
    float wi[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) wi[r] = (HAS && (FULL || r < nr)) ? gld(f.w + rbase + r) : 0.f;

    for (int j = lane; j < d8; j += 64) {
        uint4 h[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (!FULL && r >= nr) continue;
            h[r] = MKOR_SM_NT_HALF ? gld_u4_nt(P16 + (size_t)r * d + 8 * j) : gld_u4(P16 + (size_t)r * d + 8 * j);
        }
        float xv[8], wv[8];
        if constexpr (MV) {
            const float4 x0 = gld4(f.x + 8 * j), x1 = gld4(f.x + 8 * j + 4);
            xv[0] = x0.x; xv[1] = x0.y; xv[2] = x0.z; xv[3] = x0.w;
            xv[4] = x1.x; xv[5] = x1.y; xv[6] = x1.z; xv[7] = x1.w;
        }
        if constexpr (HAS) {
            const float4 w0 = gld4(f.w + 8 * j), w1 = gld4(f.w + 8 * j + 4);
            wv[0] = w0.x; wv[1] = w0.y; wv[2] = w0.z; wv[3] = w0.w;
            wv[4] = w1.x; wv[5] = w1.y; wv[6] = w1.z; wv[7] = w1.w;
        }
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (!FULL && r >= nr) break;
            float p[8];
            unpack8(h[r], p);
            if constexpr (HAS) {
#pragma unroll
                for (int e = 0; e < 8; ++e) p[e] = apply(q, p[e], wi[r], wv[e]);
                const int row = rbase + r;
                if ((row >> 3) == j) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if ((row & 7) == e) p[e] = __fadd_rn(p[e], q.c2);
                }
                const uint4 hn = pack8(p);
                if (MKOR_SM_NT_HALF) gst_u4_nt(P16 + (size_t)r * d + 8 * j, hn);
                else                 gst_u4(P16 + (size_t)r * d + 8 * j, hn);
                unpack8(hn, p);   // the stored (rounded) values are the factor from now on
            }
            if constexpr (MV) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    dot[r] = fmaf(p[e], xv[e], dot[r]);
                    nrm[r] = absacc(nrm[r], p[e], maxabs);
                }
            }
        }
    }
}

// Any d (scalar accesses).
template <int RW, bool HAS, bool MV>
__device__ __forceinline__ void pass_rows1(const FactorDesc& f, const Pending& q, int rbase, int nr,
                                           int lane, int maxabs, float (&dot)[RW], float (&nrm)[RW]) {
    const int d = f.d;
    float* __restrict__ P = static_cast<float*>(f.P) + (size_t)rbase * d;
    float wi[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) wi[r] = (HAS && r < nr) ? gld(f.w + rbase + r) : 0.f;
    for (int j = lane; j < d; j += 64) {
        const float xv = MV ? gld(f.x + j) : 0.f;
        const float wj = HAS ? gld(f.w + j) : 0.f;
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (r >= nr) break;
            float p = gld(P + (size_t)r * d + j);
            if constexpr (HAS) {
                p = apply(q, p, wi[r], wj);
                if (rbase + r == j) p = __fadd_rn(p, q.c2);
                gst(P + (size_t)r * d + j, p);
            }
            if constexpr (MV) {
                dot[r] = fmaf(p, xv, dot[r]);
                nrm[r] = absacc(nrm[r], p, maxabs);
            }
        }
    }
}

// HALF (bf16 factor, d a multiple of 64) or fp32; RW rows per wave.  A
// factor that skips the write (ST = false with HAS) or has two terms (T2) is
// lazy: fp32 with d a multiple of 64.
template <int RW, bool HALF, bool HAS, bool MV, bool ST = HAS, bool T2 = false>
__device__ __forceinline__ void pass_rows(const FactorDesc& f, const Pending& q, int rbase, int nr,
                                          int lane, int maxabs, float (&dot)[RW], float (&nrm)[RW]) {
    if constexpr (T2 || ST != HAS) {
        if constexpr (!HALF) {
            if (nr == RW) pass_rows4<RW, HAS, MV, true, ST, T2>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            else          pass_rows4<RW, HAS, MV, false, ST, T2>(f, q, rbase, nr, lane, maxabs, dot, nrm);
        }
    } else if constexpr (HALF) {
        if (nr == RW) pass_rows8h<RW, HAS, MV, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
        else          pass_rows8h<RW, HAS, MV, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
    } else if ((f.d & 3) == 0) {
        if (nr == RW) pass_rows4<RW, HAS, MV, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
        else          pass_rows4<RW, HAS, MV, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
    } else {
        pass_rows1<RW, HAS, MV>(f, q, rbase, nr, lane, maxabs, dot, nrm);
    }
}

// One row block of the pass.
// RW rows per wave: SM_ROWS_PER_WAVE for fp32 factors, SM_ROWS_PER_WAVE_HALF
// for bf16 ones (the same bytes in flight per lane).
template <int RW, bool HALF>
__device__ __forceinline__ void pass_block(const FactorDesc& f, const RowBlock& rb,
                                           float4* __restrict__ partials, int b, int maxabs,
                                           int matvec, float4* sred) {
    const Pending q = *f.pend;
    const bool has = q.has != 0;
    if (!has && !matvec) return;   // nothing pending to write, no matvec wanted
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int rbase = rb.row0 + wave * RW;
    const int nr = max(0, min(RW, f.d - rbase));

    float dot[RW], nrm[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) { dot[r] = 0.f; nrm[r] = 0.f; }
    // a lazy factor with one pending term is only read: the next term joins
    // it (finalize), and the pass of the step after writes both
    const bool two = q.has == 2, store = has && (!matvec || !f.lazy || two);
    if (nr > 0) {
        if (matvec) {
            if (!has)       pass_rows<RW, HALF, false, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            else if (two)   pass_rows<RW, HALF, true, true, true, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            else if (store) pass_rows<RW, HALF, true, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            else            pass_rows<RW, HALF, true, true, false, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
        } else {
            if (two) pass_rows<RW, HALF, true, false, true, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            else     pass_rows<RW, HALF, true, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
        }
    }
    if (!matvec) return;

#pragma unroll
    for (int r = 0; r < RW; ++r) {
        dot[r] = wave_sum(dot[r]);
        nrm[r] = maxabs ? wave_nanmax(nrm[r]) : wave_sum(nrm[r]);
    }

    if (lane == 0) {
        float mx = 0.f, sxu = 0.f, sxx = 0.f;
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (r >= nr) break;
            const int row = rbase + r;
            gst(f.u + row, dot[r]);
            const float xr = gld(f.x + row);
            mx = nanmax(mx, nrm[r]);
            sxu = fmaf(xr, dot[r], sxu);
            sxx = fmaf(xr, xr, sxx);
        }
        sred[wave] = make_float4(mx, sxu, sxx, 0.f);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float4 acc = sred[0];
        for (int w = 1; w < SM_THREADS / 64; ++w) {
            acc.x = nanmax(acc.x, sred[w].x);
            acc.y += sred[w].y;
            acc.z += sred[w].z;
        }
        gst4(reinterpret_cast<float*>(partials + b), acc);
    }
    __syncthreads();   // sred is reused by the next row block
}

// Grid-stride over the row blocks: a grid of about SM_GRID workgroups keeps
// long streams per workgroup, which measured best for this read + write
// traffic.
__global__ __launch_bounds__(SM_THREADS) void sm_pass_kernel(
    const FactorDesc* __restrict__ factors, const RowBlock* __restrict__ blocks,
    float4* __restrict__ partials, int nblocks, int maxabs, int matvec) {
    __shared__ float4 sred[SM_THREADS / 64];
    for (int b = blockIdx.x; b < nblocks; b += gridDim.x) {
        const RowBlock rb = blocks[b];
        const FactorDesc f = factors[rb.factor];
        if (f.rank > 1) continue;   // sm_pass_rank_kernel
        // a first-order layer this step: its factor is neither read nor
        // updated (a write-back pass, matvec = 0, still writes its terms)
        if (matvec && !gld_i32(f.mode)) continue;
        if (f.half) pass_block<SM_ROWS_PER_WAVE_HALF, true>(f, rb, partials, b, maxabs, matvec, sred);
        else        pass_block<SM_ROWS_PER_WAVE, false>(f, rb, partials, b, maxabs, matvec, sred);
    }
}

// ------------------------------------------------------------------ rank-r pass
// Factors with r > 1 vectors (fp32): the same stream over P, with the pending
// term (if any) of rank r,
//   P_ij = fma(c1, S_ij, t_ij) (+ c2 on the diagonal),
//   t_ij = fma(sw_r[i], w_r[j], ... fma(sw_2[i], w_2[j], sw_1[i] * w_1[j])),
// sw_l = sgn * w_l (exact), the same chain for (i, j) and (j, i) so that a
// symmetric factor stays bitwise symmetric; and r row dot products
// u_l = P x_l with the Gram partials x_l^T P x_m and x_l^T x_m of the row block.
constexpr int RR = SM_ROWS_PER_WAVE;

template <bool HAS, bool MV, bool VEC>
__device__ __forceinline__ void rank_rows(const FactorDesc& f, const Pending& q, int rbase, int nr, int lane,
                                          int maxabs, float (&dot)[RR][MAXR], float (&nrm)[RR]) {
    const int d = f.d, rk = f.rank;
    float* __restrict__ P = static_cast<float*>(f.P) + (size_t)rbase * d;
    float swi[RR][MAXR];
#pragma unroll
    for (int r = 0; r < RR; ++r)
#pragma unroll
        for (int l = 0; l < MAXR; ++l)
            swi[r][l] = (HAS && r < nr && l < rk) ? q.sgn * gld(f.w + (size_t)l * d + rbase + r) : 0.f;
    auto elem = [&](int r, int j, float v, const float (&wj)[MAXR]) {
        if constexpr (HAS) {
            float t = __fmul_rn(swi[r][0], wj[0]);
#pragma unroll
            for (int l = 1; l < MAXR; ++l)
                if (l < rk) t = __fmaf_rn(swi[r][l], wj[l], t);
            v = __fmaf_rn(q.c1, v, t);
            if (rbase + r == j) v = __fadd_rn(v, q.c2);
        }
        return v;
    };
    if constexpr (VEC) {
        const int d4 = d >> 2;
        for (int j = lane; j < d4; j += 64) {
            float4 p[RR];
#pragma unroll
            for (int r = 0; r < RR; ++r)
                if (r < nr) p[r] = gld4(P + (size_t)r * d + 4 * j);
            float4 xv[MAXR], wv[MAXR];
#pragma unroll
            for (int l = 0; l < MAXR; ++l) {
                xv[l] = make_float4(0.f, 0.f, 0.f, 0.f);
                wv[l] = xv[l];
                if (l < rk) {
                    if (MV) xv[l] = gld4(f.x + (size_t)l * d + 4 * j);
                    if (HAS) wv[l] = gld4(f.w + (size_t)l * d + 4 * j);
                }
            }
#pragma unroll
            for (int r = 0; r < RR; ++r) {
                if (r >= nr) break;
                float wj[4][MAXR];
#pragma unroll
                for (int l = 0; l < MAXR; ++l) {
                    wj[0][l] = wv[l].x; wj[1][l] = wv[l].y; wj[2][l] = wv[l].z; wj[3][l] = wv[l].w;
                }
                float v[4] = {p[r].x, p[r].y, p[r].z, p[r].w};
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = elem(r, 4 * j + c, v[c], wj[c]);
                if constexpr (HAS) gst4(P + (size_t)r * d + 4 * j, make_float4(v[0], v[1], v[2], v[3]));
                if constexpr (MV) {
#pragma unroll
                    for (int l = 0; l < MAXR; ++l) {
                        if (l >= rk) break;
                        const float xs[4] = {xv[l].x, xv[l].y, xv[l].z, xv[l].w};
#pragma unroll
                        for (int c = 0; c < 4; ++c) dot[r][l] = fmaf(v[c], xs[c], dot[r][l]);
                    }
#pragma unroll
                    for (int c = 0; c < 4; ++c) nrm[r] = absacc(nrm[r], v[c], maxabs);
                }
            }
        }
    } else {
        for (int j = lane; j < d; j += 64) {
            float wj[MAXR], xj[MAXR];
#pragma unroll
            for (int l = 0; l < MAXR; ++l) {
                wj[l] = (HAS && l < rk) ? gld(f.w + (size_t)l * d + j) : 0.f;
                xj[l] = (MV && l < rk) ? gld(f.x + (size_t)l * d + j) : 0.f;
            }
#pragma unroll
            for (int r = 0; r < RR; ++r) {
                if (r >= nr) break;
                float v = elem(r, j, gld(P + (size_t)r * d + j), wj);
                if constexpr (HAS) gst(P + (size_t)r * d + j, v);
                if constexpr (MV) {
#pragma unroll
                    for (int l = 0; l < MAXR; ++l)
                        if (l < rk) dot[r][l] = fmaf(v, xj[l], dot[r][l]);
                    nrm[r] = absacc(nrm[r], v, maxabs);
                }
            }
        }
    }
}

// MV = 1: the read pass of a step (r products, Gram partials, norms);
// MV = 0: the write of the pending rank-r term after the finalize.  Two
// kernels, so that each gets the registers of its own path (the write pass
// then holds four waves per SIMD, against two for one kernel with both
// paths).  The plan writes a rank-r term in the stage that forms it, so the
// read pass meets no pending term; should it meet one, the scalar path applies
// and writes it before the products.
template <int MV>
__global__ __launch_bounds__(SM_THREADS) void sm_pass_rank_kernel(
    const FactorDesc* __restrict__ factors, const RowBlock* __restrict__ blocks,
    float4* __restrict__ partials, float* __restrict__ gram, int nblocks, int maxabs) {
    constexpr bool matvec = MV != 0;
    __shared__ float4 sred[SM_THREADS / 64];
    __shared__ float sgram[SM_THREADS / 64][GRAM];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (int b = blockIdx.x; b < nblocks; b += gridDim.x) {
        const RowBlock rb = blocks[b];
        const FactorDesc f = factors[rb.factor];
        if (f.rank <= 1) continue;
        if (matvec && !gld_i32(f.mode)) continue;   // first-order layer this step
        const Pending q = *f.pend;
        const bool has = q.has != 0;
        if (!has && !matvec) continue;
        const int rbase = rb.row0 + wave * RR;
        const int nr = max(0, min(RR, f.d - rbase));
        const int rk = f.rank;
        float dot[RR][MAXR], nrm[RR];
#pragma unroll
        for (int r = 0; r < RR; ++r) {
            nrm[r] = 0.f;
#pragma unroll
            for (int l = 0; l < MAXR; ++l) dot[r][l] = 0.f;
        }
        // lane k < RR MAXR holds x_l[row] of the wave's row kr = k / MAXR and
        // vector kl = k % MAXR (0 past the rows or the rank), loaded ahead of
        // the stream so that the u stores and Gram partials below wait on no
        // load
        const int kr = lane / MAXR, kl = lane % MAXR;
        const bool kin = lane < RR * MAXR && kr < nr && kl < rk;
        const float xk = (matvec && kin) ? gld(f.x + (size_t)kl * f.d + rbase + kr) : 0.f;
        if (nr > 0) {
            const bool vec = (f.d & 3) == 0;
            if constexpr (matvec) {
                if (has)      rank_rows<true, true, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
                else if (vec) rank_rows<false, true, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
                else          rank_rows<false, true, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            } else {
                if (vec) rank_rows<true, false, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
                else     rank_rows<true, false, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            }
        }
        if (!matvec) continue;
#pragma unroll
        for (int r = 0; r < RR; ++r) {
#pragma unroll
            for (int l = 0; l < MAXR; ++l) dot[r][l] = wave_sum(dot[r][l]);
            nrm[r] = maxabs ? wave_nanmax(nrm[r]) : wave_sum(nrm[r]);
        }
        // u_l[row] = dot[kr][kl], one store per lane
        float dk = 0.f;
#pragma unroll
        for (int r = 0; r < RR; ++r)
#pragma unroll
            for (int l = 0; l < MAXR; ++l)
                if (lane == r * MAXR + l) dk = dot[r][l];
        if (kin) gst(f.u + (size_t)kl * f.d + rbase + kr, dk);
        // Gram entry e = lane < GRAM: e < MAXR^2 is sum_r x_l[r] (P x_m)[r],
        // the rest sum_r x_l[r] x_m[r] ((l, m) = (e / MAXR, e % MAXR) of
        // e mod MAXR^2), rows in order from 0, each term one fma
        const int e = lane % (MAXR * MAXR), gl = e / MAXR, gm = e % MAXR;
        const bool gxu_lane = lane < MAXR * MAXR;
        float gacc = 0.f;
#pragma unroll
        for (int r = 0; r < RR; ++r) {
            if (r >= nr) break;
            const float xl = __shfl(xk, r * MAXR + gl, 64);
            const float xm = __shfl(xk, r * MAXR + gm, 64);
            float dm = 0.f;
#pragma unroll
            for (int m = 0; m < MAXR; ++m)
                if (gm == m) dm = dot[r][m];
            gacc = fmaf(xl, gxu_lane ? dm : xm, gacc);
        }
        if (lane < GRAM) sgram[wave][lane] = gacc;
        if (lane == 0) {
            float mx = 0.f;
#pragma unroll
            for (int r = 0; r < RR; ++r)
                if (r < nr) mx = nanmax(mx, nrm[r]);
            sred[wave] = make_float4(mx, 0.f, 0.f, 0.f);
        }
        static_assert(RR * MAXR <= 64 && GRAM == 2 * MAXR * MAXR && GRAM <= 64, "one lane per x value and Gram entry");
        __syncthreads();
        if (threadIdx.x == 0) {
            float4 acc = sred[0];
            for (int w = 1; w < SM_THREADS / 64; ++w) acc.x = nanmax(acc.x, sred[w].x);
            gst4(reinterpret_cast<float*>(partials + b), acc);
        }
        if (threadIdx.x < GRAM) {
            float acc = sgram[0][threadIdx.x];
            for (int w = 1; w < SM_THREADS / 64; ++w) acc += sgram[w][threadIdx.x];
            gst(gram + (size_t)b * GRAM + threadIdx.x, acc);
        }
        __syncthreads();   // sred / sgram are reused by the next row block
    }
}

// ------------------------------------------------------------------ finalize
struct UpdateArgs {
    float gamma, zeta, eps;
    int   variant, guard;
};

struct SmScalars {
    float c1, c2, sgn, sqc;   // P_t = c1 P + c2 I + sgn w w^T,  w = sqc * u
    float zp, zq;             // u = zp * u_raw + zq * x
    int   stab, skip;
    float nu, s;
    int   comp;               // lazy factor whose pass left its term pending: two terms
};

// Rank-r factor: the r sequential Sherman-Morrison updates of P^(0) = P_hat /
// gamma with y_i = sqrt(1 - gamma) x_i (the paper's extension to higher ranks,
// applied to the momentum accumulation of Eq. 4/5).  Every u_i = P^(i-1) y_i
// is a combination U0 T_i of the columns of U0 = P_hat X, so all the
// recursion needs is the r x r matrix A = X^T P_hat X:
//   T_i   = (q / gamma) e_i - sum_{l<i} beta_l T_l (q T_l^T A e_i),   q = sqrt(1 - gamma)
//   beta_i = 1 / (1 + q e_i^T A T_i)
//   P_t   = P_hat / gamma - sum_i beta_i (U0 T_i)(U0 T_i)^T
// stored as the pending term c1 = zp / gamma, c2 = zq / gamma, sgn = -1,
// w_i = sqrt(beta_i) U0 T_i (U0 = zp u_raw + zq X).
__device__ void finalize_rank(const FactorDesc& f, const float4* __restrict__ partials,
                              const float* __restrict__ gram, const UpdateArgs& a) {
    const int t = threadIdx.x, rk = f.rank;
    __shared__ float s_mx[SM_THREADS];
    __shared__ double s_g[GRAM];
    __shared__ float s_coef[MAXR][MAXR];   // sqrt(beta_i) T[m][i], as [i][m]
    __shared__ float s_zp, s_zq;
    __shared__ int s_go;
    float mx = 0.f;
    for (int b = t; b < f.nblk; b += SM_THREADS) mx = nanmax(mx, partials[f.blk0 + b].x);
    s_mx[t] = mx;
    if (t < GRAM) {   // fixed-order float64 sum over the row blocks
        double acc = 0.0;
        for (int b = 0; b < f.nblk; ++b) acc += (double)gram[(size_t)(f.blk0 + b) * GRAM + t];
        s_g[t] = acc;
    }
    __syncthreads();
    for (int o = SM_THREADS / 2; o > 0; o >>= 1) {
        if (t < o) s_mx[t] = nanmax(s_mx[t], s_mx[t + o]);
        __syncthreads();
    }
    if (t == 0) {
        const double g = (double)a.gamma, q = sqrt(1.0 - g);
        const double nu = (double)s_mx[0];
        const int stab = nu > (double)a.eps ? 1 : 0;
        const double zp = stab ? (double)a.zeta : 1.0, zq = stab ? 1.0 - (double)a.zeta : 0.0;
        double A[MAXR][MAXR], T[MAXR][MAXR], beta[MAXR];
        for (int l = 0; l < MAXR; ++l)
            for (int m = 0; m < MAXR; ++m) {
                const double v = zp * s_g[l * MAXR + m] + zq * s_g[MAXR * MAXR + l * MAXR + m];
                const double vt = zp * s_g[m * MAXR + l] + zq * s_g[MAXR * MAXR + m * MAXR + l];
                A[l][m] = 0.5 * (v + vt);   // x^T P_hat x is symmetric
                T[l][m] = 0.0;
            }
        bool ok = isfinite(nu);
        for (int i = 0; i < rk; ++i) {
            T[i][i] = q / g;
            for (int l = 0; l < i; ++l) {
                double c = 0.0;   // u_l^T y_i
                for (int m = 0; m < rk; ++m) c += T[m][l] * A[m][i];
                c *= q * beta[l];
                for (int m = 0; m < rk; ++m) T[m][i] -= c * T[m][l];
            }
            double s = 0.0;       // y_i^T u_i
            for (int m = 0; m < rk; ++m) s += A[i][m] * T[m][i];
            s *= q;
            beta[i] = 1.0 / (1.0 + s);
            ok = ok && isfinite(beta[i]) && beta[i] > 0.0;
        }
        for (int i = 0; i < MAXR; ++i)
            for (int m = 0; m < MAXR; ++m)
                s_coef[i][m] = (ok && i < rk && m < rk) ? (float)(sqrt(beta[i]) * T[m][i]) : 0.f;
        s_zp = (float)zp;
        s_zq = (float)zq;
        const int skip = ok ? 0 : 1;
        if (f.stats != nullptr) {
            mkor_layer_stats* st = f.stats;
            const float nuf = (float)nu, sf = (float)A[0][0];
            if (f.side == 0) { st->nu_L = nuf; st->s_L = sf; st->stab_L = stab; st->skip_L = skip; }
            else             { st->nu_R = nuf; st->s_R = sf; st->stab_R = stab; st->skip_R = skip; }
        }
        Pending pq;
        if (skip && a.guard) { pq.c1 = 1.f; pq.c2 = 0.f; pq.sgn = 0.f; pq.has = 0; }
        else                 { pq.c1 = (float)(zp / g); pq.c2 = (float)(zq / g); pq.sgn = -1.f; pq.has = 1; }
        *f.pend = pq;
        s_go = (skip && a.guard) ? 0 : 1;
    }
    __syncthreads();
    if (!s_go) return;
    const float zp = s_zp, zq = s_zq;
    for (int k = t; k < f.d; k += SM_THREADS) {
        float um[MAXR];
#pragma unroll
        for (int m = 0; m < MAXR; ++m)
            um[m] = m < rk ? __fmaf_rn(zp, gld(f.u + (size_t)m * f.d + k), __fmul_rn(zq, gld(f.x + (size_t)m * f.d + k)))
                           : 0.f;
#pragma unroll
        for (int i = 0; i < MAXR; ++i) {
            if (i >= rk) break;
            float wv = 0.f;
#pragma unroll
            for (int m = 0; m < MAXR; ++m)
                if (m < rk) wv = __fmaf_rn(s_coef[i][m], um[m], wv);
            gst(f.w + (size_t)i * f.d + k, wv);
        }
    }
}

__global__ __launch_bounds__(SM_THREADS) void sm_finalize_kernel(
    const FactorDesc* __restrict__ factors, const float4* __restrict__ partials, const float* __restrict__ gram,
    UpdateArgs a) {
    const FactorDesc f = factors[blockIdx.x];
    if (!gld_i32(f.mode)) return;   // first-order layer this step: no update, no stats
    if (f.rank > 1) {
        finalize_rank(f, partials, gram, a);
        return;
    }
    __shared__ float s_mx[SM_THREADS];
    __shared__ double s_xu[SM_THREADS], s_xx[SM_THREADS];
    __shared__ SmScalars s_c;
    const int t = threadIdx.x;
    float mx = 0.f;
    double xu = 0.0, xx = 0.0;
    for (int b = t; b < f.nblk; b += SM_THREADS) {
        const float4 p = gld4(reinterpret_cast<const float*>(partials + f.blk0 + b));
        mx = nanmax(mx, p.x);
        xu += (double)p.y;
        xx += (double)p.z;
    }
    s_mx[t] = mx; s_xu[t] = xu; s_xx[t] = xx;
    __syncthreads();
    for (int o = SM_THREADS / 2; o > 0; o >>= 1) {
        if (t < o) {
            s_mx[t] = nanmax(s_mx[t], s_mx[t + o]);
            s_xu[t] += s_xu[t + o];
            s_xx[t] += s_xx[t + o];
        }
        __syncthreads();
    }
    if (t == 0) {
        SmScalars c;
        const double g = (double)a.gamma;
        const double nu = (double)s_mx[0];
        c.stab = (nu > (double)a.eps) ? 1 : 0;
        const double zp = c.stab ? (double)a.zeta : 1.0;
        const double zq = c.stab ? 1.0 - (double)a.zeta : 0.0;
        const double s = zp * s_xu[0] + zq * s_xx[0];
        double c1, c2, c3;
        if (a.variant == MKOR_SM_EXACT) {
            // Sherman-Morrison inverse of gamma * M_hat + (1 - gamma) x x^T
            const double k = (1.0 - g) / (g + (1.0 - g) * s);
            c1 = zp / g; c2 = zq / g; c3 = -k / g;
        } else {
            // Eq. 6/7 as printed
            const double k = (1.0 - g) / (g * g * (1.0 + g * (1.0 - g) * s));
            c1 = g * zp; c2 = g * zq; c3 = k;
        }
        c.skip = (isfinite(nu) && isfinite(s) && isfinite(c3)) ? 0 : 1;
        const Pending qp = *f.pend;   // the term the pass applied (and wrote, unless comp)
        c.comp = (f.lazy && qp.has == 1) ? 1 : 0;
        c.c1 = (float)c1; c.c2 = (float)c2;
        c.sgn = c3 < 0.0 ? -1.f : 1.f;
        c.sqc = (float)sqrt(fabs(c3));
        c.zp = (float)zp; c.zq = (float)zq;
        c.nu = (float)nu; c.s = (float)s;
        s_c = c;
        if (f.stats != nullptr) {
            mkor_layer_stats* st = f.stats;
            if (f.side == 0) { st->nu_L = c.nu; st->s_L = c.s; st->stab_L = c.stab; st->skip_L = c.skip; }
            else             { st->nu_R = c.nu; st->s_R = c.s; st->stab_R = c.stab; st->skip_R = c.skip; }
        }
        Pending q{};
        if (c.skip && a.guard) {   // leave the factor unchanged
            if (c.comp) q = qp;
            else { q.c1 = 1.f; q.c2 = 0.f; q.sgn = 0.f; q.has = 0; }
        } else if (c.comp) {   // the new term after the pending one
            q = qp;
            q.c1b = c.c1; q.c2b = c.c2; q.sgnb = c.sgn; q.has = 2;
        } else {
            q.c1 = c.c1; q.c2 = c.c2; q.sgn = c.sgn; q.has = 1;
        }
        *f.pend = q;
    }
    __syncthreads();
    const SmScalars c = s_c;
    if (c.skip && a.guard) return;
    // w = sqc * (zp * u_raw + zq * x), each rounding pinned (w2 when comp)
    float* wn = f.w + (c.comp ? f.d : 0);
    for (int i = t; i < f.d; i += SM_THREADS)
        gst(wn + i, __fmul_rn(c.sqc, __fmaf_rn(c.zp, gld(f.u + i), __fmul_rn(c.zq, gld(f.x + i)))));
}

struct ModeBits {
    uint32_t w[MODE_CHUNK / 32];
};

__global__ __launch_bounds__(256) void set_modes_kernel(int32_t* __restrict__ mode, int32_t count, ModeBits bits) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) mode[i] = (int32_t)((bits.w[i >> 5] >> (i & 31)) & 1u);
}

__global__ void sm_reset_kernel(const FactorDesc* __restrict__ factors, int32_t nfactors, int ranked_only) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < nfactors && (!ranked_only || factors[i].rank > 1)) *factors[i].pend = Pending{1.f, 0.f, 0.f, 0};
}

}  // namespace

hipError_t launch_sm_pass(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                          float4* partials, float* gram, int32_t norm_kind, int32_t matvec, int32_t ranked,
                          hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    const int32_t grid = (SM_GRID > 0 && nblocks > SM_GRID) ? SM_GRID : nblocks;
    const int maxabs = norm_kind == MKOR_NORM_MAXABS ? 1 : 0;
    hipLaunchKernelGGL(sm_pass_kernel, dim3(grid), dim3(SM_THREADS), 0, stream, factors, blocks,
                       partials, nblocks, maxabs, matvec ? 1 : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !ranked) return e;
    if (matvec)
        hipLaunchKernelGGL(sm_pass_rank_kernel<1>, dim3(grid), dim3(SM_THREADS), 0, stream, factors, blocks,
                           partials, gram, nblocks, maxabs);
    else
        hipLaunchKernelGGL(sm_pass_rank_kernel<0>, dim3(grid), dim3(SM_THREADS), 0, stream, factors, blocks,
                           partials, gram, nblocks, maxabs);
    return hipGetLastError();
}

hipError_t launch_sm_apply_rank(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                                int32_t nfactors, hipStream_t stream) {
    if (nblocks <= 0 || nfactors <= 0) return hipSuccess;
    const int32_t grid = (SM_GRID > 0 && nblocks > SM_GRID) ? SM_GRID : nblocks;
    hipLaunchKernelGGL(sm_pass_rank_kernel<0>, dim3(grid), dim3(SM_THREADS), 0, stream, factors, blocks,
                       (float4*)nullptr, (float*)nullptr, nblocks, 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sm_reset_kernel, dim3((nfactors + 255) / 256), dim3(256), 0, stream, factors,
                       nfactors, 1);
    return hipGetLastError();
}

hipError_t launch_sm_finalize(const FactorDesc* factors, int32_t nfactors, const float4* partials,
                              const float* gram, const mkor_params& p, hipStream_t stream) {
    if (nfactors <= 0) return hipSuccess;
    UpdateArgs a{p.gamma, p.zeta, p.stab_eps, p.sm_variant, p.guard_nonfinite};
    hipLaunchKernelGGL(sm_finalize_kernel, dim3(nfactors), dim3(SM_THREADS), 0, stream, factors,
                       partials, gram, a);
    return hipGetLastError();
}

hipError_t launch_set_modes(int32_t* mode, int32_t first, int32_t count, const uint32_t* bits,
                            hipStream_t stream) {
    if (count <= 0) return hipSuccess;
    if (count > MODE_CHUNK) return hipErrorInvalidValue;
    ModeBits b{};
    for (int i = 0; i < (count + 31) / 32; ++i) b.w[i] = bits[i];
    hipLaunchKernelGGL(set_modes_kernel, dim3((count + 255) / 256), dim3(256), 0, stream, mode + first, count, b);
    return hipGetLastError();
}

hipError_t launch_sm_reset(const FactorDesc* factors, int32_t nfactors, hipStream_t stream) {
    if (nfactors <= 0) return hipSuccess;
    hipLaunchKernelGGL(sm_reset_kernel, dim3((nfactors + 255) / 256), dim3(256), 0, stream, factors,
                       nfactors, 0);
    return hipGetLastError();
}

}  // namespace mkor
