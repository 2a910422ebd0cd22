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

// ------------------------------------------------------------------ pass
// Rows rbase .. rbase + nr - 1 of one fp32 factor, d a multiple of 4.  FULL: nr = R.
template <int RW, bool HAS, bool MV, bool FULL>
__device__ __forceinline__ void pass_rows4(const FactorDesc& f, const Pending& q, int rbase, int nr,
                                           int lane, int maxabs, float (&dot)[RW], float (&nrm)[RW]) {
    const int d = f.d, d4 = d >> 2;
    float* __restrict__ P = static_cast<float*>(f.P) + (size_t)rbase * d;
    float wi[RW];
#pragma unroll
    for (int r = 0; r < RW; ++r) wi[r] = (HAS && (FULL || r < nr)) ? gld(f.w + rbase + r) : 0.f;

    for (int j = lane; j < d4; j += 64) {
        float4 p[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (!FULL && r >= nr) continue;
            p[r] = MKOR_SM_NT ? gld4_nt(P + (size_t)r * d + 4 * j) : gld4(P + (size_t)r * d + 4 * j);
        }
        float4 xv = make_float4(0.f, 0.f, 0.f, 0.f), wv = xv;
        if constexpr (MV) xv = gld4(f.x + 4 * j);
        if constexpr (HAS) wv = gld4(f.w + 4 * j);
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (!FULL && r >= nr) break;
            if constexpr (HAS) {
                p[r].x = apply(q, p[r].x, wi[r], wv.x);
                p[r].y = apply(q, p[r].y, wi[r], wv.y);
                p[r].z = apply(q, p[r].z, wi[r], wv.z);
                p[r].w = apply(q, p[r].w, wi[r], wv.w);
                const int row = rbase + r;
                if ((row >> 2) == j) {
                    const int c = row & 3;
                    if (c == 0) p[r].x = __fadd_rn(p[r].x, q.c2);
                    else if (c == 1) p[r].y = __fadd_rn(p[r].y, q.c2);
                    else if (c == 2) p[r].z = __fadd_rn(p[r].z, q.c2);
                    else p[r].w = __fadd_rn(p[r].w, q.c2);
                }
                if (MKOR_SM_NT) {
                    gst4_nt(P + (size_t)r * d + 4 * j, p[r]);
                } else {
                    gst4(P + (size_t)r * d + 4 * j, p[r]);
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
            h[r] = gld_u4(P16 + (size_t)r * d + 8 * j);
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
                gst_u4(P16 + (size_t)r * d + 8 * j, hn);
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

// HALF (bf16 factor, d a multiple of 64) or fp32; RW rows per wave.
template <int RW, bool HALF, bool HAS, bool MV>
__device__ __forceinline__ void pass_rows(const FactorDesc& f, const Pending& q, int rbase, int nr,
                                          int lane, int maxabs, float (&dot)[RW], float (&nrm)[RW]) {
    if constexpr (HALF) {
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
    if (nr > 0) {
        if (matvec) {
            if (has) pass_rows<RW, HALF, true, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
            else     pass_rows<RW, HALF, false, true>(f, q, rbase, nr, lane, maxabs, dot, nrm);
        } else {
            pass_rows<RW, HALF, true, false>(f, q, rbase, nr, lane, maxabs, dot, nrm);
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
        if (f.half) pass_block<SM_ROWS_PER_WAVE_HALF, true>(f, rb, partials, b, maxabs, matvec, sred);
        else        pass_block<SM_ROWS_PER_WAVE, false>(f, rb, partials, b, maxabs, matvec, sred);
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
};

__global__ __launch_bounds__(SM_THREADS) void sm_finalize_kernel(
    const FactorDesc* __restrict__ factors, const float4* __restrict__ partials, UpdateArgs a) {
    const FactorDesc f = factors[blockIdx.x];
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
        Pending q;
        if (c.skip && a.guard) {   // leave the factor unchanged
            q.c1 = 1.f; q.c2 = 0.f; q.sgn = 0.f; q.has = 0;
        } else {
            q.c1 = c.c1; q.c2 = c.c2; q.sgn = c.sgn; q.has = 1;
        }
        *f.pend = q;
    }
    __syncthreads();
    const SmScalars c = s_c;
    if (c.skip && a.guard) return;
    // w = sqc * (zp * u_raw + zq * x), each rounding pinned
    for (int i = t; i < f.d; i += SM_THREADS)
        gst(f.w + i, __fmul_rn(c.sqc, __fmaf_rn(c.zp, gld(f.u + i), __fmul_rn(c.zq, gld(f.x + i)))));
}

__global__ void sm_reset_kernel(const FactorDesc* __restrict__ factors, int32_t nfactors) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < nfactors) *factors[i].pend = Pending{1.f, 0.f, 0.f, 0};
}

}  // namespace

hipError_t launch_sm_pass(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                          float4* partials, int32_t norm_kind, int32_t matvec, hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    const int32_t grid = (SM_GRID > 0 && nblocks > SM_GRID) ? SM_GRID : nblocks;
    hipLaunchKernelGGL(sm_pass_kernel, dim3(grid), dim3(SM_THREADS), 0, stream, factors, blocks,
                       partials, nblocks, norm_kind == MKOR_NORM_MAXABS ? 1 : 0, matvec ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_sm_finalize(const FactorDesc* factors, int32_t nfactors, const float4* partials,
                              const mkor_params& p, hipStream_t stream) {
    if (nfactors <= 0) return hipSuccess;
    UpdateArgs a{p.gamma, p.zeta, p.stab_eps, p.sm_variant, p.guard_nonfinite};
    hipLaunchKernelGGL(sm_finalize_kernel, dim3(nfactors), dim3(SM_THREADS), 0, stream, factors,
                       partials, a);
    return hipGetLastError();
}

hipError_t launch_sm_reset(const FactorDesc* factors, int32_t nfactors, hipStream_t stream) {
    if (nfactors <= 0) return hipSuccess;
    hipLaunchKernelGGL(sm_reset_kernel, dim3((nfactors + 255) / 256), dim3(256), 0, stream, factors,
                       nfactors);
    return hipGetLastError();
}

}  // namespace mkor
