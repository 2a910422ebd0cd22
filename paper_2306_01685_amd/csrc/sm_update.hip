// Grouped momentum Sherman-Morrison update of all inverse factors
// (Algorithm 1: norm-based stabilisation, then SM-based factor inversion;
// Eq. 4-7, Eq. 9-11).
//
// Two grouped launches over row blocks of every factor of every layer:
//
//   sm_matvec_kernel  reads each row of P once: u_raw_i = (P x)_i (row dot
//                     product, wave-shuffle reduction), the row's absolute sum
//                     (or max |entry|), and per-block partials
//                     {norm max, sum x_i u_raw_i, sum x_i^2}.
//   sm_update_kernel  every workgroup of a factor reduces that factor's
//                     partials in the same fixed order, so all of them take the
//                     same stabiliser decision without a host round trip, then
//                     streams its rows once:  P <- c1 P + c2 I + sgn w w^T.
//
// The stabiliser blend P_hat = zeta P + (1 - zeta) I is never materialised: it
// is folded into u = zeta u_raw + (1 - zeta) x, s = zeta x^T u_raw +
// (1 - zeta) x^T x and the coefficients c1, c2.  The rank-1 term is written as
// sgn * w_i * w_j with w = sqrt(|c3|) u so that (i,j) and (j,i) round
// identically and a symmetric factor stays bitwise symmetric.
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

// w = sqc * (zp * u_raw + zq * x) with every rounding pinned, so the row-side
// and column-side evaluations of w_i agree bit for bit.
__device__ __forceinline__ float wval(const SmScalars& c, float ur, float xv) {
    return __fmul_rn(c.sqc, __fmaf_rn(c.zp, ur, __fmul_rn(c.zq, xv)));
}

__device__ __forceinline__ float upd(const SmScalars& c, float p, float wi, float wj) {
    return __fmaf_rn(c.c1, p, c.sgn * __fmul_rn(wi, wj));
}

// ------------------------------------------------------------------ K1
__global__ __launch_bounds__(SM_THREADS) void sm_matvec_kernel(
    const FactorDesc* __restrict__ factors, const RowBlock* __restrict__ blocks,
    float4* __restrict__ partials, int maxabs) {
    const RowBlock rb = blocks[blockIdx.x];
    const FactorDesc f = factors[rb.factor];
    const int d = f.d;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int rbase = rb.row0 + wave * SM_ROWS_PER_WAVE;

    float dot[SM_ROWS_PER_WAVE], nrm[SM_ROWS_PER_WAVE];
#pragma unroll
    for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) { dot[r] = 0.f; nrm[r] = 0.f; }
    const int nr = max(0, min(SM_ROWS_PER_WAVE, d - rbase));

    if ((d & 3) == 0) {
        const int d4 = d >> 2;
        const float4* __restrict__ x4 = reinterpret_cast<const float4*>(f.x);
        const float4* __restrict__ P4 = reinterpret_cast<const float4*>(f.P) + (size_t)rbase * d4;
        if (nr == SM_ROWS_PER_WAVE) {
#pragma unroll 4
            for (int j = lane; j < d4; j += 64) {
                const float4 xv = x4[j];
#pragma unroll
                for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
                    const float4 p = P4[(size_t)r * d4 + j];
                    dot[r] = fmaf(p.x, xv.x, dot[r]);
                    dot[r] = fmaf(p.y, xv.y, dot[r]);
                    dot[r] = fmaf(p.z, xv.z, dot[r]);
                    dot[r] = fmaf(p.w, xv.w, dot[r]);
                    nrm[r] = absacc(nrm[r], p.x, maxabs);
                    nrm[r] = absacc(nrm[r], p.y, maxabs);
                    nrm[r] = absacc(nrm[r], p.z, maxabs);
                    nrm[r] = absacc(nrm[r], p.w, maxabs);
                }
            }
        } else {
            for (int j = lane; j < d4; j += 64) {
                const float4 xv = x4[j];
#pragma unroll
                for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
                    if (r >= nr) break;
                    const float4 p = P4[(size_t)r * d4 + j];
                    dot[r] = fmaf(p.x, xv.x, dot[r]);
                    dot[r] = fmaf(p.y, xv.y, dot[r]);
                    dot[r] = fmaf(p.z, xv.z, dot[r]);
                    dot[r] = fmaf(p.w, xv.w, dot[r]);
                    nrm[r] = absacc(nrm[r], p.x, maxabs);
                    nrm[r] = absacc(nrm[r], p.y, maxabs);
                    nrm[r] = absacc(nrm[r], p.z, maxabs);
                    nrm[r] = absacc(nrm[r], p.w, maxabs);
                }
            }
        }
    } else {
        const float* __restrict__ P = f.P + (size_t)rbase * d;
        for (int j = lane; j < d; j += 64) {
            const float xv = f.x[j];
#pragma unroll
            for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
                if (r >= nr) break;
                const float p = P[(size_t)r * d + j];
                dot[r] = fmaf(p, xv, dot[r]);
                nrm[r] = absacc(nrm[r], p, maxabs);
            }
        }
    }

#pragma unroll
    for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
        dot[r] = wave_sum(dot[r]);
        nrm[r] = maxabs ? wave_nanmax(nrm[r]) : wave_sum(nrm[r]);
    }

    __shared__ float4 sred[SM_THREADS / 64];
    if (lane == 0) {
        float mx = 0.f, sxu = 0.f, sxx = 0.f;
#pragma unroll
        for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
            if (r >= nr) break;
            const int row = rbase + r;
            f.u[row] = dot[r];
            const float xr = f.x[row];
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
        partials[blockIdx.x] = acc;
    }
}

// ------------------------------------------------------------------ K2
struct UpdateArgs {
    float gamma, zeta, eps;
    int   variant, guard;
};

__device__ SmScalars decide(const FactorDesc& f, const float4* __restrict__ partials,
                            const UpdateArgs& a) {
    __shared__ float s_mx[SM_THREADS];
    __shared__ double s_xu[SM_THREADS], s_xx[SM_THREADS];
    __shared__ SmScalars s_out;
    const int t = threadIdx.x;
    float mx = 0.f;
    double xu = 0.0, xx = 0.0;
    for (int b = t; b < f.nblk; b += SM_THREADS) {
        const float4 p = partials[f.blk0 + b];
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
            const double k = (1.0 - g) / (g + (1.0 - g) * s);
            c1 = zp / g; c2 = zq / g; c3 = -k / g;
        } else {
            const double k = (1.0 - g) / (g * g * (1.0 + g * (1.0 - g) * s));
            c1 = g * zp; c2 = g * zq; c3 = k;
        }
        c.skip = (isfinite(nu) && isfinite(s) && isfinite(c3)) ? 0 : 1;
        c.c1 = (float)c1; c.c2 = (float)c2;
        c.sgn = c3 < 0.0 ? -1.f : 1.f;
        c.sqc = (float)sqrt(fabs(c3));
        c.zp = (float)zp; c.zq = (float)zq;
        c.nu = (float)nu; c.s = (float)s;
        s_out = c;
    }
    __syncthreads();
    return s_out;
}

__global__ __launch_bounds__(SM_THREADS) void sm_update_kernel(
    const FactorDesc* __restrict__ factors, const RowBlock* __restrict__ blocks,
    const float4* __restrict__ partials, UpdateArgs args) {
    const RowBlock rb = blocks[blockIdx.x];
    const FactorDesc f = factors[rb.factor];
    const SmScalars c = decide(f, partials, args);

    if (rb.row0 == 0 && threadIdx.x == 0 && f.stats != nullptr) {
        mkor_layer_stats* st = f.stats;
        if (f.side == 0) { st->nu_L = c.nu; st->s_L = c.s; st->stab_L = c.stab; st->skip_L = c.skip; }
        else             { st->nu_R = c.nu; st->s_R = c.s; st->stab_R = c.stab; st->skip_R = c.skip; }
    }
    if (c.skip && args.guard) return;   // leave the factor unchanged

    const int d = f.d;
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int rbase = rb.row0 + wave * SM_ROWS_PER_WAVE;
    const int nr = max(0, min(SM_ROWS_PER_WAVE, d - rbase));
    if (nr == 0) return;

    float wi[SM_ROWS_PER_WAVE];
#pragma unroll
    for (int r = 0; r < SM_ROWS_PER_WAVE; ++r)
        wi[r] = (r < nr) ? wval(c, f.u[rbase + r], f.x[rbase + r]) : 0.f;

    if ((d & 3) == 0) {
        const int d4 = d >> 2;
        const float4* __restrict__ x4 = reinterpret_cast<const float4*>(f.x);
        const float4* __restrict__ u4 = reinterpret_cast<const float4*>(f.u);
        float4* __restrict__ P4 = reinterpret_cast<float4*>(f.P) + (size_t)rbase * d4;
        for (int j = lane; j < d4; j += 64) {
            const float4 ur = u4[j], xv = x4[j];
            const float w0 = wval(c, ur.x, xv.x), w1 = wval(c, ur.y, xv.y);
            const float w2 = wval(c, ur.z, xv.z), w3 = wval(c, ur.w, xv.w);
#pragma unroll
            for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
                if (r >= nr) break;
                float4 p = P4[(size_t)r * d4 + j];
                p.x = upd(c, p.x, wi[r], w0);
                p.y = upd(c, p.y, wi[r], w1);
                p.z = upd(c, p.z, wi[r], w2);
                p.w = upd(c, p.w, wi[r], w3);
                const int row = rbase + r;
                if ((row >> 2) == j) {
                    const int q = row & 3;
                    if (q == 0) p.x = __fadd_rn(p.x, c.c2);
                    else if (q == 1) p.y = __fadd_rn(p.y, c.c2);
                    else if (q == 2) p.z = __fadd_rn(p.z, c.c2);
                    else p.w = __fadd_rn(p.w, c.c2);
                }
                P4[(size_t)r * d4 + j] = p;
            }
        }
    } else {
        float* __restrict__ P = f.P + (size_t)rbase * d;
        for (int j = lane; j < d; j += 64) {
            const float wj = wval(c, f.u[j], f.x[j]);
#pragma unroll
            for (int r = 0; r < SM_ROWS_PER_WAVE; ++r) {
                if (r >= nr) break;
                float p = upd(c, P[(size_t)r * d + j], wi[r], wj);
                if (rbase + r == j) p = __fadd_rn(p, c.c2);
                P[(size_t)r * d + j] = p;
            }
        }
    }
}

}  // namespace

hipError_t launch_sm_matvec(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                            float4* partials, int32_t norm_kind, hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(sm_matvec_kernel, dim3(nblocks), dim3(SM_THREADS), 0, stream,
                       factors, blocks, partials, norm_kind == MKOR_NORM_MAXABS ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_sm_update(const FactorDesc* factors, const RowBlock* blocks, int32_t nblocks,
                            const float4* partials, const mkor_params& p, hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    UpdateArgs a{p.gamma, p.zeta, p.stab_eps, p.sm_variant, p.guard_nonfinite};
    hipLaunchKernelGGL(sm_update_kernel, dim3(nblocks), dim3(SM_THREADS), 0, stream,
                       factors, blocks, partials, a);
    return hipGetLastError();
}

}  // namespace mkor
