// Preconditioning for layers whose inverse factors are stored in bf16
// (half-precision factors: the paper's "half-precision" MKOR; its Table 1 halves
// the memory and the communication for it).  bf16 MFMA GEMMs
// (v_mfma_f32_32x32x16_bf16, fp32 accumulation), in the association
// dW_hat = L (G R):
//
//   stage H1:  Y = G R          A = G (d_in x d_out, bf16 or fp32 rounded to
//                               bf16), B = R (d_out x d_out), stored Y^T in bf16
//                               (d_out x d_in), plus ||G||^2 partials;
//   stage H2:  dW_hat = L Y     A = L (d_in x d_in), B = Y^T; dW_hat fp32 into
//                               dW, plus one ||dW_hat||^2 partial per tile.
//
// Both are C[m][n] = sum_k A[m][k] B[n][k] with both operands contiguous along
// k in their natural layout (the factors are symmetric, and Y is stored
// transposed), which is the layout the MFMA wants: each lane supplies 8
// consecutive k of one row.
//
// The current factor is its stored (bf16) value S plus the pending rank-1
// term of the SM update, P = c1 S + c2 I + sgn w w^T (see struct Pending).
// The GEMMs multiply with S and add the rest in the epilogue:
//   G P = c1 (G S) + c2 G + sgn (G w) w^T,   P Y = c1 (S Y) + c2 Y + sgn w (w^T Y),
// where the vector G w (or w^T Y) is summed from the other operand while it is
// staged into LDS (one fma per staged element), and G (or Y) at the output
// positions is read in the epilogue.  So the MFMA loop stays free of per-element
// arithmetic.
//
// Tiles: 256 x 256 per workgroup of 8 waves (2 x 4, each 128 x 64 = 4 x 2 MFMA
// blocks), so two waves share each SIMD and one issues MFMAs while the other
// waits on LDS or the slab barrier.  K runs in 64-deep slabs double-buffered in
// LDS (128 KB of the 160 KB) as [row][k] bf16 with the 16-byte chunk index
// XOR-swizzled by the row, so the 16-byte operand reads of a wave hit distinct
// banks.  d_in and d_out must be multiples of 64 (checked by the plan); M and
// N edges are masked.
#include "gmem.h"
#include "mkor_internal.h"

namespace mkor {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
// LDS pointers carry their address space, so every operand access is a
// ds_read / ds_write (a generic pointer would become a flat access, which
// waits on the global-load counter too).
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) mk_u4 lds_u4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf8;
typedef __attribute__((address_space(3))) float lds_float;
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int BM = HG_BM, BN = HG_BN, BK = HG_BK, NT = HG_THREADS;
constexpr int WM = HG_WM, WN = HG_WN;
constexpr int TM = BM / WM, TN = BN / WN;   // 128 x 64 per wave
constexpr int FM = TM / 32, FN = TN / 32;   // 4 x 2 MFMA blocks
constexpr int KCH = BK / 8;                 // 16-byte chunks per slab row (8)
constexpr int ACH = BM * KCH / NT;          // A chunks per thread and slab
constexpr int BCH = BN * KCH / NT;          // B chunks per thread and slab
static_assert(NT == WM * WN * 64 && KCH == 8 && TM == 128 && TN == 64, "layout");
static_assert(ACH * NT == BM * KCH && BCH * NT == BN * KCH, "staging");
static_assert(NT % KCH == 0, "a thread stages one fixed chunk column");

// byte offset of 16-byte chunk c of row r in a [rows][BK] bf16 slab
__device__ __forceinline__ int swz(int r, int c) { return r * (BK * 2) + ((c ^ (r & 7)) << 4); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

struct HgArgs {
    const HgLayer* layers;
    const GemmTile* tiles;
    float* partials;
};

// Dot of 8 staged values with 8 w values (fma chain in a fixed order).
__device__ __forceinline__ float dot8(const uint4& h, const float* w, float acc) {
    acc = fmaf(bf2f((unsigned short)(h.x & 0xffffu)), w[0], acc);
    acc = fmaf(bf2f((unsigned short)(h.x >> 16)), w[1], acc);
    acc = fmaf(bf2f((unsigned short)(h.y & 0xffffu)), w[2], acc);
    acc = fmaf(bf2f((unsigned short)(h.y >> 16)), w[3], acc);
    acc = fmaf(bf2f((unsigned short)(h.z & 0xffffu)), w[4], acc);
    acc = fmaf(bf2f((unsigned short)(h.z >> 16)), w[5], acc);
    acc = fmaf(bf2f((unsigned short)(h.w & 0xffffu)), w[6], acc);
    acc = fmaf(bf2f((unsigned short)(h.w >> 16)), w[7], acc);
    return acc;
}

__device__ __forceinline__ float sq8(const uint4& h, float acc) {
    const unsigned v[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float lo = bf2f((unsigned short)(v[i] & 0xffffu)), hi = bf2f((unsigned short)(v[i] >> 16));
        acc = fmaf(lo, lo, acc);
        acc = fmaf(hi, hi, acc);
    }
    return acc;
}

// 8 fp32 -> 8 bf16 (rounded) packed into 16 bytes
__device__ __forceinline__ uint4 pack8(const float4& a, const float4& b) {
    return make_uint4(f2bf2(a.x, a.y), f2bf2(a.z, a.w), f2bf2(b.x, b.y), f2bf2(b.z, b.w));
}

// Loads the 8 elements (row, k .. k + 7) of a row-major bf16 (or fp32,
// rounded) operand with leading dimension ld.  Rows at or past nrows are
// clamped to the last row (no branch in the K loop); their products land in
// output rows or columns the epilogue never stores.
template <bool F32>
__device__ __forceinline__ uint4 load_chunk(const void* base, int ld, int row, int nrows, int k) {
    const size_t off = (size_t)min(row, nrows - 1) * ld + k;
    if constexpr (F32) {
        const float* p = static_cast<const float*>(base) + off;
        return pack8(gld4(p), gld4(p + 4));
    } else {
        return gld_u4(static_cast<const unsigned short*>(base) + off);
    }
}

// STAGE 1: A = G (AF32: fp32 G), B = S_R (factor), rank-1 vector from A (G w_R).
// STAGE 2: A = S_L (factor), B = Y^T, rank-1 vector from B (w_L^T Y).
template <int STAGE, bool AF32, bool PEND>
__device__ void hgemm_tile(const HgLayer& L, const GemmTile& tile, const Pending& q, float* partials,
                           lds_char* smem) {
    lds_char* const A0 = smem;
    lds_char* const A1 = smem + BM * BK * 2;
    lds_char* const B0 = smem + 2 * BM * BK * 2;
    lds_char* const B1 = B0 + BN * BK * 2;
    lds_float* rvec = (lds_float*)(smem + 2 * (BM + BN) * BK * 2);   // BM (stage 1) or BN floats
    lds_float* red = rvec + (BM > BN ? BM : BN);

    const int m0 = tile.tm * BM, n0 = tile.tn * BN;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int li = lane & 31, lk = lane >> 5;
    const int M = L.M, N = L.N, K = L.K;
    const int cch = t % KCH;   // the 16-byte chunk column this thread stages
    // stage 1: ||G||^2 from the A (= G) staging of the first tile column
    const bool want_gsq = STAGE == 1 && tile.tn == 0;

    floatx16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // rank-1 partial dots of the rows this thread stages (A rows in stage 1,
    // B rows in stage 2)
    constexpr int RCH = STAGE == 1 ? ACH : BCH;
    float rdot[RCH];
#pragma unroll
    for (int i = 0; i < RCH; ++i) rdot[i] = 0.f;
    float gsq = 0.f;

    uint4 ra[ACH], rb[BCH];
    const int nslab = K / BK;
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < ACH; ++i) {
            const int row = (t + i * NT) / KCH;
            ra[i] = load_chunk<STAGE == 1 && AF32>(L.A, K, m0 + row, M, k0 + 8 * cch);
        }
#pragma unroll
        for (int i = 0; i < BCH; ++i) {
            const int row = (t + i * NT) / KCH;
            rb[i] = load_chunk<false>(L.B, K, n0 + row, N, k0 + 8 * cch);
        }
    };
    auto store = [&](int k0, lds_char* Ad, lds_char* Bd) {
        float wk[8];
        if (PEND) {
            const float4 w0 = gld4(L.w + k0 + 8 * cch), w1 = gld4(L.w + k0 + 8 * cch + 4);
            wk[0] = w0.x; wk[1] = w0.y; wk[2] = w0.z; wk[3] = w0.w;
            wk[4] = w1.x; wk[5] = w1.y; wk[6] = w1.z; wk[7] = w1.w;
        }
#pragma unroll
        for (int i = 0; i < ACH; ++i) {
            const int row = (t + i * NT) / KCH;
            *(lds_u4*)(Ad + swz(row, cch)) = mk_u4{ra[i].x, ra[i].y, ra[i].z, ra[i].w};
            if constexpr (STAGE == 1) {
                if (PEND) rdot[i] = dot8(ra[i], wk, rdot[i]);
                // ||G||^2 over real rows only (clamped rows repeat the last one)
                if (want_gsq) gsq = (m0 + row < M) ? sq8(ra[i], gsq) : gsq;
            }
        }
#pragma unroll
        for (int i = 0; i < BCH; ++i) {
            const int row = (t + i * NT) / KCH;
            *(lds_u4*)(Bd + swz(row, cch)) = mk_u4{rb[i].x, rb[i].y, rb[i].z, rb[i].w};
            if constexpr (STAGE == 2) {
                if (PEND) rdot[i] = dot8(rb[i], wk, rdot[i]);
            }
        }
    };

    // operands of one 16-deep k-step of a slab
    auto frags = [&](const lds_char* Ac, const lds_char* Bc, int ks, bf16x8 (&a)[FM], bf16x8 (&b)[FN]) {
        const int c = 2 * ks + lk;
#pragma unroll
        for (int i = 0; i < FM; ++i) a[i] = *(const lds_bf8*)(Ac + swz(wm * TM + i * 32 + li, c));
#pragma unroll
        for (int j = 0; j < FN; ++j) b[j] = *(const lds_bf8*)(Bc + swz(wn * TN + j * 32 + li, c));
    };
    auto mma = [&](const bf16x8 (&a)[FM], const bf16x8 (&b)[FN]) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };
    constexpr int KS = BK / 16;         // k-steps per slab
    constexpr int DS = FM + FN;         // LDS operand reads per k-step

    load(0);
    store(0, A0, B0);
    __syncthreads();
    for (int s = 0; s < nslab; ++s) {
        const int cur = s & 1;
        const bool more = s + 1 < nslab;
        if (more) load((s + 1) * BK);
        const lds_char* Ac = cur ? A1 : A0;
        const lds_char* Bc = cur ? B1 : B0;
        // one operand set per k-step: the other wave on the SIMD issues its
        // MFMAs while this one waits for its LDS reads
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            bf16x8 a[FM], b[FN];
            frags(Ac, Bc, ks, a, b);
            mma(a, b);
        }
        __builtin_amdgcn_sched_group_barrier(0x020, 32, 0);   // global loads of the next slab
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            __builtin_amdgcn_sched_group_barrier(0x100, DS, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, FM * FN, 0);
        }
        if (more) store((s + 1) * BK, cur ? A0 : A1, cur ? B0 : B1);
        __syncthreads();
    }

    // complete the rank-1 vector of the tile: the KCH threads of a row (adjacent
    // lanes) hold partial dots over their chunk columns
    constexpr int RROWS = STAGE == 1 ? BM : BN;
    if (PEND) {
#pragma unroll
        for (int i = 0; i < RCH; ++i) {
            float v = rdot[i];
#pragma unroll
            for (int o = 1; o < KCH; o <<= 1) v += __shfl_xor(v, o, 64);
            if (cch == 0) rvec[(t + i * NT) / KCH] = v;
        }
    }
    (void)RROWS;
    __syncthreads();

    const float c1 = PEND ? q.c1 : 1.f, c2 = PEND ? q.c2 : 0.f, sg = PEND ? q.sgn : 0.f;
    float csq = 0.f;
#pragma unroll
    for (int mi = 0; mi < FM; ++mi) {
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
            const int nl = wn * TN + ni * 32 + li, n = n0 + nl;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int ml = wm * TM + mi * 32 + 8 * g + 4 * lk, mb = m0 + ml;
                if (n >= N || mb >= M) continue;   // M, N are multiples of 64: 4 rows all in or all out
                float v[4] = {acc[mi][ni][4 * g + 0], acc[mi][ni][4 * g + 1], acc[mi][ni][4 * g + 2],
                              acc[mi][ni][4 * g + 3]};
                if constexpr (STAGE == 1) {
                    // Y = c1 (G S) + c2 G + sgn (G w) w^T, stored transposed in bf16
                    if (PEND) {
                        const float wn_ = gld(L.w + n);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const size_t go = (size_t)(mb + e) * K + n;   // G is d_in x d_out, K = d_out
                            const float gv = AF32 ? bf2f(f2bf(gld(static_cast<const float*>(L.A) + go)))
                                                  : bf2f(gld_u16(static_cast<const unsigned short*>(L.A) + go));
                            v[e] = fmaf(c1, v[e], fmaf(c2, gv, sg * rvec[ml + e] * wn_));
                        }
                    }
                    unsigned short* dst = static_cast<unsigned short*>(L.C) + (size_t)n * M + mb;
                    const uint2 h = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
                    gst_u2(dst, h);
                } else {
                    // dW_hat = c1 (S Y) + c2 Y + sgn w (w^T Y); Y[m][n] = Y^T[n][m]
                    if (PEND) {
                        const unsigned short* yt = static_cast<const unsigned short*>(L.B) + (size_t)n * K + mb;
                        const uint2 yh = gld_u2(yt);
                        const float y[4] = {bf2f((unsigned short)(yh.x & 0xffffu)), bf2f((unsigned short)(yh.x >> 16)),
                                            bf2f((unsigned short)(yh.y & 0xffffu)), bf2f((unsigned short)(yh.y >> 16))};
                        const float rn = rvec[nl];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            v[e] = fmaf(c1, v[e], fmaf(c2, y[e], sg * gld(L.w + mb + e) * rn));
                    }
                    float* dst = static_cast<float*>(L.C) + (size_t)mb * N + n;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        gst(dst + (size_t)e * N, v[e]);
                        csq = fmaf(v[e], v[e], csq);
                    }
                }
            }
        }
    }

    // partials: block-wide fixed-order sums
    const float part = STAGE == 1 ? gsq : csq;
    const float ws = wave_sum(part);
    if (lane == 0) red[wave] = ws;
    __syncthreads();
    if (t == 0 && (STAGE == 2 || want_gsq)) {
        float s = 0.f;
        for (int w = 0; w < NT / 64; ++w) s += red[w];
        if (STAGE == 1) gst(partials + L.part0 + tile.tm, s);
        else            gst(partials + L.part0 + tile.tm * L.ntn + tile.tn, s);
    }
}

constexpr int HG_SMEM = 2 * (BM + BN) * BK * 2 + 4 * ((BM > BN ? BM : BN) + NT / 64);

template <int STAGE>
__global__ __launch_bounds__(NT, 1) void hgemm_kernel(HgArgs args) {
    __shared__ __attribute__((aligned(16))) char smem_[HG_SMEM];
    lds_char* smem = (lds_char*)smem_;
    const GemmTile tile = args.tiles[blockIdx.x];
    if (tile.layer < 0) return;   // padding of the XCD interleave
    const HgLayer L = args.layers[tile.layer];
    const Pending q = *L.pend;
    if (STAGE == 1 && L.a_f32) {
        if (q.has) hgemm_tile<STAGE, true, true>(L, tile, q, args.partials, smem);
        else       hgemm_tile<STAGE, true, false>(L, tile, q, args.partials, smem);
    } else {
        if (q.has) hgemm_tile<STAGE, false, true>(L, tile, q, args.partials, smem);
        else       hgemm_tile<STAGE, false, false>(L, tile, q, args.partials, smem);
    }
}

}  // namespace

hipError_t launch_hgemm(int stage, const HgLayer* layers, const GemmTile* tiles, int32_t ntiles,
                        float* partials, hipStream_t stream) {
    if (ntiles <= 0) return hipSuccess;
    HgArgs a{layers, tiles, partials};
    if (stage == 1) hipLaunchKernelGGL(hgemm_kernel<1>, dim3(ntiles), dim3(NT), 0, stream, a);
    else            hipLaunchKernelGGL(hgemm_kernel<2>, dim3(ntiles), dim3(NT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace mkor
