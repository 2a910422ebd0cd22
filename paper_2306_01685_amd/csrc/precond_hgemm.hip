// Preconditioning for layers whose inverse factors are stored in bf16
// (half-precision factors: the paper's half-precision MKOR, whose Table 1
// halves the memory and the communication).  bf16 MFMA GEMMs
// (v_mfma_f32_32x32x16_bf16, fp32 accumulation) in the association
// dW_hat = L (G R), each stage written as  C = P_eff Q^T  with the factor as P:
//
//   stage 1:  Y^T = R G^T     P = S_R (d_out x d_out), Q = G in bf16 (d_in x
//                             d_out), C = Y^T rounded to bf16 (d_out x d_in),
//                             plus ||G||^2 partials;
//   stage 2:  dW_hat = L Y    P = S_L (d_in x d_in), Q = Y^T (d_out x d_in),
//                             C = dW_hat in fp32 (d_in x d_out), plus one
//                             ||dW_hat||^2 partial per tile.
//
// Both operands are contiguous along k in their natural layout (the factors
// are symmetric), which is what the MFMA wants: each lane supplies 8
// consecutive k of one row of P (output row i) and of Q (output column j).
//
// The factor is its stored bf16 value S plus the pending rank-1 term of the SM
// update, P_eff = c1 S + c2 I + sgn w w^T (struct Pending).  The MFMAs multiply
// with S; the epilogue adds the rest,
//   C[i][j] = c1 (S Q^T)[i][j] + c2 Q[j][i] + sgn w[i] (Q w)[j],
// where (Q w) is summed from the Q rows while they sit in LDS, and Q[j][i] is
// read at the output positions (4 consecutive i of one row j: one 8-byte load).
//
// Tiles of HG_BI x HG_BJ outputs (256 x 256), eight waves of 128 x 64 (4 x 2
// MFMA blocks), two per SIMD.  K runs in slabs of HG_BK (64) through an
// HG_NS-stage LDS ring (2 stages, 128 KB) filled by direct global-to-LDS loads
// (global_load_lds_dwordx4: lane l of a wave's instruction writes 16 bytes at
// M0 + 16 l), so the next slab streams in while one is multiplied and no
// registers hold staged data; within a slab the operand reads of k-step
// ks + 1 go out before the MFMAs of ks.  Each lane loads the global chunk
// that belongs at its LDS slot, which realises the swizzle of swz() below:
// the 16 rows of an MFMA operand read, and the rows of a rank-1 read, fall on
// 16 distinct 16-byte bank groups.  (Measured alternatives: 32-deep slabs in a
// 4-stage ring, and 256 x 128 tiles with two workgroups per CU, were within a
// few per cent, the latter moving 1.5x the bytes through the vector memory
// path.)
//
// The K loop holds no compiler-visible global access: completion of the
// direct loads is tracked by hand with s_waitcnt vmcnt (loads complete in
// order, so waiting until at most n are outstanding leaves exactly the last n
// issued), and the slab barrier is a bare s_barrier (the compiler's barrier
// would also wait for every prefetch).  d_in and d_out are multiples of 64
// (checked by the plan); tile edges are masked, rows past the edge are loaded
// clamped to the last row and never stored.
#include "gmem.h"
#include "mkor_internal.h"

namespace mkor {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
// LDS pointers carry their address space, so every operand access is a
// ds_read / ds_write (a generic pointer would become a flat access, which
// also waits on the global-load counter).
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) mk_u4 lds_u4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf8;
typedef __attribute__((address_space(3))) float lds_float;
typedef __attribute__((address_space(3))) unsigned short lds_u16;
typedef __attribute__((address_space(3))) mk_f4 lds_f4;

__device__ __forceinline__ float4 lds4(const lds_float* p) {
    const mk_f4 v = *(const lds_f4*)p;
    return make_float4(v.x, v.y, v.z, v.w);
}

constexpr int BI = HG_BI, BJ = HG_BJ, NT = HG_THREADS;
constexpr int WI = BI / 128, WJ = BJ / HG_TJ;   // wave grid
constexpr int TI = BI / WI, TJ = BJ / WJ;        // 128 x HG_TJ per wave
constexpr int FI = TI / 32, FJ = TJ / 32;        // 4 x 2 or 4 x 4 MFMA blocks
static_assert(NT == WI * WJ * 64 && TI == 128 && (TJ == 64 || TJ == 128), "wave layout");

constexpr int BK = HG_BK, NS = HG_NS;         // slab depth, ring stages
static_assert(BK == 32 || BK == 64, "slab rows of 64 or 128 bytes");
constexpr int KC = BK / 8;                    // 16-byte chunks per slab row
constexpr int RPB = 64 / KC;                  // rows per 1-KB load block
constexpr int ROWB = BK * 2;                  // bytes per slab row
constexpr int PB = BI * ROWB, QB = BJ * ROWB; // P and Q bytes per stage
constexpr int STB = PB + QB;
constexpr int WSLOT = 256;                    // w[k0 .. k0 + 64) per stage (BK used)
constexpr int NW = NT / 64;
constexpr int PBLK = PB / 1024 / NW, QBLK = QB / 1024 / NW;   // 1-KB load blocks per wave and slab
static_assert(PB % (1024 * NW) == 0 && QB % (1024 * NW) == 0, "load blocks per wave");
constexpr int TPQ = NT / BJ;                  // threads per Q row in the rank-1 reads
static_assert(TPQ * BJ == NT && (TPQ == 1 || TPQ == 2), "rank-1 reads: a whole or half Q row per thread");
constexpr int RING = NS * STB;
// Stage-1 output staging: the bf16 tile, rows of BJ * 2 bytes with the
// 16-byte chunk index XORed with the row, in the ring once the K loop is done.
constexpr int CPITCH = BJ * 2, CCH = BJ / 8;
static_assert(BI * CPITCH <= RING && (CCH & (CCH - 1)) == 0, "output staging fits in the ring");
__device__ __forceinline__ int cst(int r, int cj) { return r * CPITCH + ((cj ^ (r & (CCH - 1))) << 4); }
constexpr int SMEM = RING + NS * WSLOT + 4 * (BJ + NW + BI);   // ring, w slices, (Q w), block sums, w rows

// Row r's chunk c sits in 16-byte slot c ^ f(r): for 64-byte rows f(r) =
// (r >> 2) & 3, for 128-byte rows f(r) = (r & 7) ^ ((r >> 3) & 1).  Either way
// the 16 rows an operand read touches at one chunk fill 16 distinct 16-byte
// bank groups.
#ifndef MKOR_HG_PRIO
#define MKOR_HG_PRIO 0
#endif
#ifndef MKOR_HG_FDB
#define MKOR_HG_FDB 1
#endif

__device__ __forceinline__ int swf(int r) { return KC == 4 ? ((r >> 2) & 3) : ((r & 7) ^ ((r >> 3) & 1)); }
__device__ __forceinline__ int swz(int r, int c) { return r * ROWB + ((c ^ swf(r)) << 4); }

__device__ __forceinline__ void dma16(unsigned lds, unsigned voff, const void* base) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(base)
                 : "memory");
}
__device__ __forceinline__ void dma4(unsigned lds, unsigned voff, const void* base) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2" ::"s"(lds), "v"(voff), "s"(base)
                 : "memory");
}

// Wait until this wave's loads of a slab have landed, with `ahead` (at most
// 2) later slabs of D instructions each still in flight.
template <int D>
__device__ __forceinline__ void dma_wait(int ahead) {
    if (ahead >= 2)      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * D) : "memory");
    else if (ahead == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(D) : "memory");
    else                 asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}
static_assert(NS >= 2 && NS <= 4, "dma_wait covers up to two slabs in flight behind the awaited one");

__device__ __forceinline__ void slab_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ void unpack8(const mk_u4& h, float (&v)[8]) {
    const unsigned u[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf2f((unsigned short)(u[i] & 0xffffu));
        v[2 * i + 1] = bf2f((unsigned short)(u[i] >> 16));
    }
}

struct HgArgs {
    const HgLayer* layers;
    const GemmTile* tiles;
    float* partials;
};

template <int STAGE, bool PEND>
__device__ void hgemm_tile(const HgLayer& L, const GemmTile& tile, const Pending& q, float* partials,
                           lds_char* smem) {
    const int i0 = tile.tm * BI, j0 = tile.tn * BJ;
    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int wi = wave % WI, wj = wave / WI;
    const int li = lane & 31, lk = lane >> 5;
    const int I = L.I, J = L.J, K = L.K;
    const bool want_gsq = STAGE == 1 && tile.tm == 0;   // ||G||^2: each Q row once
    lds_float* rvec = (lds_float*)(smem + RING + NS * WSLOT);
    lds_float* red = rvec + BJ;
    lds_float* ewv = red + NW;   // w over the tile's rows, for the epilogue
    const unsigned lds0 = (unsigned)(size_t)smem;

    floatx16 acc[FI][FJ];
#pragma unroll
    for (int a = 0; a < FI; ++a)
#pragma unroll
        for (int b = 0; b < FJ; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    // this lane's load sources at k0 = 0 (byte offsets from the operand base)
    // lane l of a block writes slot l % KC of row l / KC: it loads that row's
    // chunk (l % KC) ^ f(row)
    unsigned vp[PBLK], vq[QBLK];
#pragma unroll
    for (int b = 0; b < PBLK; ++b) {
        const int r = RPB * (PBLK * wave + b) + lane / KC;
        const int c = (lane % KC) ^ swf(r);
        vp[b] = ((unsigned)min(i0 + r, I - 1) * (unsigned)K + 8u * c) * 2u;
    }
#pragma unroll
    for (int b = 0; b < QBLK; ++b) {
        const int r = RPB * (QBLK * wave + b) + lane / KC;
        const int c = (lane % KC) ^ swf(r);
        vq[b] = ((unsigned)min(j0 + r, J - 1) * (unsigned)K + 8u * c) * 2u;
    }
    const int nst = K / BK;
    constexpr int D = PBLK + QBLK;               // load instructions per wave and slab
    const bool wload = PEND && wave == 0;        // wave 0 also brings the slab's slice of w
    auto issue = [&](int st) {
        const unsigned buf = lds0 + (unsigned)(st % NS) * STB;
        const unsigned kb = (unsigned)st * ROWB;
#pragma unroll
        for (int b = 0; b < PBLK; ++b) dma16(buf + (PBLK * wave + b) * 1024, vp[b] + kb, L.P);
#pragma unroll
        for (int b = 0; b < QBLK; ++b) dma16(buf + PB + (QBLK * wave + b) * 1024, vq[b] + kb, L.Q);
        if (wload)
            dma4(lds0 + RING + (unsigned)(st % NS) * WSLOT, (unsigned)min(st * BK + lane, K - 1) * 4u, L.w);
    };

    // rank-1 dot (and ||G||^2) of this thread's part of a Q row: row t / TPQ,
    // chunks h KC / TPQ .. (h + 1) KC / TPQ - 1, summed in a fixed order over
    // the slabs.  The squares go into a short fp32 sum per slab, accumulated
    // in fp64: one fp32 chain of K / TPQ positive terms drifts low by several
    // 1e-6 relative, a bias the rescale would carry into every element of dW.
    const int rr = t / TPQ, rh = t % TPQ;
    float rdot = 0.f;
    double gsq = 0.0;
    const bool gsq_row = want_gsq && j0 + rr < J;

    for (int st = 0; st < NS - 1 && st < nst; ++st) issue(st);
    for (int s = 0; s < nst; ++s) {
        const int ahead = min(NS - 2, nst - 1 - s);
        if (wload) dma_wait<D + 1>(ahead);
        else       dma_wait<D>(ahead);
        slab_barrier();   // every wave's slab s has landed; slab s - 1 is no longer read
        if (s + NS - 1 < nst) issue(s + NS - 1);
        const lds_char* Pb = smem + (s % NS) * STB;
        const lds_char* Qb = Pb + PB;
        auto frags = [&](int ks, bf16x8 (&a)[FI], bf16x8 (&b)[FJ]) {
            const int c = 2 * ks + lk;
#pragma unroll
            for (int x = 0; x < FI; ++x) a[x] = *(const lds_bf8*)(Pb + swz(wi * TI + x * 32 + li, c));
#pragma unroll
            for (int y = 0; y < FJ; ++y) b[y] = *(const lds_bf8*)(Qb + swz(wj * TJ + y * 32 + li, c));
        };
        auto mma = [&](const bf16x8 (&a)[FI], const bf16x8 (&b)[FJ]) {
            if (MKOR_HG_PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int x = 0; x < FI; ++x)
#pragma unroll
                for (int y = 0; y < FJ; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[x], b[y], acc[x][y], 0, 0, 0);
            if (MKOR_HG_PRIO) __builtin_amdgcn_s_setprio(0);
        };
        if constexpr (MKOR_HG_FDB) {
            // two operand sets: the reads of k-step ks + 1 go out before the MFMAs of ks
            bf16x8 a0[FI], b0[FJ], a1[FI], b1[FJ];
            frags(0, a0, b0);
#pragma unroll
            for (int ks = 0; ks < BK / 16; ks += 2) {
                frags(ks + 1, a1, b1);
                mma(a0, b0);
                if (ks + 2 < BK / 16) frags(ks + 2, a0, b0);
                mma(a1, b1);
            }
        } else {
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
                bf16x8 a[FI], b[FJ];
                frags(ks, a, b);
                mma(a, b);
            }
        }
        if (PEND || want_gsq) {
            const lds_float* wsl = (const lds_float*)(smem + RING + (s % NS) * WSLOT);
            float part = 0.f;
#pragma unroll
            for (int e = 0; e < KC / TPQ; ++e) {
                const int c = (KC / TPQ) * rh + e;
                float v[8];
                const mk_u4 hv = *(const lds_u4*)(Qb + swz(rr, c));
                unpack8(hv, v);
                if (PEND) {
#pragma unroll
                    for (int x = 0; x < 8; ++x) rdot = fmaf(v[x], wsl[8 * c + x], rdot);
                }
                if (STAGE == 1 && gsq_row) {
#pragma unroll
                    for (int x = 0; x < 8; ++x) part = fmaf(v[x], v[x], part);
                }
            }
            if (STAGE == 1 && gsq_row) gsq += (double)part;
        }
    }

    if (PEND) {
        const float v = TPQ == 2 ? rdot + __shfl_xor(rdot, 1, 64) : rdot;
        if (rh == 0) rvec[rr] = v;
        // w of the tile's rows into LDS ahead of the stores: a global load
        // issued after stores shares the vector-memory counter with them, so
        // waiting for its value would also wait for those stores (rows past
        // the edge clamped; their outputs are never stored)
        for (int r = t; r < BI; r += NT) ewv[r] = gld(L.w + min(i0 + r, I - 1));
    }
    __syncthreads();   // rvec and w complete; the ring is free for the output staging

    const float c1 = PEND ? q.c1 : 1.f, c2 = PEND ? q.c2 : 0.f, sg = PEND ? q.sgn : 0.f;
    float csq = 0.f;
    // One MFMA row block (x) at a time: first the values its output groups
    // need (w from LDS; Q[j][i] from global memory, rows past the edge
    // clamped, so the loads go out together without branches), then
    // C[i][j] = c1 acc + c2 Q[j][i] + sgn w[i] (Q w)[j].  c2 is zero unless
    // the stabiliser blended the factor (Alg. 1): Q[j][i] is only read when
    // it counts (a branch on a value uniform over the tile).
    const bool qterm = PEND && c2 != 0.f;
#pragma unroll
    for (int x = 0; x < FI; ++x) {
        uint2 qh[FJ][4];
        float4 wv[4];
        if (PEND) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int il = wi * TI + x * 32 + 8 * g + 4 * lk, i = min(i0 + il, I - 4);
                wv[g] = lds4(ewv + il);
#pragma unroll
                for (int y = 0; y < FJ; ++y) {
                    const int j = min(j0 + wj * TJ + y * 32 + li, J - 1);
                    qh[y][g] = qterm ? gld_u2(static_cast<const unsigned short*>(L.Q) + (size_t)j * K + i)
                                     : make_uint2(0u, 0u);
                }
            }
        }
#pragma unroll
        for (int y = 0; y < FJ; ++y) {
            const int jl = wj * TJ + y * 32 + li, j = j0 + jl;
            const float rq = PEND ? rvec[jl] : 0.f;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int il = wi * TI + x * 32 + 8 * g + 4 * lk, i = i0 + il;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[x][y][4 * g + e];
                if (PEND) {
                    const float qv[4] = {bf2f((unsigned short)(qh[y][g].x & 0xffffu)),
                                         bf2f((unsigned short)(qh[y][g].x >> 16)),
                                         bf2f((unsigned short)(qh[y][g].y & 0xffffu)),
                                         bf2f((unsigned short)(qh[y][g].y >> 16))};
                    const float wa[4] = {wv[g].x, wv[g].y, wv[g].z, wv[g].w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = fmaf(c1, v[e], fmaf(c2, qv[e], sg * wa[e] * rq));
                }
                if constexpr (STAGE == 1) {
                    // bf16 into the staging tile (stored row by row below)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        *(lds_u16*)(smem + cst(il + e, jl >> 3) + 2 * (jl & 7)) = f2bf(v[e]);
                } else if (i < I && j < J) {   // I, J multiples of 64: 4 rows all in or all out
                    float* dst = static_cast<float*>(L.C) + (size_t)i * J + j;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        gst(dst + (size_t)e * J, v[e]);
                        csq = fmaf(v[e], v[e], csq);
                    }
                }
            }
        }
    }
    if constexpr (STAGE == 1) {
        __syncthreads();
        // Y^T rows of the tile, 16 bytes per lane
        for (int u = t; u < BI * CCH; u += NT) {
            const int il = u / CCH, cj = u % CCH;
            const int i = i0 + il, j = j0 + 8 * cj;
            if (i < I && j < J) {
                const mk_u4 h = *(const lds_u4*)(smem + cst(il, cj));
                gst_u4(static_cast<unsigned short*>(L.C) + (size_t)i * J + j, make_uint4(h.x, h.y, h.z, h.w));
            }
        }
    }

    // partials: block-wide fixed-order sums
    const float part = STAGE == 1 ? (float)gsq : csq;
    const float ws = wave_sum(part);
    if (lane == 0) red[wave] = ws;
    __syncthreads();
    if (t == 0 && (STAGE == 2 || want_gsq)) {
        float s = 0.f;
        for (int w = 0; w < NW; ++w) s += red[w];
        if (STAGE == 1) gst(partials + L.part0 + tile.tn, s);
        else            gst(partials + L.part0 + tile.tm * L.ntj + tile.tn, s);
    }
}

// 8 waves per CU (2 per SIMD): at most 256 VGPRs per lane.
template <int STAGE>
__global__ __launch_bounds__(NT, 1) void hgemm_kernel(HgArgs args) {
    __shared__ __attribute__((aligned(16))) char smem_[SMEM];
    lds_char* smem = (lds_char*)smem_;
    const GemmTile tile = args.tiles[blockIdx.x];
    if (tile.layer < 0) return;   // padding of the XCD interleave
    const HgLayer L = args.layers[tile.layer];
    if (!gld_i32(L.mode)) return;   // first-order layer this step
    const Pending q = *L.pend;
    if (q.has) hgemm_tile<STAGE, true>(L, tile, q, args.partials, smem);
    else       hgemm_tile<STAGE, false>(L, tile, q, args.partials, smem);
}

// fp32 gradients of bf16-factor layers, rounded to bf16 once per step.
__global__ __launch_bounds__(256) void cvt_bf16_kernel(const CvtItem* __restrict__ items,
                                                      const CvtBlock* __restrict__ blocks) {
    const CvtBlock b = blocks[blockIdx.x];
    const CvtItem it = items[b.item];
    if (!gld_i32(it.mode)) return;
    const int64_t end = min(b.off + (int64_t)CVT_ELEMS, it.n);
    for (int64_t e = b.off + 8 * (int64_t)threadIdx.x; e < end; e += 8 * 256) {
        const float4 x0 = gld4_nt(it.src + e), x1 = gld4_nt(it.src + e + 4);
        gst_u4(it.dst + e, make_uint4(f2bf2(x0.x, x0.y), f2bf2(x0.z, x0.w), f2bf2(x1.x, x1.y), f2bf2(x1.z, x1.w)));
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

hipError_t launch_cvt_bf16(const CvtItem* items, const CvtBlock* blocks, int32_t nblocks, hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(cvt_bf16_kernel, dim3(nblocks), dim3(256), 0, stream, items, blocks);
    return hipGetLastError();
}

}  // namespace mkor
