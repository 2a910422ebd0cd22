// Preconditioning of fp32-factor layers on the bf16 matrix cores, to fp32
// accuracy (Algorithm 1, precondition line; Eq. 2).  Every fp32 operand value
// x is carried as the sum of three bf16 values,
//
//   x = h + m + l,   h = bf16(x),  m = bf16(x - h),  l = bf16(x - h - m)
//
// (round to nearest even).  Both differences are exact in fp32 (Sterbenz), and
// x - h - m is a multiple of ulp(x) no larger than 2^-16 |x|, i.e. it has at
// most 8 significant bits, so l holds it exactly: the split is exact for
// 2^-110 <= |x| < 3.396e38 (below, l loses bits under bf16's subnormal floor;
// above, h overflows).  A product of two split values is the sum of nine bf16
// products; the three smallest (m l', l m', l l') are below 2^-23 |x x'| and are
// left out, the same order as one fp32 rounding.  Each bf16 x bf16 product is
// exact in the fp32 accumulator of v_mfma_f32_32x32x16_bf16, so the result
// carries fp32 accumulation error, like the fp32 MFMA path, at six (or, for a
// bf16 operand, which needs no split, three) bf16 MFMAs per product.  The
// bf16 matrix cores run sixteen times the fp32 rate.
//
// Association and operands as in the bf16-factor path, C = P_eff Q^T with the
// factor as P:
//   stage 1:  Y^T = R G^T     P = S_R (d_out x d_out, fp32), Q = G (d_in x
//                             d_out, bf16 or fp32), C = Y^T in fp32 (d_out x
//                             d_in); its (Q w) and the ||G||^2 partials come
//                             from the row pass ahead of it (qdot_kernel);
//   stage 2:  dW_hat = L Y    P = S_L (d_in x d_in, fp32), Q = Y^T (fp32),
//                             C = dW_hat in fp32, plus ||dW_hat||^2 partials.
// Layers with a bf16 G and d_in > d_out take the other association, so that
// their longer contraction has the bf16 operand: stage 1 X = L G (P = S_L,
// Q = G^T), stage 2 dW_hat = X R with the factor as the Q operand (P = X,
// Q = S_R).  The pending term of the SM update, P_eff = c1 S + c2 I +
// sgn w w^T, enters as
//   C[i][j] = c1 ((S + (c2 / c1) I) Q^T)[i][j] + sgn w[i] (Q w)[j]
// (factor as Q: c1 (P (S + (c2 / c1) I)^T)[i][j] + sgn w[j] (P w)[i]): the
// diagonal shift is added to the factor as it is staged (one fp32 rounding
// of each diagonal entry), c1 and the rank-1 term in the epilogue, with the
// matrix-vector product summed in fp32 from the staged rows (second GEMM)
// or by a row pass ahead of the first.
//
// Eight waves, two per SIMD, each with 128 accumulator registers (Geo: 256 x
// 256 tiles, or 128 x 512 for a bf16 Q where the layer fills them).  K runs
// in slabs (16 deep when Q is fp32, 32 when it is bf16, so that the rings fit
// in LDS): each thread loads its part of a slab row of P (and of an fp32 Q)
// into registers one slab ahead, splits it and writes the planes into a
// two-stage LDS ring with 16-byte writes.  A bf16 Q needs no
// split: its slab goes from global memory straight into a three-slot LDS ring
// (global_load_lds_dwordx4), in the same swizzle.  A plane row is BK * 2 bytes
// in 16-byte chunks; chunk c of row r sits in slot c ^ f(r).  A 16-byte LDS
// read is served 16 lanes at a time from 16 bank groups of 16 bytes, a 16-byte
// write 8 lanes at a time from 8 (address / 16 mod 8; measured with the bank
// conflict counter), so f(r) = (r >> 3) & 1 for 32-byte rows and
// ((r >> 2) & 3) ^ ((r >> 1) & 1) for 64-byte rows put the 16 rows of an MFMA
// operand read on 16 groups and the 8 lanes of a staging write on 8: no bank
// conflicts in either direction.  d_in and d_out are multiples of 64 (checked by the
// plan); rows past a tile edge are loaded clamped to the last row and never
// stored.
#include "gmem.h"
#include "mkor_internal.h"

namespace mkor {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) mk_u4 lds_u4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf8;
typedef __attribute__((address_space(3))) float lds_float;

constexpr int NT = 512;
constexpr int NW = NT / 64;

// Tile, wave layout and ring geometry (GV): an fp32 Q (GV_F32): 256 x 256
// tiles, waves of 128 x 64, six planes per slab.  A bf16 Q (three P planes,
// one Q plane) with waves of 64 x 128, which read fewer operand bytes per
// MFMA: 256 x 256 tiles (GV_H) or 128 x 512 (GV_HW), which halve the fp32 P
// bytes per output for the same accumulators (the P rows pass through
// registers and the split, the Q rows go straight into LDS) where the layer
// fills them as well.  A bf16 Q has a ring of its own, three slots of one
// plane after the P stages.
enum { GV_F32 = 0, GV_H = 1, GV_HW = 2 };
template <int GV> struct Geo {
    static constexpr bool QF = GV == GV_F32;
    static constexpr int BI = GV == GV_HW ? SG_BI1H : SG_BI, BJ = GV == GV_HW ? SG_BJ1H : SG_BJ;   // tile
    static constexpr int WI = GV == GV_H ? 4 : 2, WJ = NW / WI;   // wave grid
    static constexpr int TI = BI / WI, TJ = BJ / WJ;      // outputs per wave
    static constexpr int FI = TI / 32, FJ = TJ / 32;      // MFMA blocks per wave
    static constexpr int NQ = QF ? 3 : 1;          // Q planes
    static constexpr int BK = QF ? 16 : 32;        // slab depth
    static constexpr int KS = BK / 16;             // MFMA k-steps per slab
    static constexpr int TPR = NT / BI;            // staging threads per P row
    static constexpr int HK = BK / TPR;            // k per thread and slab
    static constexpr int ROWB = BK * 2;            // bytes per plane row
    static constexpr int PLANE = BI * ROWB;        // a P plane (an fp32 Q's too: BJ == BI)
    static constexpr int QPLANE = BJ * ROWB;       // a Q plane
    static constexpr int STB = (QF ? 6 : 3) * PLANE;   // one ring stage (P and, for an fp32 Q, Q)
    static constexpr int QRING = 2 * STB;              // bf16 Q: three slots of one plane
    static constexpr int RING = QF ? 2 * STB : QRING + 3 * QPLANE;
    static_assert(!QF || BI == BJ, "an fp32 Q is staged by the threads that stage P");
    static_assert(HK % 8 == 0, "whole 16-byte chunks per thread, row and plane");
};
constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int RING = cmax(Geo<GV_F32>::RING, cmax(Geo<GV_H>::RING, Geo<GV_HW>::RING));   // 144 KB
constexpr int BJMAX = SG_BJ > SG_BJ1H ? SG_BJ : SG_BJ1H;
constexpr int BIMAX = SG_BI > SG_BI1H ? SG_BI : SG_BI1H;
// after the ring: (P w) or (Q w) of the second GEMM's rows, the block
// reduction, and the epilogue's vectors (w over the tile's rows, or columns
// when FQ, then the second term's; (Q w) over its columns, then the second
// term's)
constexpr int EW = BJMAX + NW, EQ = EW + 2 * (BIMAX > BJMAX ? BIMAX : BJMAX);
constexpr int SMEM = RING + 4 * (EQ + 2 * BJMAX);

__device__ __forceinline__ void dma16(unsigned lds, unsigned voff, const void* base) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(base)
                 : "memory");
}

template <int ROWB>
__device__ __forceinline__ int slot(int r, int c) {
    return ROWB == 32 ? r * 32 + ((c ^ ((r >> 3) & 1)) << 4)
                      : r * 64 + ((c ^ ((r >> 2) & 3) ^ ((r >> 1) & 1)) << 4);
}

typedef __attribute__((address_space(3))) mk_f4 lds_f4;
__device__ __forceinline__ float4 lds4(const lds_float* p) {
    const mk_f4 v = *(const lds_f4*)p;
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// 8 values -> their three bf16 planes (packed pairs, element 2e in the low half)
__device__ __forceinline__ void split8(const float* v, mk_u4& hi, mk_u4& mi, mk_u4& lo) {
    unsigned h[4], m[4], l[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float x0 = v[2 * e], x1 = v[2 * e + 1];
        h[e] = f2bf2(x0, x1);
        const float r0 = __fsub_rn(x0, __uint_as_float(h[e] << 16));
        const float r1 = __fsub_rn(x1, __uint_as_float(h[e] & 0xffff0000u));
        m[e] = f2bf2(r0, r1);
        const float s0 = __fsub_rn(r0, __uint_as_float(m[e] << 16));
        const float s1 = __fsub_rn(r1, __uint_as_float(m[e] & 0xffff0000u));
        l[e] = f2bf2(s0, s1);
    }
    hi = mk_u4{h[0], h[1], h[2], h[3]};
    mi = mk_u4{m[0], m[1], m[2], m[3]};
    lo = mk_u4{l[0], l[1], l[2], l[3]};
}

struct SgArgs {
    const HgLayer* layers;
    const GemmTile* tiles;
    float* partials;
};

// GV: tile geometry (Q fp32 in three planes, or bf16 in one, exact as it
// is).  FQ: the factor is the Q operand (C = P Q_eff^T; the epilogue adds
// sgn w[j] (P w)[i], with (P w) summed from the staged P rows).
// PM: pending term of the factor: none (0), c2 = 0 (1: no stabiliser blend,
// no diagonal shift), or c2 != 0 (2).
template <int STAGE, int GV, int PM, bool FQ>
__device__ void sgemm_tile(const HgLayer& L, const GemmTile& tile, const Pending& q, float* partials,
                           lds_char* smem) {
    using G = Geo<GV>;
    constexpr bool PEND = PM != 0, DIAG = PM == 2;
    constexpr bool QF = G::QF;
    constexpr bool QDMA = !QF;   // bf16 Q (first GEMM only)
    static_assert(!QDMA || STAGE == 1, "a bf16 Q operand is the first GEMM's");
    constexpr int BI = G::BI, BJ = G::BJ, WI = G::WI, TI = G::TI, TJ = G::TJ, FI = G::FI, FJ = G::FJ;
    static_assert(NT == WI * G::WJ * 64, "wave layout");
    constexpr int NQ = G::NQ, BK = G::BK, KS = G::KS, HK = G::HK, ROWB = G::ROWB, PLANE = G::PLANE;
    constexpr int NC = HK / 8;                     // 16-byte chunks per thread and plane
    const int i0 = tile.tm * BI, j0 = tile.tn * BJ;
    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int wi = wave % WI, wj = wave / WI;
    const int li = lane & 31, lk = lane >> 5;
    const int I = L.I, J = L.J, K = L.K;
    lds_float* rvec = (lds_float*)(smem + RING);
    lds_float* red = rvec + BJMAX;
    lds_float* ew = rvec + EW;
    lds_float* eq = rvec + EQ;

    floatx16 acc[FI][FJ];
#pragma unroll
    for (int a = 0; a < FI; ++a)
#pragma unroll
        for (int b = 0; b < FJ; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

    // staging: thread t owns row sr of the P tile (and of an fp32 Q tile),
    // k part sh
    const int sr = t / G::TPR, sh = t % G::TPR;
    const float* Pp = static_cast<const float*>(L.P) + (size_t)min(i0 + sr, I - 1) * K + HK * sh;
    const size_t qoff = (size_t)min(j0 + sr, J - 1) * K + HK * sh;
    const float* Qf = static_cast<const float*>(L.Q) + qoff;
    const float* Wp = L.w + HK * sh;

    // one slab's operands staged through registers (P, and Q when it is
    // fp32), and the w slice of a slab (cached: every thread of a tile reads
    // the same one)
    struct Regs {
        float p[HK], q[QF ? HK : 1];
    };
    // stage 1 takes (Q w) from qdot_kernel: its loop stages no w slice
    constexpr bool RDOT = PEND && STAGE == 2;
    float wr[RDOT ? HK : 1];
    auto load_w = [&](int s) {
        if constexpr (RDOT) {
            const int k0 = s * BK;
#pragma unroll
            for (int c = 0; c < HK / 4; ++c) {
                const float4 v = gld4(Wp + k0 + 4 * c);
                wr[4 * c] = v.x; wr[4 * c + 1] = v.y; wr[4 * c + 2] = v.z; wr[4 * c + 3] = v.w;
            }
        }
    };
    auto wsel = [&](int e) { return wr[e]; };
    auto load = [&](Regs& R, int s) {
        const int k0 = s * BK;
#pragma unroll
        for (int c = 0; c < HK / 4; ++c) {
            const float4 v = gld4(Pp + k0 + 4 * c);
            R.p[4 * c] = v.x; R.p[4 * c + 1] = v.y; R.p[4 * c + 2] = v.z; R.p[4 * c + 3] = v.w;
        }
        if constexpr (QF) {
#pragma unroll
            for (int c = 0; c < HK / 4; ++c) {
                const float4 v = gld4(Qf + k0 + 4 * c);
                R.q[4 * c] = v.x; R.q[4 * c + 1] = v.y; R.q[4 * c + 2] = v.z; R.q[4 * c + 3] = v.w;
            }
        }
    };
    // bf16 Q of slab s into slot qs of the Q ring: wave w fills NQB 1-KB
    // blocks of 16 rows; lane l of a block lands at byte 16 l, so it loads
    // the chunk that the swizzle puts there (row r = l / 4 of the block,
    // chunk (l % 4) ^ f(r))
    constexpr int NQB = QDMA ? G::QPLANE / 1024 / NW : 1;
    unsigned qoffs[NQB];
#pragma unroll
    for (int b = 0; b < NQB; ++b) {
        const int r = 16 * (NQB * wave + b) + (lane >> 2);
        const int c = (lane & 3) ^ ((r >> 2) & 3) ^ ((r >> 1) & 1);
        qoffs[b] = ((unsigned)min(j0 + r, J - 1) * (unsigned)K) * 2u + 16u * c;
    }
    const unsigned lds_q = (unsigned)(size_t)smem + G::QRING;
    auto dma_q = [&](int s, int qs) {
        if constexpr (QDMA) {
#pragma unroll
            for (int b = 0; b < NQB; ++b)
                dma16(lds_q + qs * G::QPLANE + 1024u * (NQB * wave + b), qoffs[b] + 2u * s * BK, L.Q);
        }
    };
    float rdot = 0.f;
    // split the registers of a slab into ring stage st; (Q w) (or, FQ, (P w))
    // partial sums in a fixed order
    // The pending term's c2 I enters through the staged factor (P, or Q when
    // FQ): its diagonal entry is staged as S_ii + c2 / c1, rounded once in
    // fp32 like the c1 scaling of the output, so the epilogue reads no second
    // copy of the other operand.  frow: the factor row this thread stages.
    const int frow = FQ ? min(j0 + sr, J - 1) : min(i0 + sr, I - 1);
    const float dd = PEND ? q.c2 / q.c1 : 0.f;
    auto stage = [&](const Regs& R, int st, bool count, int sl) {
        lds_char* buf = smem + st * G::STB;
        float pv[HK], qv[QF ? HK : 1];
#pragma unroll
        for (int e = 0; e < HK; ++e) {
            pv[e] = R.p[e];
            if constexpr (QF) qv[e] = R.q[e];
        }
        if constexpr (DIAG) {   // selects, not a branch: the slab stays one basic block
            const int dk = frow - (sl * BK + HK * sh);   // the diagonal's place in this thread's part
            float* f = FQ ? qv : pv;
#pragma unroll
            for (int e = 0; e < HK; ++e) f[e] = e == dk ? __fadd_rn(f[e], dd) : f[e];
        }
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int o = slot<ROWB>(sr, NC * sh + c);
            mk_u4 hi, mi, lo;
            split8(pv + 8 * c, hi, mi, lo);
            *(lds_u4*)(buf + o) = hi;
            *(lds_u4*)(buf + PLANE + o) = mi;
            *(lds_u4*)(buf + 2 * PLANE + o) = lo;
        }
        if constexpr (QF) {
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int o = slot<ROWB>(sr, NC * sh + c);
                mk_u4 hi, mi, lo;
                split8(qv + 8 * c, hi, mi, lo);
                *(lds_u4*)(buf + 3 * PLANE + o) = hi;
                *(lds_u4*)(buf + 4 * PLANE + o) = mi;
                *(lds_u4*)(buf + 5 * PLANE + o) = lo;
            }
        }
        if constexpr (RDOT) {   // the second GEMM only, whose Q is fp32
            float r = rdot;
#pragma unroll
            for (int e = 0; e < HK; ++e) r = fmaf(FQ ? R.p[e] : R.q[e], wsel(e), r);
            rdot = count ? r : rdot;
        }
    };
    constexpr int NTERM = QF ? 6 : 3;
    // MFMA k-step ks of ring stage st: plane pairs with p + q <= 2, the small
    // terms first
    auto compute = [&](int st, int qs, int ks) {
        const lds_char* buf = smem + st * G::STB;
        const lds_char* qbuf = QDMA ? smem + G::QRING + qs * G::QPLANE : buf + 3 * PLANE;
        const int c = 2 * ks + lk;
        bf16x8 a[3][FI], b[NQ][FJ];
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
            for (int x = 0; x < FI; ++x) a[p][x] = *(const lds_bf8*)(buf + p * PLANE + slot<ROWB>(wi * TI + x * 32 + li, c));
#pragma unroll
        for (int p = 0; p < NQ; ++p)
#pragma unroll
            for (int y = 0; y < FJ; ++y)
                b[p][y] = *(const lds_bf8*)(qbuf + p * PLANE + slot<ROWB>(wj * TJ + y * 32 + li, c));
        constexpr int TP[6] = {2, 1, 0, 1, 0, 0}, TQ[6] = {0, 1, 2, 0, 1, 0};
        constexpr int UP[3] = {2, 1, 0};
#pragma unroll
        for (int u = 0; u < NTERM; ++u) {
            const int pp = QF ? TP[u] : UP[u], qq = QF ? TQ[u] : 0;
#pragma unroll
            for (int x = 0; x < FI; ++x)
#pragma unroll
                for (int y = 0; y < FJ; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[pp][x], b[qq][y], acc[x][y], 0, 0, 0);
        }
    };

    const int nst = K / BK;   // even: K is a multiple of 64
    // One basic block per slab, so that the scheduler can interleave the
    // split and LDS writes of slab s + 1 (into the other ring stage, whose
    // last reader finished before the barrier) and the loads of slab s + 2
    // with the MFMAs of slab s.  Past the end the loads are clamped to the
    // last slab, which is then re-staged into the stage nobody reads again,
    // without counting towards (Q w) and ||G||^2.
    // A bf16 Q slab goes into its slot with the loads of the P slab it pairs
    // with, one slab ahead of the split and two ahead of the MFMAs; the slot
    // is the one slab s - 1 used, whose readers finished before the last
    // barrier, and the wait ahead of the split (which also covers these DMA
    // loads, issued after the register loads it waits for) completes it one
    // barrier before compute reads it.
    Regs R;
    load(R, 0);
    load_w(0);
    dma_q(0, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    stage(R, 0, true, 0);
    load(R, 1);
    load_w(1);
    dma_q(1, 1);
    __syncthreads();
    constexpr int NMF = FI * FJ * NTERM * KS;
    for (int s = 0; s < nst; ++s) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) compute(s & 1, s % 3, ks);
        if constexpr (QDMA) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        stage(R, (s + 1) & 1, s + 1 < nst, min(s + 1, nst - 1));
        const int sl = min(s + 2, nst - 1);
        load(R, sl);
        load_w(sl);
        dma_q(sl, (s + 2) % 3);
        __builtin_amdgcn_sched_group_barrier(0x100, 3 * FI + NQ * FJ, 0);   // operand reads
#pragma unroll
        for (int i = 0; i < NMF; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);              // MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);              // VALU (measured best)
            if (i >= NMF / 2 && i < NMF / 2 + 3 + NQ)
                __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);          // LDS write
            if (i >= NMF / 2 + 3 + NQ && i < NMF / 2 + 9 + NQ)
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);          // global load
        }
        __syncthreads();
    }

    static_assert(!RDOT || G::TPR == 2, "two threads per staged row");
    if (RDOT) {
        const float v = rdot + __shfl_xor(rdot, 1, 64);
        if (sh == 0) rvec[sr] = v;
    }
    // a lazy factor (the first GEMM's) may carry a second term: w2 = w + K,
    // (Q w2) at rq + J, coefficient sgnb (q holds the composed c1, c2 and
    // the first term's c1b sgn: see sgemm_kernel)
    const bool two = STAGE == 1 && PEND && !FQ && q.has == 2;
    // The epilogue's vectors go into LDS here, ahead of its stores: a global
    // load issued after stores shares the vector-memory counter with them, so
    // waiting for its value also waits for those stores, and loads between
    // the output stores would serialise the tile's store drains.  Rows and
    // columns past the edge are clamped (their outputs are never stored).
    if constexpr (PEND) {
        if constexpr (FQ) {
            for (int c = t; c < BJ; c += NT) ew[c] = gld(L.w + min(j0 + c, J - 1));
        } else {
            for (int r = t; r < BI; r += NT) {
                ew[r] = gld(L.w + min(i0 + r, I - 1));
                if (two) ew[BI + r] = gld(L.w + K + min(i0 + r, I - 1));
            }
            if constexpr (STAGE == 1) {
                for (int c = t; c < BJ; c += NT) {
                    eq[c] = gld(L.rq + min(j0 + c, J - 1));
                    if (two) eq[BJ + c] = gld(L.rq + J + min(j0 + c, J - 1));
                }
            }
        }
    }
    __syncthreads();

    const float c1 = PEND ? q.c1 : 1.f, sg = PEND ? q.sgn : 0.f;
    float csq = 0.f;
    float* Cp = static_cast<float*>(L.C);
    // One MFMA row block (x) at a time: the w values its output groups need
    // (rows past the edge clamped), then C[i][j] = c1 acc + sgn w[i] (Q w)[j]
    // (FQ: c1 acc + sgn w[j] (P w)[i]), c2 I having entered acc through the
    // staged factor, stored as 128-byte row segments.
    const float sg2 = two ? q.sgnb : 0.f;
#pragma unroll
    for (int x = 0; x < FI; ++x) {
        float4 wv[4], wv2[4];
        float wcol[FJ];
        if (PEND) {
            if constexpr (FQ) {
#pragma unroll
                for (int y = 0; y < FJ; ++y) wcol[y] = ew[wj * TJ + y * 32 + li];
            } else {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int il = wi * TI + x * 32 + 8 * g + 4 * lk;
                    wv[g] = lds4(ew + il);
                    wv2[g] = two ? lds4(ew + BI + il) : make_float4(0.f, 0.f, 0.f, 0.f);
                }
            }
        }
#pragma unroll
        for (int y = 0; y < FJ; ++y) {
            const int jl = wj * TJ + y * 32 + li, j = j0 + jl;
            const float rq = (PEND && !FQ) ? (STAGE == 1 ? eq[jl] : rvec[jl]) : 0.f;
            const float rq2 = two ? eq[BJ + jl] : 0.f;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int il = wi * TI + x * 32 + 8 * g + 4 * lk, i = i0 + il;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[x][y][4 * g + e];
                if (PEND) {
                    if constexpr (FQ) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            v[e] = fmaf(c1, v[e], sg * wcol[y] * rvec[il + e]);
                    } else {
                        const float wa[4] = {wv[g].x, wv[g].y, wv[g].z, wv[g].w};
                        const float wb[4] = {wv2[g].x, wv2[g].y, wv2[g].z, wv2[g].w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] = fmaf(c1, v[e], fmaf(sg2 * wb[e], rq2, sg * wa[e] * rq));
                    }
                }
                if (i < I && j < J) {   // I, J multiples of 64: 4 rows all in or all out
                    float* dst = Cp + (size_t)i * J + j;
#pragma unroll
                    for (int e = 0; e < 4; ++e) gst(dst + (size_t)e * J, v[e]);
                    if (STAGE == 2) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) csq = fmaf(v[e], v[e], csq);
                    }
                }
            }
        }
    }

    // ||dW_hat||^2 partial: block-wide fixed-order sum (stage 1's ||G||^2
    // partials come from qdot_kernel).  The barrier waits for the LDS writes
    // only (a bare s_barrier): the compiler's barrier would also wait until
    // every output store of the tile has completed.
    if constexpr (STAGE == 2) {
        const float ws = wave_sum(csq);
        if (lane == 0) red[wave] = ws;
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (t == 0) {
            float s = 0.f;
            for (int w = 0; w < NW; ++w) s += red[w];
            gst(partials + L.part0 + tile.tm * L.ntj + tile.tn, s);
        }
    }
}

template <int STAGE, int GV, bool FQ>
__device__ __forceinline__ void sgemm_pm(int pm, const HgLayer& L, const GemmTile& tile, const Pending& q,
                                         float* partials, lds_char* smem) {
    if (pm == 2)      sgemm_tile<STAGE, GV, 2, FQ>(L, tile, q, partials, smem);
    else if (pm == 1) sgemm_tile<STAGE, GV, 1, FQ>(L, tile, q, partials, smem);
    else              sgemm_tile<STAGE, GV, 0, FQ>(L, tile, q, partials, smem);
}

// 8 waves per CU (2 per SIMD): at most 256 VGPRs per lane.
template <int STAGE>
__global__ __launch_bounds__(NT, 1) void sgemm_kernel(SgArgs args) {
    __shared__ __attribute__((aligned(16))) char smem_[SMEM];
    lds_char* smem = (lds_char*)smem_;
    {
        const GemmTile tile = args.tiles[blockIdx.x];
        if (tile.layer < 0) return;   // padding of the XCD interleave
        const HgLayer L = args.layers[tile.layer];
        if (!gld_i32(L.mode)) return;   // first-order layer this step
        Pending q = *L.pend;
        if (q.has == 2) {   // two terms: c1b (c1 S + c2 I + sgn w w^T) + c2b I + sgnb w2 w2^T
            q.sgn = q.c1b * q.sgn;
            q.c2 = fmaf(q.c1b, q.c2, q.c2b);
            q.c1 = q.c1b * q.c1;
        }
        const int pm = !q.has ? 0 : q.c2 != 0.f ? 2 : 1;
        if (STAGE == 2 && L.fq) {   // the second GEMM of a layer computed as X Rinv
            sgemm_pm<STAGE, GV_F32, true>(pm, L, tile, q, args.partials, smem);
        } else if (STAGE == 2 || L.qf32) {   // the second GEMM's Q (Y^T or X) is fp32
            sgemm_pm<STAGE, GV_F32, false>(pm, L, tile, q, args.partials, smem);
        } else if constexpr (STAGE == 1) {
            if (L.wide) sgemm_pm<STAGE, GV_HW, false>(pm, L, tile, q, args.partials, smem);
            else        sgemm_pm<STAGE, GV_H, false>(pm, L, tile, q, args.partials, smem);
        }
    }
}

// The sums over the wave of eight per-lane values, one per row: a butterfly
// that halves the values each lane keeps at the xor-32, -16 and -8 steps and
// sums the last over the remaining lane bits, so lanes 8 r .. 8 r + 7 end
// with row r's total (r = lane >> 3), in a fixed order.
__device__ __forceinline__ float row_sums8(const float (&v)[8], int lane) {
    const bool h5 = (lane & 32) != 0, h4 = (lane & 16) != 0, h3 = (lane & 8) != 0;
    float a[4], b[2];
#pragma unroll
    for (int k = 0; k < 4; ++k)   // rows k + 4 h5
        a[k] = (h5 ? v[k + 4] : v[k]) + __shfl_xor(h5 ? v[k] : v[k + 4], 32, 64);
#pragma unroll
    for (int k = 0; k < 2; ++k)   // rows 4 h5 + 2 h4 + k
        b[k] = (h4 ? a[k + 2] : a[k]) + __shfl_xor(h4 ? a[k] : a[k + 2], 16, 64);
    float c = (h3 ? b[1] : b[0]) + __shfl_xor(h3 ? b[0] : b[1], 8, 64);   // row 4 h5 + 2 h4 + h3
    c += __shfl_xor(c, 4, 64);
    c += __shfl_xor(c, 2, 64);
    c += __shfl_xor(c, 1, 64);
    return c;
}

template <bool TWO>
__device__ __forceinline__ void qdot_block(const HgLayer& L, const QdBlock& b, const Pending& q, float* partials,
                                           double* red, float (*rqs)[QD_MAX_ROWS]) {
    constexpr int RB = 8;   // rows in flight per wave
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int K = L.K, J = L.J;
    const float* w2 = L.w + K;
    // this lane's part of ||Q||^2: the squares of one 16-byte chunk summed in
    // fp32, the chunks accumulated in fp64, whatever K and the block's rows.
    // A long fp32 chain of positive terms (thousands of them) drifts low by
    // 1e-6 relative and more, which the rescale would carry into every
    // element of dW.
    double sq = 0.0;
    for (int r0 = wave * RB; r0 < b.rows; r0 += 4 * RB) {
        const int jb = b.rb * b.rows + r0;
        if (jb >= J) break;   // J is a multiple of 64: all RB rows in or all out
        float dot[RB], dot2[RB];
        double sqr[RB];
#pragma unroll
        for (int i = 0; i < RB; ++i) { dot[i] = dot2[i] = 0.f; sqr[i] = 0.0; }
        if (L.qf32) {
            const float* row = static_cast<const float*>(L.Q) + (size_t)jb * K;
            for (int k = 4 * lane; k < K; k += 256) {
                const float4 wv = q.has ? gld4(L.w + k) : make_float4(0.f, 0.f, 0.f, 0.f);
                const float4 wv2 = TWO ? gld4(w2 + k) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int i = 0; i < RB; ++i) {
                    const float4 v = gld4_nt(row + (size_t)i * K + k);
                    sqr[i] += (double)fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, v.w * v.w)));
                    dot[i] = fmaf(v.x, wv.x, fmaf(v.y, wv.y, fmaf(v.z, wv.z, fmaf(v.w, wv.w, dot[i]))));
                    if (TWO) dot2[i] = fmaf(v.x, wv2.x, fmaf(v.y, wv2.y, fmaf(v.z, wv2.z, fmaf(v.w, wv2.w, dot2[i]))));
                }
            }
        } else {
            const unsigned short* row = static_cast<const unsigned short*>(L.Q) + (size_t)jb * K;
            for (int k = 8 * lane; k < K; k += 512) {
                float wv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, wv2[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
                if (q.has) {
                    const float4 w0 = gld4(L.w + k), w1 = gld4(L.w + k + 4);
                    wv[0] = w0.x; wv[1] = w0.y; wv[2] = w0.z; wv[3] = w0.w;
                    wv[4] = w1.x; wv[5] = w1.y; wv[6] = w1.z; wv[7] = w1.w;
                }
                if (TWO) {
                    const float4 w0 = gld4(w2 + k), w1 = gld4(w2 + k + 4);
                    wv2[0] = w0.x; wv2[1] = w0.y; wv2[2] = w0.z; wv2[3] = w0.w;
                    wv2[4] = w1.x; wv2[5] = w1.y; wv2[6] = w1.z; wv2[7] = w1.w;
                }
#pragma unroll
                for (int i = 0; i < RB; ++i) {
                    const uint4 u = gld_u4_nt(row + (size_t)i * K + k);
                    const unsigned h[4] = {u.x, u.y, u.z, u.w};
                    float s8 = 0.f;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float v0 = __uint_as_float(h[e] << 16), v1 = __uint_as_float(h[e] & 0xffff0000u);
                        s8 = fmaf(v1, v1, fmaf(v0, v0, s8));
                        dot[i] = fmaf(v1, wv[2 * e + 1], fmaf(v0, wv[2 * e], dot[i]));
                        if (TWO) dot2[i] = fmaf(v1, wv2[2 * e + 1], fmaf(v0, wv2[2 * e], dot2[i]));
                    }
                    sqr[i] += (double)s8;
                }
            }
        }
        sq += ((sqr[0] + sqr[1]) + (sqr[2] + sqr[3])) + ((sqr[4] + sqr[5]) + (sqr[6] + sqr[7]));
        // the row results wait in LDS: a store here would hold up the next
        // rows' loads, which share the vector-memory counter with it
        const float d = row_sums8(dot, lane);
        if ((lane & 7) == 0) rqs[0][r0 + (lane >> 3)] = d;
        if (TWO) {
            const float d2 = row_sums8(dot2, lane);
            if ((lane & 7) == 0) rqs[1][r0 + (lane >> 3)] = d2;
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sq += __shfl_xor(sq, o, 64);
    if (lane == 0) red[wave] = sq;
    __syncthreads();
    if (t == 0) gst(partials + L.part0 + b.rb, (float)((red[0] + red[1]) + (red[2] + red[3])));
    const int j0 = b.rb * b.rows, nr = min(b.rows, J - j0);
    if (q.has)
        for (int r = t; r < nr; r += 256) gst(L.rq + j0 + r, rqs[0][r]);
    if (TWO)
        for (int r = t; r < nr; r += 256) gst(L.rq + J + j0 + r, rqs[1][r]);
}

// Stage-1 Q rows ahead of the first split GEMM: (Q w)[j] for each pending
// term of the factor (one, or two for a lazy factor) and the ||G||^2 partial
// of the block of rows (Q is G, or G^T: the same elements).  Four
// waves take 8 rows at a time (8 streaming loads in flight per lane); lanes
// take 16-byte chunks with a stride of 64 chunks, then fixed-order wave sums:
// deterministic.
__global__ __launch_bounds__(256) void qdot_kernel(const HgLayer* __restrict__ layers,
                                                  const QdBlock* __restrict__ blocks, float* __restrict__ partials) {
    __shared__ double red[4];
    __shared__ float rqs[2][QD_MAX_ROWS];
    const QdBlock b = blocks[blockIdx.x];
    const HgLayer L = layers[b.layer];
    if (!gld_i32(L.mode)) return;   // block-uniform
    const Pending q = *L.pend;
    if (q.has == 2) qdot_block<true>(L, b, q, partials, red, rqs);
    else            qdot_block<false>(L, b, q, partials, red, rqs);
}

// G^T of bf16 gradients, 64 x 64 tiles through LDS (rows of 64 + 2 elements,
// so the column reads of the transposed pass spread over the banks).
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const TrItem* __restrict__ items,
                                                            const TrBlock* __restrict__ blocks) {
    __shared__ unsigned short tile[64][66];
    const TrBlock b = blocks[blockIdx.x];
    const TrItem it = items[b.item];
    if (!gld_i32(it.mode)) return;   // block-uniform
    const int t = threadIdx.x, r = t >> 2, c = 16 * (t & 3);
    // 16 consecutive elements of source row r0 + r, as two 16-byte loads
    const unsigned short* s = it.src + (size_t)(b.r0 + r) * it.cols + b.c0 + c;
    const uint4 u0 = gld_u4(s), u1 = gld_u4(s + 8);
    const unsigned w[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        tile[r][c + 2 * e] = (unsigned short)(w[e] & 0xffffu);
        tile[r][c + 2 * e + 1] = (unsigned short)(w[e] >> 16);
    }
    __syncthreads();
    // destination row c0 + r holds source column c0 + r: elements r0 + c .. + 15
    unsigned o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = (unsigned)tile[c + 2 * e][r] | ((unsigned)tile[c + 2 * e + 1][r] << 16);
    unsigned short* d = it.dst + (size_t)(b.c0 + r) * it.rows + b.r0 + c;
    gst_u4(d, make_uint4(o[0], o[1], o[2], o[3]));
    gst_u4(d + 8, make_uint4(o[4], o[5], o[6], o[7]));
}

}  // namespace

hipError_t launch_qdot(const HgLayer* layers, const QdBlock* blocks, int32_t nblocks, float* partials,
                       hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(qdot_kernel, dim3(nblocks), dim3(256), 0, stream, layers, blocks, partials);
    return hipGetLastError();
}

hipError_t launch_transpose_bf16(const TrItem* items, const TrBlock* blocks, int32_t nblocks, hipStream_t stream) {
    if (nblocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(transpose_bf16_kernel, dim3(nblocks), dim3(256), 0, stream, items, blocks);
    return hipGetLastError();
}

hipError_t launch_sgemm(int stage, const HgLayer* layers, const GemmTile* tiles, int32_t ntiles,
                        float* partials, hipStream_t stream) {
    if (ntiles <= 0) return hipSuccess;
    SgArgs a{layers, tiles, partials};
    const int grid = ntiles;
    if (stage == 1) hipLaunchKernelGGL(sgemm_kernel<1>, dim3(grid), dim3(NT), 0, stream, a);
    else            hipLaunchKernelGGL(sgemm_kernel<2>, dim3(grid), dim3(NT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace mkor
