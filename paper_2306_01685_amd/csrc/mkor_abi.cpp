// C ABI of libmkor: argument validation, plan / workspace layout, launches.
//
// All validation runs on the host before the first HIP call of an entry
// point, so every error path can be exercised without a GPU.
#include "plan.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

using namespace mkor;

namespace {
thread_local char g_err[512] = "";
}  // namespace

namespace mkor {

int fail(int status, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(MKOR_HIP_ERROR, "%s: %s", what, hipGetErrorString(e));
}

void clear_error() { g_err[0] = 0; }

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Interval {
    uintptr_t lo, hi;
    bool writable;
    int layer;
    const char* what;
};

// vectors per factor update: rank 0 means 1; first-order layers have none
int32_t layer_rank(const mkor_layer& L) { return L.second_order == 1 ? std::max(1, L.rank) : 1; }

}  // namespace

int check_layers(const mkor_layer* layers, int32_t n, const void* ws, size_t ws_bytes) {
    if (n < 0) return fail(MKOR_INVALID_ARG, "n = %d is negative", n);
    if (n > 0 && layers == nullptr) return fail(MKOR_INVALID_ARG, "layers is NULL with n = %d", n);
    std::vector<Interval> iv;
    iv.reserve((size_t)n * 12 + 1);
    for (int32_t i = 0; i < n; ++i) {
        const mkor_layer& L = layers[i];
        if (L.d_in < 1 || L.d_in > MKOR_MAX_DIM || L.d_out < 1 || L.d_out > MKOR_MAX_DIM)
            return fail(MKOR_INVALID_ARG, "layer %d: d_in = %d, d_out = %d outside 1..%d", i, L.d_in,
                        L.d_out, MKOR_MAX_DIM);
        if (L.second_order != 0 && L.second_order != 1)
            return fail(MKOR_INVALID_ARG, "layer %d: second_order = %d is not 0 or 1", i, L.second_order);
        if (L.grad_dtype != MKOR_DTYPE_F32 && L.grad_dtype != MKOR_DTYPE_BF16)
            return fail(MKOR_UNSUPPORTED, "layer %d: grad_dtype = %d is not supported", i, L.grad_dtype);
        if (L.factor_dtype != MKOR_DTYPE_F32 && L.factor_dtype != MKOR_DTYPE_BF16)
            return fail(MKOR_UNSUPPORTED, "layer %d: factor_dtype = %d is not supported", i, L.factor_dtype);
        if (L.rank < 0 || L.rank > MKOR_MAX_RANK)
            return fail(MKOR_INVALID_ARG, "layer %d: rank = %d outside 0..%d", i, L.rank, MKOR_MAX_RANK);
        const bool half = L.second_order == 1 && L.factor_dtype == MKOR_DTYPE_BF16;
        const int32_t rk = layer_rank(L);
        if (rk > 1 && L.rows > 0)
            return fail(MKOR_UNSUPPORTED, "layer %d: rank %d needs rows = 0 (means are rank-1)", i, rk);
        if (rk > 1 && half)
            return fail(MKOR_UNSUPPORTED, "layer %d: rank %d needs fp32 factors", i, rk);
        if (half && (L.d_in % 64 != 0 || L.d_out % 64 != 0))
            return fail(MKOR_UNSUPPORTED, "layer %d: bf16 factors need d_in and d_out multiples of 64 (%d, %d)",
                        i, L.d_in, L.d_out);
        if (L.gemm_path != MKOR_GEMM_AUTO && L.gemm_path != MKOR_GEMM_FP32 && L.gemm_path != MKOR_GEMM_SPLIT)
            return fail(MKOR_INVALID_ARG, "layer %d: gemm_path = %d unknown", i, L.gemm_path);
        if (L.gemm_path != MKOR_GEMM_AUTO && (half || L.second_order != 1))
            return fail(MKOR_INVALID_ARG, "layer %d: gemm_path applies to second-order layers with fp32 factors",
                        i);
        if (L.gemm_path == MKOR_GEMM_SPLIT && (L.d_in % 64 != 0 || L.d_out % 64 != 0))
            return fail(MKOR_UNSUPPORTED, "layer %d: MKOR_GEMM_SPLIT needs d_in and d_out multiples of 64 (%d, %d)",
                        i, L.d_in, L.d_out);
        if (L.reserved0 != 0) return fail(MKOR_INVALID_ARG, "layer %d: reserved0 = %d must be 0", i, L.reserved0);
        if (L.rows < 0 || L.rows > MKOR_MAX_ROWS)
            return fail(MKOR_INVALID_ARG, "layer %d: rows = %d outside 0..%d", i, L.rows, MKOR_MAX_ROWS);
        const bool means = L.rows > 0;
        if (means && L.second_order != 1)
            return fail(MKOR_INVALID_ARG, "layer %d: rows > 0 needs a second-order layer", i);
        if (means && L.act_dtype != MKOR_DTYPE_F32 && L.act_dtype != MKOR_DTYPE_BF16)
            return fail(MKOR_UNSUPPORTED, "layer %d: act_dtype = %d is not supported", i, L.act_dtype);
        const size_t din = (size_t)L.d_in, dout = (size_t)L.d_out;
        const size_t gsz = din * dout * (L.grad_dtype == MKOR_DTYPE_BF16 ? 2 : 4);
        const size_t asz = means ? (size_t)L.rows * (L.act_dtype == MKOR_DTYPE_BF16 ? 2 : 4) : 0;
        struct { const void* p; size_t bytes; bool w; const char* what; bool used; } bufs[] = {
            {L.G, gsz, false, "G", true},
            {L.dW, din * dout * 4, true, "dW", true},
            {L.Linv, din * din * (half ? 2 : 4), true, "Linv", L.second_order == 1},
            {L.Rinv, dout * dout * (half ? 2 : 4), true, "Rinv", L.second_order == 1},
            {L.a, din * 4 * rk, means, "a", L.second_order == 1},
            {L.g, dout * 4 * rk, means, "g", L.second_order == 1},
            {L.stats, sizeof(mkor_layer_stats), true, "stats", L.stats != nullptr},
            {L.A, asz * din, false, "A", means},
            {L.Gout, asz * dout, false, "Gout", means},
            {L.W, din * dout * 4, true, "W", L.W != nullptr},
            {L.opt_m, din * dout * 4, true, "opt_m", L.opt_m != nullptr},
            {L.opt_v, din * dout * 4, true, "opt_v", L.opt_v != nullptr},
        };
        for (auto& b : bufs) {
            if (!b.used) continue;
            if (b.p == nullptr) return fail(MKOR_INVALID_ARG, "layer %d: %s is NULL", i, b.what);
            if (!aligned(b.p, 16))
                return fail(MKOR_INVALID_ARG, "layer %d: %s is not 16-byte aligned", i, b.what);
            const uintptr_t lo = reinterpret_cast<uintptr_t>(b.p);
            if (lo + b.bytes < lo) return fail(MKOR_INVALID_ARG, "layer %d: %s wraps the address space", i, b.what);
            iv.push_back({lo, lo + b.bytes, b.w, i, b.what});
        }
    }
    if (ws != nullptr && ws_bytes > 0) {
        const uintptr_t lo = reinterpret_cast<uintptr_t>(ws);
        iv.push_back({lo, lo + ws_bytes, true, -1, "workspace"});
    }
    // Any overlap that involves a writable buffer is an error.  After sorting
    // by start, an interval overlaps an earlier one iff its start lies below
    // the largest end seen so far; tracking that maximum separately for
    // writable intervals and for all intervals catches every such pair.
    std::sort(iv.begin(), iv.end(), [](const Interval& x, const Interval& y) { return x.lo < y.lo; });
    uintptr_t max_all = 0, max_w = 0;
    const Interval *arg_all = nullptr, *arg_w = nullptr;
    for (const Interval& c : iv) {
        if (arg_w && c.lo < max_w)
            return fail(MKOR_INVALID_ARG, "%s of layer %d overlaps writable %s of layer %d", c.what,
                        c.layer, arg_w->what, arg_w->layer);
        if (c.writable && arg_all && c.lo < max_all)
            return fail(MKOR_INVALID_ARG, "writable %s of layer %d overlaps %s of layer %d", c.what,
                        c.layer, arg_all->what, arg_all->layer);
        if (c.hi > max_all) { max_all = c.hi; arg_all = &c; }
        if (c.writable && c.hi > max_w) { max_w = c.hi; arg_w = &c; }
    }
    return MKOR_OK;
}

namespace {

// ------------------------------------------------------------------ layout

int32_t ceil_div(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }

bool is_half(const mkor_layer& L) { return L.second_order == 1 && L.factor_dtype == MKOR_DTYPE_BF16; }

// fp32 factors preconditioned on the three-way bf16 split (MKOR_GEMM_SPLIT, or
// MKOR_GEMM_AUTO where the shape allows it)
bool is_split(const mkor_layer& L) {
    if (L.second_order != 1 || L.factor_dtype != MKOR_DTYPE_F32) return false;
    if (L.gemm_path == MKOR_GEMM_SPLIT) return true;
    return L.gemm_path == MKOR_GEMM_AUTO && L.d_in % 64 == 0 && L.d_out % 64 == 0;
}

// split layers with a bf16 G and d_in > d_out take the other association,
// dW_hat = (Linv G) Rinv, so that the longer contraction (over d_in) is the
// one whose Q operand (G^T) is bf16 and needs three bf16 products per product
// instead of six
bool is_swapped(const mkor_layer& L) {
    return is_split(L) && L.grad_dtype == MKOR_DTYPE_BF16 && L.d_in > L.d_out;
}

// The factor of a split layer's first GEMM (Rinv, or Linv for the other
// association) keeps up to two pending terms, so the SM pass writes it only
// every other step; that GEMM applies both terms in its epilogue, with (Q w)
// of each from the row pass ahead of it.  Side 0: Linv, 1: Rinv.
bool lazy_factor(const mkor_layer& L, int side) {
    if (!is_split(L) || layer_rank(L) != 1) return false;
    return side == (is_swapped(L) ? 0 : 1);
}

// GEMM kernel family of a second-order layer
enum { FAM_FP32 = 0, FAM_HALF = 1, FAM_SPLIT = 2 };
int gemm_family(const mkor_layer& L) { return is_half(L) ? FAM_HALF : is_split(L) ? FAM_SPLIT : FAM_FP32; }

// Output tile grid and contraction length of a GEMM stage.  fp32 MFMA:
// stage 1 X^T = (Linv G)^T (K = d_in), stage 2 dW_hat = X Rinv (K = d_out),
// both tiled over d_in x d_out.  bf16 MFMA (bf16 factors, or fp32 factors on
// the split): stage 1 Y^T = Rinv G^T (d_out x d_in, K = d_out), stage 2
// dW_hat = Linv Y (d_in x d_out, K = d_in).
struct StageGeom {
    int32_t bm, bn;      // tile rows, columns
    int32_t rows, cols;  // output rows, columns
    int32_t K;
};
// The split's first GEMM with a bf16 Q (G or G^T) takes SG_BI1H x SG_BJ1H
// tiles (half the fp32 factor bytes per output) unless they pad the layer's
// output more than SG_BI x SG_BJ tiles do (rows: the factor's, columns: Q's).
bool split_wide(int64_t rows, int64_t cols) {
    auto padded = [&](int64_t bm, int64_t bn) { return ceil_div(rows, bm) * bm * ceil_div(cols, bn) * bn; };
    return padded(SG_BI1H, SG_BJ1H) <= padded(SG_BI, SG_BJ);
}
StageGeom stage_geom(const mkor_layer& L, int stage) {
    if (is_swapped(L)) {   // stage 1 X = Linv G (K = d_in), stage 2 dW_hat = X Rinv (K = d_out)
        if (stage == 1) {
            const bool w = split_wide(L.d_in, L.d_out);
            return StageGeom{w ? SG_BI1H : SG_BI, w ? SG_BJ1H : SG_BJ, L.d_in, L.d_out, L.d_in};
        }
        return StageGeom{SG_BI, SG_BJ, L.d_in, L.d_out, L.d_out};
    }
    const int fam = gemm_family(L);
    if (fam != FAM_FP32) {
        const int32_t bm = fam == FAM_HALF ? HG_BI : SG_BI, bn = fam == FAM_HALF ? HG_BJ : SG_BJ;
        const bool w = fam == FAM_SPLIT && L.grad_dtype == MKOR_DTYPE_BF16 && split_wide(L.d_out, L.d_in);
        if (stage == 1) return StageGeom{w ? SG_BI1H : bm, w ? SG_BJ1H : bn, L.d_out, L.d_in, L.d_out};
        return StageGeom{bm, bn, L.d_in, L.d_out, L.d_in};
    }
    const GemmShape& sh = GEMM_SHAPE[stage - 1];
    return StageGeom{sh.bm, sh.bn, L.d_in, L.d_out, stage == 1 ? L.d_in : L.d_out};
}

// Tile table of one GEMM stage over the second-order layers of one kernel
// family (FAM_*).  Each layer's tile
// grid is cut into super-tiles covering up to GEMM_SUPER x GEMM_SUPER
// outputs; super-tiles are taken longest K first and each goes whole to the
// XCD with the least work so far, so the tiles an XCD runs together share A
// and B panels in its L2 and the long tiles do not form the tail.  Workgroup
// b runs on XCD b % GEMM_XCDS, so position q * GEMM_XCDS + x of the table
// holds the q-th tile of XCD x; shorter queues are padded with tiles of layer
// -1.
std::vector<GemmTile> schedule_tiles(const mkor_layer* layers, int32_t n, int stage, int family) {
    struct Super { int32_t layer, tm0, tn0, nm, nn, K; };
    std::vector<Super> sup;
    for (int32_t i = 0; i < n; ++i) {
        const mkor_layer& L = layers[i];
        if (!L.second_order || gemm_family(L) != family) continue;
        const StageGeom g = stage_geom(L, stage);
        const int32_t sm = std::max(1, GEMM_SUPER / g.bm), sn = std::max(1, GEMM_SUPER / g.bn);
        const int32_t tm = ceil_div(g.rows, g.bm), tn = ceil_div(g.cols, g.bn);
        for (int32_t a = 0; a < tm; a += sm)
            for (int32_t b = 0; b < tn; b += sn)
                sup.push_back(Super{i, a, b, std::min(sm, tm - a), std::min(sn, tn - b), g.K});
    }
    if (sup.empty()) return {};
    std::stable_sort(sup.begin(), sup.end(), [](const Super& x, const Super& y) {
        if (x.K != y.K) return x.K > y.K;
        return x.nm * x.nn > y.nm * y.nn;
    });
    std::vector<std::vector<GemmTile>> queue(GEMM_XCDS);
    std::vector<int64_t> work(GEMM_XCDS, 0);
    for (const Super& S : sup) {
        const int x = (int)(std::min_element(work.begin(), work.end()) - work.begin());
        for (int32_t a = 0; a < S.nm; ++a)
            for (int32_t b = 0; b < S.nn; ++b)
                queue[x].push_back(GemmTile{S.layer, S.tm0 + a, S.tn0 + b, 0});
        work[x] += (int64_t)S.nm * S.nn * S.K;
    }
    size_t len = 0;
    for (const auto& q : queue) len = std::max(len, q.size());
    std::vector<GemmTile> table(len * GEMM_XCDS, GemmTile{-1, 0, 0, 0});
    for (int x = 0; x < GEMM_XCDS; ++x)
        for (size_t q = 0; q < queue[x].size(); ++q) table[q * GEMM_XCDS + x] = queue[x][q];
    return table;
}

// Rows per qdot_kernel block of a split layer: its stage-1 Q is G or G^T, rows
// of K elements in G's dtype.
int32_t qd_rows_of(const mkor_layer& L) {
    return qd_rows(stage_geom(L, 1).K, L.grad_dtype == MKOR_DTYPE_BF16 ? 2 : 4);
}

// ||G||^2 partials of a layer (one per stage-1 tile column for fp32 factors,
// one per stage-1 tile column, i.e. per block of G rows, for bf16 factors) and
// ||dW_hat||^2 partials (one per tile of the stage that writes dW_hat).
int64_t gpart_count(const mkor_layer& L) {
    const StageGeom g = stage_geom(L, 1);
    if (is_split(L)) return ceil_div(g.cols, qd_rows_of(L));   // one per qdot_kernel block
    return ceil_div(g.cols, g.bn);
}
int64_t dpart_count(const mkor_layer& L) {
    const StageGeom g = stage_geom(L, 2);
    return (int64_t)ceil_div(g.rows, g.bm) * ceil_div(g.cols, g.bn);
}

// bf16-factor layer whose gradient is fp32: the GEMMs read a bf16 copy
bool needs_cvt(const mkor_layer& L) { return is_half(L) && L.grad_dtype == MKOR_DTYPE_F32; }

// Rows per block of the column-mean partials for the whole plan: the largest
// power of two in [MEAN_ROWS_MIN, MEAN_ROWS_MAX] that still gives at least
// MEAN_MIN_BLOCKS blocks over every token-row matrix (else the minimum).
int32_t mean_rows_per_block(const mkor_layer* layers, int32_t n) {
    for (int32_t rpb = MEAN_ROWS_MAX; rpb > MEAN_ROWS_MIN; rpb /= 2) {
        int64_t blocks = 0;
        for (int32_t i = 0; i < n; ++i)
            if (layers[i].rows > 0)
                blocks += (int64_t)(ceil_div(layers[i].d_in, MEAN_COLS) + ceil_div(layers[i].d_out, MEAN_COLS)) *
                          ceil_div(layers[i].rows, rpb);
        if (blocks >= MEAN_MIN_BLOCKS) return rpb;
    }
    return MEAN_ROWS_MIN;
}

}  // namespace

int compute_layout(const mkor_layer* layers, int32_t n, Layout& Lo) {
    int64_t rowblocks = 0, g1 = 0, gpart = 0, rsb = 0, usum = 0, ncvt = 0, ncvtblk = 0, ntr = 0, ntrblk = 0;
    int64_t nqdb = 0;
    for (int32_t i = 0; i < n; ++i) {
        const mkor_layer& L = layers[i];
        rsb += ceil_div((int64_t)L.d_in * L.d_out, RS_ELEMS);
        if (needs_cvt(L)) {
            ncvt += 1;
            ncvtblk += ceil_div((int64_t)L.d_in * L.d_out, CVT_ELEMS);
        }
        if (is_swapped(L)) {
            ntr += 1;
            ntrblk += (int64_t)(L.d_in / 64) * (L.d_out / 64);
        }
        if (is_split(L)) nqdb += gpart_count(L);
        if (!L.second_order) continue;
        Lo.nsecond++;
        if (layer_rank(L) > 1) Lo.nranked++;
        const int32_t rows = is_half(L) ? SM_ROWS_HALF : SM_ROWS;
        rowblocks += ceil_div(L.d_in, rows) + ceil_div(L.d_out, rows);
        g1 += dpart_count(L);
        gpart += gpart_count(L);
        usum += L.d_in + L.d_out;
    }
    int64_t mitems = 0, mchunks = 0, mpart = 0, mmats = 0;
    Lo.mean_rpb = mean_rows_per_block(layers, n);
    for (int32_t i = 0; i < n; ++i) {
        const mkor_layer& L = layers[i];
        if (L.rows <= 0) continue;
        const int64_t nrb = ceil_div(L.rows, Lo.mean_rpb);
        for (const int32_t d : {L.d_in, L.d_out}) {
            const int64_t nch = ceil_div(d, MEAN_COLS);
            mmats += 1;
            mchunks += nch;
            mitems += nch * nrb;
            mpart += nch * nrb * MEAN_COLS;
        }
    }
    if (rowblocks > INT32_MAX || g1 > INT32_MAX || rsb > INT32_MAX || mitems > INT32_MAX || ncvtblk > INT32_MAX ||
        ntrblk > INT32_MAX || nqdb > INT32_MAX)
        return fail(MKOR_UNSUPPORTED, "layer list too large for one grouped launch");
    Lo.nmeanmat = (int32_t)mmats;
    Lo.nmeanitem = (int32_t)mitems;
    Lo.nmeanchunk = (int32_t)mchunks;
    Lo.nmeanpart = mpart;
    Lo.nfactors = 2 * Lo.nsecond;
    Lo.nrowblocks = (int32_t)rowblocks;
    const size_t t1 = schedule_tiles(layers, n, 1, FAM_FP32).size(), t2 = schedule_tiles(layers, n, 2, FAM_FP32).size();
    const size_t h1 = schedule_tiles(layers, n, 1, FAM_HALF).size(), h2 = schedule_tiles(layers, n, 2, FAM_HALF).size();
    const size_t s1 = schedule_tiles(layers, n, 1, FAM_SPLIT).size(), s2 = schedule_tiles(layers, n, 2, FAM_SPLIT).size();
    if (t1 > INT32_MAX || t2 > INT32_MAX || h1 > INT32_MAX || h2 > INT32_MAX || s1 > INT32_MAX || s2 > INT32_MAX)
        return fail(MKOR_UNSUPPORTED, "layer list too large for one grouped launch");
    Lo.ns1 = (int32_t)s1;
    Lo.ns2 = (int32_t)s2;
    Lo.ng1 = (int32_t)t1;
    Lo.ng2 = (int32_t)t2;
    Lo.nh1 = (int32_t)h1;
    Lo.nh2 = (int32_t)h2;
    Lo.ngpart = (int32_t)gpart;
    Lo.ndpart = (int32_t)g1;
    Lo.nrsblocks = (int32_t)rsb;
    Lo.ncvt = (int32_t)ncvt;
    Lo.ncvtblk = (int32_t)ncvtblk;
    Lo.ntr = (int32_t)ntr;
    Lo.ntrblk = (int32_t)ntrblk;
    Lo.nqdb = (int32_t)nqdb;

    size_t o = 0;
    auto take = [&](size_t bytes) { o = align_up(o, 256); size_t r = o; o += bytes; return r; };
    Lo.off_factors = take(sizeof(FactorDesc) * Lo.nfactors);
    Lo.off_rowblocks = take(sizeof(RowBlock) * Lo.nrowblocks);
    Lo.off_g1l = take(sizeof(GemmLayer) * n);
    Lo.off_g1t = take(sizeof(GemmTile) * Lo.ng1);
    Lo.off_g2l = take(sizeof(GemmLayer) * n);
    Lo.off_g2t = take(sizeof(GemmTile) * Lo.ng2);
    Lo.off_h1l = take(sizeof(HgLayer) * n);
    Lo.off_h1t = take(sizeof(GemmTile) * Lo.nh1);
    Lo.off_h2l = take(sizeof(HgLayer) * n);
    Lo.off_h2t = take(sizeof(GemmTile) * Lo.nh2);
    Lo.off_s1l = take(sizeof(HgLayer) * n);
    Lo.off_s1t = take(sizeof(GemmTile) * Lo.ns1);
    Lo.off_s2l = take(sizeof(HgLayer) * n);
    Lo.off_s2t = take(sizeof(GemmTile) * Lo.ns2);
    Lo.off_rsl = take(sizeof(RescaleLayer) * n);
    Lo.off_rsb = take(sizeof(RescaleBlock) * Lo.nrsblocks);
    Lo.off_mmat = take(sizeof(MeanMat) * Lo.nmeanmat);
    Lo.off_mitem = take(sizeof(MeanItem) * Lo.nmeanitem);
    Lo.off_mchunk = take(sizeof(MeanItem) * Lo.nmeanchunk);
    Lo.off_cvti = take(sizeof(CvtItem) * Lo.ncvt);
    Lo.off_cvtb = take(sizeof(CvtBlock) * Lo.ncvtblk);
    Lo.off_tri = take(sizeof(TrItem) * Lo.ntr);
    Lo.off_trb = take(sizeof(TrBlock) * Lo.ntrblk);
    Lo.off_qdb = take(sizeof(QdBlock) * Lo.nqdb);
    // pending terms start out empty (has = 0), the mode words as planned:
    // the upload initialises them
    Lo.off_pend = take(sizeof(Pending) * Lo.nfactors);
    Lo.off_mode = take(sizeof(int32_t) * (size_t)n);
    Lo.table_bytes = align_up(o, 256);
    Lo.off_smpart = take(sizeof(float4) * Lo.nrowblocks);
    Lo.off_gram = take(Lo.nranked > 0 ? sizeof(float) * GRAM * (size_t)Lo.nrowblocks : 0);
    Lo.off_lpart = take(sizeof(float2) * (size_t)Lo.nrsblocks);
    Lo.off_trust = take(sizeof(float) * (size_t)n);
    Lo.off_gpart = take(sizeof(float) * Lo.ngpart);
    Lo.off_dpart = take(sizeof(float) * Lo.ndpart);
    Lo.off_mpart = take(sizeof(double) * (size_t)Lo.nmeanpart);
    Lo.u_off.clear();
    Lo.w_off.clear();
    Lo.x_off.assign(n, 0);
    for (int32_t i = 0; i < n; ++i) {
        if (!layers[i].second_order) continue;
        for (int side = 0; side < 2; ++side) {
            const int32_t d = side == 0 ? layers[i].d_in : layers[i].d_out;
            Lo.u_off.push_back(take(sizeof(float) * d * layer_rank(layers[i])));
            Lo.w_off.push_back(take(sizeof(float) * d * (lazy_factor(layers[i], side) ? 2 : layer_rank(layers[i]))));
        }
    }
    for (int32_t i = 0; i < n; ++i) {
        if (!layers[i].second_order) continue;
        // X^T or Y^T (fp32) of fp32-factor layers, Y^T (bf16) of bf16-factor layers
        Lo.x_off[i] = take((is_half(layers[i]) ? 2 : 4) * (size_t)layers[i].d_in * layers[i].d_out);
    }
    Lo.gh_off.assign(n, 0);
    for (int32_t i = 0; i < n; ++i)
        if (needs_cvt(layers[i])) Lo.gh_off[i] = take(2 * (size_t)layers[i].d_in * layers[i].d_out);
    Lo.gt_off.assign(n, 0);
    for (int32_t i = 0; i < n; ++i)
        if (is_swapped(layers[i])) Lo.gt_off[i] = take(2 * (size_t)layers[i].d_in * layers[i].d_out);
    Lo.rq_off.assign(n, 0);
    for (int32_t i = 0; i < n; ++i)
        if (is_split(layers[i]))   // (Q w) of the first GEMM's factor, one row per pending term
            Lo.rq_off[i] = take(sizeof(float) * 2 * (size_t)stage_geom(layers[i], 1).cols);
    Lo.total = align_up(o, 256);
    (void)usum;
    return MKOR_OK;
}

int check_params(const mkor_params* p) {
    if (p == nullptr) return fail(MKOR_INVALID_ARG, "params is NULL");
    if (!(p->gamma > 0.f && p->gamma < 1.f))
        return fail(MKOR_INVALID_ARG, "gamma = %g outside (0, 1)", (double)p->gamma);
    if (!(p->zeta > 0.f && p->zeta <= 1.f))
        return fail(MKOR_INVALID_ARG, "zeta = %g outside (0, 1]", (double)p->zeta);
    if (std::isnan(p->stab_eps) || p->stab_eps < 0.f)
        return fail(MKOR_INVALID_ARG, "stab_eps = %g must be >= 0 or +inf", (double)p->stab_eps);
    if (p->norm_kind != MKOR_NORM_INF && p->norm_kind != MKOR_NORM_MAXABS)
        return fail(MKOR_INVALID_ARG, "norm_kind = %d unknown", p->norm_kind);
    if (p->sm_variant != MKOR_SM_EXACT && p->sm_variant != MKOR_SM_PAPER_EQ6)
        return fail(MKOR_INVALID_ARG, "sm_variant = %d unknown", p->sm_variant);
    if (p->rescale != 0 && p->rescale != 1)
        return fail(MKOR_INVALID_ARG, "rescale = %d is not 0 or 1", p->rescale);
    if (p->guard_nonfinite != 0 && p->guard_nonfinite != 1)
        return fail(MKOR_INVALID_ARG, "guard_nonfinite = %d is not 0 or 1", p->guard_nonfinite);
    return MKOR_OK;
}


// Descriptor tables of a plan whose workspace starts at device address
// `base`: the bytes [0, lo.table_bytes) of that workspace, built on the host.
void build_tables(const mkor_layer* layers, int32_t n, char* base, const Layout& lo, std::vector<char>& host) {
    host.assign(lo.table_bytes, 0);
    FactorDesc* fd = reinterpret_cast<FactorDesc*>(host.data() + lo.off_factors);
    RowBlock* rb = reinterpret_cast<RowBlock*>(host.data() + lo.off_rowblocks);
    GemmLayer* g1l = reinterpret_cast<GemmLayer*>(host.data() + lo.off_g1l);
    GemmLayer* g2l = reinterpret_cast<GemmLayer*>(host.data() + lo.off_g2l);
    GemmTile* g1t = reinterpret_cast<GemmTile*>(host.data() + lo.off_g1t);
    GemmTile* g2t = reinterpret_cast<GemmTile*>(host.data() + lo.off_g2t);
    HgLayer* h1l = reinterpret_cast<HgLayer*>(host.data() + lo.off_h1l);
    HgLayer* h2l = reinterpret_cast<HgLayer*>(host.data() + lo.off_h2l);
    GemmTile* h1t = reinterpret_cast<GemmTile*>(host.data() + lo.off_h1t);
    GemmTile* h2t = reinterpret_cast<GemmTile*>(host.data() + lo.off_h2t);
    HgLayer* s1l = reinterpret_cast<HgLayer*>(host.data() + lo.off_s1l);
    HgLayer* s2l = reinterpret_cast<HgLayer*>(host.data() + lo.off_s2l);
    GemmTile* s1t = reinterpret_cast<GemmTile*>(host.data() + lo.off_s1t);
    GemmTile* s2t = reinterpret_cast<GemmTile*>(host.data() + lo.off_s2t);
    CvtItem* cvi = reinterpret_cast<CvtItem*>(host.data() + lo.off_cvti);
    CvtBlock* cvb = reinterpret_cast<CvtBlock*>(host.data() + lo.off_cvtb);
    int32_t nci = 0, ncb = 0;
    TrItem* tri = reinterpret_cast<TrItem*>(host.data() + lo.off_tri);
    TrBlock* trb = reinterpret_cast<TrBlock*>(host.data() + lo.off_trb);
    int32_t nti = 0, ntb = 0;
    QdBlock* qdb = reinterpret_cast<QdBlock*>(host.data() + lo.off_qdb);
    int32_t nqb = 0;
    RescaleLayer* rsl = reinterpret_cast<RescaleLayer*>(host.data() + lo.off_rsl);
    RescaleBlock* rsb = reinterpret_cast<RescaleBlock*>(host.data() + lo.off_rsb);
    Pending* pend_h = reinterpret_cast<Pending*>(host.data() + lo.off_pend);
    MeanMat* mm = reinterpret_cast<MeanMat*>(host.data() + lo.off_mmat);
    MeanItem* mi = reinterpret_cast<MeanItem*>(host.data() + lo.off_mitem);
    MeanItem* mc = reinterpret_cast<MeanItem*>(host.data() + lo.off_mchunk);
    int32_t* mode_h = reinterpret_cast<int32_t*>(host.data() + lo.off_mode);
    const int32_t* mode_d = reinterpret_cast<const int32_t*>(base + lo.off_mode);
    for (int32_t i = 0; i < n; ++i) mode_h[i] = layers[i].second_order;
    {
        int32_t k = 0, ki = 0, kc = 0;
        int64_t p0 = 0;
        for (int32_t i = 0; i < n; ++i) {
            const mkor_layer& L = layers[i];
            if (L.rows <= 0) continue;
            for (int side = 0; side < 2; ++side) {
                MeanMat& M = mm[k];
                M.X = side == 0 ? L.A : L.Gout;
                M.out = side == 0 ? L.a : L.g;
                M.rows = L.rows;
                M.cols = side == 0 ? L.d_in : L.d_out;
                M.bf16 = L.act_dtype == MKOR_DTYPE_BF16;
                M.vec = (M.cols % 8) == 0;
                M.nchunk = ceil_div(M.cols, MEAN_COLS);
                M.nrb = ceil_div(M.rows, lo.mean_rpb);
                M.rpb = lo.mean_rpb;
                M._pad = 0;
                M.part0 = p0;
                M.mode = mode_d + i;
                p0 += (int64_t)M.nchunk * M.nrb * MEAN_COLS;
                for (int32_t rb = 0; rb < M.nrb; ++rb)
                    for (int32_t c = 0; c < M.nchunk; ++c) mi[ki++] = MeanItem{k, c, rb, 0};
                for (int32_t c = 0; c < M.nchunk; ++c) mc[kc++] = MeanItem{k, c, 0, 0};
                ++k;
            }
        }
    }
    Pending* pend_d = reinterpret_cast<Pending*>(base + lo.off_pend);

    int32_t fi = 0, bi = 0, gp = 0, dp = 0, rbi = 0;
    for (int32_t i = 0; i < n; ++i) {
        const mkor_layer& L = layers[i];
        mkor_layer_stats* stats = static_cast<mkor_layer_stats*>(L.stats);
        RescaleLayer& R = rsl[i];
        R.G = L.G;
        R.dW = L.dW;
        R.stats = stats;
        R.numel = (int64_t)L.d_in * L.d_out;
        R.second_order = L.second_order;
        R.g_bf16 = L.grad_dtype == MKOR_DTYPE_BF16;
        R.first_blk = rbi;
        for (int64_t s = 0; s < R.numel; s += RS_ELEMS) rsb[rbi++] = RescaleBlock{i, 0, s};
        R.nblk = rbi - R.first_blk;
        R.W = L.W;
        R.m = L.opt_m;
        R.v = L.opt_v;
        R.mode = mode_d + i;
        if (!L.second_order) continue;
        const bool half = is_half(L);
        for (int side = 0; side < 2; ++side) {
            FactorDesc& f = fd[fi];
            f.P = side == 0 ? L.Linv : L.Rinv;
            f.x = side == 0 ? L.a : L.g;
            f.u = reinterpret_cast<float*>(base + lo.u_off[fi]);
            f.w = reinterpret_cast<float*>(base + lo.w_off[fi]);
            f.pend = pend_d + fi;
            pend_h[fi] = Pending{1.f, 0.f, 0.f, 0};
            f.stats = stats;
            f.d = side == 0 ? L.d_in : L.d_out;
            f.blk0 = bi;
            const int32_t rows = half ? SM_ROWS_HALF : SM_ROWS;
            f.nblk = ceil_div(f.d, rows);
            f.side = side;
            f.half = half ? 1 : 0;
            f.rank = layer_rank(L);
            f.lazy = lazy_factor(L, side) ? 1 : 0;
            f.mode = mode_d + i;
            for (int32_t r = 0; r < f.nblk; ++r) rb[bi++] = RowBlock{fi, r * rows};
            ++fi;
        }
        const bool bf16 = L.grad_dtype == MKOR_DTYPE_BF16;
        const FactorDesc& fL = fd[fi - 2];
        const FactorDesc& fR = fd[fi - 1];
        const int32_t ngp = (int32_t)gpart_count(L), ndp = (int32_t)dpart_count(L);
        R.gpart0 = gp; R.ngpart = ngp;
        R.dpart0 = dp; R.ndpart = ndp;
        if (half) {
            // Y^T = R G^T (stored bf16 in the workspace), then dW_hat = L Y;
            // an fp32 G is first copied to bf16 in the workspace
            void* Yt = base + lo.x_off[i];
            const void* Gq = L.G;
            if (needs_cvt(L)) {
                unsigned short* gh = reinterpret_cast<unsigned short*>(base + lo.gh_off[i]);
                const int64_t ne = (int64_t)L.d_in * L.d_out;
                cvi[nci] = CvtItem{static_cast<const float*>(L.G), gh, ne, mode_d + i};
                for (int64_t o = 0; o < ne; o += CVT_ELEMS) cvb[ncb++] = CvtBlock{nci, 0, o};
                ++nci;
                Gq = gh;
            }
            const StageGeom s1 = stage_geom(L, 1), s2 = stage_geom(L, 2);
            HgLayer& A = h1l[i];
            A.P = L.Rinv; A.Q = Gq; A.C = Yt;
            A.pend = fR.pend; A.w = fR.w;
            A.I = s1.rows; A.J = s1.cols; A.K = s1.K;
            A.part0 = gp; A.ntj = ceil_div(s1.cols, s1.bn);
            A.mode = mode_d + i;
            HgLayer& B = h2l[i];
            B.P = L.Linv; B.Q = Yt; B.C = L.dW;
            B.pend = fL.pend; B.w = fL.w;
            B.I = s2.rows; B.J = s2.cols; B.K = s2.K;
            B.part0 = dp; B.ntj = ceil_div(s2.cols, s2.bn);
            B.mode = mode_d + i;
            gp += ngp;
            dp += ndp;
            continue;
        }
        if (is_swapped(L)) {
            // X = L G with Q = G^T (bf16, transposed into the workspace), then
            // dW_hat = X R with the factor R as the Q operand
            void* X = base + lo.x_off[i];
            unsigned short* Gt = reinterpret_cast<unsigned short*>(base + lo.gt_off[i]);
            tri[nti] = TrItem{static_cast<const unsigned short*>(L.G), Gt, L.d_in, L.d_out, mode_d + i};
            for (int32_t r0 = 0; r0 < L.d_in; r0 += 64)
                for (int32_t c0 = 0; c0 < L.d_out; c0 += 64) trb[ntb++] = TrBlock{nti, r0, c0, 0};
            ++nti;
            const StageGeom s1 = stage_geom(L, 1), s2 = stage_geom(L, 2);
            HgLayer& A = s1l[i];
            A.P = L.Linv; A.Q = Gt; A.C = X;
            A.pend = fL.pend; A.w = fL.w;
            A.I = s1.rows; A.J = s1.cols; A.K = s1.K;
            A.part0 = gp; A.ntj = ceil_div(s1.cols, s1.bn);
            A.qf32 = 0; A.fq = 0; A.wide = s1.bm == SG_BI1H;
            A.rq = reinterpret_cast<float*>(base + lo.rq_off[i]);
            A.mode = mode_d + i;
            for (int32_t r = 0; r < ngp; ++r) qdb[nqb++] = QdBlock{i, r, qd_rows_of(L)};
            HgLayer& B = s2l[i];
            B.P = X; B.Q = L.Rinv; B.C = L.dW;
            B.pend = fR.pend; B.w = fR.w;
            B.I = s2.rows; B.J = s2.cols; B.K = s2.K;
            B.part0 = dp; B.ntj = ceil_div(s2.cols, s2.bn);
            B.qf32 = 1; B.fq = 1;
            B.mode = mode_d + i;
            gp += ngp;
            dp += ndp;
            continue;
        }
        if (is_split(L)) {
            // Y^T = R G^T (fp32 in the workspace), then dW_hat = L Y, both on
            // the bf16 split of the fp32 operands
            void* Yt = base + lo.x_off[i];
            const StageGeom s1 = stage_geom(L, 1), s2 = stage_geom(L, 2);
            HgLayer& A = s1l[i];
            A.P = L.Rinv; A.Q = L.G; A.C = Yt;
            A.pend = fR.pend; A.w = fR.w;
            A.I = s1.rows; A.J = s1.cols; A.K = s1.K;
            A.part0 = gp; A.ntj = ceil_div(s1.cols, s1.bn);
            A.qf32 = bf16 ? 0 : 1; A.fq = 0; A.wide = s1.bm == SG_BI1H;
            A.rq = reinterpret_cast<float*>(base + lo.rq_off[i]);
            A.mode = mode_d + i;
            for (int32_t r = 0; r < ngp; ++r) qdb[nqb++] = QdBlock{i, r, qd_rows_of(L)};
            HgLayer& B = s2l[i];
            B.P = L.Linv; B.Q = Yt; B.C = L.dW;
            B.pend = fL.pend; B.w = fL.w;
            B.I = s2.rows; B.J = s2.cols; B.K = s2.K;
            B.part0 = dp; B.ntj = ceil_div(s2.cols, s2.bn);
            B.qf32 = 1; B.fq = 0;
            B.mode = mode_d + i;
            gp += ngp;
            dp += ndp;
            continue;
        }
        float* X = reinterpret_cast<float*>(base + lo.x_off[i]);
        const int32_t tn1 = ceil_div(L.d_out, GEMM_SHAPE[0].bn);
        const int32_t tn2 = ceil_div(L.d_out, GEMM_SHAPE[1].bn);
        GemmLayer& A = g1l[i];
        A.At = static_cast<const float*>(L.Linv); A.B = L.G; A.C = X;
        A.pend = fL.pend; A.w = fL.w;
        A.M = L.d_in; A.N = L.d_out; A.K = L.d_in;
        A.b_bf16 = bf16;
        A.vec = (L.d_in % 4 == 0) && (L.d_out % 4 == 0);
        A.part0 = gp; A.ntn = tn1;
        A.mode = mode_d + i;
        GemmLayer& B = g2l[i];
        B.At = X; B.B = L.Rinv; B.C = L.dW;
        B.pend = fR.pend; B.w = fR.w;
        B.M = L.d_in; B.N = L.d_out; B.K = L.d_out;
        B.b_bf16 = 0;
        B.vec = (L.d_in % 4 == 0) && (L.d_out % 4 == 0);
        B.part0 = dp; B.ntn = tn2;
        B.mode = mode_d + i;
        gp += ngp;
        dp += ndp;
    }
    const std::vector<GemmTile> t1 = schedule_tiles(layers, n, 1, FAM_FP32), t2 = schedule_tiles(layers, n, 2, FAM_FP32);
    std::copy(t1.begin(), t1.end(), g1t);
    std::copy(t2.begin(), t2.end(), g2t);
    const std::vector<GemmTile> u1 = schedule_tiles(layers, n, 1, FAM_HALF), u2 = schedule_tiles(layers, n, 2, FAM_HALF);
    std::copy(u1.begin(), u1.end(), h1t);
    std::copy(u2.begin(), u2.end(), h2t);
    const std::vector<GemmTile> v1 = schedule_tiles(layers, n, 1, FAM_SPLIT), v2 = schedule_tiles(layers, n, 2, FAM_SPLIT);
    std::copy(v1.begin(), v1.end(), s1t);
    std::copy(v2.begin(), v2.end(), s2t);

}

int run_stage(const WsView& v, const mkor_params* prm, int32_t stage, hipStream_t s) {
    const Layout& lo = *v.lo;
    char* ws = v.ws;
    const FactorDesc* fd = reinterpret_cast<const FactorDesc*>(ws + lo.off_factors);
    const RowBlock* rb = reinterpret_cast<const RowBlock*>(ws + lo.off_rowblocks);
    float4* smpart = reinterpret_cast<float4*>(ws + lo.off_smpart);
    float* gram = reinterpret_cast<float*>(ws + lo.off_gram);
    float* gpart = reinterpret_cast<float*>(ws + lo.off_gpart);
    float* dpart = reinterpret_cast<float*>(ws + lo.off_dpart);
    hipError_t e = hipSuccess;
    switch (stage) {
        case MKOR_STAGE_MEANS:
            if (lo.nmeanitem == 0) return MKOR_OK;
            e = launch_colmean(reinterpret_cast<const MeanMat*>(ws + lo.off_mmat),
                               reinterpret_cast<const MeanItem*>(ws + lo.off_mitem), lo.nmeanitem,
                               reinterpret_cast<const MeanItem*>(ws + lo.off_mchunk), lo.nmeanchunk,
                               reinterpret_cast<double*>(ws + lo.off_mpart), s);
            if (e != hipSuccess) return hip_fail(e, "colmean launch");
            return MKOR_OK;
        case MKOR_STAGE_SM_PASS:
            if (lo.nrowblocks == 0) return MKOR_OK;
            e = launch_sm_pass(fd, rb, lo.nrowblocks, smpart, gram, prm->norm_kind, 1, lo.nranked > 0, s);
            if (e != hipSuccess) return hip_fail(e, "sm_pass launch");
            return MKOR_OK;
        case MKOR_STAGE_SM_FINALIZE:
            if (lo.nfactors == 0) return MKOR_OK;
            e = launch_sm_finalize(fd, lo.nfactors, smpart, gram, *prm, s);
            if (e != hipSuccess) return hip_fail(e, "sm_finalize launch");
            // rank-r updates are written into their factors at once
            if (lo.nranked > 0) e = launch_sm_apply_rank(fd, rb, lo.nrowblocks, lo.nfactors, s);
            if (e != hipSuccess) return hip_fail(e, "rank-r apply launch");
            return MKOR_OK;
        case MKOR_STAGE_GEMM_PREP:
            e = launch_cvt_bf16(reinterpret_cast<const CvtItem*>(ws + lo.off_cvti),
                                reinterpret_cast<const CvtBlock*>(ws + lo.off_cvtb), lo.ncvtblk, s);
            if (e != hipSuccess) return hip_fail(e, "bf16 gradient copy launch");
            e = launch_transpose_bf16(reinterpret_cast<const TrItem*>(ws + lo.off_tri),
                                      reinterpret_cast<const TrBlock*>(ws + lo.off_trb), lo.ntrblk, s);
            if (e != hipSuccess) return hip_fail(e, "bf16 gradient transpose launch");
            e = launch_qdot(reinterpret_cast<const HgLayer*>(ws + lo.off_s1l),
                            reinterpret_cast<const QdBlock*>(ws + lo.off_qdb), lo.nqdb, gpart, s);
            if (e != hipSuccess) return hip_fail(e, "split gemm row pass launch");
            return MKOR_OK;
        case MKOR_STAGE_GEMM_XT:
            e = launch_gemm_xt(reinterpret_cast<const GemmLayer*>(ws + lo.off_g1l),
                               reinterpret_cast<const GemmTile*>(ws + lo.off_g1t), lo.ng1, gpart, s);
            if (e != hipSuccess) return hip_fail(e, "gemm_xt launch");
            e = launch_hgemm(1, reinterpret_cast<const HgLayer*>(ws + lo.off_h1l),
                             reinterpret_cast<const GemmTile*>(ws + lo.off_h1t), lo.nh1, gpart, s);
            if (e != hipSuccess) return hip_fail(e, "bf16 gemm (R G^T) launch");
            e = launch_sgemm(1, reinterpret_cast<const HgLayer*>(ws + lo.off_s1l),
                             reinterpret_cast<const GemmTile*>(ws + lo.off_s1t), lo.ns1, gpart, s);
            if (e != hipSuccess) return hip_fail(e, "split gemm (R G^T) launch");
            return MKOR_OK;
        case MKOR_STAGE_GEMM_DW:
            e = launch_gemm_dw(reinterpret_cast<const GemmLayer*>(ws + lo.off_g2l),
                               reinterpret_cast<const GemmTile*>(ws + lo.off_g2t), lo.ng2, dpart, s);
            if (e != hipSuccess) return hip_fail(e, "gemm_dw launch");
            e = launch_hgemm(2, reinterpret_cast<const HgLayer*>(ws + lo.off_h2l),
                             reinterpret_cast<const GemmTile*>(ws + lo.off_h2t), lo.nh2, dpart, s);
            if (e != hipSuccess) return hip_fail(e, "bf16 gemm (L Y) launch");
            e = launch_sgemm(2, reinterpret_cast<const HgLayer*>(ws + lo.off_s2l),
                             reinterpret_cast<const GemmTile*>(ws + lo.off_s2t), lo.ns2, dpart, s);
            if (e != hipSuccess) return hip_fail(e, "split gemm (L Y) launch");
            return MKOR_OK;
        case MKOR_STAGE_RESCALE:
            e = launch_rescale(reinterpret_cast<const RescaleLayer*>(ws + lo.off_rsl),
                               reinterpret_cast<const RescaleBlock*>(ws + lo.off_rsb), lo.nrsblocks, gpart,
                               dpart, prm->rescale, s);
            if (e != hipSuccess) return hip_fail(e, "rescale launch");
            return MKOR_OK;
        default:
            return fail(MKOR_INVALID_ARG, "stage = %d unknown", stage);
    }
}

int run_range(const WsView& v, const mkor_params* prm, int32_t first, int32_t last, hipStream_t s) {
    if (v.n == 0) return MKOR_OK;
    for (int32_t st = first; st <= last; ++st) {
        const int r = run_stage(v, prm, st, s);
        if (r != MKOR_OK) return r;
    }
    return MKOR_OK;
}

// Writes every pending term into its factor buffer and clears the terms.
int sync_factors(const WsView& v, hipStream_t s) {
    const Layout& lo = *v.lo;
    if (v.n == 0 || lo.nfactors == 0) return MKOR_OK;
    const FactorDesc* fd = reinterpret_cast<const FactorDesc*>(v.ws + lo.off_factors);
    const RowBlock* rb = reinterpret_cast<const RowBlock*>(v.ws + lo.off_rowblocks);
    float4* smpart = reinterpret_cast<float4*>(v.ws + lo.off_smpart);
    hipError_t e = launch_sm_pass(fd, rb, lo.nrowblocks, smpart, nullptr, MKOR_NORM_INF, 0, lo.nranked > 0, s);
    if (e != hipSuccess) return hip_fail(e, "sm_pass launch");
    e = launch_sm_reset(fd, lo.nfactors, s);
    if (e != hipSuccess) return hip_fail(e, "sm_reset launch");
    return MKOR_OK;
}

// Parameters valid, and valid for a layer list with `nranked` rank-r layers:
// those exist for the EXACT variant only.
int check_run_params(const mkor_params* params, int32_t nranked) {
    const int st = check_params(params);
    if (st != MKOR_OK) return st;
    if (nranked > 0 && params->sm_variant != MKOR_SM_EXACT)
        return fail(MKOR_UNSUPPORTED, "rank-r layers need sm_variant = MKOR_SM_EXACT");
    return MKOR_OK;
}

}  // namespace mkor

struct mkor_plan {
    int32_t n = 0;
    char* ws = nullptr;
    Layout lo;
    std::vector<uint8_t> optbuf;   // per layer: 1 W, 2 opt_m, 4 opt_v
    std::vector<uint8_t> planned;  // per layer: 1 second-order at creation (has factors)
    std::vector<uint8_t> rank1;    // per layer: second-order with a rank-1 update (leaves pending terms)
    std::vector<int32_t> mode;     // per layer: the mode word as the calls on the plan set it
    int32_t pending = 0;           // a factor update ran since creation or the last sync
};

extern "C" {

int mkor_abi_version(void) { return MKOR_ABI_VERSION; }

const char* mkor_status_string(int status) {
    switch (status) {
        case MKOR_OK: return "MKOR_OK";
        case MKOR_INVALID_ARG: return "MKOR_INVALID_ARG";
        case MKOR_WORKSPACE_TOO_SMALL: return "MKOR_WORKSPACE_TOO_SMALL";
        case MKOR_UNSUPPORTED: return "MKOR_UNSUPPORTED";
        case MKOR_HIP_ERROR: return "MKOR_HIP_ERROR";
        default: return "MKOR_UNKNOWN_STATUS";
    }
}

const char* mkor_last_error(void) { return g_err; }

int mkor_params_check(const mkor_params* params) {
    g_err[0] = 0;
    return check_params(params);
}

int mkor_workspace_size(const mkor_layer* layers, int32_t n, size_t* bytes) {
    g_err[0] = 0;
    if (bytes == nullptr) return fail(MKOR_INVALID_ARG, "bytes is NULL");
    int st = check_layers(layers, n, nullptr, 0);
    if (st != MKOR_OK) return st;
    Layout lo;
    st = compute_layout(layers, n, lo);
    if (st != MKOR_OK) return st;
    *bytes = lo.total;
    return MKOR_OK;
}

int mkor_plan_create(const mkor_layer* layers, int32_t n, void* d_workspace, size_t ws_bytes,
                     mkor_plan** out) {
    const TraceRange range("mkor_plan_create");
    g_err[0] = 0;
    if (out == nullptr) return fail(MKOR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    int st = check_layers(layers, n, nullptr, 0);
    if (st != MKOR_OK) return st;
    Layout lo;
    st = compute_layout(layers, n, lo);
    if (st != MKOR_OK) return st;
    if (lo.total > 0) {
        if (d_workspace == nullptr) return fail(MKOR_INVALID_ARG, "workspace is NULL");
        if (!aligned(d_workspace, 256)) return fail(MKOR_INVALID_ARG, "workspace is not 256-byte aligned");
        if (ws_bytes < lo.total)
            return fail(MKOR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, the plan needs %zu", ws_bytes,
                        lo.total);
        st = check_layers(layers, n, d_workspace, lo.total);
        if (st != MKOR_OK) return st;
    }

    std::vector<char> host;
    build_tables(layers, n, static_cast<char*>(d_workspace), lo, host);
    char* base = static_cast<char*>(d_workspace);

    mkor_plan* plan = new (std::nothrow) mkor_plan;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "out of host memory");
    plan->n = n;
    plan->ws = base;
    plan->lo = lo;
    plan->optbuf.resize(n);
    plan->planned.resize(n);
    plan->rank1.resize(n);
    plan->mode.resize(n);
    for (int32_t i = 0; i < n; ++i) {
        const mkor_layer& L = layers[i];
        plan->optbuf[i] = (uint8_t)((L.W ? 1 : 0) | (L.opt_m ? 2 : 0) | (L.opt_v ? 4 : 0));
        plan->planned[i] = (uint8_t)L.second_order;
        plan->rank1[i] = (uint8_t)(L.second_order == 1 && L.rank <= 1);
        plan->mode[i] = L.second_order;
    }
    if (lo.table_bytes > 0) {
        hipError_t e = hipMemcpy(base, host.data(), lo.table_bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            delete plan;
            return hip_fail(e, "uploading plan descriptors");
        }
    }
    *out = plan;
    return MKOR_OK;
}

static WsView view(const mkor_plan* p) { return WsView{p->ws, &p->lo, p->n}; }

static int check_plan_params(const mkor_plan* plan, const mkor_params* params) {
    return check_run_params(params, plan->lo.nranked);
}

// A range that includes the factor update leaves pending terms on the
// rank-1 factors of the layers whose mode is second-order.
static void note_update(mkor_plan* p, int32_t first, int32_t last) {
    if (first > MKOR_STAGE_SM_FINALIZE || last < MKOR_STAGE_SM_FINALIZE) return;
    for (int32_t i = 0; i < p->n; ++i)
        if (p->rank1[i] && p->mode[i]) p->pending = 1;
}

static int run_range(mkor_plan* p, const mkor_params* prm, int32_t first, int32_t last, hipStream_t s) {
    const int st = run_range(view(p), prm, first, last, s);
    if (st == MKOR_OK) note_update(p, first, last);
    return st;
}

static int check_opt(const mkor_opt_params* o) {
    if (o == nullptr) return fail(MKOR_INVALID_ARG, "opt is NULL");
    if (o->kind != MKOR_OPT_SGD && o->kind != MKOR_OPT_LAMB)
        return fail(MKOR_INVALID_ARG, "opt kind = %d unknown", o->kind);
    if (!(o->lr >= 0.f) || !std::isfinite(o->lr)) return fail(MKOR_INVALID_ARG, "lr = %g must be finite and >= 0", (double)o->lr);
    if (!(o->weight_decay >= 0.f) || !std::isfinite(o->weight_decay))
        return fail(MKOR_INVALID_ARG, "weight_decay = %g must be finite and >= 0", (double)o->weight_decay);
    if (o->store_dw != 0 && o->store_dw != 1) return fail(MKOR_INVALID_ARG, "store_dw = %d is not 0 or 1", o->store_dw);
    if (o->reserved != 0) return fail(MKOR_INVALID_ARG, "reserved = %d must be 0", o->reserved);
    if (o->kind == MKOR_OPT_SGD && !(o->momentum >= 0.f && o->momentum < 1.f))
        return fail(MKOR_INVALID_ARG, "momentum = %g outside [0, 1)", (double)o->momentum);
    if (o->kind == MKOR_OPT_LAMB) {
        if (!(o->beta1 >= 0.f && o->beta1 < 1.f) || !(o->beta2 >= 0.f && o->beta2 < 1.f))
            return fail(MKOR_INVALID_ARG, "betas = (%g, %g) outside [0, 1)", (double)o->beta1, (double)o->beta2);
        if (!(o->eps > 0.f) || !std::isfinite(o->eps)) return fail(MKOR_INVALID_ARG, "eps = %g must be > 0", (double)o->eps);
        if (o->step < 1) return fail(MKOR_INVALID_ARG, "step = %d must be >= 1", o->step);
    }
    return MKOR_OK;
}

// The fused rescale + optimizer stage (in place of MKOR_STAGE_RESCALE).
static int run_rescale_opt(mkor_plan* p, const mkor_params* prm, const mkor_opt_params* o, hipStream_t s) {
    const Layout& lo = p->lo;
    char* ws = p->ws;
    OptArgs a{};
    a.kind = o->kind;
    a.store_dw = o->store_dw;
    a.lr = o->lr; a.mom = o->momentum; a.b1 = o->beta1; a.b2 = o->beta2; a.eps = o->eps;
    a.wd = o->weight_decay;
    a.bc1 = o->kind == MKOR_OPT_LAMB ? (float)(1.0 / (1.0 - std::pow((double)o->beta1, (double)o->step))) : 1.f;
    a.bc2 = o->kind == MKOR_OPT_LAMB ? (float)(1.0 / (1.0 - std::pow((double)o->beta2, (double)o->step))) : 1.f;
    const hipError_t e = launch_rescale_opt(reinterpret_cast<const RescaleLayer*>(ws + lo.off_rsl), p->n,
                                            reinterpret_cast<const RescaleBlock*>(ws + lo.off_rsb), lo.nrsblocks,
                                            reinterpret_cast<const float*>(ws + lo.off_gpart),
                                            reinterpret_cast<const float*>(ws + lo.off_dpart), prm->rescale, a,
                                            reinterpret_cast<float2*>(ws + lo.off_lpart),
                                            reinterpret_cast<float*>(ws + lo.off_trust), s);
    if (e != hipSuccess) return hip_fail(e, "rescale + optimizer launch");
    return MKOR_OK;
}

static int check_opt_plan(const mkor_plan* plan, const mkor_opt_params* o) {
    const int st = check_opt(o);
    if (st != MKOR_OK) return st;
    const uint8_t need = o->kind == MKOR_OPT_SGD ? 2 : 6;
    for (int32_t i = 0; i < plan->n; ++i)
        if ((plan->optbuf[i] & 1) && (plan->optbuf[i] & need) != need)
            return fail(MKOR_INVALID_ARG, "layer %d has W but not the %s state", i,
                        o->kind == MKOR_OPT_SGD ? "opt_m" : "opt_m / opt_v");
    return MKOR_OK;
}

int mkor_update_factors(mkor_plan* plan, const mkor_params* params, void* stream) {
    const TraceRange range("mkor_update_factors");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    int st = check_plan_params(plan, params);
    if (st != MKOR_OK) return st;
    return run_range(plan, params, MKOR_STAGE_MEANS, MKOR_STAGE_SM_FINALIZE,
                     static_cast<hipStream_t>(stream));
}

int mkor_precondition(mkor_plan* plan, const mkor_params* params, void* stream) {
    const TraceRange range("mkor_precondition");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    int st = check_plan_params(plan, params);
    if (st != MKOR_OK) return st;
    return run_range(plan, params, MKOR_STAGE_GEMM_PREP, MKOR_STAGE_RESCALE,
                     static_cast<hipStream_t>(stream));
}

int mkor_step(mkor_plan* plan, const mkor_params* params, void* stream) {
    const TraceRange range("mkor_step");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    int st = check_plan_params(plan, params);
    if (st != MKOR_OK) return st;
    return run_range(plan, params, MKOR_STAGE_MEANS, MKOR_STAGE_RESCALE,
                     static_cast<hipStream_t>(stream));
}

int mkor_opt_params_check(const mkor_opt_params* opt) {
    g_err[0] = 0;
    return check_opt(opt);
}

int mkor_step_opt(mkor_plan* plan, const mkor_params* params, const mkor_opt_params* opt, void* stream) {
    const TraceRange range("mkor_step_opt");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    int st = check_plan_params(plan, params);
    if (st != MKOR_OK) return st;
    st = check_opt_plan(plan, opt);
    if (st != MKOR_OK) return st;
    if (plan->n == 0) return MKOR_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = run_range(plan, params, MKOR_STAGE_MEANS, MKOR_STAGE_GEMM_DW, s);
    if (st != MKOR_OK) return st;
    return run_rescale_opt(plan, params, opt, s);
}

int mkor_precondition_opt(mkor_plan* plan, const mkor_params* params, const mkor_opt_params* opt,
                          void* stream) {
    const TraceRange range("mkor_precondition_opt");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    int st = check_plan_params(plan, params);
    if (st != MKOR_OK) return st;
    st = check_opt_plan(plan, opt);
    if (st != MKOR_OK) return st;
    if (plan->n == 0) return MKOR_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = run_range(plan, params, MKOR_STAGE_GEMM_PREP, MKOR_STAGE_GEMM_DW, s);
    if (st != MKOR_OK) return st;
    return run_rescale_opt(plan, params, opt, s);
}

int mkor_run_stage(mkor_plan* plan, const mkor_params* params, int32_t stage, void* stream) {
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    int st = check_plan_params(plan, params);
    if (st != MKOR_OK) return st;
    if (stage < 0 || stage >= MKOR_NUM_STAGES) return fail(MKOR_INVALID_ARG, "stage = %d unknown", stage);
    if (plan->n == 0) return MKOR_OK;
    static const char* const names[MKOR_NUM_STAGES] = {
        "mkor_run_stage: means", "mkor_run_stage: sm_pass", "mkor_run_stage: sm_finalize", "mkor_run_stage: gemm_prep",
        "mkor_run_stage: gemm_xt", "mkor_run_stage: gemm_dw", "mkor_run_stage: rescale"};
    const TraceRange range(names[stage]);
    st = run_stage(view(plan), params, stage, static_cast<hipStream_t>(stream));
    if (st == MKOR_OK) note_update(plan, stage, stage);
    return st;
}

int mkor_sync_factors(mkor_plan* plan, void* stream) {
    const TraceRange range("mkor_sync_factors");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    const int st = sync_factors(view(plan), static_cast<hipStream_t>(stream));
    if (st == MKOR_OK) plan->pending = 0;
    return st;
}

int mkor_factors_pending(const mkor_plan* plan, int32_t* pending) {
    g_err[0] = 0;
    if (plan == nullptr || pending == nullptr) return fail(MKOR_INVALID_ARG, "plan or pending is NULL");
    *pending = plan->pending;
    return MKOR_OK;
}

int mkor_set_second_order(mkor_plan* plan, const int32_t* flags, void* stream) {
    const TraceRange range("mkor_set_second_order");
    g_err[0] = 0;
    if (plan == nullptr) return fail(MKOR_INVALID_ARG, "plan is NULL");
    if (plan->n == 0) return MKOR_OK;
    if (flags == nullptr) return fail(MKOR_INVALID_ARG, "flags is NULL");
    for (int32_t i = 0; i < plan->n; ++i) {
        if (flags[i] != 0 && flags[i] != 1)
            return fail(MKOR_INVALID_ARG, "flags[%d] = %d is not 0 or 1", i, flags[i]);
        if (flags[i] == 1 && !plan->planned[i])
            return fail(MKOR_INVALID_ARG, "layer %d was planned first-order (it has no factors)", i);
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t* mode_d = reinterpret_cast<int32_t*>(plan->ws + plan->lo.off_mode);
    for (int32_t first = 0; first < plan->n; first += MODE_CHUNK) {
        const int32_t count = std::min<int32_t>(MODE_CHUNK, plan->n - first);
        uint32_t bits[MODE_CHUNK / 32] = {};
        for (int32_t k = 0; k < count; ++k) bits[k >> 5] |= (uint32_t)flags[first + k] << (k & 31);
        const hipError_t e = launch_set_modes(mode_d, first, count, bits, s);
        if (e != hipSuccess) return hip_fail(e, "mode word launch");
    }
    std::copy(flags, flags + plan->n, plan->mode.begin());
    return MKOR_OK;
}

void mkor_plan_destroy(mkor_plan* plan) { delete plan; }

}  // extern "C"
