// Host-side plan machinery of libmkor, shared by the C ABI entry points:
// argument validation, the workspace layout, the descriptor tables, and the
// launch of each kernel of a step against a workspace.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "mkor_internal.h"

namespace mkor {

// A roctx range over the host-side span of an entry point (its launches), so
// that a trace (rocprofv3 --marker-trace) groups each call's kernels under
// its name.  Costs a function call when no tool is attached.
struct TraceRange {
    explicit TraceRange(const char* name) { roctxRangePush(name); }
    ~TraceRange() { roctxRangePop(); }
    TraceRange(const TraceRange&) = delete;
    TraceRange& operator=(const TraceRange&) = delete;
};

// Records the thread-local error text (mkor_last_error) and returns `status`.
int fail(int status, const char* fmt, ...);
int hip_fail(hipError_t e, const char* what);
void clear_error();

// Byte offsets of every table and buffer in a plan's workspace, and the
// element counts of the grouped launches.
struct Layout {
    size_t off_factors = 0, off_rowblocks = 0, off_pend = 0, off_smpart = 0;
    size_t off_g1l = 0, off_g1t = 0, off_g2l = 0, off_g2t = 0, off_gpart = 0, off_dpart = 0;
    size_t off_rsl = 0, off_rsb = 0, off_x = 0;
    size_t off_mmat = 0, off_mitem = 0, off_mchunk = 0, off_mpart = 0;
    size_t off_h1l = 0, off_h1t = 0, off_h2l = 0, off_h2t = 0;   // bf16-factor GEMMs
    size_t off_s1l = 0, off_s1t = 0, off_s2l = 0, off_s2t = 0;   // fp32 factors on the bf16 split
    size_t off_cvti = 0, off_cvtb = 0;                           // fp32 -> bf16 gradient copies
    size_t off_tri = 0, off_trb = 0;                             // G^T of swapped split layers
    size_t off_qdb = 0;                                          // stage-1 (Q w) row blocks (split)
    size_t off_gram = 0;                                         // rank-r Gram partials
    size_t off_lpart = 0, off_trust = 0;                         // LAMB block sums, per-layer ratios
    size_t off_mode = 0;                                         // per-layer mode words (int32)
    size_t table_bytes = 0;   // descriptor tables [0, table_bytes) are uploaded
    size_t total = 0;
    int32_t nfactors = 0, nrowblocks = 0, ng1 = 0, ng2 = 0, ngpart = 0, ndpart = 0, nrsblocks = 0;
    int32_t nh1 = 0, nh2 = 0;
    int32_t ns1 = 0, ns2 = 0;
    int32_t ncvt = 0, ncvtblk = 0;
    int32_t ntr = 0, ntrblk = 0;
    int32_t nqdb = 0;
    int32_t nsecond = 0;
    int32_t nranked = 0;      // second-order layers with rank > 1
    int32_t nmeanmat = 0, nmeanitem = 0, nmeanchunk = 0;
    int32_t mean_rpb = MEAN_ROWS_MIN;   // rows per block of the mean partials
    int64_t nmeanpart = 0;   // doubles
    std::vector<size_t> u_off, w_off, x_off;   // per factor / per layer offsets (bytes)
    std::vector<size_t> gh_off;                // per layer: bf16 copy of an fp32 G (bf16 factors)
    std::vector<size_t> gt_off;                // per layer: G^T (bf16) of swapped split layers
    std::vector<size_t> rq_off;                // per layer: stage-1 (Q w) of split layers
};

int check_params(const mkor_params* p);
// `params` valid, and valid for a layer list with `nranked` rank-r layers
int check_run_params(const mkor_params* params, int32_t nranked);
// Sizes, pointers, alignment, and overlaps among the buffers of the layers
// and the workspace [ws, ws + ws_bytes) (ws may be NULL).
int check_layers(const mkor_layer* layers, int32_t n, const void* ws, size_t ws_bytes);
int compute_layout(const mkor_layer* layers, int32_t n, Layout& lo);
// The descriptor tables of a workspace that starts at device address `base`:
// host.size() == lo.table_bytes, to be copied to [base, base + table_bytes).
// Every pending term starts empty.
void build_tables(const mkor_layer* layers, int32_t n, char* base, const Layout& lo, std::vector<char>& host);

// A workspace holding the tables of `n` layers laid out as *lo.
struct WsView {
    char*         ws;
    const Layout* lo;
    int32_t       n;
};
// One kernel of a step (MKOR_STAGE_*), or the stages first..last in order.
int run_stage(const WsView& v, const mkor_params* prm, int32_t stage, hipStream_t s);
int run_range(const WsView& v, const mkor_params* prm, int32_t first, int32_t last, hipStream_t s);
// Writes every pending term into its factor buffer and clears the terms.
int sync_factors(const WsView& v, hipStream_t s);

}  // namespace mkor
