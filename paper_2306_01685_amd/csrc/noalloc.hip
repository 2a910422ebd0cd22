// mkor_step_noalloc: one full step for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops).  The workspace
// a plan would keep in caller memory lives in a fixed device array of this
// library instead, `scratch`, one per GPU, held until the process ends.
//
// Every call lays the tables of its layer list out in that array, uploads
// them with kernel launches that carry the bytes as arguments (stream-ordered,
// no host buffer outlives the call, nothing to allocate), runs the stages of
// a step, and writes the updated factors into the caller's buffers: the same
// kernels, in the same order, as a fresh plan's mkor_step followed by
// mkor_sync_factors.  Nothing carries over from one call to the next, so the
// array's earlier contents do not matter; the pending-term table, the only
// part read before it is written, starts out empty with the tables.
#include "plan.h"

#include <algorithm>
#include <cstring>
#include <mutex>

namespace mkor {
namespace {

static __device__ __align__(256) unsigned char scratch[MKOR_NOALLOC_MAX_BYTES];

// Host-side device addresses of `scratch`, one per device (the array's name in
// host code is only a stand-in for the symbol and must never be passed on).
constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void* g_scratch[MAX_DEVICES] = {};

int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= MAX_DEVICES)
        return fail(MKOR_UNSUPPORTED, "device %d: the no-allocation entry point supports devices 0..%d", dev,
                    MAX_DEVICES - 1);
    std::lock_guard<std::mutex> lock(g_mu);
    if (g_scratch[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (p == nullptr) return fail(MKOR_HIP_ERROR, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return MKOR_OK;
}

// Table bytes travel as kernel arguments, UP_WORDS 4-byte words per launch.
constexpr int UP_WORDS = 256;
struct UpChunk {
    uint32_t w[UP_WORDS];
};

__global__ __launch_bounds__(UP_WORDS) void upload_kernel(uint32_t* __restrict__ dst, UpChunk c, int nwords) {
    const int i = threadIdx.x;
    if (i < nwords) dst[i] = c.w[i];
}

int upload(char* dst, const std::vector<char>& host, hipStream_t s) {
    const size_t nw = host.size() / 4;   // table_bytes is a multiple of 256
    const uint32_t* src = reinterpret_cast<const uint32_t*>(host.data());
    for (size_t o = 0; o < nw; o += UP_WORDS) {
        const int k = (int)std::min<size_t>(UP_WORDS, nw - o);
        UpChunk c{};
        std::memcpy(c.w, src + o, 4 * (size_t)k);
        hipLaunchKernelGGL(upload_kernel, dim3(1), dim3(UP_WORDS), 0, s, reinterpret_cast<uint32_t*>(dst) + o, c,
                           k);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(e, "table upload launch");
    }
    return MKOR_OK;
}

}  // namespace
}  // namespace mkor

using namespace mkor;

extern "C" int mkor_step_noalloc(const mkor_layer* layers, int32_t n, const mkor_params* params, void* stream) {
    const TraceRange range("mkor_step_noalloc");
    clear_error();
    int st = check_layers(layers, n, nullptr, 0);
    if (st != MKOR_OK) return st;
    Layout lo;
    st = compute_layout(layers, n, lo);
    if (st != MKOR_OK) return st;
    st = check_run_params(params, lo.nranked);
    if (st != MKOR_OK) return st;
    if (n == 0) return MKOR_OK;
    if (lo.total > (size_t)MKOR_NOALLOC_MAX_BYTES)
        return fail(MKOR_WORKSPACE_TOO_SMALL,
                    "the layer list needs %zu bytes of workspace; mkor_step_noalloc holds at most %zu "
                    "(use a plan with a caller workspace)",
                    lo.total, (size_t)MKOR_NOALLOC_MAX_BYTES);
    void* ptr = nullptr;
    st = scratch_address(&ptr);
    if (st != MKOR_OK) return st;
    char* ws = static_cast<char*>(ptr);
    st = check_layers(layers, n, ws, lo.total);   // no caller buffer may lie inside the array
    if (st != MKOR_OK) return st;

    std::vector<char> host;
    build_tables(layers, n, ws, lo, host);
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = upload(ws, host, s);
    if (st != MKOR_OK) return st;
    const WsView v{ws, &lo, n};
    st = run_range(v, params, MKOR_STAGE_MEANS, MKOR_STAGE_RESCALE, s);
    if (st != MKOR_OK) return st;
    return sync_factors(v, s);
}
