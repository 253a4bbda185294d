// Launch timing: when enabled, every kernel launch of the library is
// bracketed by a pair of HIP events recorded on the launch's own stream and
// labelled with its kernel class and algorithmic work (flops, bytes).
// Events come from a pool created at enable time; reading synchronises on
// the recorded events and folds them into per-class totals.
#include <atomic>
#include <mutex>
#include <vector>

#include "prof.h"

namespace gcn {
namespace {

struct Record {
    int kind;
    double flops, bytes;
    hipEvent_t a, b;
};

std::mutex g_mu;
std::atomic<bool> g_on{false};
std::vector<hipEvent_t> g_pool;
size_t g_used = 0;
std::vector<Record> g_recs;
int64_t g_dropped = 0;

}  // namespace

const char* kind_name(int k) {
    switch (k) {
        case K_PAIR_SUMS: return "pair_sums";
        case K_LIST_SUMS: return "list_sums";
        case K_GEMM_FWD: return "gemm_fwd";
        case K_GEMM_CLS: return "gemm_cls";
        case K_GEMM_DX: return "gemm_dx";
        case K_GEMM_CLS_DX: return "gemm_cls_dx";
        case K_GEMM_DW: return "gemm_dw";
        case K_GEMM_CLS_DW: return "gemm_cls_dw";
        case K_SGD: return "sgd_reduce";
        case K_LOSS_ROWS: return "loss_rows";
        case K_LOSS_MEAN: return "loss_mean";
        case K_SPLITK_FINISH: return "splitk_finish";
        case K_GEMM_FWD_BF16: return "gemm_fwd_bf16";
        case K_GEMM_CLS_BF16: return "gemm_cls_bf16";
        case K_GEMM_DX_BF16: return "gemm_dx_bf16";
        case K_GEMM_CLS_DX_BF16: return "gemm_cls_dx_bf16";
        case K_GEMM_DW_BF16: return "gemm_dw_bf16";
        case K_GEMM_CLS_DW_BF16: return "gemm_cls_dw_bf16";
        case K_TO_BF16: return "to_bf16";
        case K_GEMM_FWD_IN: return "gemm_fwd_in";
        case K_GEMM_DW_IN: return "gemm_dw_in";
        case K_GEMM_FWD_IN_BF16: return "gemm_fwd_in_bf16";
        case K_GEMM_DW_IN_BF16: return "gemm_dw_in_bf16";
        case K_GATHER: return "gather_rows";
        case K_READ_PROBE: return "read_probe";
        default: return "other";
    }
}

ProfScope::ProfScope(hipStream_t s, int kind, double flops, double bytes)
    : s_(s), idx_(-1) {
    if (!g_on) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_on || g_used + 2 > g_pool.size()) {
        ++g_dropped;
        return;
    }
    Record r{kind, flops, bytes, g_pool[g_used], g_pool[g_used + 1]};
    g_used += 2;
    if (hipEventRecord(r.a, s) != hipSuccess) return;
    idx_ = (int64_t)g_recs.size();
    g_recs.push_back(r);
}

ProfScope::~ProfScope() {
    if (idx_ < 0) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (idx_ < (int64_t)g_recs.size()) (void)hipEventRecord(g_recs[idx_].b, s_);
}

// Read-only streaming kernel: every 16-byte word of the buffer is loaded
// once, four words in flight per thread, and summed; each wavefront's sum
// (reduced across lanes, so no load is dead) goes to its own word of the
// sink. The bandwidth it reaches on a buffer far beyond the 256 MB
// Infinity Cache is what a kernel that only reads can get from HBM.
constexpr int kProbeBlocks = 4096, kProbeThreads = 256;
static_assert(GCN_READ_PROBE_SINK == kProbeBlocks * (kProbeThreads / 64), "sink size");

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const float4* __restrict__ p,
                                                                   int64_t n4,
                                                                   float* __restrict__ sink) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    float s = 0.f;
    for (; i + 3 * stride < n4; i += 4 * stride) {
        const float4 a = p[i], b = p[i + stride], c = p[i + 2 * stride], d = p[i + 3 * stride];
        s += ((a.x + a.y) + (a.z + a.w)) + ((b.x + b.y) + (b.z + b.w)) +
             ((c.x + c.y) + (c.z + c.w)) + ((d.x + d.y) + (d.z + d.w));
    }
    for (; i < n4; i += stride) {
        const float4 a = p[i];
        s += (a.x + a.y) + (a.z + a.w);
    }
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if ((threadIdx.x & 63) == 0) sink[blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6)] = s;
}

}  // namespace gcn

using namespace gcn;

extern "C" {

int gcn_profile_enable(int32_t capacity) {
    GCN_CHECK_ARG(capacity >= 1 && capacity <= (1 << 20),
                  "gcn_profile_enable: capacity %d outside [1, 2^20]", capacity);
    std::lock_guard<std::mutex> lk(g_mu);
    for (hipEvent_t e : g_pool) (void)hipEventDestroy(e);
    g_pool.clear();
    g_recs.clear();
    g_used = 0;
    g_dropped = 0;
    g_pool.reserve(2 * (size_t)capacity);
    for (int32_t i = 0; i < 2 * capacity; ++i) {
        hipEvent_t e;
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) {
            set_error("gcn_profile_enable: hipEventCreate failed (%s)", hipGetErrorString(err));
            for (hipEvent_t x : g_pool) (void)hipEventDestroy(x);
            g_pool.clear();
            g_on = false;
            return GCN_E_HIP;
        }
        g_pool.push_back(e);
    }
    g_recs.reserve(capacity);
    g_on = true;
    return GCN_OK;
}

int gcn_profile_disable(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_on = false;
    return GCN_OK;
}

int gcn_profile_read(gcn_profile_entry* out, int32_t max_entries, int32_t* count,
                     int32_t reset) {
    GCN_CHECK_ARG(count != nullptr, "gcn_profile_read: count is NULL");
    GCN_CHECK_ARG(max_entries >= 0 && (out != nullptr || max_entries == 0),
                  "gcn_profile_read: bad output buffer");
    std::lock_guard<std::mutex> lk(g_mu);
    gcn_profile_entry acc[K_COUNT];
    for (int k = 0; k < K_COUNT; ++k) {
        acc[k] = gcn_profile_entry{};
        acc[k].kind = k;
        acc[k].name = kind_name(k);
        acc[k].min_ms = 1e30;
    }
    for (const Record& r : g_recs) {
        hipError_t e = hipEventSynchronize(r.b);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
        if (e != hipSuccess) {
            set_error("gcn_profile_read: %s", hipGetErrorString(e));
            return GCN_E_HIP;
        }
        gcn_profile_entry& a = acc[r.kind];
        a.launches += 1;
        a.total_ms += ms;
        a.min_ms = ms < a.min_ms ? ms : a.min_ms;
        a.max_ms = ms > a.max_ms ? ms : a.max_ms;
        a.flops += r.flops;
        a.bytes += r.bytes;
    }
    int32_t n = 0;
    for (int k = 0; k < K_COUNT; ++k) {
        if (acc[k].launches == 0) continue;
        if (n < max_entries) out[n] = acc[k];
        ++n;
    }
    *count = n;
    const bool dropped = g_dropped != 0;
    if (reset) {
        g_recs.clear();
        g_used = 0;
        g_dropped = 0;
    }
    if (dropped) {
        set_error("gcn_profile_read: launches went untimed (capacity exhausted)");
        return GCN_E_INTERNAL;
    }
    return GCN_OK;
}

int gcn_read_probe(const void* buf, size_t bytes, float* sink, gcn_stream_t stream) {
    GCN_CHECK_ARG(buf != nullptr && sink != nullptr, "gcn_read_probe: NULL pointer");
    GCN_CHECK_ARG(((uintptr_t)buf & 15) == 0 && (bytes & 15) == 0 && bytes > 0,
                  "gcn_read_probe: buffer must be 16-byte aligned, bytes a positive multiple "
                  "of 16 (got %zu)", bytes);
    GCN_CHECK_ARG(((uintptr_t)sink & 3) == 0, "gcn_read_probe: sink not 4-byte aligned");
    hipStream_t s = (hipStream_t)stream;
    {
        ProfScope prof(s, K_READ_PROBE, (double)bytes / 4, (double)bytes);
        read_probe_kernel<<<dim3(kProbeBlocks), dim3(kProbeThreads), 0, s>>>(
            (const float4*)buf, (int64_t)(bytes / 16), sink);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error("gcn_read_probe: launch failed (%s)", hipGetErrorString(e));
        return GCN_E_HIP;
    }
    return GCN_OK;
}

}  // extern "C"
