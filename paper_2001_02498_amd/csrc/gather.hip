// Row gather for a sampled minibatch (Section 4.1: the accelerator receives
// the input features of the minibatch's vertices). With the full graph's
// features resident in device memory, a minibatch's rows are copied from
// them by vertex id: one wavefront per row, each lane moving consecutive
// 16-, 4- or 1-byte words, so a row is read and written in contiguous runs.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "prof.h"

using gcn::set_error;

namespace {

constexpr int kRowsPerBlock = 4;   // one wavefront per row, 256 threads

template <class Word>
__global__ __launch_bounds__(256) void gather_rows_kernel(
    const char* __restrict__ src, int64_t ld_src, int64_t n_src, const int32_t* __restrict__ idx,
    int32_t n, int64_t words, char* __restrict__ dst, int64_t ld_dst) {
    const int lane = threadIdx.x & 63;
    for (int64_t k = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6); k < n;
         k += (int64_t)gridDim.x * kRowsPerBlock) {
        const int64_t v = idx[k];
        if (v < 0 || v >= n_src) continue;
        const Word* s = reinterpret_cast<const Word*>(src + v * ld_src);
        Word* d = reinterpret_cast<Word*>(dst + k * ld_dst);
        for (int64_t w = lane; w < words; w += 64) d[w] = s[w];
    }
}

}  // namespace

extern "C" int gcn_gather_rows(const void* src, int64_t ld_src, int64_t n_src,
                               const int32_t* idx, int32_t n, int64_t row_bytes, void* dst,
                               int64_t ld_dst, gcn_stream_t stream) {
    GCN_CHECK_ARG(n >= 0 && n_src >= 0 && row_bytes >= 0, "gcn_gather_rows: negative size");
    GCN_CHECK_ARG(row_bytes <= ld_src && row_bytes <= ld_dst,
                  "gcn_gather_rows: row_bytes %lld above a stride (%lld, %lld)",
                  (long long)row_bytes, (long long)ld_src, (long long)ld_dst);
    if (n == 0 || row_bytes == 0) return GCN_OK;
    GCN_CHECK_ARG(src && idx && dst, "gcn_gather_rows: NULL argument");
    const uintptr_t align = (uintptr_t)src | (uintptr_t)dst | (uintptr_t)ld_src |
                            (uintptr_t)ld_dst | (uintptr_t)row_bytes;
    const hipStream_t s = (hipStream_t)stream;
    const int64_t blocks = std::min<int64_t>((n + kRowsPerBlock - 1) / kRowsPerBlock, 65536);
    const dim3 grid((unsigned)blocks), block(256);
    const char* sp = static_cast<const char*>(src);
    char* dp = static_cast<char*>(dst);
    {
        gcn::ProfScope prof(s, gcn::K_GATHER, 0.0, 2.0 * n * row_bytes + 4.0 * n);
        if ((align & 15) == 0)
            gather_rows_kernel<uint4><<<grid, block, 0, s>>>(sp, ld_src, n_src, idx, n,
                                                             row_bytes / 16, dp, ld_dst);
        else if ((align & 3) == 0)
            gather_rows_kernel<uint32_t><<<grid, block, 0, s>>>(sp, ld_src, n_src, idx, n,
                                                                row_bytes / 4, dp, ld_dst);
        else
            gather_rows_kernel<uint8_t><<<grid, block, 0, s>>>(sp, ld_src, n_src, idx, n,
                                                               row_bytes, dp, ld_dst);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) {
        set_error("gcn_gather_rows: %s", hipGetErrorString(e));
        return GCN_E_HIP;
    }
    return GCN_OK;
}
