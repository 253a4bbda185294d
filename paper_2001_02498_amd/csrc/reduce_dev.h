// Device redundancy reduction (reduce_dev.hip): the rounds of Algorithms
// 1-3 run on the GPU; results come back to the host in the same form as
// the host reduction produces them.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "graph_types.h"

namespace gcn {

struct DeviceReduceResult {
    int32_t naux = 0;
    std::vector<int32_t> rowptr, col, pairs, round_offsets;
    std::vector<gcn_rr_round> stats;
};

// Workspace bytes for reducing the lists rowptr[0..n] (their lengths bound
// every buffer).
int redundancy_reduce_device_bytes(const int32_t* rowptr, int64_t n, const gcn_rr_params* p,
                                   size_t* bytes);

// Runs the rounds on stream s (synchronising it once per round, after the
// pair counting) and downloads the reduced lists.
int redundancy_reduce_device(const int32_t* rowptr, const int32_t* col, int64_t n,
                             const gcn_rr_params* p, void* ws, size_t ws_bytes, hipStream_t s,
                             DeviceReduceResult* out);

}  // namespace gcn
