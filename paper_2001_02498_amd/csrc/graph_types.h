// Host graph objects behind the opaque handles of gcn_act.h, shared by the
// host preprocessing and the device reduction driver.
#pragma once

#include <cstdint>
#include <vector>

#include "common.h"

struct gcn_graph {
    int32_t n = 0;
    std::vector<int32_t> rowptr;  // n + 1
    std::vector<int32_t> col;
};

struct gcn_reduced {
    int32_t n = 0, naux = 0, rounds = 0;
    std::vector<int32_t> rowptr, col, pairs, round_offsets, deg;
    std::vector<gcn_rr_round> stats;
};
