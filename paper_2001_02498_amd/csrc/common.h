// Internal helpers shared by the host and device halves of the library.
#pragma once

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/gcn_act.h"

namespace gcn {

void set_error(const char* fmt, ...);
void clear_error();

// Fails the calling entry point with GCN_E_INVALID_ARG and a message.
#define GCN_CHECK_ARG(cond, ...)                 \
    do {                                         \
        if (!(cond)) {                           \
            ::gcn::set_error(__VA_ARGS__);       \
            return GCN_E_INVALID_ARG;            \
        }                                        \
    } while (0)

inline int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// Layout of the packed device image of a reduced graph. All sections start
// on 256-byte boundaries; the header is stored at offset 0.
struct ImageHeader {
    uint32_t magic;
    int32_t n, naux, rounds, seg_len;
    int32_t nseg, nbins, nmulti, max_row;
    int32_t nhub;
    int64_t nnz, exp_nnz;
    int64_t off_rowptr, off_col, off_pairs, off_inv_deg, off_seg, off_bins;
    int64_t off_exp_col, off_exp_seg;
    int64_t total;
    int32_t round_offsets[GCN_MAX_ROUNDS + 1];
};
constexpr uint32_t kImageMagic = 0x47434e33u;  // "GCN3"
constexpr int kDefaultSegLen = 32;
// Pieces per bin of the list-sum work list: the lane groups of one
// aggregation workgroup. A list split into pieces lies in one bin.
constexpr int kBinGroups = GCN_BIN_GROUPS;

}  // namespace gcn
