// Redundancy reduction on the GPU (Section 3.2: Algorithms 1-3 applied in
// rounds), with results identical to the host version in host_graph.cpp.
//
// One round:
//   Algorithm 1  transposed index of the lists (for each id, the stretch
//                after it in every list holding it), then one workgroup
//                per id x counts, in 16-bit LDS
//                counters (65,536 ids per pass), every larger id y that
//                follows x in a list holding x; pairs above the threshold
//                leave as 64-bit keys ordered by (weight descending, x, y).
//   Algorithm 2  the keys are radix-sorted (rocPRIM); one workgroup scans
//                them in blocks, drops pairs with a used endpoint in
//                parallel and takes the rest in key order with one wavefront:
//                the greedy matching under the budget, pair by pair as the
//                host takes it.
//   Algorithm 3  every list is rewritten by one workgroup (its ids marked
//                in an LDS bitmap): entries whose partner is in the same
//                list are replaced by the pair's new id; kept entries keep
//                their order and the new ids (all larger) follow in
//                increasing order.
// The host enqueues the rounds back to back; the kernels read the ids and
// the budget left from a small device-side state, so the host waits once
// per round, after the pair counting (the sort needs the candidate count).
#include <rocprim/device/device_radix_sort.hpp>

#include <algorithm>
#include <climits>
#include <cstring>
#include <new>
#include <vector>

#include "common.h"
#include "reduce_dev.h"

namespace gcn {
namespace {

constexpr int kBlock = 256;
constexpr int kScanThreads = 1024;
constexpr int kScanPer = 4;                           // consecutive values per thread per tile
constexpr int kGreedyThreads = 1024;
constexpr int kGreedyPer = 4;                         // keys per thread per block
constexpr int kGreedyBurst = 256;                     // survivors taken between refilters
constexpr int kGreedyBlock = kGreedyThreads * kGreedyPer;
// ids per reduction: the greedy scan's used set fills at most 64 KB of LDS
// (beside its 64 KB of survivor buffers); pair keys hold 20-bit ids
constexpr int kMaxIds = 1 << 19;
// Candidate sort: rocPRIM's merge sort up to kMergeSortMax keys, its
// onesweep radix sort above (the library's default switches at 2^20)
#ifndef GCN_MERGE_SORT_MAX
#define GCN_MERGE_SORT_MAX 262144
#endif
constexpr size_t kMergeSortMax = GCN_MERGE_SORT_MAX;
using SortConfig = rocprim::radix_sort_config<rocprim::default_config, rocprim::default_config,
                                              rocprim::default_config, kMergeSortMax>;
// ids counted per pass of Algorithm 1: 16-bit counters in 128 KB of LDS
constexpr int kCountWindow = 65536;

// Device-side counters of one round (and the error flag).
struct RoundCounters {
    unsigned long long ncand;   // candidates emitted (may exceed capacity: overflow)
    long long taken, wsum;
    unsigned long long num_add;
    long long nnz;              // list entries after the round's rewrite
};

// Device-side state of a reduction: the rounds run back to back on the
// stream, each reading the ids issued so far from here, so the host waits
// only once per round (for the candidate count the sort needs).
struct DevState {
    long long naux;             // pairs taken in all rounds so far
    int done;                   // a round took no pair, or the budget is spent
    int error;                  // 1: candidate capacity, 2: id out of range,
                                // 3: ids reach kMaxIds, or a pair count
                                //    exceeds 16 bits
    RoundCounters round[GCN_MAX_ROUNDS];
};

__device__ __forceinline__ uint64_t cand_key(uint32_t w, uint32_t x, uint32_t y) {
    return ((uint64_t)(0xFFFFu - w) << 40) | ((uint64_t)x << 20) | (uint64_t)y;
}

// ------------------------------------------------------------------ scan
// out[0] = 0, out[i + 1] = in[0] + .. + in[i] (one workgroup, tiles of
// kScanPer consecutive values per thread, all loaded before any is used: a
// scan inside the thread, one across the wavefront by shuffles, one across
// the 16 wavefront totals). cur, when set, also receives the exclusive
// prefix out[i] wherever in[i] is nonzero; it may be in itself, since every
// value is read by the thread that overwrites it, before it does (a zero
// count then stays zero). With num_add,
// also the sum of max(in[i] - 1, 0) (numAdd of Section 3.2 when in holds
// list lengths).
__global__ __launch_bounds__(kScanThreads) void scan_kernel(const int32_t* in,
                                                            int32_t* __restrict__ out, int len,
                                                            int32_t* cur,
                                                            unsigned long long* num_add,
                                                            long long* total) {
    constexpr int kWaves = kScanThreads / 64;
    __shared__ int32_t wsum[kWaves];
    __shared__ unsigned long long adds[kWaves];
    const int t = threadIdx.x, lane = t % 64, wave = t / 64;
    int32_t carry = 0;   // sum of the earlier tiles
    unsigned long long a = 0;
    if (t == 0) out[0] = 0;
    for (int base = 0; base < len; base += kScanPer * kScanThreads) {
        const int i0 = base + kScanPer * t;
        int32_t v[kScanPer], incl[kScanPer];
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) v[j] = i0 + j < len ? in[i0 + j] : 0;
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            a += v[j] > 1 ? (unsigned long long)(v[j] - 1) : 0ull;
            incl[j] = (j ? incl[j - 1] : 0) + v[j];
        }
        int32_t inc = incl[kScanPer - 1];
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t y = __shfl_up(inc, off);
            if (lane >= off) inc += y;
        }
        if (lane == 63) wsum[wave] = inc;
        __syncthreads();
        int32_t before = carry, tile = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int32_t x = wsum[w];
            before += w < wave ? x : 0;
            tile += x;
        }
        const int32_t ex = before + inc - incl[kScanPer - 1];   // values before this thread's
#pragma unroll
        for (int j = 0; j < kScanPer; ++j) {
            if (i0 + j < len) {
                out[i0 + j + 1] = ex + incl[j];
                if (cur && v[j]) cur[i0 + j] = ex + incl[j] - v[j];
            }
        }
        carry += tile;
        __syncthreads();   // wsum is rewritten by the next tile
    }
    if (num_add) {
        for (int off = 32; off > 0; off >>= 1) a += __shfl_xor(a, off);
        if (lane == 0) adds[wave] = a;
        __syncthreads();
        if (t == 0) {
            unsigned long long tot = 0;
            for (int w = 0; w < kWaves; ++w) tot += adds[w];
            *num_add = tot;
        }
    }
    if (total && t == 0) *total = carry;
}

// A reduction's starting state: no id paired yet, every transposed-index
// count zero (each round's pair counting zeroes them again as it passes).
__global__ void init_kernel(int32_t* __restrict__ partner, int32_t* __restrict__ newid,
                            int32_t* __restrict__ tcnt, int64_t len) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < len) {
        partner[i] = -1;
        newid[i] = -1;
        tcnt[i] = 0;
    }
}

// ------------------------------------------------------------ Algorithm 1
// one wavefront per list
__global__ __launch_bounds__(kBlock) void tcount_kernel(int n, const int32_t* __restrict__ rowptr,
                                                        const int32_t* __restrict__ col,
                                                        int32_t* __restrict__ tcnt,
                                                        DevState* st) {
    const int w = blockIdx.x * (kBlock / 64) + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (w >= n || st->done) return;
    const int ncols = n + (int)st->naux;
    for (int e = rowptr[w] + lane; e < rowptr[w + 1]; e += 64) {
        const int c = col[e];
        if (c < 0 || c >= ncols) {
            st->error = 2;
            continue;
        }
        atomicAdd(&tcnt[c], 1);
    }
}

// For k in [tptr[c], tptr[c + 1]), one per list holding id c (any order
// inside: the counts do not depend on it): tnext[k], the position in col of
// the entry after c in that list, and tend[k], the list's end, so the pair
// counting reads the stretch after c without looking up the list.
__global__ __launch_bounds__(kBlock) void tfill_kernel(int n, const int32_t* __restrict__ rowptr,
                                                       const int32_t* __restrict__ col,
                                                       int32_t* __restrict__ tcur,
                                                       int32_t* __restrict__ tnext,
                                                       int32_t* __restrict__ tend,
                                                       const DevState* st) {
    const int w = blockIdx.x * (kBlock / 64) + threadIdx.x / 64;
    const int lane = threadIdx.x % 64;
    if (w >= n || st->done) return;
    const int ncols = n + (int)st->naux;
    const int end = rowptr[w + 1];
    for (int e = rowptr[w] + lane; e < end; e += 64) {
        const int c = col[e];
        if (c < 0 || c >= ncols) continue;
        const int k = atomicAdd(&tcur[c], 1);
        tnext[k] = e + 1;
        tend[k] = end;
    }
}

// The same two steps with the counts gathered per workgroup first, for id
// ranges whose counters fit LDS: a workgroup takes kTransLists consecutive
// lists (one wavefront per list), counts their ids in LDS, then adds each
// nonzero count to the global one, so an id held by many lists (a hub)
// costs one global atomic per workgroup instead of one per list. The fill
// reserves each id's run of slots the same way, then hands the slots out
// from LDS.
constexpr int kTransLists = 32;
constexpr int kTransMaxIds = 16384;   // 64 KB of LDS counters

__device__ __forceinline__ void trans_count(int n, int nc, const int32_t* __restrict__ rowptr,
                                            const int32_t* __restrict__ col, int32_t* cnt,
                                            DevState* st) {
    const int ncols = min(n + (int)st->naux, nc);
    for (int i = threadIdx.x; i < nc; i += kBlock) cnt[i] = 0;
    __syncthreads();
    const int lane = threadIdx.x % 64;
    const int w1 = min(n, (int)(blockIdx.x + 1) * kTransLists);
    for (int w = blockIdx.x * kTransLists + threadIdx.x / 64; w < w1; w += kBlock / 64) {
        for (int e = rowptr[w] + lane; e < rowptr[w + 1]; e += 64) {
            const int c = col[e];
            if (c < 0 || c >= ncols) {
                st->error = 2;
                continue;
            }
            atomicAdd(&cnt[c], 1);
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(kBlock) void tcount_lds_kernel(int n, int nc,
                                                            const int32_t* __restrict__ rowptr,
                                                            const int32_t* __restrict__ col,
                                                            int32_t* __restrict__ tcnt,
                                                            DevState* st) {
    extern __shared__ int32_t trans_cnt[];
    if (st->done) return;
    trans_count(n, nc, rowptr, col, trans_cnt, st);
    for (int i = threadIdx.x; i < nc; i += kBlock) {
        const int v = trans_cnt[i];
        if (v) atomicAdd(&tcnt[i], v);
    }
}

__global__ __launch_bounds__(kBlock) void tfill_lds_kernel(int n, int nc,
                                                           const int32_t* __restrict__ rowptr,
                                                           const int32_t* __restrict__ col,
                                                           int32_t* __restrict__ tcur,
                                                           int32_t* __restrict__ tnext,
                                                           int32_t* __restrict__ tend,
                                                           DevState* st) {
    extern __shared__ int32_t trans_cnt[];
    if (st->done) return;
    trans_count(n, nc, rowptr, col, trans_cnt, st);
    // this workgroup's slots of id i start where the cursor stood (eight
    // ids per thread at a time, so their atomics are in flight together)
    for (int i0 = threadIdx.x; i0 < nc; i0 += 8 * kBlock) {
        int v[8], r[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * kBlock;
            v[u] = i < nc ? trans_cnt[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (v[u]) r[u] = atomicAdd(&tcur[i0 + u * kBlock], v[u]);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (v[u]) trans_cnt[i0 + u * kBlock] = r[u];
    }
    __syncthreads();
    const int ncols = min(n + (int)st->naux, nc);
    const int lane = threadIdx.x % 64;
    const int w1 = min(n, (int)(blockIdx.x + 1) * kTransLists);
    for (int w = blockIdx.x * kTransLists + threadIdx.x / 64; w < w1; w += kBlock / 64) {
        const int end = rowptr[w + 1];
        for (int e = rowptr[w] + lane; e < end; e += 64) {
            const int c = col[e];
            if (c < 0 || c >= ncols) continue;
            const int k = atomicAdd(&trans_cnt[c], 1);
            tnext[k] = e + 1;
            tend[k] = end;
        }
    }
}

// One workgroup per id x (grid-stride): counts, for every y > x, the lists
// holding both, in 16-bit counters packed two per LDS word; pairs whose
// count exceeds theta (and 1: weight-1 pairs are no edges of G_a) are
// emitted. The ids are counted in windows of kCountWindow (one window when
// there are fewer ids); a window takes, by binary search, the stretch of
// every (sorted) list tail that falls in it. The parts of the lists after x
// are staged (start, prefix of lengths) in LDS, kCountStage lists at a
// time, and all threads sweep their concatenation, so a hub with thousands
// of lists keeps every lane busy. A count is at most the number of lists:
// with 65,535 lists or more a counter that would pass 16 bits is reported
// (error 3) instead of wrapping.
constexpr int kCountThreads = 512;
constexpr int kCountStage = 1024;

// first index in [b, e) of the ascending array a whose value is >= v
__device__ __forceinline__ int lower_bound_dev(const int32_t* __restrict__ a, int b, int e,
                                               int v) {
    while (b < e) {
        const int mid = (b + e) >> 1;
        if (a[mid] < v)
            b = mid + 1;
        else
            e = mid;
    }
    return b;
}

__global__ __launch_bounds__(kCountThreads) void count_pairs_kernel(
    int n, int theta, const int32_t* __restrict__ col,
    const int32_t* __restrict__ tptr, const int32_t* __restrict__ tnext,
    const int32_t* __restrict__ tend, int32_t* __restrict__ tcur, uint64_t* __restrict__ cand,
    int64_t cap,
    DevState* st, int round) {
    extern __shared__ uint32_t cnt[];
    __shared__ int32_t s_start[kCountStage];
    __shared__ int32_t s_off[kCountStage + 1];
    __shared__ int32_t s_wave[kCountThreads / 64];
    if (st->done) return;
    const int ncols = n + (int)st->naux;
    if (ncols >= kMaxIds) {   // pair keys and the greedy scan's used set
        if (threadIdx.x == 0 && blockIdx.x == 0) st->error = 3;
        return;
    }
    RoundCounters* rc = &st->round[round];
    const bool windowed = ncols > kCountWindow;
    const int win = windowed ? kCountWindow : ncols;
    const bool check = n >= 65535;   // counts can reach 2^16 only with that many lists
    const int t = threadIdx.x, lane = t % 64, wave = t / 64;
    for (int i = t; i < (win + 1) / 2; i += kCountThreads) cnt[i] = 0;
    __syncthreads();
    for (int x = blockIdx.x; x < ncols; x += gridDim.x) {
        // the fill cursors are done with: zero them as the next round's counts
        if (t == 0) tcur[x] = 0;
        const int tb = tptr[x], te = tptr[x + 1];
        if (te - tb < 2) continue;   // uniform: x in fewer than two lists
        // the windows [y0, y0 + win) holding ids above x
        for (int y0 = windowed ? (x + 1) / win * win : 0; y0 < ncols; y0 += win) {
            const int y1 = min(ncols, y0 + win);
            const int nw = (y1 - y0 + 1) / 2;
            for (int kb = tb; kb < te; kb += kCountStage) {
                const int m = min(kCountStage, te - kb);
                // thread t stages lists 2t, 2t + 1 of this pass
                int len[2], sum = 0;
                for (int j = 0; j < 2; ++j) {
                    const int i = 2 * t + j;
                    len[j] = 0;
                    if (i < m) {
                        const int k = kb + i;
                        int b = tnext[k], e = tend[k];
                        if (windowed) {
                            b = lower_bound_dev(col, b, e, y0);
                            e = lower_bound_dev(col, b, e, y1);
                        }
                        s_start[i] = b;
                        len[j] = e - b;
                    }
                    sum += len[j];
                }
                int incl = sum;
                for (int off = 1; off < 64; off <<= 1) {
                    const int v = __shfl_up(incl, off);
                    if (lane >= off) incl += v;
                }
                if (lane == 63) s_wave[wave] = incl;
                __syncthreads();
                int before = 0;
                for (int v = 0; v < wave; ++v) before += s_wave[v];
                int run = before + incl - sum;
                for (int j = 0; j < 2; ++j) {
                    const int i = 2 * t + j;
                    if (i < m) s_off[i] = run;
                    run += len[j];
                }
                if (t == kCountThreads - 1) s_off[m] = run;   // total (run after the last thread)
                __syncthreads();
                const int total = s_off[m];
                int k = 0;
                for (int v = t; v < total; v += kCountThreads) {
                    // the staged list holding visit v: the last k with s_off[k] <= v
                    int lo = k, hi = m - 1;
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (s_off[mid] <= v)
                            lo = mid;
                        else
                            hi = mid - 1;
                    }
                    k = lo;
                    const int y = col[s_start[k] + (v - s_off[k])] - y0;
                    if ((unsigned)y < (unsigned)(y1 - y0)) {
                        const int sh = (y & 1) * 16;
                        if (check) {
                            const uint32_t old = atomicAdd(&cnt[y >> 1], 1u << sh);
                            if (((old >> sh) & 0xFFFFu) == 0xFFFFu) st->error = 3;
                        } else {
                            atomicAdd(&cnt[y >> 1], 1u << sh);
                        }
                    }
                }
                __syncthreads();
            }
            // Emit the pairs of x in the window (counters of y > x, from
            // the word holding x + 1): count them, reserve one range of
            // slots for the workgroup, then write each thread's pairs at
            // its prefix and clear.
            const int w0 = x + 1 > y0 ? (x + 1 - y0) >> 1 : 0;
            auto emits = [&](uint32_t v, int wd, int h) {
                const int y = y0 + 2 * wd + h;
                const uint32_t c = (v >> (16 * h)) & 0xFFFFu;
                return y > x && (int)c > theta && c >= 2;
            };
            int mine = 0;
            for (int wd = w0 + t; wd < nw; wd += kCountThreads) {
                const uint32_t v = cnt[wd];
                if (v) mine += emits(v, wd, 0) + emits(v, wd, 1);
            }
            int incl = mine;
            for (int off = 1; off < 64; off <<= 1) {
                const int v = __shfl_up(incl, off);
                if (lane >= off) incl += v;
            }
            if (lane == 63) s_wave[wave] = incl;
            __syncthreads();
            __shared__ unsigned long long s_base;
            if (t == 0) {
                int tot = 0;
                for (int v = 0; v < kCountThreads / 64; ++v) tot += s_wave[v];
                s_base = tot ? atomicAdd(&rc->ncand, (unsigned long long)tot) : 0ull;
            }
            __syncthreads();
            int before = 0;
            for (int v = 0; v < wave; ++v) before += s_wave[v];
            unsigned long long slot = s_base + (unsigned long long)(before + incl - mine);
            for (int wd = w0 + t; wd < nw; wd += kCountThreads) {
                const uint32_t v = cnt[wd];
                if (!v) continue;
                cnt[wd] = 0;
                for (int h = 0; h < 2; ++h) {
                    if (!emits(v, wd, h)) continue;
                    if ((int64_t)slot < cap)
                        cand[slot] = cand_key((v >> (16 * h)) & 0xFFFFu, (uint32_t)x,
                                              (uint32_t)(y0 + 2 * wd + h));
                    else
                        st->error = 1;
                    ++slot;
                }
            }
            __syncthreads();
        }
    }
}

// ------------------------------------------------------------ Algorithm 2
// Workgroup barrier for LDS traffic only: waits for this wave's LDS
// operations but leaves its global loads and stores in flight (the key
// prefetch and the pair stores of the greedy scan), which __syncthreads
// would drain at every barrier.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// set bits of m in the lanes below this one
__device__ __forceinline__ int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Exclusive prefix (for this wavefront) and total of the greedy scan's 16
// per-wavefront counts, after the barrier that published them: one LDS
// read and a four-step scan across lanes 0-15 (one DPP row).
static_assert(kGreedyThreads == 1024, "the wavefront counts fill one 16-lane DPP row");
__device__ __forceinline__ void wave_prefix(const int32_t* wave_sum, int wave, int lane,
                                            int* before, int* total) {
    int v = lane < 16 ? wave_sum[lane] : 0;
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);   // row_shr:8
    *total = __builtin_amdgcn_readlane(v, 15);
    *before = wave ? __builtin_amdgcn_readlane(v, wave - 1) : 0;
}

// The greedy matching over keys sorted ascending, i.e. weight descending,
// then (x, y): a pair is taken when neither endpoint is used, while fewer
// than `budget` pairs were taken this round. Blocks of keys are first
// filtered in parallel against the used set; one wavefront then takes the
// survivors in order, 64 at a time. Taken pairs go to pairs[2 i],
// pairs[2 i + 1].

__global__ __launch_bounds__(kGreedyThreads) void greedy_kernel(
    const uint64_t* __restrict__ keys, int64_t nc, int n, int64_t max_aux, int64_t pairs_cap,
    int32_t* __restrict__ all_pairs, DevState* st, int round) {
    extern __shared__ uint32_t used[];   // (ncols + 31) / 32 words
    __shared__ uint64_t surv[2][kGreedyBlock];
    __shared__ int32_t wave_sum[kGreedyThreads / 64];
    __shared__ int stop;
    __shared__ long long s_taken, s_wsum;
    const int t = threadIdx.x, lane = t % 64, wave = t / 64;
    // this round's ids and budget follow from the pairs of earlier rounds
    const long long naux0 = st->naux;
    const int ncols = n + (int)naux0;
    const long long budget_left = max_aux < 0 ? LLONG_MAX : max_aux - naux0;
    const long long budget = min(budget_left, (long long)pairs_cap - naux0);
    int32_t* __restrict__ pairs = all_pairs + 2 * naux0;
    RoundCounters* rc = &st->round[round];
    for (int i = t; i < (ncols + 31) / 32; i += kGreedyThreads) used[i] = 0;
    if (t == 0) {
        stop = budget <= 0;
        s_taken = 0;
        s_wsum = 0;
    }
    lds_barrier();
    auto is_used = [&](uint32_t v) { return (used[v >> 5] >> (v & 31)) & 1u; };
    // both endpoints free (no short-circuit: no branch, both reads in flight)
    auto free_pair = [&](uint64_t key) {
        const uint32_t x = (uint32_t)(key >> 20) & 0xFFFFFu, y = (uint32_t)key & 0xFFFFFu;
        return (is_used(x) | is_used(y)) == 0u;
    };
    // Keys of the next block are loaded while this one is filtered and
    // taken. Loads are unconditional (clamped index, so every key read is a
    // real one with ids below ncols); a slot past nc is dropped by its
    // index only, so nothing waits for a load before its block is used.
    auto load_raw = [&](int64_t i) { return keys[i < nc ? i : nc - 1]; };
    uint64_t k_raw[kGreedyPer];
#pragma unroll
    for (int j = 0; j < kGreedyPer; ++j) k_raw[j] = load_raw((int64_t)t * kGreedyPer + j);
    for (int64_t base = 0; base < nc && !stop; base += kGreedyBlock) {
        uint64_t k[kGreedyPer];
        bool live[kGreedyPer];
#pragma unroll
        for (int j = 0; j < kGreedyPer; ++j) {
            const int64_t i = base + (int64_t)t * kGreedyPer + j;
            k[j] = k_raw[j];
            live[j] = i < nc;
            k_raw[j] = load_raw(i + kGreedyBlock);
        }
#pragma unroll
        for (int j = 0; j < kGreedyPer; ++j) live[j] = live[j] & free_pair(k[j]);
        // survivors keep their order (thread-major, then j): the prefix
        // inside a wave from one ballot per key slot, across waves from the
        // per-wave totals
        int excl = 0, wtot = 0;
#pragma unroll
        for (int j = 0; j < kGreedyPer; ++j) {
            const uint64_t mj = __ballot(live[j]);
            excl += lanes_below(mj);
            wtot += __popcll(mj);
        }
        if (lane == 0) wave_sum[wave] = wtot;
        lds_barrier();
        int before, nsurv;
        wave_prefix(wave_sum, wave, lane, &before, &nsurv);
        int wpos = before + excl;
#pragma unroll
        for (int j = 0; j < kGreedyPer; ++j)
            if (live[j]) surv[0][wpos++] = k[j];
        lds_barrier();
        int buf = 0, pos = 0, cnt = nsurv;
        while (pos < cnt) {
            const uint64_t* S = surv[buf];
            const int end = min(cnt, pos + kGreedyBurst);
            if (wave == 0) {
                long long taken = s_taken, wsum = s_wsum;
                bool halt = false;
                for (int c0 = pos; c0 < end && !halt; c0 += 64) {
                    const int si = c0 + lane;
                    const uint64_t kv = S[si < end ? si : end - 1];
                    const uint32_t x = (uint32_t)(kv >> 20) & 0xFFFFFu, y = (uint32_t)kv & 0xFFFFFu;
                    const uint32_t w = 0xFFFFu - (uint32_t)(kv >> 40);
                    // live lanes as one wave-uniform mask: the first is
                    // taken and every lane sharing an endpoint with it
                    // leaves the mask (one compare per lane and a ballot
                    // per pair; the used set and the output follow after
                    // the chunk)
                    uint64_t m = __builtin_amdgcn_ballot_w64((si < end) & free_pair(kv));
                    uint64_t tm = 0;
                    const long long room = budget - taken;
                    long long got = 0;
                    while (m) {
                        if (got >= room) {
                            halt = true;
                            break;
                        }
                        const int j = (int)__builtin_ctzll(m);
                        const uint32_t xj = __builtin_amdgcn_readlane(x, j);
                        const uint32_t yj = __builtin_amdgcn_readlane(y, j);
                        wsum += __builtin_amdgcn_readlane(w, j);
                        tm |= 1ull << j;
                        ++got;
                        m &= ~(__builtin_amdgcn_ballot_w64(x == xj) |
                               __builtin_amdgcn_ballot_w64(x == yj) |
                               __builtin_amdgcn_ballot_w64(y == xj) |
                               __builtin_amdgcn_ballot_w64(y == yj));
                    }
                    const long long first = taken;
                    taken += got;
                    if ((tm >> lane) & 1ull) {
                        const long long r = first + lanes_below(tm);
                        atomicOr(&used[x >> 5], 1u << (x & 31));
                        atomicOr(&used[y >> 5], 1u << (y & 31));
                        pairs[2 * r] = (int32_t)x;
                        pairs[2 * r + 1] = (int32_t)y;
                    }
                }
                if (lane == 0) {
                    s_taken = taken;
                    s_wsum = wsum;
                    if (halt || taken >= budget) stop = 1;
                }
            }
            lds_barrier();
            if (stop) break;
            pos = end;
            if (cnt - pos > kGreedyBurst) {
                // order-preserving filter of S[pos, cnt) into the other buffer
                const int rem = cnt - pos;
                const int per = (rem + kGreedyThreads - 1) / kGreedyThreads;
                uint64_t kk[kGreedyPer];
                bool lv[kGreedyPer];
                int a = 0;
#pragma unroll
                for (int j = 0; j < kGreedyPer; ++j) {
                    const int i = pos + t * per + j;
                    lv[j] = false;
                    kk[j] = 0;
                    if (j < per && i < cnt) {
                        kk[j] = S[i];
                        lv[j] = free_pair(kk[j]);
                    }
                    a += lv[j];
                }
                int inc = a;
                for (int off = 1; off < 64; off <<= 1) {
                    const int v = __shfl_up(inc, off);
                    if (lane >= off) inc += v;
                }
                if (lane == 63) wave_sum[wave] = inc;
                lds_barrier();
                int before, total;
                wave_prefix(wave_sum, wave, lane, &before, &total);
                int o = before + inc - a;
                uint64_t* D = surv[buf ^ 1];
#pragma unroll
                for (int j = 0; j < kGreedyPer; ++j)
                    if (lv[j]) D[o++] = kk[j];
                lds_barrier();
                buf ^= 1;
                pos = 0;
                cnt = total;
            }
        }
        lds_barrier();
        if (stop) break;
    }
    if (t == 0) {
        rc->taken = s_taken;
        rc->wsum = s_wsum;
        st->naux = naux0 + s_taken;
        // no pair taken, or the budget spent: the later rounds do nothing
        st->done = s_taken == 0 || s_taken >= budget_left;
    }
}

// ------------------------------------------------------------ Algorithm 3
// The pairs of round `round` (the last `taken` of all pairs so far) mark
// their ids with the partner and the pair's new id, after the previous
// round's marks are cleared (its ids may pair again). One workgroup, so the
// barrier orders the clears before the marks; nothing reads the marks
// between one round's rewrite and the next round's marking, and a call
// starts from cleared arrays.
__global__ __launch_bounds__(kScanThreads) void set_partner_kernel(
    const int32_t* __restrict__ all_pairs, int n, const DevState* st, int round,
    int32_t* __restrict__ partner, int32_t* __restrict__ newid) {
    const long long taken = st->round[round].taken, naux0 = st->naux - taken;
    if (round > 0) {
        const long long prev = st->round[round - 1].taken;
        const int32_t* pp = all_pairs + 2 * (naux0 - prev);
        for (long long i = threadIdx.x; i < prev; i += kScanThreads) {
            const int32_t x = pp[2 * i], y = pp[2 * i + 1];
            partner[x] = partner[y] = -1;
            newid[x] = newid[y] = -1;
        }
        __syncthreads();
    }
    const int32_t* pairs = all_pairs + 2 * naux0;
    for (long long i = threadIdx.x; i < taken; i += kScanThreads) {
        const int32_t x = pairs[2 * i], y = pairs[2 * i + 1];
        partner[x] = y;
        partner[y] = x;
        newid[x] = newid[y] = n + (int32_t)(naux0 + i);
    }
}

// One workgroup per list; the list's ids are marked in an LDS bitmap
// (ncols bits, cleared first: LDS starts with whatever the previous
// workgroup left) so that "is my partner in this list" is one LDS read.
constexpr int kRowThreads = 256;
constexpr int kRowIds = 4096;   // new ids of one list ranked in LDS (beyond: scratch)

__device__ __forceinline__ void mark_row(uint32_t* bits, int nwords,
                                         const int32_t* __restrict__ row, int d) {
    for (int i = threadIdx.x; i < nwords; i += kRowThreads) bits[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < d; i += kRowThreads) {
        const int32_t c = row[i];
        atomicOr(&bits[c >> 5], 1u << (c & 31));
    }
}

__device__ __forceinline__ bool has(const uint32_t* bits, int32_t v) {
    return (bits[v >> 5] >> (v & 31)) & 1u;
}

// block-wide exclusive prefix of a 0/1 flag (order = thread order); returns
// the prefix and writes the block total
__device__ __forceinline__ int block_prefix(bool f, int32_t* s_wave, int* total) {
    const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
    const uint64_t m = __ballot(f);
    if (lane == 0) s_wave[wave] = __popcll(m);
    __syncthreads();
    int before = 0, all = 0;
    for (int w = 0; w < kRowThreads / 64; ++w) {
        const int v = s_wave[w];
        if (w < wave) before += v;
        all += v;
    }
    __syncthreads();
    *total = all;
    return before + __popcll(m & ((1ull << lane) - 1));
}

// new length of every list
__global__ __launch_bounds__(kRowThreads) void rewrite_count_kernel(
    int n, const DevState* st, int round, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ col, const int32_t* __restrict__ partner,
    int32_t* __restrict__ rowlen) {
    extern __shared__ uint32_t bits[];
    __shared__ int32_t s_wave[kRowThreads / 64];
    const int ncols = n + (int)(st->naux - st->round[round].taken);   // ids before the round
    const int w = blockIdx.x;
    const int b = rowptr[w], d = rowptr[w + 1] - b;
    const int32_t* row = col + b;
    mark_row(bits, (ncols + 31) / 32, row, d);
    __syncthreads();
    int pairs_here = 0;
    for (int i = threadIdx.x; i < d; i += kRowThreads) {
        const int32_t c = row[i], p = partner[c];
        if (p >= 0 && c < p && has(bits, p)) ++pairs_here;
    }
    for (int off = 32; off > 0; off >>= 1) pairs_here += __shfl_xor(pairs_here, off);
    if (threadIdx.x % 64 == 0) s_wave[threadIdx.x / 64] = pairs_here;
    __syncthreads();
    if (threadIdx.x == 0) {
        int tot = 0;
        for (int v = 0; v < kRowThreads / 64; ++v) tot += s_wave[v];
        rowlen[w] = d - tot;
    }
}

// kept entries in order, then the new ids in increasing order (each placed
// by its rank among the list's new ids)
__global__ __launch_bounds__(kRowThreads) void rewrite_fill_kernel(
    int n, const DevState* st, int round, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ col, const int32_t* __restrict__ partner,
    const int32_t* __restrict__ newid, const int32_t* __restrict__ rowptr_new,
    int32_t* __restrict__ col_new, int32_t* __restrict__ scratch) {
    extern __shared__ uint32_t bits[];
    __shared__ int32_t s_wave[kRowThreads / 64];
    __shared__ int32_t ids[kRowIds];
    const int ncols = n + (int)(st->naux - st->round[round].taken);   // ids before the round
    const int w = blockIdx.x;
    const int b = rowptr[w], d = rowptr[w + 1] - b;
    const int out = rowptr_new[w], len = rowptr_new[w + 1] - out;
    const int nadd = d - len, kept_total = len - nadd;
    const int32_t* row = col + b;
    // new ids wait in LDS, or in the list's own stretch of scratch when many
    int32_t* idbuf = nadd <= kRowIds ? ids : scratch + out + kept_total;
    mark_row(bits, (ncols + 31) / 32, row, d);
    __syncthreads();
    int kept = 0, added = 0;
    for (int i0 = 0; i0 < d; i0 += kRowThreads) {
        const int i = i0 + threadIdx.x;
        int32_t c = -1, p = -1;
        if (i < d) {
            c = row[i];
            p = partner[c];
        }
        const bool pair_in = p >= 0 && has(bits, p);
        const bool keep = i < d && !pair_in;
        const bool add = pair_in && c < p;
        int nk, na;
        const int pk = block_prefix(keep, s_wave, &nk);
        const int pa = block_prefix(add, s_wave, &na);
        if (keep) col_new[out + kept + pk] = c;
        if (add) idbuf[added + pa] = newid[c];
        kept += nk;
        added += na;
    }
    __syncthreads();   // (also orders the scratch writes before the reads below)
    for (int j = threadIdx.x; j < nadd; j += kRowThreads) {
        const int32_t id = idbuf[j];
        int rank = 0;
        for (int i = 0; i < nadd; ++i) rank += idbuf[i] < id;
        col_new[out + kept_total + rank] = id;
    }
}

}  // namespace

// Algorithm 3's rewrite with one wavefront per list, for rounds whose ids
// and new ids fit a wavefront's share of LDS: the list's ids go to the
// wave's own bitmap and the pairs it keeps to a bitmap of the round's new
// ids, so prefixes come from ballots and the new ids are written in
// increasing order by scanning that bitmap, with no workgroup barrier. A
// wavefront's LDS operations run in program order, so its clears, marks
// and reads need no wait between them.
constexpr int kListsPerGroup = kRowThreads / 64;
constexpr int kWaveMaxIds = 32768;    // ids before the round (1,024 bitmap words)
constexpr int kWaveMaxNew = 8192;     // pairs the round may take (256 words)

__global__ __launch_bounds__(kRowThreads) void rewrite_fill_wave_kernel(
    int n, const DevState* st, int round, const int32_t* __restrict__ rowptr,
    const int32_t* __restrict__ col, const int32_t* __restrict__ partner,
    const int32_t* __restrict__ newid, const int32_t* __restrict__ rowptr_new,
    int32_t* __restrict__ col_new, int wstride, int wids) {
    extern __shared__ uint32_t wbits[];
    const int lane = threadIdx.x % 64;
    const int w = blockIdx.x * kListsPerGroup + threadIdx.x / 64;
    if (w >= n) return;   // the whole wavefront
    uint32_t* bits = wbits + (threadIdx.x / 64) * wstride;
    uint32_t* nbits = bits + wids;   // the round's new ids, from ncols on
    const long long taken = st->round[round].taken;
    const int ncols = n + (int)(st->naux - taken);   // ids before the round = first new id
    const int nnew = (int)((taken + 31) / 32);
    const int b = rowptr[w], d = rowptr[w + 1] - b;
    const int out = rowptr_new[w], len = rowptr_new[w + 1] - out;
    const int kept_total = len - (d - len);
    const int32_t* row = col + b;
    for (int i = lane; i < (ncols + 31) / 32; i += 64) bits[i] = 0;
    for (int i = lane; i < nnew; i += 64) nbits[i] = 0;
    for (int i = lane; i < d; i += 64) {
        const int32_t c = row[i];
        atomicOr(&bits[c >> 5], 1u << (c & 31));
    }
    int kept = 0;
    for (int i0 = 0; i0 < d; i0 += 64) {
        const int i = i0 + lane;
        int32_t c = -1, p = -1;
        if (i < d) {
            c = row[i];
            p = partner[c];
        }
        const bool pair_in = p >= 0 && has(bits, p);
        const bool keep = i < d && !pair_in;
        const uint64_t mk = __ballot(keep);
        if (keep) col_new[out + kept + lanes_below(mk)] = c;
        kept += __popcll(mk);
        if (pair_in && c < p) {
            const int q = newid[c] - ncols;
            atomicOr(&nbits[q >> 5], 1u << (q & 31));
        }
    }
    // the new ids after the kept entries, in increasing order
    int added = 0;
    for (int j0 = 0; j0 < nnew; j0 += 64) {
        const int j = j0 + lane;
        uint32_t word = j < nnew ? nbits[j] : 0u;
        const int cnt = __popc(word);
        int incl = cnt;
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(incl, off);
            if (lane >= off) incl += y;
        }
        int pos = out + kept_total + added + incl - cnt;
        while (word) {
            const int bit = __ffs(word) - 1;
            col_new[pos++] = ncols + 32 * j + bit;
            word &= word - 1;
        }
        added += __shfl(incl, 63);
    }
}

// ------------------------------------------------------------ host driver

namespace {

struct DevPlan {
    int64_t n, nnz, pairs_cap, ncols_cap, cand_cap;
    size_t sort_tmp;
    // byte offsets in the workspace
    size_t rowptr[2], col[2], rowlen, scratch, tptr, tcur, tnext, tend, partner, newid,
        keys_in, keys_out, pairs, counters, sort, total;
};

int64_t visits_of(const int32_t* rowptr, int64_t n) {
    int64_t s = 0;
    for (int64_t w = 0; w < n; ++w) {
        const int64_t d = rowptr[w + 1] - rowptr[w];
        s += d * (d - 1) / 2;
    }
    return s;
}

int plan(const int32_t* rowptr, int64_t n, const gcn_rr_params* p, DevPlan* dp) {
    std::memset(dp, 0, sizeof(*dp));
    dp->n = n;
    dp->nnz = rowptr[n];
    dp->pairs_cap = dp->nnz / 2;   // every pair removes >= 2 list entries
    if (p->max_aux >= 0) dp->pairs_cap = std::min<int64_t>(dp->pairs_cap, p->max_aux);
    dp->ncols_cap = n + dp->pairs_cap;
    // every candidate has weight >= max(theta + 1, 2), and the pair visits
    // (sum of C(d, 2) over the lists) never grow from round to round
    dp->cand_cap = std::max<int64_t>(1, visits_of(rowptr, n) / std::max(p->theta + 1, 2));
    // the sort's scratch: the most either of its algorithms needs (merge
    // sort up to kMergeSortMax keys, onesweep above)
    const int64_t sizes[2] = {std::min<int64_t>(dp->cand_cap, UINT32_MAX),
                              std::min<int64_t>(dp->cand_cap, (int64_t)kMergeSortMax)};
    dp->sort_tmp = 0;
    for (const int64_t sz : sizes) {
        size_t tmp = 0;
        if (rocprim::radix_sort_keys<SortConfig>(nullptr, tmp, (uint64_t*)nullptr,
                                                 (uint64_t*)nullptr, (unsigned)sz, 0, 56,
                                                 (hipStream_t)0) != hipSuccess)
            return GCN_E_HIP;
        dp->sort_tmp = std::max(dp->sort_tmp, tmp);
    }
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = (off + std::max<size_t>(bytes, 4) + 255) / 256 * 256;
        return o;
    };
    for (int i = 0; i < 2; ++i) {
        dp->rowptr[i] = take(4 * (size_t)(n + 1));
        dp->col[i] = take(4 * (size_t)dp->nnz);
    }
    dp->rowlen = take(4 * (size_t)n);
    dp->scratch = take(4 * (size_t)dp->nnz);
    dp->tptr = take(4 * (size_t)(dp->ncols_cap + 1));
    dp->tcur = take(4 * (size_t)dp->ncols_cap);
    dp->tnext = take(4 * (size_t)dp->nnz);
    dp->tend = take(4 * (size_t)dp->nnz);
    dp->partner = take(4 * (size_t)dp->ncols_cap);
    dp->newid = take(4 * (size_t)dp->ncols_cap);
    dp->keys_in = take(8 * (size_t)dp->cand_cap);
    dp->keys_out = take(8 * (size_t)dp->cand_cap);
    dp->pairs = take(8 * (size_t)std::max<int64_t>(dp->pairs_cap, 1));
    dp->counters = take(sizeof(DevState));
    dp->sort = take(dp->sort_tmp);
    dp->total = off;
    return GCN_OK;
}

dim3 waves_grid(int64_t rows) { return dim3((unsigned)((rows + kBlock / 64 - 1) / (kBlock / 64))); }
dim3 items_grid(int64_t items) { return dim3((unsigned)std::max<int64_t>(1, (items + kBlock - 1) / kBlock)); }

}  // namespace

int redundancy_reduce_device_bytes(const int32_t* rowptr, int64_t n, const gcn_rr_params* p,
                                   size_t* bytes) {
    DevPlan dp;
    int rc = plan(rowptr, n, p, &dp);
    if (rc) return rc;
    *bytes = dp.total;
    return GCN_OK;
}

int redundancy_reduce_device(const int32_t* rowptr_h, const int32_t* col_h, int64_t n,
                             const gcn_rr_params* p, void* ws, size_t ws_bytes,
                             hipStream_t s, DeviceReduceResult* out) {
    DevPlan dp;
    int rc = plan(rowptr_h, n, p, &dp);
    if (rc) {
        set_error("gcn_redundancy_reduce_device: rocPRIM sort planning failed");
        return rc;
    }
    if (ws_bytes < dp.total) {
        set_error("gcn_redundancy_reduce_device: workspace of %zu bytes, need %zu", ws_bytes,
                  dp.total);
        return GCN_E_WORKSPACE;
    }
    if (n >= kMaxIds) {
        set_error("gcn_redundancy_reduce_device: %lld vertices; the device reduction "
                  "handles fewer than %d",
                  (long long)n, kMaxIds);
        return GCN_E_UNSUPPORTED;
    }
    char* base = static_cast<char*>(ws);
    auto I = [&](size_t off) { return reinterpret_cast<int32_t*>(base + off); };
    int32_t* rowptr[2] = {I(dp.rowptr[0]), I(dp.rowptr[1])};
    int32_t* col[2] = {I(dp.col[0]), I(dp.col[1])};
    uint64_t* keys_in = reinterpret_cast<uint64_t*>(base + dp.keys_in);
    uint64_t* keys_out = reinterpret_cast<uint64_t*>(base + dp.keys_out);
    int32_t* pairs = I(dp.pairs);
    DevState* dst = reinterpret_cast<DevState*>(base + dp.counters);
    auto fail = [&](hipError_t e, const char* what) {
        set_error("gcn_redundancy_reduce_device: %s: HIP error %d (%s)", what, (int)e,
                  hipGetErrorString(e));
        return GCN_E_HIP;
    };
#define GCN_DR(call, what)                         \
    do {                                           \
        hipError_t e_ = (call);                    \
        if (e_ != hipSuccess) return fail(e_, what); \
    } while (0)

    const int64_t nnz = dp.nnz;
    out->round_offsets.assign(1, 0);
    out->stats.clear();
    if (n == 0 || nnz == 0 || p->max_rounds == 0 || p->max_aux == 0) {   // no pairs: the lists as given
        out->naux = 0;
        out->rowptr.assign(rowptr_h, rowptr_h + n + 1);
        out->col.assign(col_h, col_h + nnz);
        out->pairs.clear();
        return GCN_OK;
    }
    GCN_DR(hipMemcpyAsync(rowptr[0], rowptr_h, 4 * (size_t)(n + 1), hipMemcpyHostToDevice, s),
           "upload");
    GCN_DR(hipMemcpyAsync(col[0], col_h, 4 * (size_t)nnz, hipMemcpyHostToDevice, s), "upload");
    GCN_DR(hipMemsetAsync(dst, 0, sizeof(DevState), s), "state");
    init_kernel<<<items_grid(dp.ncols_cap), kBlock, 0, s>>>(I(dp.partner), I(dp.newid),
                                                             I(dp.tcur), dp.ncols_cap);
    GCN_DR(hipGetLastError(), "init");

    // The host knows the ids exactly at each round's wait (after the pair
    // counting); the round after may add at most its budget of new ids.
    int64_t naux_known = 0;
    int64_t ncols_ub = n;   // bound on the ids the next round sees
    int cur = 0, rounds = 0;
    DevState hs;
    for (int round = 0; round < p->max_rounds; ++round) {
        const int32_t nc_ub = (int32_t)std::min<int64_t>(ncols_ub, dp.ncols_cap);
        // Algorithm 1: transposed index, then pair counts per id
        const bool trans_lds = nc_ub <= kTransMaxIds;
        const dim3 trans_grid((unsigned)((n + kTransLists - 1) / kTransLists));
        if (trans_lds && 4 * (size_t)nc_ub > 48 * 1024) {
            GCN_DR(hipFuncSetAttribute((const void*)tcount_lds_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       4 * kTransMaxIds),
                   "transposed index LDS");
            GCN_DR(hipFuncSetAttribute((const void*)tfill_lds_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       4 * kTransMaxIds),
                   "transposed index LDS");
        }
        if (trans_lds)
            tcount_lds_kernel<<<trans_grid, kBlock, 4 * (size_t)nc_ub, s>>>(
                (int)n, nc_ub, rowptr[cur], col[cur], I(dp.tcur), dst);
        else
            tcount_kernel<<<waves_grid(n), kBlock, 0, s>>>((int)n, rowptr[cur], col[cur],
                                                            I(dp.tcur), dst);
        // tptr from the counts; the counts become the fill cursors
        scan_kernel<<<1, kScanThreads, 0, s>>>(I(dp.tcur), I(dp.tptr), nc_ub, I(dp.tcur), nullptr,
                                               nullptr);
        if (trans_lds)
            tfill_lds_kernel<<<trans_grid, kBlock, 4 * (size_t)nc_ub, s>>>(
                (int)n, nc_ub, rowptr[cur], col[cur], I(dp.tcur), I(dp.tnext), I(dp.tend), dst);
        else
            tfill_kernel<<<waves_grid(n), kBlock, 0, s>>>((int)n, rowptr[cur], col[cur],
                                                           I(dp.tcur), I(dp.tnext), I(dp.tend),
                                                           dst);
        const size_t lds = 4 * (size_t)((std::min<int64_t>(nc_ub, kCountWindow) + 1) / 2);
        if (lds > 48 * 1024)
            GCN_DR(hipFuncSetAttribute((const void*)count_pairs_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds),
                   "pair counting LDS");
        const unsigned grid = (unsigned)std::min<int64_t>(nc_ub, 4096);
        count_pairs_kernel<<<grid, kCountThreads, lds, s>>>((int)n, p->theta, col[cur],
                                                            I(dp.tptr), I(dp.tnext),
                                                            I(dp.tend), I(dp.tcur), keys_in,
                                                            dp.cand_cap,
                                                            dst, round);
        GCN_DR(hipGetLastError(), "pair counting");
        // the one wait of the round: the sort needs the candidate count
        GCN_DR(hipMemcpyAsync(&hs, dst, sizeof(hs), hipMemcpyDeviceToHost, s), "state");
        GCN_DR(hipStreamSynchronize(s), "pair counting");
        if (hs.error) {
            set_error("gcn_redundancy_reduce_device: %s in round %d",
                      hs.error == 1   ? "candidate capacity exceeded"
                      : hs.error == 2 ? "list id out of range"
                                      : "ids reach the device reduction's range (2^19) or a "
                                        "pair count exceeds 16 bits",
                      round + 1);
            return hs.error == 3 ? GCN_E_UNSUPPORTED : GCN_E_INTERNAL;
        }
        if (hs.done) break;   // the previous round ended the reduction
        naux_known = hs.naux;
        const int64_t nc = (int64_t)hs.round[round].ncand;
        if (nc == 0) break;
        // Algorithm 2: sort by (weight descending, x, y), then the greedy scan
        size_t tmp = dp.sort_tmp;
        GCN_DR(rocprim::radix_sort_keys<SortConfig>(base + dp.sort, tmp, keys_in, keys_out,
                                                    (unsigned)nc, 0, 56, s),
               "candidate sort");
        // the used set: one bit per id issued so far
        const size_t used = 4 * (size_t)((n + naux_known + 31) / 32);
        if (used > 48 * 1024)
            GCN_DR(hipFuncSetAttribute((const void*)greedy_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)used),
                   "matching LDS");
        greedy_kernel<<<1, kGreedyThreads, used, s>>>(keys_out, nc, (int)n, p->max_aux,
                                                      dp.pairs_cap, pairs, dst, round);
        GCN_DR(hipGetLastError(), "matching");
        // Algorithm 3: rewrite every list (a round that took no pair
        // copies the lists unchanged)
        // pairs this round can take: within the budget and the capacity,
        // and a matching over the ids so far has at most half as many
        const int64_t budget_ub =
            std::min<int64_t>({p->max_aux < 0 ? INT64_MAX : p->max_aux - naux_known,
                               dp.pairs_cap - naux_known, (n + naux_known) / 2});
        const int nxt = cur ^ 1;
        const size_t bits = 4 * (size_t)((std::min<int64_t>(n + naux_known, kMaxIds) + 31) / 32);
        if (bits > 48 * 1024) {
            GCN_DR(hipFuncSetAttribute((const void*)rewrite_count_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bits),
                   "rewrite LDS");
            GCN_DR(hipFuncSetAttribute((const void*)rewrite_fill_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bits),
                   "rewrite LDS");
        }
        set_partner_kernel<<<1, kScanThreads, 0, s>>>(pairs, (int)n, dst, round, I(dp.partner),
                                                      I(dp.newid));
        // the rewrite: one wavefront per list where its bitmaps fit, else one
        // workgroup (the new lengths: one workgroup per list, which measured
        // faster than a wavefront per list)
        const bool wave_rows = n + naux_known <= kWaveMaxIds && budget_ub <= kWaveMaxNew;
        const int wids = (int)((n + naux_known + 31) / 32);
        const int wstride = wids + (int)((std::max<int64_t>(budget_ub, 0) + 31) / 32);
        const dim3 wave_grid((unsigned)((n + kListsPerGroup - 1) / kListsPerGroup));
        const size_t wave_lds = 4 * (size_t)kListsPerGroup * wstride;
        rewrite_count_kernel<<<(unsigned)n, kRowThreads, bits, s>>>(
            (int)n, dst, round, rowptr[cur], col[cur], I(dp.partner), I(dp.rowlen));
        scan_kernel<<<1, kScanThreads, 0, s>>>(I(dp.rowlen), rowptr[nxt], (int)n, nullptr,
                                               &dst->round[round].num_add,
                                               &dst->round[round].nnz);
        if (wave_rows)
            rewrite_fill_wave_kernel<<<wave_grid, kRowThreads, wave_lds, s>>>(
                (int)n, dst, round, rowptr[cur], col[cur], I(dp.partner), I(dp.newid),
                rowptr[nxt], col[nxt], wstride, wids);
        else
            rewrite_fill_kernel<<<(unsigned)n, kRowThreads, bits, s>>>(
                (int)n, dst, round, rowptr[cur], col[cur], I(dp.partner), I(dp.newid),
                rowptr[nxt], col[nxt], I(dp.scratch));
        GCN_DR(hipGetLastError(), "rewrite");
        cur = nxt;
        rounds = round + 1;
        ncols_ub = n + naux_known + budget_ub;
    }
    // the rounds' results (a round that took nothing ends the list)
    GCN_DR(hipMemcpyAsync(&hs, dst, sizeof(hs), hipMemcpyDeviceToHost, s), "state");
    GCN_DR(hipStreamSynchronize(s), "rounds");
    int64_t naux = 0, cur_nnz = nnz;
    for (int r = 0; r < rounds; ++r) {
        const RoundCounters& rc = hs.round[r];
        if (rc.taken == 0) break;
        naux += rc.taken;
        cur_nnz = rc.nnz;
        out->round_offsets.push_back((int32_t)naux);
        out->stats.push_back({rc.taken, rc.wsum, rc.nnz, (int64_t)rc.num_add});
    }
    if (naux != hs.naux) {
        set_error("gcn_redundancy_reduce_device: pair count mismatch (%lld vs %lld)",
                  (long long)naux, (long long)hs.naux);
        return GCN_E_INTERNAL;
    }
    out->naux = (int32_t)naux;
    out->rowptr.resize(n + 1);
    out->col.resize(cur_nnz);
    out->pairs.resize(2 * naux);
    GCN_DR(hipMemcpyAsync(out->rowptr.data(), rowptr[cur], 4 * (size_t)(n + 1),
                          hipMemcpyDeviceToHost, s),
           "download");
    if (cur_nnz)
        GCN_DR(hipMemcpyAsync(out->col.data(), col[cur], 4 * (size_t)cur_nnz, hipMemcpyDeviceToHost, s),
               "download");
    if (naux)
        GCN_DR(hipMemcpyAsync(out->pairs.data(), pairs, 8 * (size_t)naux, hipMemcpyDeviceToHost, s),
               "download");
    GCN_DR(hipStreamSynchronize(s), "download");
#undef GCN_DR
    return GCN_OK;
}

}  // namespace gcn

// ------------------------------------------------------------ C ABI
using gcn::set_error;

extern "C" {

int gcn_redundancy_reduce_device_bytes(gcn_graph_t g, const gcn_rr_params* params,
                                       size_t* bytes) {
    GCN_CHECK_ARG(g && params && bytes, "gcn_redundancy_reduce_device_bytes: NULL argument");
    GCN_CHECK_ARG(params->theta >= 0, "gcn_redundancy_reduce_device_bytes: theta < 0");
    const int rc = gcn::redundancy_reduce_device_bytes(g->rowptr.data(), g->n, params, bytes);
    if (rc) set_error("gcn_redundancy_reduce_device_bytes: sort planning failed");
    return rc;
}

int gcn_redundancy_reduce_device(gcn_graph_t g, const gcn_rr_params* params, void* ws,
                                 size_t ws_bytes, gcn_stream_t stream, gcn_reduced_t* out) {
    GCN_CHECK_ARG(g && params && out, "gcn_redundancy_reduce_device: NULL argument");
    GCN_CHECK_ARG(params->theta >= 0, "gcn_redundancy_reduce_device: theta < 0");
    GCN_CHECK_ARG(params->max_rounds >= 0 && params->max_rounds <= GCN_MAX_ROUNDS,
                  "gcn_redundancy_reduce_device: max_rounds %d outside [0, %d]",
                  params->max_rounds, GCN_MAX_ROUNDS);
    GCN_CHECK_ARG(ws != nullptr && ((uintptr_t)ws % 256) == 0,
                  "gcn_redundancy_reduce_device: workspace NULL or not 256-byte aligned");
    try {
        gcn::DeviceReduceResult res;
        const int rc = gcn::redundancy_reduce_device(g->rowptr.data(), g->col.data(), g->n,
                                                     params, ws, ws_bytes,
                                                     (hipStream_t)stream, &res);
        if (rc) return rc;
        auto* r = new gcn_reduced;
        r->n = g->n;
        r->naux = res.naux;
        r->rounds = (int32_t)res.stats.size();
        r->rowptr = std::move(res.rowptr);
        r->col = std::move(res.col);
        r->pairs = std::move(res.pairs);
        r->round_offsets = std::move(res.round_offsets);
        r->stats = std::move(res.stats);
        r->deg.resize(g->n);
        for (int32_t v = 0; v < g->n; ++v) r->deg[v] = g->rowptr[v + 1] - g->rowptr[v];
        *out = r;
        gcn::clear_error();
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_redundancy_reduce_device: out of host memory");
        return GCN_E_OOM;
    }
}

}  // extern "C"
