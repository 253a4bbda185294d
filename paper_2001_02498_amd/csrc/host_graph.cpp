// Host-side graph preprocessing: subgraph construction (Section 2.1,
// Section 3.1) and the redundancy reduction of Section 3.2 (Algorithms 1-3
// applied in rounds), plus packing of the device image. CPU only: nothing
// here calls the HIP runtime, so it also builds and runs without a GPU.
#include <algorithm>
#include <array>
#include <atomic>
#include <cstring>
#include <exception>
#include <emmintrin.h>
#include <new>
#include <numeric>
#include <thread>
#include <vector>

#include "common.h"
#include "graph_types.h"

namespace gcn {

static thread_local std::string g_err;

void set_error(const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
}

void clear_error() { g_err.clear(); }

}  // namespace gcn

using gcn::set_error;


namespace {

// Runs body(t) on `threads` threads (inline when threads == 1).
template <class F>
void parallel_run(int threads, F&& body) {
    if (threads <= 1) {
        body(0);
        return;
    }
    std::vector<std::thread> pool;
    pool.reserve(threads);
    for (int t = 0; t < threads; ++t) pool.emplace_back([&, t] { body(t); });
    for (auto& th : pool) th.join();
}

int pick_threads(int requested, int64_t work) {
    int hw = (int)std::thread::hardware_concurrency();
    if (hw <= 0) hw = 1;
    int t = requested > 0 ? requested : hw;
    t = std::min(t, 64);
    // small problems are not worth the thread start-up
    int64_t cap = std::max<int64_t>(1, work / 200000);
    return (int)std::max<int64_t>(1, std::min<int64_t>(t, cap));
}

// Bit i set when blk[i] > floor, for i < len <= 64.
inline uint64_t above(const int32_t* blk, int32_t len, int32_t floor) {
    uint64_t bits = 0;
    for (int32_t i = 0; i < len; ++i) bits |= (uint64_t)(blk[i] > floor) << i;
    return bits;
}

// 16-bit counters: eight per SSE2 compare (blk[i] - floor saturates at zero
// exactly when blk[i] <= floor); a whole block of 64 is eight compares.
inline uint64_t above(const uint16_t* blk, int32_t len, uint16_t floor) {
    if (len < 64) {
        uint64_t bits = 0;
        for (int32_t i = 0; i < len; ++i) bits |= (uint64_t)(blk[i] > floor) << i;
        return bits;
    }
    const __m128i f = _mm_set1_epi16((short)floor);
    const __m128i zero = _mm_setzero_si128();
    uint64_t le_bits = 0;   // bit i: blk[i] <= floor
    for (int q = 0; q < 4; ++q) {
        const __m128i a = _mm_loadu_si128(reinterpret_cast<const __m128i*>(blk + 16 * q));
        const __m128i b = _mm_loadu_si128(reinterpret_cast<const __m128i*>(blk + 16 * q + 8));
        // all-ones lanes where the count does not exceed floor, packed to
        // one byte per lane (saturation keeps -1 and 0), one bit per byte
        const __m128i le = _mm_packs_epi16(_mm_cmpeq_epi16(_mm_subs_epu16(a, f), zero),
                                           _mm_cmpeq_epi16(_mm_subs_epu16(b, f), zero));
        le_bits |= (uint64_t)(uint32_t)_mm_movemask_epi8(le) << (16 * q);
    }
    return ~le_bits;
}

struct Candidate {
    int32_t w;   // lists holding both (at most the number of lists)
    int32_t x, y;
};

// Lists of the aggregators in CSR form; ids in [0, ncols).
struct Lists {
    int32_t n = 0, ncols = 0;
    std::vector<int64_t> ptr;
    std::vector<int32_t> col;
};

// Algorithm 1, keeping only pairs whose count exceeds theta: for each x,
// walk the lists that hold x and count every larger id y that follows x in
// the same (sorted) list; the count of {x, y} is the number of lists holding
// both. A dense counter per thread plays the hash table.
template <class Count>
std::vector<Candidate> count_pairs_t(const Lists& L, int theta, int threads) {
    const int32_t ncols = L.ncols;
    // transposed index: for each id, the (list, position) pairs holding it
    std::vector<int64_t> tptr(ncols + 1, 0);
    for (int64_t e = 0; e < L.ptr[L.n]; ++e) tptr[L.col[e] + 1]++;
    for (int32_t c = 0; c < ncols; ++c) tptr[c + 1] += tptr[c];
    std::vector<int32_t> tlist(L.ptr[L.n]), tpos(L.ptr[L.n]);
    {
        std::vector<int64_t> fill(tptr.begin(), tptr.end() - 1);
        for (int32_t w = 0; w < L.n; ++w)
            for (int64_t e = L.ptr[w]; e < L.ptr[w + 1]; ++e) {
                int64_t k = fill[L.col[e]]++;
                tlist[k] = w;
                tpos[k] = (int32_t)(e - L.ptr[w]);
            }
    }
    int64_t work = 0;
    for (int32_t w = 0; w < L.n; ++w) {
        int64_t d = L.ptr[w + 1] - L.ptr[w];
        work += d * (d - 1) / 2;
    }
    int nt = pick_threads(threads, work);
    // Candidates come out per chunk of 32 consecutive x, each x's pairs
    // sorted by y, so concatenating the chunks gives (x, y) order.
    const int32_t chunk = 32;
    const int32_t nchunks = (ncols + chunk - 1) / chunk;
    std::vector<std::vector<Candidate>> out(nchunks);
    std::atomic<int32_t> next{0};
    const int32_t nwords = (ncols + 63) / 64;
    parallel_run(nt, [&](int) {
        std::vector<Count> cnt(ncols, 0);
        std::vector<uint64_t> seen(nwords, 0);   // ids touched for the current x
        std::vector<Candidate> mine;
        for (;;) {
            const int32_t c = next.fetch_add(1);
            if (c >= nchunks) break;
            const int32_t x0 = c * chunk, x1 = std::min(ncols, x0 + chunk);
            mine.clear();
            for (int32_t x = x0; x < x1; ++x) {
                if (tptr[x + 1] - tptr[x] < 2) continue;   // in < 2 lists: no pair
                // visits of x: the tails after x in the lists holding it
                int64_t visits = 0;
                for (int64_t k = tptr[x]; k < tptr[x + 1]; ++k) {
                    const int32_t w = tlist[k];
                    visits += (L.ptr[w + 1] - L.ptr[w]) - tpos[k] - 1;
                }
                // Dense when the counters after x are few against the visits:
                // count without marking, then sweep every counter after x in
                // blocks of 64 (a vectorisable compare gives the block's
                // candidate bits; the block is cleared with plain stores).
                // Sparse otherwise: mark touched ids in the bitmap and visit
                // only those. Both emit the same pairs in ascending y.
                const bool dense = (int64_t)(ncols - x - 1) <= 8 * visits;
                for (int64_t k = tptr[x]; k < tptr[x + 1]; ++k) {
                    int32_t w = tlist[k];
                    const int32_t* row = L.col.data() + L.ptr[w];
                    int32_t d = (int32_t)(L.ptr[w + 1] - L.ptr[w]);
                    if (dense) {
                        for (int32_t p = tpos[k] + 1; p < d; ++p) cnt[row[p]]++;
                    } else {
                        for (int32_t p = tpos[k] + 1; p < d; ++p) {
                            int32_t y = row[p];
                            cnt[y]++;
                            seen[y >> 6] |= uint64_t(1) << (y & 63);
                        }
                    }
                }
                // weight-1 pairs are not edges of G_a (Alg. 1 drops them)
                const Count floor = (Count)std::max(theta, 1);
                if (dense) {
                    for (int32_t y0 = x + 1; y0 < ncols; y0 += 64) {
                        const int32_t len = std::min<int32_t>(64, ncols - y0);
                        Count* blk = cnt.data() + y0;
                        const uint64_t bits = above(blk, len, floor);
                        for (uint64_t b = bits; b;) {
                            const int32_t i = __builtin_ctzll(b);
                            b &= b - 1;
                            mine.push_back({(int32_t)blk[i], x, y0 + i});
                        }
                        std::memset(blk, 0, sizeof(Count) * len);
                    }
                } else {
                    // touched ids in ascending order (all exceed x)
                    for (int32_t wd = (x + 1) >> 6; wd < nwords; ++wd) {
                        uint64_t bits = seen[wd];
                        if (!bits) continue;
                        seen[wd] = 0;
                        while (bits) {
                            const int32_t y = (wd << 6) + __builtin_ctzll(bits);
                            bits &= bits - 1;
                            if (cnt[y] > floor) mine.push_back({(int32_t)cnt[y], x, y});
                            cnt[y] = 0;
                        }
                    }
                }
            }
            out[c] = mine;
        }
    });
    std::vector<Candidate> all;
    size_t total = 0;
    for (auto& v : out) total += v.size();
    all.reserve(total);
    for (auto& v : out) all.insert(all.end(), v.begin(), v.end());
    return all;
}

// A pair's count is at most the number of lists: 16-bit counters when that
// fits (half the bytes for the dense sweep).
std::vector<Candidate> count_pairs(const Lists& L, int theta, int threads) {
    // a count is at most the number of lists, so theta >= L.n leaves no pair
    // (and keeps every floor below within the counter type)
    if ((int64_t)theta >= (int64_t)L.n) return {};
    if (L.n < 65536) return count_pairs_t<uint16_t>(L, theta, threads);
    return count_pairs_t<int32_t>(L, theta, threads);
}

// Candidates in Algorithm 2's order (weight descending, then (x, y)):
// with weights below 2^16 and ids below 2^24 the order is that of the
// 64-bit key (65535 - w, x, y), sorted by four stable passes of 16-bit
// digits, least significant first; a comparison sort otherwise.
void sort_candidates(std::vector<Candidate>& c, int32_t ncols) {
    int32_t wmax = 0;
    for (const Candidate& e : c) wmax = std::max(wmax, e.w);
    if (wmax >= 65536 || ncols > (1 << 24) || c.size() < 4096) {
        std::sort(c.begin(), c.end(), [](const Candidate& a, const Candidate& b) {
            if (a.w != b.w) return a.w > b.w;
            return a.x != b.x ? a.x < b.x : a.y < b.y;
        });
        return;
    }
    const size_t n = c.size();
    std::vector<uint64_t> key(n), tmp(n);
    for (size_t i = 0; i < n; ++i)
        key[i] = ((uint64_t)(65535 - c[i].w) << 48) | ((uint64_t)c[i].x << 24) |
                 (uint64_t)c[i].y;
    std::vector<uint32_t> count(65536);
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 16 * pass;
        std::fill(count.begin(), count.end(), 0u);
        for (size_t i = 0; i < n; ++i) count[(key[i] >> shift) & 0xFFFF]++;
        uint32_t run = 0;
        for (uint32_t& k : count) {
            const uint32_t v = k;
            k = run;
            run += v;
        }
        for (size_t i = 0; i < n; ++i) tmp[count[(key[i] >> shift) & 0xFFFF]++] = key[i];
        key.swap(tmp);
    }
    for (size_t i = 0; i < n; ++i) {
        const uint64_t k = key[i];
        c[i] = {(int32_t)(65535 - (int32_t)(k >> 48)), (int32_t)((k >> 24) & 0xFFFFFF),
                (int32_t)(k & 0xFFFFFF)};
    }
}

// Algorithm 1 after a round whose greedy scan ran to the end of its
// candidates. Every pair counted above theta then had an endpoint taken
// (the matching is maximal), and a pair with neither endpoint taken nor new
// is held by the same lists as before, so its count is unchanged: no such
// pair exceeds theta now. The candidates are therefore the pairs with an
// endpoint in `touched` (the previous round's matched ids and new ids): for
// each u in it, the whole lists holding u are counted and every counter is
// swept; a pair of two touched ids is kept from its smaller one. Returned in
// Algorithm 2's order (weight descending, then (x, y)).
template <class Count>
std::vector<Candidate> count_touched_t(const Lists& L, int theta, int threads,
                                       const std::vector<int32_t>& touched) {
    const int32_t ncols = L.ncols;
    std::vector<char> in_t(ncols, 0);
    for (int32_t u : touched) in_t[u] = 1;
    std::vector<int64_t> tptr(ncols + 1, 0);
    for (int64_t e = 0; e < L.ptr[L.n]; ++e) tptr[L.col[e] + 1]++;
    for (int32_t c = 0; c < ncols; ++c) tptr[c + 1] += tptr[c];
    std::vector<int32_t> tlist(L.ptr[L.n]);
    {
        std::vector<int64_t> fill(tptr.begin(), tptr.end() - 1);
        for (int32_t w = 0; w < L.n; ++w)
            for (int64_t e = L.ptr[w]; e < L.ptr[w + 1]; ++e) tlist[fill[L.col[e]]++] = w;
    }
    int64_t work = 0;
    for (int32_t u : touched)
        for (int64_t k = tptr[u]; k < tptr[u + 1]; ++k) work += L.ptr[tlist[k] + 1] - L.ptr[tlist[k]];
    const int nt = pick_threads(threads, work);
    const int32_t nu = (int32_t)touched.size(), chunk = 16;
    const int32_t nchunks = (nu + chunk - 1) / chunk;
    std::vector<std::vector<Candidate>> out(nchunks);
    std::atomic<int32_t> next{0};
    const Count floor = (Count)std::max(theta, 1);
    parallel_run(nt, [&](int) {
        std::vector<Count> cnt(ncols, 0);
        for (;;) {
            const int32_t c = next.fetch_add(1);
            if (c >= nchunks) break;
            std::vector<Candidate>& mine = out[c];
            for (int32_t i = c * chunk; i < std::min(nu, (c + 1) * chunk); ++i) {
                const int32_t u = touched[i];
                if (tptr[u + 1] - tptr[u] < 2) continue;   // in < 2 lists: no pair
                for (int64_t k = tptr[u]; k < tptr[u + 1]; ++k) {
                    const int32_t w = tlist[k];
                    for (int64_t e = L.ptr[w]; e < L.ptr[w + 1]; ++e) cnt[L.col[e]]++;
                }
                cnt[u] = 0;
                for (int32_t y0 = 0; y0 < ncols; y0 += 64) {
                    const int32_t len = std::min<int32_t>(64, ncols - y0);
                    Count* blk = cnt.data() + y0;
                    for (uint64_t b = above(blk, len, floor); b;) {
                        const int32_t j = __builtin_ctzll(b);
                        b &= b - 1;
                        const int32_t y = y0 + j;
                        if (in_t[y] && y < u) continue;
                        mine.push_back({(int32_t)blk[j], std::min(u, y), std::max(u, y)});
                    }
                    std::memset(blk, 0, sizeof(Count) * len);
                }
            }
        }
    });
    std::vector<Candidate> all;
    size_t total = 0;
    for (auto& v : out) total += v.size();
    all.reserve(total);
    for (auto& v : out) all.insert(all.end(), v.begin(), v.end());
    sort_candidates(all, ncols);
    return all;
}

std::vector<Candidate> count_touched(const Lists& L, int theta, int threads,
                                     const std::vector<int32_t>& touched) {
    if ((int64_t)theta >= (int64_t)L.n) return {};
    if (L.n < 65536) return count_touched_t<uint16_t>(L, theta, threads, touched);
    return count_touched_t<int32_t>(L, theta, threads, touched);
}

// Orders candidates by decreasing weight, keeping the (x, y) order among
// equal weights: a stable counting sort on the (small, integer) weights.
std::vector<Candidate> order_by_weight(const std::vector<Candidate>& c) {
    int64_t wmax = 0;
    for (const Candidate& e : c) wmax = std::max<int64_t>(wmax, e.w);
    std::vector<int64_t> start(wmax + 2, 0);
    for (const Candidate& e : c) start[wmax - e.w + 1]++;
    for (int64_t i = 0; i <= wmax; ++i) start[i + 1] += start[i];
    std::vector<Candidate> out(c.size());
    for (const Candidate& e : c) out[start[wmax - e.w]++] = e;
    return out;
}

// Algorithm 3 for one round: rewrite every list, replacing each matched pair
// it holds by the pair's new id; lists stay sorted (new ids exceed all older
// ones, and the few new ids of a list are sorted among themselves).
Lists rewrite(const Lists& L, const std::vector<int32_t>& partner,
              const std::vector<int32_t>& newid, int32_t ncols_new,
              int threads) {
    Lists out;
    out.n = L.n;
    out.ncols = ncols_new;
    out.ptr.assign(L.n + 1, 0);
    int nt = pick_threads(threads, L.ptr[L.n] * 4);
    auto pass = [&](bool fill) {
        std::atomic<int32_t> next{0};
        parallel_run(nt, [&](int) {
            std::vector<int32_t> stamp(L.ncols, -1);
            std::vector<int32_t> added;
            for (;;) {
                int32_t w0 = next.fetch_add(256);
                if (w0 >= L.n) break;
                int32_t w1 = std::min(L.n, w0 + 256);
                for (int32_t w = w0; w < w1; ++w) {
                    const int32_t* row = L.col.data() + L.ptr[w];
                    int32_t d = (int32_t)(L.ptr[w + 1] - L.ptr[w]);
                    for (int32_t i = 0; i < d; ++i) stamp[row[i]] = w;
                    int32_t* dst = fill ? out.col.data() + out.ptr[w] : nullptr;
                    int32_t kept = 0;
                    added.clear();
                    for (int32_t i = 0; i < d; ++i) {
                        int32_t c = row[i];
                        int32_t p = partner[c];
                        if (p >= 0 && stamp[p] == w) {
                            if (c < p) added.push_back(newid[c]);
                            continue;
                        }
                        if (fill) dst[kept] = c;
                        ++kept;
                    }
                    if (fill) {
                        std::sort(added.begin(), added.end());
                        std::copy(added.begin(), added.end(), dst + kept);
                    } else {
                        out.ptr[w + 1] = kept + (int32_t)added.size();
                    }
                }
            }
        });
    };
    pass(false);
    for (int32_t w = 0; w < L.n; ++w) out.ptr[w + 1] += out.ptr[w];
    out.col.resize(out.ptr[L.n]);
    pass(true);
    return out;
}

int64_t num_add(const Lists& L) {
    int64_t s = 0;
    for (int32_t w = 0; w < L.n; ++w) {
        int64_t d = L.ptr[w + 1] - L.ptr[w];
        if (d >= 1) s += d - 1;
    }
    return s;
}

}  // namespace

extern "C" {

const char* gcn_last_error(void) { return gcn::g_err.c_str(); }

int gcn_abi_version(void) { return GCN_ABI_VERSION; }

int gcn_subgraph_build(int64_t n_full, const int64_t* src, const int64_t* dst,
                       int64_t n_edges, const int64_t* vertices,
                       int64_t n_vertices, gcn_graph_t* out) {
    GCN_CHECK_ARG(out != nullptr, "gcn_subgraph_build: out is NULL");
    GCN_CHECK_ARG(n_full >= 0 && n_full < INT32_MAX,
                  "gcn_subgraph_build: n_full %lld outside [0, 2^31-1)",
                  (long long)n_full);
    GCN_CHECK_ARG(n_edges >= 0, "gcn_subgraph_build: negative n_edges");
    GCN_CHECK_ARG(n_edges == 0 || (src && dst),
                  "gcn_subgraph_build: src/dst NULL with n_edges > 0");
    GCN_CHECK_ARG(vertices == nullptr || (n_vertices >= 0 && n_vertices <= n_full),
                  "gcn_subgraph_build: n_vertices outside [0, n_full]");
    try {
        const int32_t n = vertices ? (int32_t)n_vertices : (int32_t)n_full;
        std::vector<int32_t> relabel;
        if (vertices) {
            relabel.assign((size_t)n_full, -1);
            for (int64_t k = 0; k < n_vertices; ++k) {
                int64_t v = vertices[k];
                GCN_CHECK_ARG(v >= 0 && v < n_full,
                              "gcn_subgraph_build: vertex %lld out of range",
                              (long long)v);
                GCN_CHECK_ARG(relabel[v] < 0,
                              "gcn_subgraph_build: vertex %lld repeated",
                              (long long)v);
                relabel[v] = (int32_t)k;
            }
        }
        std::vector<int64_t> cnt((size_t)n + 1, 0);
        for (int64_t i = 0; i < n_edges; ++i) {
            int64_t a = src[i], b = dst[i];
            GCN_CHECK_ARG(a >= 0 && a < n_full && b >= 0 && b < n_full,
                          "gcn_subgraph_build: edge %lld (%lld, %lld) out of range",
                          (long long)i, (long long)a, (long long)b);
        }
        auto map = [&](int64_t v) -> int32_t {
            return vertices ? relabel[v] : (int32_t)v;
        };
        for (int64_t i = 0; i < n_edges; ++i) {
            int32_t a = map(src[i]), b = map(dst[i]);
            if (a < 0 || b < 0 || a == b) continue;
            cnt[a + 1]++;
            cnt[b + 1]++;
        }
        for (int32_t v = 0; v < n; ++v) cnt[v + 1] += cnt[v];
        std::vector<int32_t> adj(cnt[n]);
        std::vector<int64_t> fill(cnt.begin(), cnt.end() - 1);
        for (int64_t i = 0; i < n_edges; ++i) {
            int32_t a = map(src[i]), b = map(dst[i]);
            if (a < 0 || b < 0 || a == b) continue;
            adj[fill[a]++] = b;
            adj[fill[b]++] = a;
        }
        auto* g = new gcn_graph;
        g->n = n;
        g->rowptr.assign((size_t)n + 1, 0);
        int64_t total = 0;
        for (int32_t v = 0; v < n; ++v) {
            auto b = adj.begin() + cnt[v], e = adj.begin() + cnt[v + 1];
            std::sort(b, e);
            auto last = std::unique(b, e);
            total += last - b;
            if (total >= INT32_MAX) {
                delete g;
                set_error("gcn_subgraph_build: more than 2^31-1 list entries");
                return GCN_E_INVALID_ARG;
            }
            g->rowptr[v + 1] = (int32_t)total;
        }
        g->col.resize(total);
        for (int32_t v = 0; v < n; ++v) {
            int64_t d = g->rowptr[v + 1] - g->rowptr[v];
            std::copy(adj.begin() + cnt[v], adj.begin() + cnt[v] + d,
                      g->col.begin() + g->rowptr[v]);
        }
        *out = g;
        gcn::clear_error();
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_subgraph_build: out of host memory");
        return GCN_E_OOM;
    }
}

int gcn_graph_info(gcn_graph_t g, int32_t* n, int64_t* nnz,
                   const int32_t** rowptr, const int32_t** col) {
    GCN_CHECK_ARG(g != nullptr, "gcn_graph_info: NULL graph");
    if (n) *n = g->n;
    if (nnz) *nnz = g->rowptr[g->n];
    if (rowptr) *rowptr = g->rowptr.data();
    if (col) *col = g->col.data();
    return GCN_OK;
}

void gcn_graph_free(gcn_graph_t g) { delete g; }

int gcn_redundancy_reduce(gcn_graph_t g, const gcn_rr_params* params,
                          gcn_reduced_t* out) {
    GCN_CHECK_ARG(g != nullptr && params != nullptr && out != nullptr,
                  "gcn_redundancy_reduce: NULL argument");
    GCN_CHECK_ARG(params->theta >= 0, "gcn_redundancy_reduce: theta < 0");
    GCN_CHECK_ARG(params->max_rounds >= 0 && params->max_rounds <= GCN_MAX_ROUNDS,
                  "gcn_redundancy_reduce: max_rounds %d outside [0, %d]",
                  params->max_rounds, GCN_MAX_ROUNDS);
    GCN_CHECK_ARG(params->num_threads >= 0, "gcn_redundancy_reduce: num_threads < 0");
    try {
        const int32_t n = g->n;
        Lists L;
        L.n = n;
        L.ncols = n;
        L.ptr.assign(g->rowptr.begin(), g->rowptr.end());
        L.col = g->col;
        auto* r = new gcn_reduced;
        r->n = n;
        r->deg.resize(n);
        for (int32_t v = 0; v < n; ++v) r->deg[v] = g->rowptr[v + 1] - g->rowptr[v];
        r->round_offsets.push_back(0);
        const int64_t max_aux = params->max_aux;
        std::vector<int32_t> touched;
        for (int round = 0; round < params->max_rounds; ++round) {
            int64_t naux = (int64_t)r->pairs.size() / 2;
            int64_t budget_left = max_aux < 0 ? INT64_MAX : max_aux - naux;
            if (budget_left <= 0) break;
            if ((int64_t)L.ncols + std::min<int64_t>(budget_left, L.ncols) >= INT32_MAX) {
                delete r;
                set_error("gcn_redundancy_reduce: vertex ids would exceed 2^31-1");
                return GCN_E_INVALID_ARG;
            }
            // Algorithm 1 (candidates above theta only), from the ids the last
            // round touched when they are few; Algorithm 2 scans by
            // decreasing weight, then (x, y) ascending
            const bool incremental =
                round > 0 && (int64_t)touched.size() * 5 <= (int64_t)L.ncols;
            const std::vector<Candidate> cand =
                incremental ? count_touched(L, params->theta, params->num_threads, touched)
                            : order_by_weight(count_pairs(L, params->theta, params->num_threads));
            std::vector<char> used(L.ncols, 0);
            std::vector<int32_t> partner(L.ncols, -1), newid(L.ncols, -1);
            int64_t taken = 0, wsum = 0;
            bool exhausted = false;
            for (const Candidate& c : cand) {
                if (taken >= budget_left) {
                    exhausted = true;
                    break;
                }
                if (used[c.x] || used[c.y]) continue;
                used[c.x] = used[c.y] = 1;
                int32_t id = L.ncols + (int32_t)taken;
                partner[c.x] = c.y;
                partner[c.y] = c.x;
                newid[c.x] = newid[c.y] = id;
                r->pairs.push_back(c.x);
                r->pairs.push_back(c.y);
                wsum += c.w;
                ++taken;
            }
            if (taken == 0) break;
            // the ids this round touched: its matched ids and its new ids
            touched.clear();
            for (int32_t v = 0; v < L.ncols; ++v)
                if (used[v]) touched.push_back(v);
            for (int32_t k = 0; k < (int32_t)taken; ++k) touched.push_back(L.ncols + k);
            // Algorithm 3
            L = rewrite(L, partner, newid, L.ncols + (int32_t)taken, params->num_threads);
            r->round_offsets.push_back((int32_t)(r->pairs.size() / 2));
            r->stats.push_back({taken, wsum, L.ptr[n], num_add(L)});
            if (exhausted) break;
        }
        r->naux = (int32_t)(r->pairs.size() / 2);
        r->rounds = (int32_t)r->stats.size();
        if (L.ptr[n] >= INT32_MAX) {
            delete r;
            set_error("gcn_redundancy_reduce: list entries exceed 2^31-1");
            return GCN_E_INVALID_ARG;
        }
        r->rowptr.resize(n + 1);
        for (int32_t v = 0; v <= n; ++v) r->rowptr[v] = (int32_t)L.ptr[v];
        r->col = std::move(L.col);
        *out = r;
        gcn::clear_error();
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_redundancy_reduce: out of host memory");
        return GCN_E_OOM;
    }
}

int gcn_reduced_info(gcn_reduced_t r, int32_t* n, int32_t* naux,
                     int32_t* rounds, int64_t* nnz, const int32_t** rowptr,
                     const int32_t** col, const int32_t** pairs,
                     const int32_t** round_offsets,
                     const gcn_rr_round** per_round, const int32_t** deg) {
    GCN_CHECK_ARG(r != nullptr, "gcn_reduced_info: NULL handle");
    if (n) *n = r->n;
    if (naux) *naux = r->naux;
    if (rounds) *rounds = r->rounds;
    if (nnz) *nnz = r->rowptr[r->n];
    if (rowptr) *rowptr = r->rowptr.data();
    if (col) *col = r->col.data();
    if (pairs) *pairs = r->pairs.data();
    if (round_offsets) *round_offsets = r->round_offsets.data();
    if (per_round) *per_round = r->stats.data();
    if (deg) *deg = r->deg.data();
    return GCN_OK;
}

void gcn_reduced_free(gcn_reduced_t r) { delete r; }

// ----------------------------------------------------------- device image

// Work-list bins. A row of d entries is ceil(d / seg_len) pieces (one when
// d <= seg_len, d == 0 included). A row of more than kBinGroups pieces (a
// hub) is a bin of its own; rows of 2..kBinGroups pieces are packed
// next-fit, largest first, into bins of kBinGroups pieces; single-piece
// rows, longest first, fill what those bins leave, then bins of their own.
// So every row's pieces sit in one bin, the hub bins come first, then the
// other bins holding split rows, and the groups of one bin have lists of
// similar length (a workgroup lasts as long as its longest group).
struct BinLayout {
    std::vector<int32_t> rows;      // rows in work-list order
    std::vector<int64_t> bin_rows;  // bin b: rows[bin_rows[b] .. bin_rows[b + 1])
    int64_t nseg = 0;
    int32_t nhub = 0, nmulti = 0, max_row = 0;
};

static int64_t row_pieces(gcn_reduced_t r, int32_t w, int32_t seg_len) {
    const int64_t d = r->rowptr[w + 1] - r->rowptr[w];
    return d <= seg_len ? 1 : (d + seg_len - 1) / seg_len;
}

static BinLayout layout_bins(gcn_reduced_t r, int32_t seg_len) {
    const int64_t G = gcn::kBinGroups;
    BinLayout L;
    std::vector<int32_t> multi, single;
    L.bin_rows.push_back(0);
    for (int32_t w = 0; w < r->n; ++w) {
        L.max_row = std::max(L.max_row, r->rowptr[w + 1] - r->rowptr[w]);
        const int64_t k = row_pieces(r, w, seg_len);
        L.nseg += k;
        if (k > G) {
            L.rows.push_back(w);
            L.bin_rows.push_back((int64_t)L.rows.size());
            ++L.nhub;
        } else if (k > 1) {
            multi.push_back(w);
        } else {
            single.push_back(w);
        }
    }
    std::stable_sort(multi.begin(), multi.end(), [&](int32_t a, int32_t b) {
        return row_pieces(r, a, seg_len) > row_pieces(r, b, seg_len);
    });
    auto len = [&](int32_t w) { return r->rowptr[w + 1] - r->rowptr[w]; };
    std::stable_sort(single.begin(), single.end(),
                     [&](int32_t a, int32_t b) { return len(a) > len(b); });
    std::vector<std::vector<int32_t>> mb;
    std::vector<int64_t> used;
    for (int32_t w : multi) {
        const int64_t k = row_pieces(r, w, seg_len);
        if (mb.empty() || used.back() + k > G) {
            mb.emplace_back();
            used.push_back(0);
        }
        mb.back().push_back(w);
        used.back() += k;
    }
    size_t si = 0;
    for (size_t b = 0; b < mb.size(); ++b) {
        for (; used[b] < G && si < single.size(); ++used[b]) mb[b].push_back(single[si++]);
        L.rows.insert(L.rows.end(), mb[b].begin(), mb[b].end());
        L.bin_rows.push_back((int64_t)L.rows.size());
    }
    L.nmulti = (int32_t)(L.bin_rows.size() - 1);
    for (; si < single.size(); si += (size_t)G) {
        const size_t e = std::min(single.size(), si + (size_t)G);
        L.rows.insert(L.rows.end(), single.begin() + (int64_t)si, single.begin() + (int64_t)e);
        L.bin_rows.push_back((int64_t)L.rows.size());
    }
    return L;
}

static int plan_image(gcn_reduced_t r, int32_t seg_len, gcn::ImageHeader* h) {
    GCN_CHECK_ARG(r != nullptr, "graph image: NULL reduced graph");
    if (seg_len == 0) seg_len = gcn::kDefaultSegLen;
    GCN_CHECK_ARG(seg_len >= 1 && seg_len <= 65536,
                  "graph image: seg_len %d outside [1, 65536]", seg_len);
    std::memset(h, 0, sizeof(*h));
    h->magic = gcn::kImageMagic;
    h->n = r->n;
    h->naux = r->naux;
    h->rounds = r->rounds;
    h->seg_len = seg_len;
    h->nnz = r->rowptr[r->n];
    const BinLayout L = layout_bins(r, seg_len);
    GCN_CHECK_ARG(L.nseg < INT32_MAX, "graph image: too many segments");
    h->nseg = (int32_t)L.nseg;
    h->nbins = (int32_t)(L.bin_rows.size() - 1);
    h->nmulti = L.nmulti;
    h->nhub = L.nhub;
    h->max_row = L.max_row;
    const int64_t nbins = h->nbins;
    int64_t off = gcn::round_up(sizeof(gcn::ImageHeader), 256);
    auto take = [&](int64_t bytes) {
        int64_t o = off;
        off = gcn::round_up(off + std::max<int64_t>(bytes, 1), 256);
        return o;
    };
    h->off_rowptr = take(4 * ((int64_t)r->n + 1));
    h->off_col = take(4 * h->nnz);
    h->off_pairs = take(8 * (int64_t)r->naux);
    h->off_inv_deg = take(4 * (int64_t)r->n);
    h->off_seg = take(16 * L.nseg);
    h->off_bins = take(4 * (nbins + 1));
    // expansion sizes: |E(k)| = |E(p_k)| + |E(q_k)|, originals count 1
    int64_t exp_nnz = 0;
    {
        std::vector<int64_t> sz(r->naux);
        for (int32_t k = 0; k < r->naux; ++k) {
            int64_t t = 0;
            for (int e = 0; e < 2; ++e) {
                const int32_t c = r->pairs[2 * k + e];
                t += c < r->n ? 1 : sz[c - r->n];
            }
            sz[k] = t;
            exp_nnz += t;
        }
    }
    GCN_CHECK_ARG(exp_nnz < INT32_MAX, "graph image: pair-sum expansions too long");
    h->exp_nnz = exp_nnz;
    h->off_exp_col = take(4 * exp_nnz);
    h->off_exp_seg = take(16 * (int64_t)r->naux);
    h->total = off;
    for (int i = 0; i <= r->rounds; ++i) h->round_offsets[i] = r->round_offsets[i];
    return GCN_OK;
}

int gcn_graph_image_bytes(gcn_reduced_t r, int32_t seg_len, size_t* bytes) {
    GCN_CHECK_ARG(bytes != nullptr, "gcn_graph_image_bytes: NULL bytes");
    gcn::ImageHeader h;
    int rc = plan_image(r, seg_len, &h);
    if (rc) return rc;
    *bytes = (size_t)h.total;
    return GCN_OK;
}

int gcn_graph_pack(gcn_reduced_t r, int32_t seg_len, void* host_buf,
                   size_t bytes) {
    GCN_CHECK_ARG(host_buf != nullptr, "gcn_graph_pack: NULL buffer");
    gcn::ImageHeader h;
    int rc = plan_image(r, seg_len, &h);
    if (rc) return rc;
    GCN_CHECK_ARG(bytes >= (size_t)h.total,
                  "gcn_graph_pack: buffer of %zu bytes, image needs %lld",
                  bytes, (long long)h.total);
    char* base = static_cast<char*>(host_buf);
    std::memset(base, 0, (size_t)h.total);
    std::memcpy(base, &h, sizeof(h));
    std::memcpy(base + h.off_rowptr, r->rowptr.data(), 4 * ((size_t)r->n + 1));
    if (h.nnz) std::memcpy(base + h.off_col, r->col.data(), 4 * (size_t)h.nnz);
    if (r->naux) std::memcpy(base + h.off_pairs, r->pairs.data(), 8 * (size_t)r->naux);
    float* inv = reinterpret_cast<float*>(base + h.off_inv_deg);
    for (int32_t v = 0; v < r->n; ++v)
        inv[v] = r->deg[v] > 0 ? (float)(1.0 / (double)r->deg[v]) : 0.0f;
    // Work list, bin by bin (see layout_bins): a row's pieces are
    // consecutive, the first carrying the piece count, the others 0.
    const BinLayout L = layout_bins(r, h.seg_len);
    int32_t* seg = reinterpret_cast<int32_t*>(base + h.off_seg);
    int32_t* bins = reinterpret_cast<int32_t*>(base + h.off_bins);
    int64_t s = 0;
    for (int32_t bi = 0; bi < h.nbins; ++bi) {
        bins[bi] = (int32_t)s;
        for (int64_t x = L.bin_rows[bi]; x < L.bin_rows[bi + 1]; ++x) {
            const int32_t w = L.rows[x];
            const int32_t b = r->rowptr[w], e = r->rowptr[w + 1];
            const int64_t k = row_pieces(r, w, h.seg_len);
            for (int64_t j = 0; j < k; ++j) {
                seg[4 * s + 0] = w;
                seg[4 * s + 1] = (int32_t)std::min<int64_t>(e, b + j * h.seg_len);
                seg[4 * s + 2] = (int32_t)std::min<int64_t>(e, b + (j + 1) * h.seg_len);
                seg[4 * s + 3] = j == 0 ? (int32_t)k : 0;
                ++s;
            }
        }
    }
    bins[h.nbins] = (int32_t)s;
    // Expansion of every pair sum into original vertices, ascending: the
    // members of pair k are the members of its two parts (earlier ids).
    int32_t* ecol = reinterpret_cast<int32_t*>(base + h.off_exp_col);
    int32_t* eseg = reinterpret_cast<int32_t*>(base + h.off_exp_seg);
    int32_t pos = 0;
    for (int32_t k = 0; k < r->naux; ++k) {
        const int32_t b = pos;
        for (int e = 0; e < 2; ++e) {
            const int32_t c = r->pairs[2 * k + e];
            if (c < r->n) {
                ecol[pos++] = c;
            } else {
                const int32_t* src = eseg + 4 * (c - r->n);
                for (int32_t i = src[1]; i < src[2]; ++i) ecol[pos++] = ecol[i];
            }
        }
        std::sort(ecol + b, ecol + pos);
        eseg[4 * k + 0] = k;
        eseg[4 * k + 1] = b;
        eseg[4 * k + 2] = pos;
        eseg[4 * k + 3] = -1;
    }
    // Longest expansions first (each entry names its pair sum, so the order
    // is free): the pair sums of the last rounds, the longest, start first
    // instead of forming the launch's tail.
    {
        std::vector<std::array<int32_t, 4>> ent(r->naux);
        for (int32_t k = 0; k < r->naux; ++k)
            for (int j = 0; j < 4; ++j) ent[k][j] = eseg[4 * k + j];
        std::stable_sort(ent.begin(), ent.end(), [](const auto& a, const auto& b) {
            return a[2] - a[1] > b[2] - b[1];
        });
        for (int32_t k = 0; k < r->naux; ++k)
            for (int j = 0; j < 4; ++j) eseg[4 * k + j] = ent[k][j];
    }
    return GCN_OK;
}

int gcn_graph_describe(const void* host_image, size_t bytes,
                       const void* dev_buf, gcn_dgraph* out) {
    GCN_CHECK_ARG(host_image && dev_buf && out, "gcn_graph_describe: NULL argument");
    GCN_CHECK_ARG(bytes >= sizeof(gcn::ImageHeader), "gcn_graph_describe: image too small");
    gcn::ImageHeader h;
    std::memcpy(&h, host_image, sizeof(h));
    GCN_CHECK_ARG(h.magic == gcn::kImageMagic, "gcn_graph_describe: not a graph image");
    GCN_CHECK_ARG((size_t)h.total <= bytes, "gcn_graph_describe: image truncated");
    GCN_CHECK_ARG(((uintptr_t)dev_buf & 255) == 0,
                  "gcn_graph_describe: device buffer not 256-byte aligned");
    const char* d = static_cast<const char*>(dev_buf);
    std::memset(out, 0, sizeof(*out));
    out->n = h.n;
    out->naux = h.naux;
    out->rounds = h.rounds;
    out->seg_len = h.seg_len;
    out->nseg = h.nseg;
    out->nbins = h.nbins;
    out->nmulti = h.nmulti;
    out->nhub = h.nhub;
    out->max_row = h.max_row;
    out->nnz = h.nnz;
    out->rowptr = reinterpret_cast<const int32_t*>(d + h.off_rowptr);
    out->col = reinterpret_cast<const int32_t*>(d + h.off_col);
    out->pairs = reinterpret_cast<const int32_t*>(d + h.off_pairs);
    out->inv_deg = reinterpret_cast<const float*>(d + h.off_inv_deg);
    out->seg = reinterpret_cast<const int32_t*>(d + h.off_seg);
    out->bins = reinterpret_cast<const int32_t*>(d + h.off_bins);
    out->exp_nnz = h.exp_nnz;
    out->exp_col = reinterpret_cast<const int32_t*>(d + h.off_exp_col);
    out->exp_seg = reinterpret_cast<const int32_t*>(d + h.off_exp_seg);
    for (int i = 0; i <= h.rounds; ++i) out->round_offsets[i] = h.round_offsets[i];
    return GCN_OK;
}

}  // extern "C"
