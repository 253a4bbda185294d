// Minibatch vertex sets by frontier sampling, and the subgraph induced on a
// vertex set (Section 3.1: a minibatch is the subgraph induced on vertices
// drawn from the training graph by a graph sampler; the paper names the
// multi-dimensional random walk of Ribeiro and Towsley, IMC 2010, as one).
// Host C++ only: a walk is a chain of dependent steps (each picks from the
// frontier that the previous step left), which a CPU core runs at cache
// latency; independent minibatches run on independent host threads.
#include <algorithm>
#include <cstring>
#include <memory>
#include <new>
#include <vector>

#include "common.h"
#include "graph_types.h"

using gcn::set_error;

namespace {

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) as a counter-based
// generator: output i of seed s finalises s + (i + 1) * golden gamma.
struct SplitMix64 {
    uint64_t seed;
    uint64_t count = 0;
    explicit SplitMix64(uint64_t s) : seed(s) {}
    uint64_t next() {
        uint64_t z = seed + (count + 1) * 0x9E3779B97F4A7C15ull;
        ++count;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    // uniform integer in [0, bound): the high word of output * bound
    uint64_t below(uint64_t bound) {
        return (uint64_t)(((unsigned __int128)next() * bound) >> 64);
    }
};

// Open-addressing map from vertex id to a small int (-1: absent), sized
// for at most `cap` keys at load <= 1/2.
class IdMap {
public:
    explicit IdMap(int64_t cap) {
        size_t s = 16;
        while ((int64_t)s < 2 * cap) s <<= 1;
        mask_ = s - 1;
        keys_.assign(s, -1);
        vals_.assign(s, -1);
    }
    // inserts key -> val unless present; returns true if inserted
    bool insert(int32_t key, int32_t val) {
        size_t i = slot(key);
        while (keys_[i] != -1) {
            if (keys_[i] == key) return false;
            i = (i + 1) & mask_;
        }
        keys_[i] = key;
        vals_[i] = val;
        return true;
    }
    int32_t find(int32_t key) const {
        size_t i = slot(key);
        while (keys_[i] != -1) {
            if (keys_[i] == key) return vals_[i];
            i = (i + 1) & mask_;
        }
        return -1;
    }

private:
    size_t slot(int32_t key) const {
        return (size_t)(((uint64_t)(uint32_t)key * 0x9E3779B97F4A7C15ull) >> 20) & mask_;
    }
    size_t mask_ = 0;
    std::vector<int32_t> keys_, vals_;
};

// Running sums of the frontier's degrees (a Fenwick tree over the slots):
// O(log m) update of one slot and O(log m) search for the first slot whose
// running sum exceeds a draw.
class DegreeSums {
public:
    explicit DegreeSums(int32_t m) : m_(m), t_(m + 1, 0) {
        top_ = 1;
        while (top_ * 2 <= m_) top_ *= 2;
    }
    void add(int32_t slot, int64_t delta) {
        for (int32_t i = slot + 1; i <= m_; i += i & -i) t_[i] += delta;
    }
    // first slot s (0-based) with deg[0] + ... + deg[s] > r, for 0 <= r < total
    int32_t first_exceeding(int64_t r) const {
        int32_t pos = 0;
        for (int32_t step = top_; step; step >>= 1)
            if (pos + step <= m_ && t_[pos + step] <= r) {
                pos += step;
                r -= t_[pos];
            }
        return pos;
    }

private:
    int32_t m_, top_;
    std::vector<int64_t> t_;
};

}  // namespace

extern "C" {

int gcn_sample_frontier(gcn_graph_t full, int32_t m, int32_t budget, uint64_t seed,
                        int64_t max_steps, int32_t* vertices, int32_t* n_out,
                        int64_t* steps_out) {
    GCN_CHECK_ARG(full && vertices && n_out, "gcn_sample_frontier: NULL argument");
    const int32_t n = full->n;
    GCN_CHECK_ARG(m >= 1 && m <= budget && budget <= n,
                  "gcn_sample_frontier: need 1 <= m (%d) <= budget (%d) <= n (%d)", m, budget,
                  n);
    GCN_CHECK_ARG(max_steps >= 0, "gcn_sample_frontier: negative max_steps");
    try {
        const int32_t* rowptr = full->rowptr.data();
        const int32_t* col = full->col.data();
        SplitMix64 rng(seed);
        IdMap sampled(budget);
        int32_t count = 0;

        // initial frontier: m distinct vertices drawn uniformly (a draw that
        // repeats a vertex already taken is dropped and drawn again)
        std::vector<int32_t> frontier(m);
        DegreeSums sums(m);
        int64_t total = 0;
        for (int32_t s = 0; s < m;) {
            const int32_t v = (int32_t)rng.below((uint64_t)n);
            if (!sampled.insert(v, count)) continue;
            vertices[count++] = v;
            frontier[s] = v;
            const int64_t d = rowptr[v + 1] - rowptr[v];
            sums.add(s, d);
            total += d;
            ++s;
        }

        // each step moves the frontier vertex picked in proportion to its
        // degree along a uniformly chosen edge
        int64_t steps = 0;
        while (count < budget && steps < max_steps && total > 0) {
            const int32_t s = sums.first_exceeding((int64_t)rng.below((uint64_t)total));
            const int32_t u = frontier[s];
            const int64_t du = rowptr[u + 1] - rowptr[u];
            const int32_t v = col[rowptr[u] + (int64_t)rng.below((uint64_t)du)];
            const int64_t dv = rowptr[v + 1] - rowptr[v];
            frontier[s] = v;
            sums.add(s, dv - du);
            total += dv - du;
            if (sampled.insert(v, count)) vertices[count++] = v;
            ++steps;
        }
        std::sort(vertices, vertices + count);
        *n_out = count;
        if (steps_out) *steps_out = steps;
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_sample_frontier: out of host memory");
        return GCN_E_OOM;
    }
}

int gcn_subgraph_induce(gcn_graph_t full, const int32_t* vertices, int32_t n_vertices,
                        gcn_graph_t* out) {
    GCN_CHECK_ARG(full && out, "gcn_subgraph_induce: NULL argument");
    GCN_CHECK_ARG(n_vertices >= 0 && n_vertices <= full->n && (n_vertices == 0 || vertices),
                  "gcn_subgraph_induce: n_vertices %d outside [0, %d] or NULL vertices",
                  n_vertices, full->n);
    try {
        // Membership as a bitmap over the full graph's ids with a running
        // count per 64-bit word, so the rank of a member among the subset's
        // ids (ascending) is a popcount; rank_to_k maps it to the member's
        // position in `vertices`. Most neighbours of a sampled vertex are not
        // sampled: they cost one bit test in a cache-resident bitmap.
        const int64_t nwords = ((int64_t)full->n + 63) / 64;
        std::vector<uint64_t> bits((size_t)nwords, 0);
        for (int32_t k = 0; k < n_vertices; ++k) {
            const int32_t v = vertices[k];
            GCN_CHECK_ARG(v >= 0 && v < full->n, "gcn_subgraph_induce: vertex %d out of range",
                          v);
            const uint64_t b = uint64_t(1) << (v & 63);
            GCN_CHECK_ARG(!(bits[v >> 6] & b), "gcn_subgraph_induce: vertex %d repeated", v);
            bits[v >> 6] |= b;
        }
        std::vector<int32_t> before((size_t)nwords);   // members in earlier words
        int32_t run = 0;
        for (int64_t w = 0; w < nwords; ++w) {
            before[w] = run;
            run += __builtin_popcountll(bits[w]);
        }
        auto rank = [&](int32_t v) {
            return before[v >> 6] +
                   __builtin_popcountll(bits[v >> 6] & ((uint64_t(1) << (v & 63)) - 1));
        };
        std::vector<int32_t> rank_to_k((size_t)n_vertices);
        bool ascending = true;
        for (int32_t k = 0; k < n_vertices; ++k) {
            rank_to_k[rank(vertices[k])] = k;
            ascending = ascending && (k == 0 || vertices[k - 1] < vertices[k]);
        }

        auto g = std::make_unique<gcn_graph>();
        g->n = n_vertices;
        g->rowptr.assign((size_t)n_vertices + 1, 0);
        const int32_t* rowptr = full->rowptr.data();
        const int32_t* col = full->col.data();
        // one pass: an edge stays when both ends are in the subset; a
        // symmetric full graph gives a symmetric subgraph. Full lists are
        // sorted, so an ascending subset yields sorted rows directly.
        for (int32_t k = 0; k < n_vertices; ++k) {
            const int32_t v = vertices[k];
            const size_t first = g->col.size();
            for (int32_t e = rowptr[v]; e < rowptr[v + 1]; ++e) {
                const int32_t w = col[e];
                if (bits[w >> 6] & (uint64_t(1) << (w & 63))) g->col.push_back(rank_to_k[rank(w)]);
            }
            if (!ascending) std::sort(g->col.begin() + first, g->col.end());
            g->rowptr[k + 1] = (int32_t)g->col.size();
        }
        *out = g.release();
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_subgraph_induce: out of host memory");
        return GCN_E_OOM;
    }
}

}  // extern "C"
