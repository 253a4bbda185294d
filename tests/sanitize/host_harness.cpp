// CPU driver of the host half of the library (subgraph build, redundancy
// reduction, image packing, frontier sampling, induced subgraphs), built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitizers.py. It checks nothing numerically (the oracle tests
// do that); it walks every host path, including error paths and the
// threaded pair counting, so the sanitizers see each access.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "gcn_act.h"

namespace {

int failures = 0;

void expect(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "harness: %s (%s)\n", what, gcn_last_error());
        ++failures;
    }
}

// Edges with repeats, self-loops and a few hubs (power-law-like degrees).
void random_edges(std::mt19937_64& rng, int64_t n, int64_t m, std::vector<int64_t>& s,
                  std::vector<int64_t>& d) {
    s.clear();
    d.clear();
    if (n == 0) return;
    std::uniform_int_distribution<int64_t> any(0, n - 1);
    std::uniform_int_distribution<int64_t> hub(0, std::min<int64_t>(n, 5) - 1);
    std::uniform_real_distribution<double> u(0.0, 1.0);
    for (int64_t e = 0; e < m; ++e) {
        s.push_back(u(rng) < 0.3 ? hub(rng) : any(rng));
        d.push_back(any(rng));
    }
}

void walk_reduced(gcn_reduced_t r) {
    int32_t n = 0, naux = 0, rounds = 0;
    int64_t nnz = 0;
    const int32_t *rp, *cl, *pairs, *ro, *deg;
    const gcn_rr_round* st;
    expect(gcn_reduced_info(r, &n, &naux, &rounds, &nnz, &rp, &cl, &pairs, &ro, &st, &deg) ==
               GCN_OK,
           "reduced_info");
    int64_t sum = 0;
    for (int64_t i = 0; i < nnz; ++i) sum += cl[i];
    for (int32_t k = 0; k < 2 * naux; ++k) sum += pairs[k];
    for (int32_t w = 0; w < n; ++w) sum += deg[w] + rp[w + 1] - rp[w];
    for (int32_t i = 0; i < rounds; ++i) sum += st[i].matched + ro[i + 1];
    if (sum == -1) std::puts("");
    for (int32_t seg : {0, 3, 16}) {
        size_t bytes = 0;
        expect(gcn_graph_image_bytes(r, seg, &bytes) == GCN_OK, "image_bytes");
        // 256-byte aligned, as a device image buffer must be
        const size_t cap = (bytes + 255) / 256 * 256;
        unsigned char* img = static_cast<unsigned char*>(std::aligned_alloc(256, cap));
        expect(gcn_graph_pack(r, seg, img, bytes) == GCN_OK, "pack");
        gcn_dgraph dg;
        expect(gcn_graph_describe(img, bytes, img, &dg) == GCN_OK, "describe");
        expect(gcn_graph_pack(r, seg, img, bytes / 2) != GCN_OK, "pack: short buffer");
        std::free(img);
    }
}

}  // namespace

int main() {
    std::mt19937_64 rng(20010249);
    std::vector<int64_t> s, d;
    // random graphs, vertex subsets, every reduction knob, 1-4 threads
    for (int trial = 0; trial < 120; ++trial) {
        const int64_t n = (int64_t)(rng() % 300);
        random_edges(rng, n, (int64_t)(rng() % (12 * n + 1)), s, d);
        std::vector<int64_t> subset;
        const bool use_subset = n > 2 && trial % 3 == 0;
        if (use_subset)
            for (int64_t v = 0; v < n; v += 2) subset.push_back(v);
        gcn_graph_t g = nullptr;
        expect(gcn_subgraph_build(n, s.data(), d.data(), (int64_t)s.size(),
                                  use_subset ? subset.data() : nullptr,
                                  use_subset ? (int64_t)subset.size() : 0, &g) == GCN_OK,
               "subgraph_build");
        if (!g) continue;
        int32_t gn = 0;
        int64_t gnnz = 0;
        const int32_t *rp, *cl;
        expect(gcn_graph_info(g, &gn, &gnnz, &rp, &cl) == GCN_OK, "graph_info");
        gcn_rr_params p{(int32_t)(rng() % 4), (int32_t)(rng() % 7),
                        (int64_t)(rng() % 3 == 0 ? -1 : (int64_t)(rng() % 40)),
                        (int32_t)(1 + rng() % 4), 0};
        gcn_reduced_t r = nullptr;
        expect(gcn_redundancy_reduce(g, &p, &r) == GCN_OK, "reduce");
        if (r) walk_reduced(r);
        gcn_reduced_free(r);
        // frontier sampling and the induced subgraph on it
        if (gn > 4) {
            const int32_t budget = gn / 2, m = std::max(1, budget / 4);
            std::vector<int32_t> out(budget);
            int32_t count = 0;
            int64_t steps = 0;
            expect(gcn_sample_frontier(g, m, budget, rng(), 10 * budget, out.data(), &count,
                                       &steps) == GCN_OK,
                   "sample_frontier");
            gcn_graph_t sub = nullptr;
            expect(gcn_subgraph_induce(g, out.data(), count, &sub) == GCN_OK, "induce");
            gcn_graph_free(sub);
        }
        gcn_graph_free(g);
    }
    // a heavy hub (K_{2,R}: one pair of weight R, 16-bit counters) and a
    // threshold beyond the counters' range
    {
        const int64_t R = 40000, n = R + 2;
        s.clear();
        d.clear();
        for (int64_t v = 2; v < n; ++v) {
            s.push_back(0);
            d.push_back(v);
            s.push_back(1);
            d.push_back(v);
        }
        gcn_graph_t g = nullptr;
        expect(gcn_subgraph_build(n, s.data(), d.data(), (int64_t)s.size(), nullptr, 0, &g) ==
                   GCN_OK,
               "hub build");
        for (int32_t theta : {2, 70000}) {
            gcn_rr_params p{theta, 3, -1, 4, 0};
            gcn_reduced_t r = nullptr;
            expect(gcn_redundancy_reduce(g, &p, &r) == GCN_OK, "hub reduce");
            if (r) walk_reduced(r);
            gcn_reduced_free(r);
        }
        gcn_graph_free(g);
    }
    // error paths: every call must refuse without touching memory
    {
        gcn_graph_t g = nullptr;
        int64_t bad_s[2] = {0, 5}, bad_d[2] = {1, 1};
        expect(gcn_subgraph_build(3, bad_s, bad_d, 2, nullptr, 0, &g) != GCN_OK,
               "build: id out of range");
        expect(gcn_subgraph_build(3, nullptr, bad_d, 2, nullptr, 0, &g) != GCN_OK,
               "build: NULL src");
        int64_t ok_s[1] = {0}, ok_d[1] = {1};
        expect(gcn_subgraph_build(3, ok_s, ok_d, 1, nullptr, 0, &g) == GCN_OK, "build");
        gcn_rr_params p{-1, 2, -1, 1, 0};
        gcn_reduced_t r = nullptr;
        expect(gcn_redundancy_reduce(g, &p, &r) != GCN_OK, "reduce: theta < 0");
        p = gcn_rr_params{2, GCN_MAX_ROUNDS + 1, -1, 1, 0};
        expect(gcn_redundancy_reduce(g, &p, &r) != GCN_OK, "reduce: too many rounds");
        int32_t out[4];
        int32_t count = 0;
        int64_t steps = 0;
        expect(gcn_sample_frontier(g, 5, 2, 1, 10, out, &count, &steps) != GCN_OK,
               "sample: m > budget");
        int32_t verts[2] = {0, 7};
        gcn_graph_t sub = nullptr;
        expect(gcn_subgraph_induce(g, verts, 2, &sub) != GCN_OK, "induce: id out of range");
        gcn_graph_free(g);
    }
    std::printf("host harness: %d failures\n", failures);
    return failures ? 1 : 0;
}
