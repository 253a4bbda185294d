// CPU driver of the preparation pipeline's worker pool (and the threaded
// pair counting of the reduction), built with ThreadSanitizer by
// tests/test_sanitizers.py: several pipelines with 1-6 host workers build,
// reduce and pack subgraphs (edge lists and frontier samples of a full
// graph) while the caller takes and releases them in order; one pipeline is
// destroyed with jobs still queued. No GPU is used: the device reduction is
// replaced by a stub that the host-only workers never call.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "gcn_act.h"

extern "C" {
int gcn_redundancy_reduce_device_bytes(gcn_graph_t, const gcn_rr_params*, size_t*) {
    return GCN_E_UNSUPPORTED;
}
int gcn_redundancy_reduce_device(gcn_graph_t, const gcn_rr_params*, void*, size_t,
                                 gcn_stream_t, gcn_reduced_t*) {
    return GCN_E_UNSUPPORTED;
}
}

namespace {

int failures = 0;

void expect(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "harness: %s (%s)\n", what, gcn_last_error());
        ++failures;
    }
}

void edges(std::mt19937_64& rng, int64_t n, int64_t m, std::vector<int64_t>& s,
           std::vector<int64_t>& d) {
    s.resize(m);
    d.resize(m);
    for (int64_t e = 0; e < m; ++e) {
        s[e] = (int64_t)(rng() % (uint64_t)n);
        d[e] = (rng() % 4 == 0) ? (int64_t)(rng() % 4) : (int64_t)(rng() % (uint64_t)n);
    }
}

}  // namespace

int main() {
    std::mt19937_64 rng(4404);
    std::vector<int64_t> s, d;
    edges(rng, 5000, 40000, s, d);
    gcn_graph_t full = nullptr;
    expect(gcn_subgraph_build(5000, s.data(), d.data(), (int64_t)s.size(), nullptr, 0, &full) ==
               GCN_OK,
           "full graph");
    for (int32_t workers : {1, 3, 6}) {
        gcn_rr_params p{2, 4, -1, 2, 0};
        gcn_pipeline_t pipe = nullptr;
        expect(gcn_pipeline_create(&p, 16, workers, 4, 0, nullptr, 0, &pipe) == GCN_OK,
               "create");
        if (!pipe) continue;
        const int jobs = 24;
        for (int j = 0; j < jobs; ++j) {
            int64_t id = -1;
            if (j % 3 == 2) {
                expect(gcn_pipeline_submit_sample(pipe, full, 40, 600, (uint64_t)(j + 1), 20000,
                                                  &id) == GCN_OK,
                       "submit_sample");
            } else {
                edges(rng, 700, 6000, s, d);
                expect(gcn_pipeline_submit(pipe, 700, s.data(), d.data(), (int64_t)s.size(),
                                           nullptr, 0, &id) == GCN_OK,
                       "submit");
            }
        }
        std::vector<int64_t> held;
        for (int j = 0; j < jobs; ++j) {
            int64_t id = -1;
            const void* img = nullptr;
            size_t bytes = 0;
            gcn_pipeline_info info;
            expect(gcn_pipeline_next(pipe, &id, &img, &bytes, &info) == GCN_OK, "next");
            expect(id == j && img != nullptr && bytes > 0, "next: order / image");
            held.push_back(id);
            if (held.size() >= 2) {
                expect(gcn_pipeline_release(pipe, held.front()) == GCN_OK, "release");
                held.erase(held.begin());
            }
        }
        for (int64_t id : held) expect(gcn_pipeline_release(pipe, id) == GCN_OK, "release");
        gcn_pipeline_destroy(pipe);
    }
    // destroyed while jobs are still queued and running
    {
        gcn_rr_params p{2, 3, -1, 1, 0};
        gcn_pipeline_t pipe = nullptr;
        expect(gcn_pipeline_create(&p, 0, 4, 2, 0, nullptr, 0, &pipe) == GCN_OK, "create");
        for (int j = 0; j < 10 && pipe; ++j) {
            edges(rng, 2000, 20000, s, d);
            expect(gcn_pipeline_submit(pipe, 2000, s.data(), d.data(), (int64_t)s.size(),
                                       nullptr, 0, nullptr) == GCN_OK,
                   "submit");
        }
        gcn_pipeline_destroy(pipe);
    }
    gcn_graph_free(full);
    std::printf("pipeline harness: %d failures\n", failures);
    return failures ? 1 : 0;
}
