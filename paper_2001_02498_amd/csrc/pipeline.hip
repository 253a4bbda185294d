// Host side of the per-minibatch schedule (Section 4.4): while the device
// trains on one subgraph, host threads prepare the next ones — subgraph
// construction (from an edge list, or by frontier sampling of a full graph
// and the induced subgraph, Section 3.1), redundancy reduction (Algorithms 1-3 in rounds, on the host
// or driven on the GPU from the worker's own stream) and packing of the
// device image into (optionally pinned) host memory — each worker on its
// own subgraph, since minibatches are independent. The consumer takes
// prepared images in submission order and uploads them itself.
#include <hip/hip_runtime.h>

#include <chrono>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "common.h"

using gcn::set_error;

namespace {

struct Buffer {
    void* ptr = nullptr;
    size_t cap = 0;
};

struct Job {
    int64_t id = 0;
    int64_t n_full = 0;
    std::vector<int64_t> src, dst, verts;
    bool has_verts = false;
    // sampled jobs: frontier sampling on a full graph the caller keeps alive
    gcn_graph_t full = nullptr;
    int32_t m = 0, budget = 0;
    uint64_t seed = 0;
    int64_t max_steps = 0;
    // results
    bool done = false;
    int status = GCN_OK;
    std::string error;
    Buffer buf;
    size_t bytes = 0;
    gcn_pipeline_info info{};
};

}  // namespace

struct gcn_pipeline {
    gcn_rr_params rr{};
    int32_t seg_len = 0;
    int32_t depth = 1;
    bool pinned = false;
    bool device_reduce = false;
    int device = 0;
    std::mutex mu;
    std::condition_variable cv_work, cv_done;
    std::deque<std::shared_ptr<Job>> todo;
    std::map<int64_t, std::shared_ptr<Job>> jobs;   // submitted, not released
    std::vector<Buffer> free_bufs;
    int64_t next_id = 0, next_pop = 0;
    int64_t prepared_unreleased = 0;                // started, not released
    int64_t held = 0;                               // taken by the caller, not released
    bool stop = false;
    std::vector<std::thread> workers;

    void alloc(Buffer& b, size_t bytes) {
        if (b.cap >= bytes) return;
        release_buffer(b);
        if (pinned) {
            if (hipHostMalloc(&b.ptr, bytes, hipHostMallocDefault) != hipSuccess) b.ptr = nullptr;
        } else {
            b.ptr = std::malloc(bytes);
        }
        b.cap = b.ptr ? bytes : 0;
    }
    void release_buffer(Buffer& b) {
        if (!b.ptr) return;
        if (pinned)
            (void)hipHostFree(b.ptr);
        else
            std::free(b.ptr);
        b.ptr = nullptr;
        b.cap = 0;
    }

    // caller-owned device workspace of the GPU-reducing workers, split
    // evenly between them (256-byte-aligned shares)
    char* dev_ws = nullptr;
    size_t dev_share = 0;

    // per-worker device state of the device reduction
    struct DevState {
        bool device = false;   // this worker reduces on the GPU
        hipStream_t stream = nullptr;
        void* ws = nullptr;
        size_t cap = 0;
    };

    void run(bool device_worker, int32_t index) {
        DevState ds;
        ds.device = device_worker;
        if (device_worker) {
            (void)hipSetDevice(device);
            if (hipStreamCreate(&ds.stream) != hipSuccess) ds.stream = nullptr;
            ds.ws = dev_ws + (size_t)index * dev_share;
            ds.cap = dev_share;
        }
        run_jobs(ds);
        if (ds.stream) (void)hipStreamDestroy(ds.stream);
    }

    // device reduction in the worker's share of the caller's workspace; a
    // job that needs more fails (nothing is allocated while jobs run)
    int reduce_on_device(gcn_graph_t g, DevState& ds, gcn_reduced_t* r) {
        if (!ds.stream) {
            set_error("gcn_pipeline: worker stream not created");
            return GCN_E_HIP;
        }
        size_t need = 0;
        int rc = gcn_redundancy_reduce_device_bytes(g, &rr, &need);
        if (rc) return rc;
        if (need > ds.cap) {
            set_error("gcn_pipeline: the device reduction needs %zu bytes, a worker's share of "
                      "the pipeline's device workspace is %zu",
                      need, ds.cap);
            return GCN_E_WORKSPACE;
        }
        return gcn_redundancy_reduce_device(g, &rr, ds.ws, ds.cap, ds.stream, r);
    }

    void run_jobs(DevState& ds) {
        for (;;) {
            std::shared_ptr<Job> job;
            Buffer buf;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv_work.wait(lk, [&] {
                    return stop || (!todo.empty() && prepared_unreleased < depth);
                });
                if (stop) return;
                job = todo.front();
                todo.pop_front();
                ++prepared_unreleased;
                if (!free_bufs.empty()) {
                    buf = free_bufs.back();
                    free_bufs.pop_back();
                }
            }
            prepare(*job, buf, ds);
            {
                std::lock_guard<std::mutex> lk(mu);
                job->done = true;
            }
            cv_done.notify_all();
        }
    }

    void prepare(Job& job, Buffer& buf, DevState& ds) {
        using clock = std::chrono::steady_clock;
        const auto t0 = clock::now();
        gcn_graph_t g = nullptr;
        gcn_reduced_t r = nullptr;
        int rc = GCN_OK;
        std::vector<int32_t> sampled;
        auto ts = t0;
        if (job.full) {
            // the walk, then the subgraph induced on its vertices
            int32_t count = 0;
            int64_t steps = 0;
            try {
                sampled.resize((size_t)job.budget);
            } catch (const std::bad_alloc&) {
                set_error("gcn_pipeline: out of host memory");
                rc = GCN_E_OOM;
            }
            if (rc == GCN_OK)
                rc = gcn_sample_frontier(job.full, job.m, job.budget, job.seed, job.max_steps,
                                         sampled.data(), &count, &steps);
            sampled.resize(rc == GCN_OK ? (size_t)count : 0);
            job.info.steps = steps;
            ts = clock::now();
            if (rc == GCN_OK) rc = gcn_subgraph_induce(job.full, sampled.data(), count, &g);
        } else {
            rc = gcn_subgraph_build(job.n_full, job.src.data(), job.dst.data(),
                                    (int64_t)job.src.size(),
                                    job.has_verts ? job.verts.data() : nullptr,
                                    (int64_t)job.verts.size(), &g);
        }
        const auto t1 = clock::now();
        if (rc == GCN_OK)
            rc = ds.device ? reduce_on_device(g, ds, &r) : gcn_redundancy_reduce(g, &rr, &r);
        const auto t2 = clock::now();
        size_t img = 0, bytes = 0;
        if (rc == GCN_OK) rc = gcn_graph_image_bytes(r, seg_len, &img);
        // a sampled job's vertex ids follow the image (256-byte aligned), so
        // one copy moves both
        const size_t voff = job.full ? (size_t)gcn::round_up((int64_t)img, 256) : img;
        bytes = voff + sizeof(int32_t) * sampled.size();
        if (rc == GCN_OK) {
            alloc(buf, bytes);
            if (!buf.ptr) {
                set_error("gcn_pipeline: host buffer of %zu bytes not allocated", bytes);
                rc = GCN_E_OOM;
            }
        }
        if (rc == GCN_OK) rc = gcn_graph_pack(r, seg_len, buf.ptr, img);
        if (rc == GCN_OK && job.full) {
            std::memset(static_cast<char*>(buf.ptr) + img, 0, voff - img);
            if (!sampled.empty())
                std::memcpy(static_cast<char*>(buf.ptr) + voff, sampled.data(),
                            sizeof(int32_t) * sampled.size());
        }
        job.info.image_bytes = (int64_t)img;
        job.info.vertices_offset = job.full ? (int64_t)voff : -1;
        const auto t3 = clock::now();
        if (rc == GCN_OK) {
            int32_t n = 0, naux = 0, rounds = 0;
            int64_t nnz = 0;
            gcn_reduced_info(r, &n, &naux, &rounds, &nnz, nullptr, nullptr, nullptr, nullptr,
                             nullptr, nullptr);
            job.info.n = n;
            job.info.naux = naux;
            job.info.rounds = rounds;
            job.info.nnz = nnz;
            int32_t gn = 0;
            int64_t gnnz = 0;
            gcn_graph_info(g, &gn, &gnnz, nullptr, nullptr);
            job.info.nnz_direct = gnnz;
        }
        auto ms = [](auto a, auto b) {
            return std::chrono::duration<double, std::milli>(b - a).count();
        };
        job.info.sample_ms = ms(t0, ts);
        job.info.build_ms = ms(ts, t1);
        job.info.reduce_ms = ms(t1, t2);
        job.info.pack_ms = ms(t2, t3);
        job.status = rc;
        if (rc != GCN_OK) job.error = gcn_last_error();
        job.buf = buf;
        job.bytes = rc == GCN_OK ? bytes : 0;
        gcn_graph_free(g);
        gcn_reduced_free(r);
        // the edge lists are no longer needed
        std::vector<int64_t>().swap(job.src);
        std::vector<int64_t>().swap(job.dst);
        std::vector<int64_t>().swap(job.verts);
    }
};

extern "C" {

int gcn_pipeline_create_mixed(const gcn_rr_params* params, int32_t seg_len,
                              int32_t host_workers, int32_t device_workers, int32_t depth,
                              int32_t flags, void* dev_ws, size_t dev_ws_bytes,
                              gcn_pipeline_t* out) {
    GCN_CHECK_ARG(params && out, "gcn_pipeline_create: NULL argument");
    GCN_CHECK_ARG(host_workers >= 0 && device_workers >= 0 &&
                      host_workers + device_workers >= 1 && host_workers + device_workers <= 256,
                  "gcn_pipeline_create: workers outside [1, 256]");
    GCN_CHECK_ARG(depth >= 1 && depth <= 4096, "gcn_pipeline_create: depth outside [1, 4096]");
    GCN_CHECK_ARG(params->theta >= 0 && params->max_rounds >= 0 &&
                      params->max_rounds <= GCN_MAX_ROUNDS && params->num_threads >= 0,
                  "gcn_pipeline_create: bad reduction parameters");
    GCN_CHECK_ARG(seg_len == 0 || (seg_len >= 1 && seg_len <= 65536),
                  "gcn_pipeline_create: seg_len outside [1, 65536]");
    GCN_CHECK_ARG((flags & ~GCN_PIPE_PINNED) == 0, "gcn_pipeline_create: unknown flags 0x%x",
                  flags);
    const size_t share =
        device_workers > 0 ? dev_ws_bytes / (size_t)device_workers / 256 * 256 : 0;
    GCN_CHECK_ARG(device_workers == 0 ||
                      (dev_ws != nullptr && ((uintptr_t)dev_ws & 255) == 0 && share > 0),
                  "gcn_pipeline_create: GPU-reducing workers need a 256-byte-aligned device "
                  "workspace of at least 256 bytes each");
    try {
        auto* p = new gcn_pipeline;
        p->rr = *params;
        p->seg_len = seg_len;
        p->depth = depth;
        p->pinned = (flags & GCN_PIPE_PINNED) != 0;
        p->device_reduce = device_workers > 0;
        p->dev_ws = static_cast<char*>(dev_ws);
        p->dev_share = share;
        if (p->device_reduce && hipGetDevice(&p->device) != hipSuccess) {
            delete p;
            set_error("gcn_pipeline_create: no current GPU for the device reduction");
            return GCN_E_HIP;
        }
        for (int32_t i = 0; i < device_workers; ++i)
            p->workers.emplace_back([p, i] { p->run(true, i); });
        for (int32_t i = 0; i < host_workers; ++i)
            p->workers.emplace_back([p, i] { p->run(false, i); });
        *out = p;
        return GCN_OK;
    } catch (const std::exception& e) {
        set_error("gcn_pipeline_create: %s", e.what());
        return GCN_E_OOM;
    }
}

int gcn_pipeline_create(const gcn_rr_params* params, int32_t seg_len, int32_t workers,
                        int32_t depth, int32_t flags, void* dev_ws, size_t dev_ws_bytes,
                        gcn_pipeline_t* out) {
    GCN_CHECK_ARG((flags & ~(GCN_PIPE_PINNED | GCN_PIPE_DEVICE_REDUCE)) == 0,
                  "gcn_pipeline_create: unknown flags 0x%x", flags);
    GCN_CHECK_ARG(workers >= 1 && workers <= 256, "gcn_pipeline_create: workers outside [1, 256]");
    const bool dev = (flags & GCN_PIPE_DEVICE_REDUCE) != 0;
    return gcn_pipeline_create_mixed(params, seg_len, dev ? 0 : workers, dev ? workers : 0, depth,
                                     flags & GCN_PIPE_PINNED, dev_ws, dev_ws_bytes, out);
}

int gcn_pipeline_submit(gcn_pipeline_t p, int64_t n_full, const int64_t* src,
                        const int64_t* dst, int64_t n_edges, const int64_t* vertices,
                        int64_t n_vertices, int64_t* job_id) {
    GCN_CHECK_ARG(p != nullptr, "gcn_pipeline_submit: NULL pipeline");
    GCN_CHECK_ARG(n_edges >= 0 && (n_edges == 0 || (src && dst)),
                  "gcn_pipeline_submit: bad edge arrays");
    GCN_CHECK_ARG(vertices == nullptr || n_vertices >= 0, "gcn_pipeline_submit: bad subset");
    try {
        auto job = std::make_shared<Job>();
        job->n_full = n_full;
        job->src.assign(src, src + n_edges);
        job->dst.assign(dst, dst + n_edges);
        if (vertices) {
            job->has_verts = true;
            job->verts.assign(vertices, vertices + n_vertices);
        }
        {
            std::lock_guard<std::mutex> lk(p->mu);
            job->id = p->next_id++;
            p->jobs[job->id] = job;
            p->todo.push_back(job);
            if (job_id) *job_id = job->id;
        }
        p->cv_work.notify_one();
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_pipeline_submit: out of host memory");
        return GCN_E_OOM;
    }
}

int gcn_pipeline_submit_sample(gcn_pipeline_t p, gcn_graph_t full, int32_t m,
                               int32_t budget, uint64_t seed, int64_t max_steps,
                               int64_t* job_id) {
    GCN_CHECK_ARG(p && full, "gcn_pipeline_submit_sample: NULL argument");
    int32_t n = 0;
    int64_t nnz = 0;
    if (int rc = gcn_graph_info(full, &n, &nnz, nullptr, nullptr)) return rc;
    GCN_CHECK_ARG(m >= 1 && m <= budget && budget <= n,
                  "gcn_pipeline_submit_sample: need 1 <= m (%d) <= budget (%d) <= n (%d)", m,
                  budget, n);
    GCN_CHECK_ARG(max_steps >= 0, "gcn_pipeline_submit_sample: negative max_steps");
    try {
        auto job = std::make_shared<Job>();
        job->full = full;
        job->m = m;
        job->budget = budget;
        job->seed = seed;
        job->max_steps = max_steps;
        {
            std::lock_guard<std::mutex> lk(p->mu);
            job->id = p->next_id++;
            p->jobs[job->id] = job;
            p->todo.push_back(job);
            if (job_id) *job_id = job->id;
        }
        p->cv_work.notify_one();
        return GCN_OK;
    } catch (const std::bad_alloc&) {
        set_error("gcn_pipeline_submit_sample: out of host memory");
        return GCN_E_OOM;
    }
}

int gcn_pipeline_next(gcn_pipeline_t p, int64_t* job_id, const void** image, size_t* bytes,
                      gcn_pipeline_info* info) {
    GCN_CHECK_ARG(p && job_id && image && bytes, "gcn_pipeline_next: NULL argument");
    std::shared_ptr<Job> job;
    {
        std::unique_lock<std::mutex> lk(p->mu);
        GCN_CHECK_ARG(p->next_pop < p->next_id, "gcn_pipeline_next: nothing submitted");
        auto it = p->jobs.find(p->next_pop);
        GCN_CHECK_ARG(it != p->jobs.end(), "gcn_pipeline_next: job already released");
        GCN_CHECK_ARG(p->held < p->depth,
                      "gcn_pipeline_next: %lld jobs held (depth %d): release one first",
                      (long long)p->held, p->depth);
        job = it->second;
        // Jobs start in submission order and fewer than `depth` are held, so
        // this job is running, done, or next to start: the wait ends.
        p->cv_done.wait(lk, [&] { return job->done; });
        ++p->next_pop;
        ++p->held;
    }
    *job_id = job->id;
    *image = job->buf.ptr;
    *bytes = job->bytes;
    if (info) *info = job->info;
    if (job->status != GCN_OK) {
        set_error("gcn_pipeline_next: job %lld: %s", (long long)job->id, job->error.c_str());
        return job->status;
    }
    return GCN_OK;
}

int gcn_pipeline_release(gcn_pipeline_t p, int64_t job_id) {
    GCN_CHECK_ARG(p != nullptr, "gcn_pipeline_release: NULL pipeline");
    {
        std::lock_guard<std::mutex> lk(p->mu);
        auto it = p->jobs.find(job_id);
        GCN_CHECK_ARG(it != p->jobs.end() && it->second->done && job_id < p->next_pop,
                      "gcn_pipeline_release: job %lld not taken or already released",
                      (long long)job_id);
        if (it->second->buf.ptr) p->free_bufs.push_back(it->second->buf);
        p->jobs.erase(it);
        --p->prepared_unreleased;
        --p->held;
    }
    p->cv_work.notify_all();
    return GCN_OK;
}

void gcn_pipeline_destroy(gcn_pipeline_t p) {
    if (!p) return;
    {
        std::lock_guard<std::mutex> lk(p->mu);
        p->stop = true;
    }
    p->cv_work.notify_all();
    for (auto& t : p->workers) t.join();
    for (auto& kv : p->jobs) p->release_buffer(kv.second->buf);
    for (auto& b : p->free_bufs) p->release_buffer(b);
    delete p;
}

}  // extern "C"
