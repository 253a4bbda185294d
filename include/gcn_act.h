/*
 * gcn_act.h - C ABI of the MI355X subgraph GCN training hot path.
 *
 * Method: GraphACT (Zeng & Prasanna, FPGA '20). A minibatch is a subgraph
 * G_s induced on sampled vertices (Section 3.1); every layer aggregates
 * neighbour features with D^-1 A and transforms them with two weight
 * matrices (Eq. 1); gradients follow Eq. 2a-2c; the aggregation may run on
 * the redundancy-reduced graph G_s^# whose extra vertices are pre-computed
 * sums of neighbour pairs (Section 3.2, Algorithms 1-3; Section 4.2).
 *
 * Conventions (every entry point):
 *   - Returns GCN_OK (0) or a negative status; gcn_last_error() gives a
 *     thread-local message for the last failing call on this thread.
 *   - All arguments are validated before anything is enqueued; on error no
 *     device work is launched and no output is touched.
 *   - Host objects (gcn_graph_t, gcn_reduced_t) are created and freed by the
 *     library. Calls on distinct objects may run concurrently from different
 *     threads.
 *   - Device buffers are caller-owned. Dense matrices are row-major float32
 *     with an explicit leading dimension ld (in elements): ld >= width,
 *     ld % 4 == 0, base pointer 16-byte aligned. Weight matrices are dense
 *     with ld == width. The library never allocates device memory: scratch
 *     space is the caller's `ws` buffer (256-byte aligned) of `ws_bytes`
 *     (gcn_aggregate_noalloc alone uses a fixed array per device that the
 *     loaded library holds).
 *   - Device entry points take a stream (a hipStream_t passed as void*; NULL
 *     is the null stream), only enqueue work on it, never synchronise, and
 *     return before the work completes.
 *   - Vertex indices are int32; sizes that can exceed 2^31 are int64.
 *   - Columns of an output beyond its logical width are never written.
 */
#ifndef GCN_ACT_H
#define GCN_ACT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status */
#define GCN_OK              0
#define GCN_E_INVALID_ARG  (-1)  /* bad pointer, size, layout or graph     */
#define GCN_E_HIP          (-2)  /* a HIP runtime call failed              */
#define GCN_E_OOM          (-3)  /* host allocation failed                 */
#define GCN_E_UNSUPPORTED  (-4)  /* valid request this build cannot serve  */
#define GCN_E_WORKSPACE    (-5)  /* ws_bytes below the required size       */
#define GCN_E_INTERNAL     (-6)
#define GCN_E_NONFINITE    (-7)  /* the loss of a call was inf or NaN      */

#define GCN_MAX_ROUNDS 64
#define GCN_MAX_LAYERS 8
#define GCN_BIN_GROUPS 16        /* pieces per work-list bin (see image)  */

#define GCN_LOSS_SOFTMAX_CE 0    /* labels: int32[n] class ids            */
#define GCN_LOSS_SIGMOID_BCE 1   /* labels: uint8[n*C] 0/1, row-major     */

#define GCN_PREC_FP32 0          /* fp32 MFMA for the dense products      */
#define GCN_PREC_BF16 1          /* bf16 MFMA operands, fp32 accumulation */

#define GCN_AGG_MEAN 0           /* Y = D^-1 A X        (forward, Eq. 1)   */
#define GCN_AGG_TRANSPOSED 1     /* Y = A D^-1 X        (backward, Eq. 2c) */

typedef void* gcn_stream_t;      /* hipStream_t */

/* Message of the last failing call on this thread ("" if none). */
const char* gcn_last_error(void);

/* ABI version of this header (bumped on incompatible change). */
int gcn_abi_version(void);
#define GCN_ABI_VERSION 7

/* ------------------------------------------------ subgraph (host, a1)
 * gcn_subgraph_build - undirected simple subgraph in CSR form.
 * Section 2.1: the input graph is undirected, A is its 0/1 adjacency and D
 * the diagonal degree matrix. Section 3.1: a minibatch is the subgraph
 * induced on a vertex subset, used by every layer.
 *   n_full      vertices of the full graph (ids 0..n_full-1), < 2^31
 *   src,dst     host int64[n_edges]; edge i joins src[i] and dst[i], either
 *               direction; repeats and self-loops are allowed and dropped
 *   vertices    host int64[n_vertices] subset (vertex vertices[k] becomes k)
 *               or NULL for all n_full vertices
 *   out         receives a new graph; free with gcn_graph_free
 * Errors: GCN_E_INVALID_ARG for out-of-range or repeated ids, negative
 * sizes or NULL pointers with nonzero sizes; GCN_E_OOM.
 */
typedef struct gcn_graph* gcn_graph_t;
int gcn_subgraph_build(int64_t n_full, const int64_t* src, const int64_t* dst,
                       int64_t n_edges, const int64_t* vertices,
                       int64_t n_vertices, gcn_graph_t* out);

/* Borrowed views (valid until gcn_graph_free): rowptr int32[n+1], col
 * int32[nnz], each row sorted ascending, symmetric, no self-loops. */
int gcn_graph_info(gcn_graph_t g, int32_t* n, int64_t* nnz,
                   const int32_t** rowptr, const int32_t** col);
void gcn_graph_free(gcn_graph_t g);

/* ------------------------------------------ minibatch sampling (host)
 * gcn_sample_frontier - the vertex set of one minibatch, drawn from the full
 * training graph by frontier sampling. Section 3.1 forms a minibatch as the
 * subgraph induced on vertices that a graph sampler draws from the training
 * graph, and names the multi-dimensional random walk of the cited work
 * (Ribeiro and Towsley, IMC 2010) as such a sampler. As run here:
 *   1. a frontier of m distinct vertices is drawn uniformly (a draw that
 *      repeats a taken vertex is dropped and drawn again); they are sampled;
 *   2. each step picks frontier slot s with probability deg(u_s) / (sum of
 *      the frontier's degrees) - the first slot whose running degree sum
 *      exceeds a uniform draw r in [0, sum) - moves along a uniformly chosen
 *      edge (u_s, v), puts v in slot s and samples v;
 *   3. it stops once `budget` distinct vertices are sampled, after
 *      max_steps steps, or when every frontier vertex is isolated.
 * Random numbers: SplitMix64 of `seed` (Steele, Lea and Flood, OOPSLA
 * 2014) as a counter-based generator, output i = mix(seed + (i+1) *
 * 0x9E3779B97F4A7C15); a draw in [0, b) is the high 64 bits of output * b;
 * outputs are used in the order: the initial frontier's draws, then per step
 * the slot draw and the edge draw.
 *   full       graph from gcn_subgraph_build (vertices = NULL); read only,
 *              so concurrent calls on one graph are safe
 *   m, budget  1 <= m <= budget <= n of `full`
 *   max_steps  >= 0
 *   vertices   host int32[budget]: receives the sampled ids, ascending
 *   n_out      receives their count (budget unless the walk stopped early)
 *   steps_out  NULL, or receives the number of steps taken
 * Errors: GCN_E_INVALID_ARG (NULL, sizes as above); GCN_E_OOM.
 */
int gcn_sample_frontier(gcn_graph_t full, int32_t m, int32_t budget, uint64_t seed,
                        int64_t max_steps, int32_t* vertices, int32_t* n_out,
                        int64_t* steps_out);

/* gcn_subgraph_induce - the subgraph of `full` induced on a vertex subset
 * (Section 3.1): vertex vertices[k] becomes k, an edge is kept when both
 * ends are in the subset, lists sorted. The same graph as gcn_subgraph_build
 * on the full graph's edges with this subset, in time proportional to the
 * subset's degree sum.
 *   vertices   host int32[n_vertices], distinct, each in [0, n of full)
 *   out        receives a new graph; free with gcn_graph_free
 * Errors: GCN_E_INVALID_ARG (NULL, out-of-range or repeated id); GCN_E_OOM.
 */
int gcn_subgraph_induce(gcn_graph_t full, const int32_t* vertices, int32_t n_vertices,
                        gcn_graph_t* out);

/* gcn_gather_rows - rows of the full graph's arrays for the minibatch's
 * vertices (Section 4.1: the accelerator receives the input features of the
 * minibatch's vertices; their labels likewise): dst row k = src row idx[k].
 *   src       device, rows of row_bytes bytes at a stride of ld_src bytes,
 *             n_src rows
 *   idx       device int32[n]
 *   dst       device, n rows at a stride of ld_dst bytes; bytes of a row
 *             beyond row_bytes are never written
 * Rows whose idx lies outside [0, n_src) are not written. 16-byte copies
 * when both pointers, both strides and row_bytes are multiples of 16, else
 * 4-byte copies when they are multiples of 4, else single bytes.
 * Errors: GCN_E_INVALID_ARG (NULL with n > 0, negative sizes, row_bytes
 * above a stride); GCN_E_HIP.
 */
int gcn_gather_rows(const void* src, int64_t ld_src, int64_t n_src, const int32_t* idx,
                    int32_t n, int64_t row_bytes, void* dst, int64_t ld_dst,
                    gcn_stream_t stream);

/* ------------------------------------- redundancy reduction (host, a2)
 * gcn_redundancy_reduce - rounds of Algorithms 1-3 (Section 3.2).
 * Each round counts, for every pair of vertices, the neighbour lists that
 * hold both (Alg. 1); takes pairs greedily by decreasing count while the
 * count exceeds theta, skipping pairs with an endpoint already taken
 * (Alg. 2; equal counts in ascending (smaller id, larger id) order); gives
 * the k-th taken pair of the round the id n + (pairs of earlier rounds) + k
 * and replaces the pair by that id in every list holding both (Alg. 3);
 * lists stay sorted. Rounds stop at max_rounds, at an empty matching, or
 * when max_aux new vertices exist (a pair is taken only while the total is
 * below max_aux; < 0 means no cap). max_rounds == 0 gives the input graph
 * unchanged (direct aggregation).
 *   num_threads  host threads for the pair counting (0: all hardware
 *                threads, capped at 64); results do not depend on it
 * Errors: GCN_E_INVALID_ARG (theta < 0, max_rounds outside
 * [0, GCN_MAX_ROUNDS], NULL); GCN_E_OOM.
 */
typedef struct {
    int32_t theta;        /* default 2 */
    int32_t max_rounds;   /* default 5 */
    int64_t max_aux;      /* default -1 (no cap) */
    int32_t num_threads;  /* default 0 */
    int32_t reserved;
} gcn_rr_params;

typedef struct {
    int64_t matched;      /* |M| of the round                        */
    int64_t weight_sum;   /* sum of the taken pairs' counts          */
    int64_t nnz;          /* numRead of the lists after the round    */
    int64_t num_add;      /* numAdd of the lists after the round     */
} gcn_rr_round;

typedef struct gcn_reduced* gcn_reduced_t;
int gcn_redundancy_reduce(gcn_graph_t g, const gcn_rr_params* params,
                          gcn_reduced_t* out);

/* Borrowed views (valid until gcn_reduced_free):
 *   rowptr int32[n+1], col int32[nnz]  lists of G_s^# for the n original
 *                     vertices; ids >= n name pair sums
 *   pairs  int32[naux*2]  pair k = (pairs[2k], pairs[2k+1]), smaller first;
 *                     its sum is vertex n+k
 *   round_offsets int32[rounds+1]; per_round gcn_rr_round[rounds]
 *   deg    int32[n]   degrees of the ORIGINAL subgraph (D of Eq. 1)      */
int gcn_reduced_info(gcn_reduced_t r, int32_t* n, int32_t* naux,
                     int32_t* rounds, int64_t* nnz, const int32_t** rowptr,
                     const int32_t** col, const int32_t** pairs,
                     const int32_t** round_offsets,
                     const gcn_rr_round** per_round, const int32_t** deg);
void gcn_reduced_free(gcn_reduced_t r);

/* ----------------------------- redundancy reduction on the device (a2)
 * gcn_redundancy_reduce_device - the same rounds of Algorithms 1-3
 * (Section 3.2) run on the GPU; the result object is identical, field by
 * field, to what gcn_redundancy_reduce returns for the same graph and
 * parameters (the same pairs, ids, lists and per-round counts). Per round:
 * the pair counts of Algorithm 1 per vertex in LDS counters; the pairs
 * above theta sorted by (count descending, smaller id, larger id); the
 * greedy scan of Algorithm 2 under the max_aux cap; the list rewrite of
 * Algorithm 3, one workgroup per list. Synchronous: uploads the lists,
 * runs on `stream` (synchronising it twice per round to size the next
 * launches), downloads the result, and returns.
 *   ws, ws_bytes  device workspace, 256-byte aligned, of at least
 *                 gcn_redundancy_reduce_device_bytes(g, params) bytes;
 *                 caller-owned, reusable once the call returned
 *   num_threads   ignored
 * Limits: fewer than 524288 (2^19) vertex ids (original plus pair sums)
 * in any round, and pair counts below 65536 (GCN_E_UNSUPPORTED beyond;
 * the host reduction has neither limit).
 * Errors: GCN_E_INVALID_ARG (as gcn_redundancy_reduce, or a NULL /
 * misaligned workspace); GCN_E_WORKSPACE; GCN_E_UNSUPPORTED; GCN_E_HIP;
 * GCN_E_INTERNAL (a device-side capacity or range check failed); GCN_E_OOM.
 */
int gcn_redundancy_reduce_device_bytes(gcn_graph_t g, const gcn_rr_params* params,
                                       size_t* bytes);
int gcn_redundancy_reduce_device(gcn_graph_t g, const gcn_rr_params* params, void* ws,
                                 size_t ws_bytes, gcn_stream_t stream, gcn_reduced_t* out);

/* ------------------------------------------------ device graph image
 * The device form of G_s^# (what the accelerator receives in Section 4.1:
 * the lists, the pairs and D), plus a work list that splits long lists
 * into pieces of at most `seg_len` entries for load balance, and each pair
 * sum's expansion into original vertices (the pair sum of Section 4.2 step 1
 * is the sum of those rows), so that all pair sums of all rounds can be
 * formed in one pass instead of one dependent pass per round.
 * Work list: `seg` holds nseg pieces (row, begin, end, lead) into col, with
 * lead = the row's piece count on its first piece and 0 on the others; a
 * row of at most seg_len entries is one piece (lead 1). `bins` (nbins + 1
 * ascending piece offsets) cuts it into bins of at most GCN_BIN_GROUPS
 * pieces, or one bin for a single row of more pieces (a hub); every row's
 * pieces are consecutive and in one bin, the nhub hub bins come first, then
 * the other bins holding a split row (nmulti bins in all), so the pieces of
 * a split row are added within one workgroup (a hub's list within each of
 * the workgroups that share its columns).
 * gcn_graph_image_bytes - size of the packed image (host and device).
 * gcn_graph_pack        - write the image into a caller host buffer (may
 *                         be pinned); the reduced object may then be freed.
 * gcn_graph_upload      - copy `bytes` bytes from host_image (the image
 *                         and anything the caller placed after it, such as
 *                         a sampled pipeline job's vertex ids) to a caller
 *                         device buffer of at least `bytes` bytes on
 *                         `stream` (hipMemcpyAsync; the host buffer must
 *                         stay valid until the copy completes) and fill the
 *                         descriptor, whose pointers are into dev_buf.
 * seg_len: 0 selects the default (32); otherwise 1..65536.
 */
typedef struct {
    int32_t n, naux, rounds, seg_len;
    int32_t nseg, nbins, nmulti, nhub;
    int32_t max_row, reserved;
    int64_t nnz;
    int64_t exp_nnz;           /* total expansion length             */
    const int32_t* rowptr;     /* device int32[n+1]                  */
    const int32_t* col;        /* device int32[nnz]                  */
    const int32_t* pairs;      /* device int32[2*naux]               */
    const float* inv_deg;      /* device float[n], 1/d (0 if d == 0) */
    const int32_t* seg;        /* device int32[4*nseg]               */
    const int32_t* bins;       /* device int32[nbins+1]              */
    const int32_t* exp_col;    /* device int32[exp_nnz]: original
                                  vertices of pair sum k, ascending  */
    const int32_t* exp_seg;    /* device int32[4*naux]: (k, begin,
                                  end, -1) into exp_col, longest
                                  expansion first                    */
    int32_t round_offsets[GCN_MAX_ROUNDS + 1];   /* host copy        */
} gcn_dgraph;

int gcn_graph_image_bytes(gcn_reduced_t r, int32_t seg_len, size_t* bytes);
int gcn_graph_pack(gcn_reduced_t r, int32_t seg_len, void* host_buf,
                   size_t bytes);
int gcn_graph_upload(const void* host_image, size_t bytes, void* dev_buf,
                     gcn_dgraph* out, gcn_stream_t stream);
/* Fill the descriptor for an image already resident at dev_buf (host_image
 * is the same image's host copy; nothing is copied). */
int gcn_graph_describe(const void* host_image, size_t bytes,
                       const void* dev_buf, gcn_dgraph* out);

/* ---------------------------------------- host preparation pipeline (a13)
 * Section 4.4: subgraphs are independent, so while the device trains on one
 * minibatch the host prepares the next ones, several at once. A pipeline
 * owns `workers` host threads; each submitted subgraph is built
 * (gcn_subgraph_build), reduced (gcn_redundancy_reduce with `params`) and
 * packed (gcn_graph_pack) into a host buffer (page-locked with
 * GCN_PIPE_PINNED, so uploads are asynchronous DMA). Results come back in
 * submission order.
 *   flags  GCN_PIPE_PINNED: page-locked image buffers.
 *          GCN_PIPE_DEVICE_REDUCE: each worker reduces on the GPU that is
 *          current when the pipeline is created
 *          (gcn_redundancy_reduce_device, same result), on a stream of its
 *          own (default priority), in its share of dev_ws.
 *   dev_ws, dev_ws_bytes  device workspace of the GPU-reducing workers,
 *          caller-owned, 256-byte aligned, kept alive until destroy: split
 *          evenly between them (256-byte-aligned shares). Size it up front
 *          from gcn_redundancy_reduce_device_bytes of the largest subgraph
 *          to be submitted: a job needing more than a share fails with
 *          GCN_E_WORKSPACE (from gcn_pipeline_next); nothing is allocated
 *          or freed on the device while jobs run. NULL, 0 without
 *          GPU-reducing workers.
 * gcn_pipeline_submit - copies the edge arrays (the caller may free them on
 *   return) and queues the job; *job_id receives its number (0, 1, ...).
 * gcn_pipeline_submit_sample - queues a job that samples its vertex set
 *   from `full` (gcn_sample_frontier with these arguments) and induces the
 *   subgraph on it (gcn_subgraph_induce) before the reduction and packing.
 *   `full` is borrowed: keep it alive until the job has been taken. The
 *   job's buffer holds the image and, at info.vertices_offset, the sampled
 *   ids (the induced subgraph's vertex k is the k-th), and `bytes` from
 *   gcn_pipeline_next covers both, so one copy uploads them together.
 * gcn_pipeline_next - waits for the oldest job not yet taken and returns its
 *   image (valid until gcn_pipeline_release) and timings. A failed job
 *   returns its error code (the pipeline keeps going). At most `depth` jobs
 *   are prepared ahead or held by the caller: release taken jobs to let the
 *   workers continue; taking a job while holding `depth` others returns
 *   GCN_E_INVALID_ARG instead of waiting forever.
 * gcn_pipeline_release - returns a taken job's buffer to the pool (after any
 *   asynchronous copy from it has completed).
 * gcn_pipeline_destroy - stops the workers (after their current job) and
 *   frees every buffer.
 */
typedef struct gcn_pipeline* gcn_pipeline_t;
typedef struct {
    int32_t n, naux, rounds, reserved;
    int64_t nnz;          /* list entries of G_s^#     */
    int64_t nnz_direct;   /* list entries of G_s       */
    double build_ms, reduce_ms, pack_ms;   /* wall time of this job's steps */
    double sample_ms;     /* sampled jobs: the walk (0 otherwise)         */
    int64_t image_bytes;  /* the graph image, at the buffer's start       */
    int64_t vertices_offset;  /* sampled jobs: byte offset of the sampled
                             ids, int32[n] ascending, in the buffer (a
                             multiple of 256); -1 otherwise              */
    int64_t steps;        /* sampled jobs: walk steps taken               */
} gcn_pipeline_info;

#define GCN_PIPE_PINNED 1
#define GCN_PIPE_DEVICE_REDUCE 2
int gcn_pipeline_create(const gcn_rr_params* params, int32_t seg_len,
                        int32_t workers, int32_t depth, int32_t flags,
                        void* dev_ws, size_t dev_ws_bytes, gcn_pipeline_t* out);
/* gcn_pipeline_create_mixed - the same pipeline with host_workers reducing
 * on the host and device_workers on the GPU (as GCN_PIPE_DEVICE_REDUCE);
 * every job goes to whichever worker is free, and since both reductions give
 * the same result, so do the jobs. flags: GCN_PIPE_PINNED only.
 * Errors: GCN_E_INVALID_ARG (no worker, more than 256, other flags); as
 * gcn_pipeline_create otherwise. */
int gcn_pipeline_create_mixed(const gcn_rr_params* params, int32_t seg_len,
                              int32_t host_workers, int32_t device_workers, int32_t depth,
                              int32_t flags, void* dev_ws, size_t dev_ws_bytes,
                              gcn_pipeline_t* out);
int gcn_pipeline_submit(gcn_pipeline_t p, int64_t n_full, const int64_t* src,
                        const int64_t* dst, int64_t n_edges,
                        const int64_t* vertices, int64_t n_vertices,
                        int64_t* job_id);
int gcn_pipeline_submit_sample(gcn_pipeline_t p, gcn_graph_t full, int32_t m,
                               int32_t budget, uint64_t seed, int64_t max_steps,
                               int64_t* job_id);
int gcn_pipeline_next(gcn_pipeline_t p, int64_t* job_id, const void** image,
                      size_t* bytes, gcn_pipeline_info* info);
int gcn_pipeline_release(gcn_pipeline_t p, int64_t job_id);
void gcn_pipeline_destroy(gcn_pipeline_t p);

/* ------------------------------------------------------- scratch size
 * Bytes of `ws` needed by gcn_aggregate / gcn_layer_fwd / gcn_layer_bwd /
 * gcn_classifier_* / gcn_loss for widths up to max_width and row count of
 * the graph (g may be NULL for the classifier and loss alone, then n is
 * taken from `n`). */
int gcn_scratch_bytes(const gcn_dgraph* g, int32_t n, int32_t max_width,
                      size_t* bytes);

/* ---------------------------------------------- aggregation (a3 a4 a10)
 * gcn_aggregate - Y = D^-1 A X (GCN_AGG_MEAN, forward aggregation of Eq. 1)
 * or Y = A D^-1 X (GCN_AGG_TRANSPOSED, the aggregation inside Eq. 2c), run
 * on G_s^#: the pair sums of every round are formed first (Section 4.2 step
 * 1; each from its expansion into original rows, in one pass), then the
 * lists are summed (step 2) and scaled by the original 1/d (step 3, after
 * the sum for MEAN; on the gathered original rows for TRANSPOSED).
 * Vertices with d == 0 get zero rows.
 *   X  device [n x F] ld ldx;  Y  device [n x F] ld ldy (X and Y must not
 *   overlap). Scratch: the pair sums. A split list's pieces are added in
 *   one workgroup, in a fixed order, so results do not vary from run to run.
 */
int gcn_aggregate(const gcn_dgraph* g, int32_t mode, int32_t F,
                  const float* X, int64_t ldx, float* Y, int64_t ldy,
                  void* ws, size_t ws_bytes, gcn_stream_t stream);

/* gcn_aggregate_noalloc - gcn_aggregate without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation). Same operation,
 * kernels and results as gcn_aggregate. Its scratch (the pair sums, each
 * written before it is read) is a fixed array of
 * GCN_AGG_NOALLOC_SCRATCH_BYTES per device, held by the library on every
 * device it runs on until the process ends; its device address is looked
 * up (hipGetSymbolAddress) on the first call on each device, the only
 * call that may touch the runtime beyond launches. Calls allocate nothing.
 * Every call on one device shares that device's array: calls that overlap
 * on one device (concurrent streams or threads) race and give wrong
 * results; serialise them. Errors: GCN_E_INVALID_ARG as gcn_aggregate,
 * and when the scratch needed, 4 r4(F) naux bytes in 256-byte-aligned
 * regions, exceeds the fixed size (nothing launched);
 * GCN_E_HIP if the address lookup or a launch fails. */
#define GCN_AGG_NOALLOC_SCRATCH_BYTES (64ll << 20)
int gcn_aggregate_noalloc(const gcn_dgraph* g, int32_t mode, int32_t F,
                          const float* X, int64_t ldx, float* Y, int64_t ldy,
                          gcn_stream_t stream);

/* ------------------------------------------------- layer forward (a3-a5)
 * gcn_layer_fwd - one graph convolutional layer, Eq. 1:
 *   AH    = D^-1 A H_in                         (saved for Eq. 2b)
 *   H_out = ReLU( H_in W_self | AH W_neigh  (+ bias) )
 *   H_in  [n x F] ld ld_in;  W_self, W_neigh [F x h];  bias [2h] or NULL
 *   AH    [n x F] ld ld_ah;  H_out [n x 2h] ld ld_out (self half first)
 *   precision GCN_PREC_FP32, or GCN_PREC_BF16: operands of every dense product
 *   rounded to bfloat16 (nearest, ties to even), float32 accumulation
 */
int gcn_layer_fwd(const gcn_dgraph* g, int32_t F, int32_t h,
                  const float* H_in, int64_t ld_in, const float* W_self,
                  const float* W_neigh, const float* bias, float* AH,
                  int64_t ld_ah, float* H_out, int64_t ld_out,
                  int32_t precision, void* ws, size_t ws_bytes,
                  gcn_stream_t stream);

/* --------------------------------------------- classifier + loss (a6)
 * gcn_classifier_fwd - logits = H W_cls (+ b_cls), a linear layer on the
 * last layer's output (Section 2.1, node classifier).
 *   H [n x K] ld ldh; W_cls [K x C]; b_cls [C] or NULL; logits [n x C] ldz
 *   Scratch (split-K slices when n x C is too small to fill the GPU):
 *   gcn_scratch_bytes(NULL, n, max(K, C)).
 */
int gcn_classifier_fwd(int32_t n, int32_t K, int32_t C, const float* H,
                       int64_t ldh, const float* W_cls, const float* b_cls,
                       float* logits, int64_t ldz, int32_t precision,
                       void* ws, size_t ws_bytes, gcn_stream_t stream);

/* gcn_loss - loss and its gradient w.r.t. the logits (Section 2.1: softmax
 * with cross-entropy; its gradient is a subtraction).
 *   SOFTMAX_CE : loss = mean_v (logsumexp(z_v) - z_v[y_v]),
 *                dz   = (softmax(z) - onehot(y)) / n;   labels int32[n]
 *   SIGMOID_BCE: loss = mean over n*C of
 *                       max(z,0) - z y + log(1 + exp(-|z|)),
 *                dz   = (sigmoid(z) - y) / (n C);        labels uint8[n*C]
 *   logits, dlogits [n x C] (ld ldz, ldd; may be the same buffer);
 *   loss_out device float[1]. Deterministic (fixed summation order).
 *   C <= 512 (GCN_E_UNSUPPORTED above; the same limit holds for the
 *   training step).
 * Status: the call writes a status word, the first int32 of ws, on the
 * device (bit 0: a label is invalid -- a class outside [0, C), or a
 * multi-label byte other than 0 or 1 -- which gives a wrong loss but no
 * out-of-bounds access; bit 1: the loss is not finite). gcn_status_check
 * reads it at the caller's next host sync. */
int gcn_loss(int32_t n, int32_t C, int32_t kind, const float* logits,
             int64_t ldz, const void* labels, float* dlogits, int64_t ldd,
             float* loss_out, void* ws, size_t ws_bytes, gcn_stream_t stream);

/* ---------------------------------------- classifier backward (a7, a12)
 * gcn_classifier_bwd - with dZ = dL/dlogits:
 *   G_out  = (dZ W_cls^T) * [H > 0]      (dL/dH masked by the ReLU that
 *                                         produced H; NULL to skip)
 *   dW_cls = H^T dZ,  db_cls = 1^T dZ
 *   W_cls -= lr dW_cls, b_cls -= lr db_cls   (after G_out has read W_cls)
 *   dW_cls_out / db_cls_out: optional copies of the gradients (NULL ok)
 * Deterministic: split sums are combined in a fixed order. */
int gcn_classifier_bwd(int32_t n, int32_t K, int32_t C, const float* dZ,
                       int64_t ldd, const float* H, int64_t ldh, float* W_cls,
                       float* b_cls, float lr, float* G_out, int64_t ldg,
                       float* dW_cls_out, float* db_cls_out, int32_t precision,
                       void* ws, size_t ws_bytes, gcn_stream_t stream);

/* ---------------------------------------- layer backward (a8-a12)
 * gcn_layer_bwd - Eq. 2a-2c for one layer. G is this layer's masked output
 * gradient, G = dL/dH_out * [H_out > 0] (n x 2h, self half first).
 *   dW_self  = H_in^T G[:, :h]                       (Eq. 2a)
 *   dW_neigh = AH^T  G[:, h:]                        (Eq. 2b)
 *   db       = 1^T G                                 (when bias != NULL)
 *   G_in     = ( G[:, :h] W_self^T + A D^-1 G[:, h:] W_neigh^T ) * [H_in > 0]
 *              (Eq. 2c, masked by the ReLU that produced H_in; NULL for the
 *              first layer, whose input has no gradient)
 *   W -= lr dW for W_self, W_neigh (and bias), after G_in has read them.
 *   H_in [n x F] ld ld_in; AH [n x F] ld ld_ah; G [n x 2h] ld ldg;
 *   G_in [n x F] ld ldgi; dW*_out optional gradient copies (NULL ok).
 */
int gcn_layer_bwd(const gcn_dgraph* g, int32_t F, int32_t h, const float* G,
                  int64_t ldg, const float* H_in, int64_t ld_in,
                  const float* AH, int64_t ld_ah, float* W_self,
                  float* W_neigh, float* bias, float lr, float* G_in,
                  int64_t ldgi, float* dW_self_out, float* dW_neigh_out,
                  float* db_out, int32_t precision, void* ws, size_t ws_bytes,
                  gcn_stream_t stream);

/* ---------------------------------------------- full step (a3-a12)
 * gcn_train_step - forward through L layers (Eq. 1), classifier, loss,
 * backward (Eq. 2a-2c) and the gradient-descent update of every weight, on
 * one subgraph. Weights in `params` are updated in place.
 *   X       device [n x f_in] ld desc->ld_x
 *   labels  device, as for gcn_loss
 *   loss_out device float[1]
 *   grads   optional device buffers receiving every gradient (NULL, or
 *           individual NULL members, to skip)
 *   ws      >= gcn_workspace_bytes(); activations live at the offsets
 *           reported by gcn_workspace_layout (valid after the step).
 * Every weight is updated by one launch at the end of the backward pass,
 * after all input gradients have read the weights; each layer's and the
 * classifier's gradient slices keep a workspace region of their own until
 * then.
 * order GCN_ORDER_PAPER: every layer aggregates first, D^-1 A (H W_neigh)
 *   as D^-1 A H then times W_neigh (Eq. 1), and keeps AH for Eq. 2b.
 * order GCN_ORDER_NARROW: a layer whose input is wider than h (F > h)
 *   transforms first and aggregates the h-wide product, D^-1 A (H W_neigh),
 *   with the bias and ReLU applied after the aggregation; its neighbour
 *   weight gradient becomes H^T (A D^-1 G_neigh) = (D^-1 A H)^T G_neigh,
 *   the same product reassociated, and its AH region holds H W_neigh
 *   instead. Equal results up to rounding, with every aggregation at width
 *   h. Not with has_bias (GCN_E_UNSUPPORTED).
 * precision GCN_PREC_BF16 with h a multiple of 8 (either order):
 *   the step keeps a bf16 copy (rounded to nearest even) of every operand
 *   of a dense product, written by the kernel that produces the operand
 *   (X and the weights are rounded once at the start of the step), and the
 *   products read those copies: the same rounded operands as the per-layer
 *   entry points' bf16 products, at half the operand bytes. A paper-order
 *   layer's AH, read only by products, is then stored in bf16 only (layout
 *   field ah_bytes = 2). Only what an fp32 aggregation reads is kept in
 *   fp32: a layer output only when the next layer aggregates it first
 *   (layout H[l] is -1 otherwise; H16 holds every output), a gradient only
 *   in its neighbour half [h, 2h) and only when its layer aggregates it
 *   (G16 holds the full gradients). The backward's ReLU masks are read
 *   from H16, which has the fp32 sign except for activations in
 *   (0, 2^-134]. With h % 8 != 0 the products round fp32 operands on the
 *   way, as in the per-layer entry points.
 */
#define GCN_ORDER_PAPER 0
#define GCN_ORDER_NARROW 1
typedef struct {
    int32_t L, f_in, h, C;
    int32_t loss;         /* GCN_LOSS_*  */
    int32_t precision;    /* GCN_PREC_*  */
    int32_t has_bias;     /* biases on every layer and the classifier */
    int32_t order;        /* GCN_ORDER_* */
    int64_t ld_x;
} gcn_model_desc;

typedef struct {          /* device pointers, row-major, ld == width */
    float* W_self[GCN_MAX_LAYERS];    /* layer l: [F_l x h]          */
    float* W_neigh[GCN_MAX_LAYERS];   /* layer l: [F_l x h]          */
    float* b[GCN_MAX_LAYERS];         /* layer l: [2h] (has_bias)    */
    float* W_cls;                     /* [2h x C]                    */
    float* b_cls;                     /* [C] (has_bias)              */
} gcn_params;

typedef struct {          /* byte offsets into ws, -1 when absent */
    int64_t AH[GCN_MAX_LAYERS];       /* [n x F_l], ld ld_AH[l] (narrow
                                         layers: H W_neigh [n x h])  */
    int64_t H[GCN_MAX_LAYERS];        /* layer outputs [n x 2h]      */
    int64_t ld_AH[GCN_MAX_LAYERS];
    int64_t ld_H;
    int64_t logits, dlogits, ld_C;    /* [n x C]                     */
    int64_t G[GCN_MAX_LAYERS];        /* masked grads of layer outputs;
                                         ping-pong, so only the last
                                         two written stay valid      */
    int64_t scratch, scratch_bytes, total_bytes;
    int64_t ah_bytes;                 /* bytes per AH element of the
                                         layers that aggregate first: 4
                                         (float), 2 (bf16, see
                                         gcn_train_step); a narrow
                                         layer's region is float */
    int64_t H16[GCN_MAX_LAYERS];      /* bf16 step with operand copies
                                         (ah_bytes = 2): bf16 copies of
                                         H[l] and of G[l], ld ld_H (G16
                                         ping-pongs like G); -1 else */
    int64_t G16[GCN_MAX_LAYERS];
    int64_t status;                   /* the step's loss status word (int32;
                                         see gcn_loss), for
                                         gcn_status_check */
} gcn_ws_layout;

int gcn_workspace_layout(const gcn_dgraph* g, const gcn_model_desc* desc,
                         gcn_ws_layout* out);
int gcn_workspace_bytes(const gcn_dgraph* g, const gcn_model_desc* desc,
                        size_t* bytes);
int gcn_train_step(const gcn_dgraph* g, const gcn_model_desc* desc,
                   const gcn_params* params, const float* X,
                   const void* labels, float lr, float* loss_out,
                   const gcn_params* grads, void* ws, size_t ws_bytes,
                   gcn_stream_t stream);

/* ------------------------------------------------------- inference
 * gcn_infer - the forward pass of gcn_train_step alone, finished into
 * logits: Eq. 1 through the L layers and the classifier (logits plus b_cls),
 * no loss and no update. The paper's conclusion names inference on large,
 * un-sampled graphs as the method's extension, with the redundancy
 * reduction applied to the whole graph: `g` is then the reduced (or direct)
 * image of that graph, built exactly as for a training subgraph. Same
 * descriptor, parameters (read only), precision and order as the step, and
 * the same workspace (gcn_workspace_bytes); the activations it leaves at
 * the gcn_workspace_layout offsets are those of the step's forward pass.
 *   X       device [n x f_in] ld desc->ld_x
 *   logits  device [n x C] ld ld_logits (>= C, a multiple of 4, 16-byte
 *           aligned)
 * Errors: as gcn_train_step (GCN_E_INVALID_ARG before any launch).
 */
int gcn_infer(const gcn_dgraph* g, const gcn_model_desc* desc,
              const gcn_params* params, const float* X, float* logits,
              int64_t ld_logits, void* ws, size_t ws_bytes, gcn_stream_t stream);

/* ------------------------------------------------------ optimisers
 * gcn_train_step_optim - gcn_train_step with every weight (and bias)
 * updated by the optimiser `opt` instead of plain gradient descent.
 * Section 4.1 names the state each optimiser keeps beside the weights:
 * none for gradient descent, the earlier steps' weight gradients for
 * gradient descent with momentum, first and second moment estimates for
 * Adam; the update rules are those of the cited methods, with g the
 * weight's gradient of this step and t = opt->step:
 *   GCN_OPT_SGD       W <- W - lr g                       (gcn_train_step)
 *   GCN_OPT_MOMENTUM  u <- mu u + g;  W <- W - lr u
 *   GCN_OPT_ADAM      m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
 *                     W <- W - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
 * The update runs where the weight-gradient slices are summed, so each
 * weight and each state word is read and written once per step.
 *   opt     host struct; step counts updates from 1 (Adam's bias
 *           correction); momentum in [0, 1); beta1, beta2 in [0, 1);
 *           eps > 0; lr finite
 *   state1  momentum: u, Adam: m; state2: Adam's v (NULL otherwise).
 *           Device buffers shaped like `params` (every member the model
 *           uses non-NULL), zero before the first step, updated in place;
 *           owned by the caller. SGD reads neither.
 * Errors: GCN_E_INVALID_ARG for an unknown kind, a value out of range or a
 * missing state buffer (nothing launched); otherwise as gcn_train_step.
 */
#define GCN_OPT_SGD 0
#define GCN_OPT_MOMENTUM 1
#define GCN_OPT_ADAM 2
typedef struct {
    int32_t kind;         /* GCN_OPT_* */
    int32_t step;         /* Adam: 1 for the first update */
    float lr;
    float momentum;       /* GCN_OPT_MOMENTUM: mu */
    float beta1, beta2, eps;   /* GCN_OPT_ADAM */
    float reserved;
} gcn_optim;

int gcn_train_step_optim(const gcn_dgraph* g, const gcn_model_desc* desc,
                         const gcn_params* params, const float* X,
                         const void* labels, const gcn_optim* opt,
                         const gcn_params* state1, const gcn_params* state2,
                         float* loss_out, const gcn_params* grads, void* ws,
                         size_t ws_bytes, gcn_stream_t stream);

/* ---------------------------------------------------- launch timing
 * Tracing for measurement: when enabled, every kernel launch made by the
 * entry points above is bracketed by two HIP events on its own stream and
 * labelled with its kernel class and algorithmic work.
 * gcn_profile_enable - start timing with room for `capacity` launches
 *   (1..2^20); clears earlier records; creates the events (host call, not
 *   for use while another thread launches through the library).
 * gcn_profile_disable - stop timing new launches (records are kept).
 * gcn_profile_read - wait for the timed launches and report, per kernel
 *   class with at least one launch: launches, total / min / max
 *   milliseconds, and the summed algorithmic flops and bytes (bytes: each
 *   operand element read or written once, list gathers counted per list
 *   entry). Writes up to max_entries entries and sets *count to the number
 *   of classes; reset != 0 clears the records. Returns GCN_E_INTERNAL if
 *   launches went untimed because the capacity ran out.
 */
typedef struct {
    int32_t kind;
    int32_t launches;
    const char* name;     /* static string, e.g. "gemm_dw" */
    double total_ms, min_ms, max_ms;
    double flops, bytes;
} gcn_profile_entry;

int gcn_profile_enable(int32_t capacity);
int gcn_profile_disable(void);
int gcn_profile_read(gcn_profile_entry* out, int32_t max_entries,
                     int32_t* count, int32_t reset);

/* gcn_status_check - the host side of the loss status word that gcn_loss
 * (the first int32 of its ws) and gcn_train_step / gcn_train_step_optim
 * (at ws + layout.status) write on the device every call: waits for
 * `stream`, reads the word and returns GCN_OK, GCN_E_INVALID_ARG if a label
 * of the last call was invalid, or GCN_E_NONFINITE if its loss was inf or
 * NaN (message in gcn_last_error). A device-side check, so the step itself
 * never waits on the host. `status` is a device pointer. */
int gcn_status_check(const void* status, gcn_stream_t stream);

/* ---------------------------------------------------- bandwidth probe
 * gcn_read_probe - measurement helper, not part of the training step: one
 *   launch on `stream` that reads every 16-byte word of `buf` (device
 *   memory, 16-byte aligned, `bytes` a positive multiple of 16) once and
 *   sums it, writing one float per wavefront to `sink` (device memory,
 *   GCN_READ_PROBE_SINK floats, caller-owned). Timed over a buffer far
 *   larger than the 256 MB Infinity Cache it gives the HBM bandwidth a
 *   kernel that only reads can reach: the denominator for the aggregation's
 *   compulsory bytes. Timed as class "read_probe". GCN_E_INVALID_ARG on bad
 *   pointers or sizes (nothing launched), GCN_E_HIP if the launch fails.
 */
#define GCN_READ_PROBE_SINK 16384
int gcn_read_probe(const void* buf, size_t bytes, float* sink, gcn_stream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* GCN_ACT_H */
