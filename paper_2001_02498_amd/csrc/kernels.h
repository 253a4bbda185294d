// Internal launch interface between the entry points (api.hip) and the
// kernel files. Every launcher only enqueues work on `s` and returns the
// hipGetLastError() status of its launches.
#pragma once

#include <hip/hip_runtime.h>

#include "common.h"

namespace gcn {

// ---------------------------------------------------------------- aggregation
// Extended row source: vertex c < n reads X row c, c >= n reads aux row c-n.
struct RowSource {
    const float* X;
    int64_t ldx;
    const float* aux;
    int64_t ldaux;
    int32_t n;
};

// Pair sums of all rounds in one pass: aux[k] = sum over the original
// vertices v of pair k's expansion of s(v) X[v], s(v) = 1/d_v when
// prescale, else 1.
hipError_t launch_pair_sums(const gcn_dgraph* g, RowSource src, bool prescale,
                            float* aux, int64_t ldaux, int32_t F, hipStream_t s);

// What a finished list sum becomes.
enum AggEpi : int {
    AGG_SUM = 0,             // Y_w = sum
    AGG_MEAN = 1,            // Y_w = (1/d_w) sum
    AGG_MEAN_BIAS_RELU = 2,  // Y_w = max((1/d_w) sum + bias, 0)  (bias may be NULL)
};

// Sums of the G_s^# lists (the binned work list of gcn_graph_pack; a split
// list's pieces are added within its bin's workgroup), finished as `epi`
// says; prescale (with AGG_SUM only): gathered original rows are multiplied
// by their 1/d.
// Yh != NULL: the finished rows go to Yh as bf16 (rounded to nearest even;
// leading dimension ldyh) instead of to Y.
hipError_t launch_list_sums(const gcn_dgraph* g, RowSource src, bool prescale, AggEpi epi,
                            const float* bias, float* Y, int64_t ldy, int32_t F, hipStream_t s,
                            __bf16* Yh = nullptr, int64_t ldyh = 0);

// ---------------------------------------------------------------- GEMM
enum ALayout : int { A_MK = 0, A_KM = 1 };   // A(m,k) = A[m*lda+k] | A[k*lda+m]
enum BLayout : int { B_KN = 0, B_NK = 1 };   // B(k,n) = B[k*ldb+n] | B[n*ldb+k]
enum Epilogue : int {
    EPI_STORE = 0,      // C = acc
    EPI_BIAS_RELU = 1,  // C = max(acc + bias[n], 0)   (bias may be NULL; no_relu: no max)
    EPI_BIAS = 2,       // C = acc + bias[n]            (bias may be NULL)
    EPI_MASK = 3,       // C = acc * [mask[m,n] > 0]
    EPI_PARTIAL = 4,    // C + split*part_stride = acc over the split's K range
};

struct GemmProblem {
    int32_t M, N, K;
    // A, optionally concatenated along K: k < ksplitA reads A0, else A1 at
    // k - ksplitA (ksplitA % 4 == 0); A_KM may append a row of ones (m == M-1)
    const float* A0;
    const float* A1;
    int64_t lda0, lda1;
    int32_t ksplitA;
    int32_t ones_row;
    const float* B0;
    const float* B1;
    int64_t ldb0, ldb1;
    int32_t ksplitB;
    int32_t splits;       // split-K factor (EPI_PARTIAL: from gemm_split_plan)
    float* C;
    int64_t ldc;
    const float* bias;
    const float* mask;
    int64_t ldmask;
    int64_t part_stride;  // floats between split slices
    int32_t kchunk;       // K per split (EPI_PARTIAL: from gemm_split_plan)
    int32_t tiles_m, tiles_n, tile_begin;
    int32_t a_vec, b_vec; // operand rows 16-byte aligned: float4 loads
    int32_t no_relu;      // EPI_BIAS_RELU: this problem stores acc + bias only
    // bf16 copies of the operands (launch_gemm with bf16 and hA0 != NULL):
    // the same elements as A0/A1/B0/B1, rounded to bf16, with their own
    // leading dimensions (multiples of 8, rows 16-byte aligned; a K
    // concatenation point must then be a multiple of 8)
    const __bf16* hA0;
    const __bf16* hA1;
    int64_t hlda0, hlda1;
    const __bf16* hB0;
    const __bf16* hB1;
    int64_t hldb0, hldb1;
    // optional bf16 copy of the finished output (EPI_BIAS_RELU, EPI_MASK),
    // leading dimension a multiple of 4
    __bf16* hC;
    int64_t ldhc;
    // with hC: the fp32 output C is written only for columns >= c_from (a
    // multiple of 4; N or more: not at all, C may then be NULL)
    int32_t c_from;
    // EPI_MASK in the copies kernel: the mask read from this bf16 matrix
    // (leading dimension a multiple of 4) instead of `mask`, when set
    const __bf16* hmask;
    int64_t ldhmask;
};

constexpr int kMaxProblems = 2;
struct GemmBatch {
    GemmProblem p[kMaxProblems];
    int32_t nprob;
    int32_t total_tiles;
    // tile rows asked for by the caller: 0 (the planner's 128-row tiles),
    // 32 (32 x 128 tiles of the fp32 kernel: the weight gradients of the
    // classifier and of the first layer) or 64 (64 x 128, fp32: the
    // classifier's logits); the bf16 kernels always take 128
    int32_t tbm;
};

// Split-K plan for `nprob` problems of one shape launched together
// (deterministic in the shapes): K is cut into `splits` ranges of `kchunk`
// (a multiple of the K tile), the last one possibly shorter; every range is
// non-empty when K > 0.
void gemm_split_plan(int32_t M, int32_t N, int32_t K, int32_t nprob, int32_t* splits,
                     int32_t* kchunk);
// The same for `tiles` output tiles of any shape.
void gemm_split_plan_tiles(int64_t tiles, int32_t K, int32_t* splits, int32_t* kchunk);

// Which product of the step a launch computes (its own kernel name and
// timing class; the code depends only on layouts and epilogue).
enum GemmRole : int {
    ROLE_FWD = 0,     // layer transforms            [H W_self | AH W_neigh]
    ROLE_CLS_FWD,     // classifier logits            H W_cls
    ROLE_DX,          // layer input gradient         [G_s | T][W_s; W_n]^T
    ROLE_CLS_DX,      // classifier input gradient    dZ W_cls^T
    ROLE_DW,          // layer weight gradients       H^T G_s, AH^T G_n
    ROLE_CLS_DW,      // classifier weight gradient   H^T dZ
    ROLE_FWD_IN,      // first layer's transforms     (K = f_in)
    ROLE_DW_IN,       // first layer's weight grads   (M = f_in)
};

// Launch C = A B for 1-2 problems of identical layouts / epilogue; bf16:
// operands rounded to bf16 for the matrix cores, fp32 accumulation. With
// bf16 and operand copies (hA0 set in every problem) the products read the
// copies; otherwise they read the fp32 operands and round them on the way.
hipError_t launch_gemm(GemmBatch& b, ALayout al, BLayout bl, Epilogue ep, GemmRole role,
                       bool bf16, hipStream_t s);

// Sum of split-K slices in slice order plus an optional bias:
//   C[m][n] = sum_j part[j*stride + m*ldp + n] (+ bias[n]).
hipError_t launch_splitk_finish(const float* part, int64_t part_stride, int64_t ldp,
                                int32_t splits, int32_t M, int32_t N, const float* bias,
                                float* C, int64_t ldc, hipStream_t s);

// Deterministic sum of split-K slices + gradient-descent update:
//   d = sum_j part[j] (j ascending);  W[m][n] -= lr d  (m < Mw);
//   bias row m == Mw (when b != NULL): b[n] -= lr d.  Optional copies of d.
struct SgdProblem {
    const float* part;
    int64_t part_stride;
    int64_t ldp;
    int32_t splits, Mw, N;
    float* W;
    float* b;
    float* dW_out;
    float* db_out;
    // optimiser state of W and of the bias row (momentum: s1 = velocity;
    // Adam: s1 = first, s2 = second moment); NULL for plain descent
    float* s1;
    float* s2;
    float* s1b;
    float* s2b;
};
// Weight update applied where the gradient slices are summed.
enum OptKind : int32_t { OPT_SGD = 0, OPT_MOMENTUM = 1, OPT_ADAM = 2 };
struct OptimArgs {
    int32_t kind;
    float lr, mu, b1, b2, eps;
    float c1, c2;   // Adam bias corrections 1 / (1 - b1^t), 1 / (1 - b2^t)
};
// Up to kMaxSgdProblems weights (both branches of every layer and the
// classifier) in one launch.
constexpr int kMaxSgdProblems = 2 * GCN_MAX_LAYERS + 1;
hipError_t launch_sgd_reduce(const SgdProblem* p, int nprob, const OptimArgs& o,
                             hipStream_t s);

// Rounding of fp32 matrices to bf16 copies (nearest even), up to
// kMaxConvJobs matrices in one launch: dst[r][c] = bf16(src[r][c]) for
// c < cols, 0 for cols <= c < ldd (ldd a multiple of 8).
constexpr int kMaxConvJobs = 2 * GCN_MAX_LAYERS + 2;
struct ConvJob {
    const float* src;
    int64_t lds;
    __bf16* dst;
    int64_t ldd;
    int32_t rows, cols;
};
hipError_t launch_to_bf16(const ConvJob* jobs, int njobs, hipStream_t s);

// ---------------------------------------------------------------- loss
constexpr int kMaxLossVPL = 8;   // classes per lane: C <= 512
// rowflag [n] (per-row invalid-label flags) and status (one int32: bit 0 an
// invalid label, bit 1 a non-finite loss, written every call) may be NULL.
hipError_t launch_loss(int32_t n, int32_t C, int32_t kind, const float* z,
                       int64_t ldz, const void* labels, float* dz,
                       int64_t ldd, float* rowloss, int32_t* rowflag, int32_t* status,
                       float* loss_out, hipStream_t s);
// The same with logits = sum of `splits` slices (stride apart, ld ldp) plus
// bias, written to z_out.
// dzh != NULL: also a bf16 copy of dz (leading dimension lddh).
hipError_t launch_loss_parts(int32_t n, int32_t C, int32_t kind, const float* part,
                             int64_t stride, int32_t splits, int64_t ldp, const float* bias,
                             float* z_out, int64_t ldz, const void* labels, float* dz,
                             int64_t ldd, float* rowloss, int32_t* rowflag, int32_t* status,
                             float* loss_out, hipStream_t s, __bf16* dzh = nullptr,
                             int64_t lddh = 0);

}  // namespace gcn
