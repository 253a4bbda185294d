// Device entry points of gcn_act.h: argument validation, scratch planning
// and the composition of aggregation, GEMMs, loss and update into layer and
// training-step calls. Every check runs before the first launch.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "kernels.h"

using namespace gcn;

namespace {

constexpr int64_t kAlign = 256;

inline int64_t r4(int64_t x) { return round_up(x, 4); }
inline int64_t r8(int64_t x) { return round_up(x, 8); }

// Scratch regions (bytes from the start of ws) for widths up to W. The
// loss status word (one int32) comes first, at offset 0.
struct ScratchPlan {
    int64_t status, aux, T, gemm_part, rowloss, rowflag, total;
    int64_t gemm_part_floats;   // per problem
    int64_t ld_max;             // widest row (floats) of the aux / T regions
};

// Split-K partial sums of product pair `region` (two problems each): the
// training step keeps every layer's weight gradients (region l) and the
// classifier's (region L) until its single update launch at the end.
float* part_region(void* ws, const ScratchPlan& sp, int region) {
    return reinterpret_cast<float*>(static_cast<char*>(ws) + sp.gemm_part) +
           (int64_t)region * 2 * sp.gemm_part_floats;
}

// Weight updates collected over a step for one launch.
struct SgdList {
    SgdProblem p[kMaxSgdProblems];
    int n = 0;
};

// Launches q[0..nq) now, or appends them to `defer`.
hipError_t sgd_now_or_later(const SgdProblem* q, int nq, const OptimArgs& oa, SgdList* defer,
                            hipStream_t s) {
    if (!defer) return launch_sgd_reduce(q, nq, oa, s);
    if (defer->n + nq > kMaxSgdProblems) return hipErrorInvalidValue;
    for (int i = 0; i < nq; ++i) defer->p[defer->n++] = q[i];
    return hipSuccess;
}

int64_t gemm_part_bound(int64_t W) {
    // split factor * tiles <= 512 + tiles, each tile 128 x 128 floats
    const int64_t tiles = ((W + 1 + 127) / 128) * ((W + 127) / 128);
    return (512 + tiles) * 128 * 128;
}

ScratchPlan plan_scratch(int64_t n, int64_t naux, int64_t W, int64_t part_regions = 1) {
    ScratchPlan p{};
    const int64_t ldW = r4(std::max<int64_t>(W, 1));
    int64_t off = 0;
    auto take = [&](int64_t bytes) {
        int64_t o = off;
        off = round_up(off + std::max<int64_t>(bytes, 1), kAlign);
        return o;
    };
    p.ld_max = ldW;
    p.status = take(4);
    p.aux = take(4 * naux * ldW);
    p.T = take(4 * n * ldW);
    p.gemm_part_floats = gemm_part_bound(W);
    p.gemm_part = take(4 * 2 * p.gemm_part_floats * part_regions);
    p.rowloss = take(4 * std::max<int64_t>(n, 1));
    p.rowflag = take(4 * std::max<int64_t>(n, 1));
    p.total = off;
    return p;
}

// Scratch of gcn_aggregate_noalloc: one fixed array per device, resolved
// to its device address once per device (the name is a host-side stand-in;
// only the address from hipGetSymbolAddress may reach a kernel or a copy).
constexpr int64_t kAggStaticBytes = GCN_AGG_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kAggStaticBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int hip_fail(hipError_t e, const char* where);

// Device address of the current device's scratch array, looked up on the
// first call on that device.
int static_scratch(const char* fn, void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, fn);
    GCN_CHECK_ARG(dev >= 0 && dev < kMaxDevices, "%s: device %d beyond %d", fn, dev,
                  kMaxDevices);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, fn);
        if (!p) {
            set_error("%s: no device address for the scratch array", fn);
            return GCN_E_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return GCN_OK;
}

int hip_fail(hipError_t e, const char* where) {
    set_error("%s: HIP error %d (%s)", where, (int)e, hipGetErrorString(e));
    return GCN_E_HIP;
}

#define GCN_HIP(call, where)                          \
    do {                                              \
        hipError_t e_ = (call);                       \
        if (e_ != hipSuccess) return hip_fail(e_, where); \
    } while (0)

// Dense matrix argument check: rows x width, leading dimension ld.
int check_mat(const char* fn, const char* name, const void* p, int64_t rows,
              int64_t width, int64_t ld) {
    if (rows <= 0 || width <= 0) return GCN_OK;
    GCN_CHECK_ARG(p != nullptr, "%s: %s is NULL", fn, name);
    GCN_CHECK_ARG(((uintptr_t)p & 15) == 0, "%s: %s not 16-byte aligned", fn, name);
    GCN_CHECK_ARG(ld >= width, "%s: ld of %s (%lld) < width %lld", fn, name,
                  (long long)ld, (long long)width);
    GCN_CHECK_ARG(ld % 4 == 0, "%s: ld of %s (%lld) not a multiple of 4", fn,
                  name, (long long)ld);
    return GCN_OK;
}

int check_vec(const char* fn, const char* name, const void* p, int64_t len) {
    if (len <= 0) return GCN_OK;
    GCN_CHECK_ARG(p != nullptr, "%s: %s is NULL", fn, name);
    GCN_CHECK_ARG(((uintptr_t)p & 3) == 0, "%s: %s not 4-byte aligned", fn, name);
    return GCN_OK;
}

int check_graph(const char* fn, const gcn_dgraph* g) {
    GCN_CHECK_ARG(g != nullptr, "%s: graph descriptor is NULL", fn);
    GCN_CHECK_ARG(g->n >= 0 && g->naux >= 0 && g->rounds >= 0 &&
                      g->rounds <= GCN_MAX_ROUNDS && g->nseg >= 0 &&
                      g->nbins >= 0 && g->nmulti >= 0 && g->nmulti <= g->nbins &&
                      g->nhub >= 0 && g->nhub <= g->nmulti &&
                      (g->n == 0 || g->nbins >= 1),
                  "%s: malformed graph descriptor", fn);
    GCN_CHECK_ARG(g->round_offsets[0] == 0 && g->round_offsets[g->rounds] == g->naux,
                  "%s: graph descriptor round offsets inconsistent", fn);
    GCN_CHECK_ARG(g->n == 0 || (g->rowptr && g->inv_deg && g->seg && g->bins),
                  "%s: graph descriptor has NULL arrays", fn);
    GCN_CHECK_ARG(g->naux == 0 || (g->exp_col && g->exp_seg && g->exp_nnz >= 2 * (int64_t)g->naux),
                  "%s: graph descriptor lacks pair-sum expansions", fn);
    return GCN_OK;
}

int check_ws(const char* fn, const void* ws, size_t ws_bytes, int64_t need) {
    GCN_CHECK_ARG(ws != nullptr || need == 0, "%s: workspace is NULL", fn);
    GCN_CHECK_ARG(((uintptr_t)ws % kAlign) == 0, "%s: workspace not 256-byte aligned", fn);
    if ((int64_t)ws_bytes < need) {
        set_error("%s: workspace of %zu bytes, need %lld", fn, ws_bytes, (long long)need);
        return GCN_E_WORKSPACE;
    }
    return GCN_OK;
}

int check_precision(const char* fn, int32_t precision) {
    GCN_CHECK_ARG(precision == GCN_PREC_FP32 || precision == GCN_PREC_BF16,
                  "%s: unknown precision %d", fn, precision);
    return GCN_OK;
}

#define GCN_TRY(x)                \
    do {                          \
        int rc_ = (x);            \
        if (rc_ != GCN_OK) return rc_; \
    } while (0)

__bf16* hptr(void* ws, int64_t off) {
    return reinterpret_cast<__bf16*>(static_cast<char*>(ws) + off);
}

float* fptr(void* ws, int64_t off) {
    return reinterpret_cast<float*>(static_cast<char*>(ws) + off);
}

int32_t* iptr(void* ws, int64_t off) {
    return reinterpret_cast<int32_t*>(static_cast<char*>(ws) + off);
}

// ------------------------------------------------------------ internals
// (arguments already validated)

// transposed: Y = A D^-1 X (Eq. 2c); else Y = epi(D^-1 A X) (Eq. 1), with
// epi AGG_MEAN or AGG_MEAN_BIAS_RELU
int do_aggregate(const char* fn, const gcn_dgraph* g, bool transposed, int32_t F,
                 const float* X, int64_t ldx, float* Y, int64_t ldy,
                 const ScratchPlan& sp, void* ws, hipStream_t s,
                 AggEpi epi = AGG_MEAN, const float* bias = nullptr, __bf16* Yh = nullptr,
                 int64_t ldyh = 0) {
    if (transposed) epi = AGG_SUM;
    const int64_t ldaux = r4(F);
    float* aux = fptr(ws, sp.aux);
    RowSource src{X, ldx, aux, ldaux, g->n};
    GCN_HIP(launch_pair_sums(g, src, transposed, aux, ldaux, F, s), fn);
    GCN_HIP(launch_list_sums(g, src, transposed, epi, bias, Y, ldy, F, s, Yh, ldyh), fn);
    return GCN_OK;
}

GemmProblem gp_zero() {
    GemmProblem p;
    std::memset(&p, 0, sizeof(p));
    p.splits = 1;
    return p;
}

// bf16 copies of a layer's product operands (the step's bf16 variant):
// the inputs are read by the products, the outputs written beside (or, for
// AH and T, instead of) their fp32 versions. Leading dimensions in elements.
struct LayerCopies {
    const __bf16* Hin;   // layer input                      [n x F]
    int64_t ld_hin;
    __bf16* AH;          // its aggregation, bf16 only        [n x F]
    int64_t ld_ah;
    const __bf16* Ws;    // weights                           [F x h], ld h
    const __bf16* Wn;
    __bf16* Hout;        // layer output (forward)            [n x 2h]
    int64_t ld_hout;
    bool hout_fp32;      // the fp32 output is read later (by an aggregation)
    const __bf16* G;     // output gradient (backward)        [n x 2h]
    int64_t ldg;
    __bf16* T;           // aggregated neighbour gradient, bf16 only
    int64_t ldt;
    __bf16* Gin;         // input gradient (backward)         [n x F]
    int64_t ldgi;
    int32_t gin_fp32_from;   // first column of Gin also kept in fp32
};

int do_layer_fwd(const char* fn, const gcn_dgraph* g, int32_t F, int32_t h,
                 const float* H_in, int64_t ld_in, const float* Ws,
                 const float* Wn, const float* bias, float* AH, int64_t ld_ah,
                 float* H_out, int64_t ld_out, bool bf16, const ScratchPlan& sp, void* ws,
                 hipStream_t s, const LayerCopies* c = nullptr, bool first = false) {
    GCN_TRY(do_aggregate(fn, g, false, F, H_in, ld_in, AH, ld_ah, sp, ws, s, AGG_MEAN, nullptr,
                         c ? c->AH : nullptr, c ? c->ld_ah : 0));
    GemmBatch b;
    std::memset(&b, 0, sizeof(b));
    b.nprob = 2;
    for (int i = 0; i < 2; ++i) {
        GemmProblem p = gp_zero();
        p.M = g->n;
        p.N = h;
        p.K = F;
        p.A0 = p.A1 = i == 0 ? H_in : AH;
        p.lda0 = p.lda1 = i == 0 ? ld_in : ld_ah;
        p.ksplitA = F;
        p.B0 = p.B1 = i == 0 ? Ws : Wn;
        p.ldb0 = p.ldb1 = h;
        p.ksplitB = F;
        p.C = H_out + (i == 0 ? 0 : h);
        p.ldc = ld_out;
        p.bias = bias ? bias + (i == 0 ? 0 : h) : nullptr;
        if (c) {
            p.hA0 = p.hA1 = i == 0 ? c->Hin : c->AH;
            p.hlda0 = p.hlda1 = i == 0 ? c->ld_hin : c->ld_ah;
            p.hB0 = p.hB1 = i == 0 ? c->Ws : c->Wn;
            p.hldb0 = p.hldb1 = h;
            p.hC = c->Hout + (i == 0 ? 0 : h);
            p.ldhc = c->ld_hout;
            p.c_from = c->hout_fp32 ? 0 : h;
        }
        b.p[i] = p;
    }
    GCN_HIP(launch_gemm(b, A_MK, B_KN, EPI_BIAS_RELU, first ? ROLE_FWD_IN : ROLE_FWD, bf16, s),
            fn);
    return GCN_OK;
}

// Logits as split-K slices (or in place when not split): slices j at
// part + j*stride, leading dimension ldp; bias not yet added when split.
struct Logits {
    const float* part;
    int64_t stride, ldp;
    int32_t splits;
};

int do_classifier_fwd(const char* fn, int32_t n, int32_t K, int32_t C,
                      const float* H, int64_t ldh, const float* Wc,
                      const float* bc, float* Z, int64_t ldz, bool bf16, const ScratchPlan& sp,
                      void* ws, hipStream_t s, bool finish, Logits* out,
                      const __bf16* Hb = nullptr, int64_t ldhb = 0, const __bf16* Wb = nullptr,
                      int64_t ldwb = 0) {
    GemmBatch b;
    std::memset(&b, 0, sizeof(b));
    b.nprob = 1;
    GemmProblem p = gp_zero();
    p.M = n;
    p.N = C;
    p.K = K;
    p.A0 = p.A1 = H;
    p.lda0 = p.lda1 = ldh;
    p.ksplitA = K;
    p.B0 = p.B1 = Wc;
    p.ldb0 = p.ldb1 = C;
    p.ksplitB = K;
    if (Hb) {
        p.hA0 = p.hA1 = Hb;
        p.hlda0 = p.hlda1 = ldhb;
        p.hB0 = p.hB1 = Wb;
        p.hldb0 = p.hldb1 = ldwb;
    }
    // A few output tiles cannot fill the GPU: split K, then sum the slices
    // (with the bias) either here or inside the loss kernel. fp32 takes
    // 64 x 128 tiles: twice the row tiles, so half the slices to write and
    // sum. (32-row tiles without slices were slower: a K step then holds
    // too few MFMAs per wavefront to cover the loads of H two steps ahead.)
    const int tm = bf16 ? 128 : 64;
    b.tbm = bf16 ? 0 : 64;
    const int64_t tiles = (int64_t)((n + tm - 1) / tm) * ((C + 127) / 128);
    int32_t splits = 1, kchunk = 0;
    if (tiles < (bf16 ? 192 : 256)) gemm_split_plan_tiles(tiles, K, &splits, &kchunk);
    if (splits > 1) {
        p.splits = splits;
        p.kchunk = kchunk;
        p.C = fptr(ws, sp.gemm_part);
        p.ldc = r4(C);
        p.part_stride = (int64_t)n * p.ldc;
        b.p[0] = p;
        GCN_HIP(launch_gemm(b, A_MK, B_KN, EPI_PARTIAL, ROLE_CLS_FWD, bf16, s), fn);
        if (out) *out = Logits{p.C, p.part_stride, p.ldc, splits};
        if (finish)
            GCN_HIP(launch_splitk_finish(p.C, p.part_stride, p.ldc, splits, n, C, bc, Z, ldz, s),
                    fn);
        return GCN_OK;
    }
    p.C = Z;
    p.ldc = ldz;
    p.bias = bc;
    b.p[0] = p;
    GCN_HIP(launch_gemm(b, A_MK, B_KN, EPI_BIAS, ROLE_CLS_FWD, bf16, s), fn);
    if (out) *out = Logits{Z, 0, ldz, 1};
    return GCN_OK;
}

// dW = A^T B over K = n rows with split-K slices in scratch slot `which`,
// planned for output tiles of tm x 128.
GemmProblem dw_problem(int32_t n, int32_t Mw, bool ones, int32_t N,
                       const float* A, int64_t lda, const float* B, int64_t ldb,
                       float* part, int32_t nprob, int32_t tm = 128) {
    GemmProblem p = gp_zero();
    p.M = Mw + (ones ? 1 : 0);
    p.N = N;
    p.K = n;
    p.A0 = p.A1 = A;
    p.lda0 = p.lda1 = lda;
    p.ones_row = ones ? 1 : 0;
    p.B0 = p.B1 = B;
    p.ldb0 = p.ldb1 = ldb;
    gemm_split_plan_tiles((int64_t)((p.M + tm - 1) / tm) * ((p.N + 127) / 128) * nprob, p.K,
                          &p.splits, &p.kchunk);
    p.C = part;
    p.ldc = r4(N);
    p.part_stride = (int64_t)p.M * p.ldc;
    return p;
}

SgdProblem sgd_problem(const GemmProblem& gpb, int32_t Mw, int32_t N, float* W,
                       float* b, float* dW_out, float* db_out) {
    SgdProblem q;
    q.part = gpb.C;
    q.part_stride = gpb.part_stride;
    q.ldp = gpb.ldc;
    q.splits = gpb.splits;
    q.Mw = Mw;
    q.N = N;
    q.W = W;
    q.b = b;
    q.dW_out = dW_out;
    q.db_out = db_out;
    q.s1 = q.s2 = q.s1b = q.s2b = nullptr;
    return q;
}

// Optimiser state of one weight and of the bias it shares a reduction with
// (NULL members: plain gradient descent keeps none).
struct OptState {
    float* s1 = nullptr;
    float* s2 = nullptr;
    float* s1b = nullptr;
    float* s2b = nullptr;
};

SgdProblem with_state(SgdProblem q, const OptState& st) {
    q.s1 = st.s1;
    q.s2 = st.s2;
    q.s1b = st.s1b;
    q.s2b = st.s2b;
    return q;
}

OptimArgs sgd_args(float lr) {
    OptimArgs o{};
    o.kind = OPT_SGD;
    o.lr = lr;
    return o;
}

// bf16 copies of the classifier's operands (the step's bf16 variant).
struct ClsCopies {
    const __bf16* H;    // classifier input          [n x K]
    int64_t ldh;
    const __bf16* W;    // W_cls                     [K x C]
    int64_t ldw;
    const __bf16* dZ;   // logit gradient            [n x C]
    int64_t lddz;
    __bf16* G;          // input gradient, written    [n x K]
    int64_t ldg;
    int32_t g_fp32_from;   // first column of G also kept in fp32
};

int do_classifier_bwd(const char* fn, int32_t n, int32_t K, int32_t C,
                      const float* dZ, int64_t ldd, const float* H, int64_t ldh,
                      float* Wc, float* bc, const OptimArgs& oa, const OptState& st,
                      float* G_out, int64_t ldg, float* dWc_out, float* dbc_out, bool bf16,
                      const ScratchPlan& sp, void* ws, hipStream_t s,
                      const ClsCopies* c = nullptr, SgdList* defer = nullptr,
                      int region = 0) {
    if (G_out) {
        GemmBatch b;
        std::memset(&b, 0, sizeof(b));
        b.nprob = 1;
        GemmProblem p = gp_zero();
        p.M = n;
        p.N = K;
        p.K = C;
        p.A0 = p.A1 = dZ;
        p.lda0 = p.lda1 = ldd;
        p.ksplitA = C;
        p.B0 = p.B1 = Wc;       // B(k=c, n=j) = W_cls[j][c]
        p.ldb0 = p.ldb1 = C;
        p.ksplitB = C;
        p.mask = H;
        p.ldmask = ldh;
        p.C = G_out;
        p.ldc = ldg;
        if (c) {
            p.hA0 = p.hA1 = c->dZ;
            p.hlda0 = p.hlda1 = c->lddz;
            p.hB0 = p.hB1 = c->W;
            p.hldb0 = p.hldb1 = c->ldw;
            p.hC = c->G;
            p.ldhc = c->ldg;
            p.c_from = c->g_fp32_from;
            p.hmask = c->H;   // the ReLU mask of H from its bf16 copy
            p.ldhmask = c->ldh;
        }
        b.p[0] = p;
        GCN_HIP(launch_gemm(b, A_MK, B_NK, EPI_MASK, ROLE_CLS_DX, bf16, s), fn);
    }
    // fp32: 32 x 128 tiles (fewer K slices to write and sum than 128-row
    // tiles of a classifier-wide product)
    GemmBatch b;
    std::memset(&b, 0, sizeof(b));
    b.nprob = 1;
    b.tbm = bf16 ? 0 : 32;
    b.p[0] = dw_problem(n, K, bc != nullptr, C, H, ldh, dZ, ldd, part_region(ws, sp, region), 1,
                        bf16 ? 128 : 32);
    if (c) {
        b.p[0].hA0 = b.p[0].hA1 = c->H;
        b.p[0].hlda0 = b.p[0].hlda1 = c->ldh;
        b.p[0].hB0 = b.p[0].hB1 = c->dZ;
        b.p[0].hldb0 = b.p[0].hldb1 = c->lddz;
    }
    GCN_HIP(launch_gemm(b, A_KM, B_KN, EPI_PARTIAL, ROLE_CLS_DW, bf16, s), fn);
    SgdProblem q = with_state(sgd_problem(b.p[0], K, C, Wc, bc, dWc_out, dbc_out), st);
    GCN_HIP(sgd_now_or_later(&q, 1, oa, defer, s), fn);
    return GCN_OK;
}

int do_layer_bwd(const char* fn, const gcn_dgraph* g, int32_t F, int32_t h,
                 const float* G, int64_t ldg, const float* H_in, int64_t ld_in,
                 const float* AH, int64_t ld_ah, float* Ws, float* Wn,
                 float* bias, const OptimArgs& oa, const OptState& st_self,
                 const OptState& st_neigh, float* G_in, int64_t ldgi,
                 float* dWs_out, float* dWn_out, float* db_out, bool bf16,
                 const ScratchPlan& sp, void* ws, hipStream_t s,
                 const LayerCopies* c = nullptr, bool first = false, SgdList* defer = nullptr,
                 int region = 0) {
    const int32_t n = g->n;
    if (G_in) {
        // T = A D^-1 G[:, h:]  (Eq. 2c), then G_in = [G_self | T] [W_self; W_neigh]^T;
        // T takes G's leading dimension when the scratch rows are that wide
        // (equal strides across the K concatenation keep the GEMM's loads
        // on its fast path)
        float* T = fptr(ws, sp.T);
        const int64_t ldt = ldg <= sp.ld_max ? ldg : r4(h);
        GCN_TRY(do_aggregate(fn, g, true, h, G + h, ldg, T, ldt, sp, ws, s, AGG_SUM, nullptr,
                             c ? c->T : nullptr, c ? c->ldt : 0));
        GemmBatch b;
        std::memset(&b, 0, sizeof(b));
        b.nprob = 1;
        GemmProblem p = gp_zero();
        p.M = n;
        p.N = F;
        p.K = 2 * h;
        p.A0 = G;
        p.lda0 = ldg;
        p.A1 = T;
        p.lda1 = ldt;
        p.ksplitA = h;
        p.B0 = Ws;
        p.ldb0 = h;
        p.B1 = Wn;
        p.ldb1 = h;
        p.ksplitB = h;
        p.mask = H_in;
        p.ldmask = ld_in;
        p.C = G_in;
        p.ldc = ldgi;
        if (c) {
            p.hA0 = c->G;
            p.hlda0 = c->ldg;
            p.hA1 = c->T;
            p.hlda1 = c->ldt;
            p.hB0 = c->Ws;
            p.hB1 = c->Wn;
            p.hldb0 = p.hldb1 = h;
            p.hC = c->Gin;
            p.ldhc = c->ldgi;
            p.c_from = c->gin_fp32_from;
            p.hmask = c->Hin;   // the ReLU mask of H_in from its bf16 copy
            p.ldhmask = c->ld_hin;
        }
        b.p[0] = p;
        GCN_HIP(launch_gemm(b, A_MK, B_NK, EPI_MASK, ROLE_DX, bf16, s), fn);
    }
    GemmBatch b;
    std::memset(&b, 0, sizeof(b));
    b.nprob = 2;
    float* part0 = part_region(ws, sp, region);
    float* part1 = part0 + sp.gemm_part_floats;
    const bool ones = bias != nullptr;
    // fp32 first layer: 32 x 128 tiles (M = f_in + bias row is padded to a
    // multiple of 32 instead of 128, and needs fewer K slices)
    const int tm = (first && !bf16) ? 32 : 128;
    b.tbm = tm == 32 ? 32 : 0;
    b.p[0] = dw_problem(n, F, ones, h, H_in, ld_in, G, ldg, part0, 2, tm);
    b.p[1] = dw_problem(n, F, ones, h, AH, ld_ah, G + h, ldg, part1, 2, tm);
    if (c) {
        for (int i = 0; i < 2; ++i) {
            b.p[i].hA0 = b.p[i].hA1 = i == 0 ? c->Hin : c->AH;
            b.p[i].hlda0 = b.p[i].hlda1 = i == 0 ? c->ld_hin : c->ld_ah;
            b.p[i].hB0 = b.p[i].hB1 = c->G + (i == 0 ? 0 : h);
            b.p[i].hldb0 = b.p[i].hldb1 = c->ldg;
        }
    }
    GCN_HIP(launch_gemm(b, A_KM, B_KN, EPI_PARTIAL, first ? ROLE_DW_IN : ROLE_DW, bf16, s), fn);
    SgdProblem q[2] = {
        with_state(sgd_problem(b.p[0], F, h, Ws, bias, dWs_out, db_out), st_self),
        with_state(sgd_problem(b.p[1], F, h, Wn, bias ? bias + h : nullptr, dWn_out,
                               db_out ? db_out + h : nullptr),
                   st_neigh)};
    GCN_HIP(sgd_now_or_later(q, 2, oa, defer, s), fn);
    return GCN_OK;
}

// Narrow-side order (GCN_ORDER_NARROW) for a layer with F > h: the
// grouped GEMM writes ReLU(H W_self) and Z = H W_neigh, then the h-wide
// aggregation finishes the neighbour half as ReLU(D^-1 A^# Z).
int do_layer_fwd_narrow(const char* fn, const gcn_dgraph* g, int32_t F, int32_t h,
                        const float* H_in, int64_t ld_in, const float* Ws, const float* Wn,
                        float* Z, int64_t ldz, float* H_out, int64_t ld_out, bool bf16,
                        const ScratchPlan& sp, void* ws, hipStream_t s,
                        const LayerCopies* c = nullptr, bool first = false) {
    GemmBatch b;
    std::memset(&b, 0, sizeof(b));
    b.nprob = 2;
    for (int i = 0; i < 2; ++i) {
        GemmProblem p = gp_zero();
        p.M = g->n;
        p.N = h;
        p.K = F;
        p.A0 = p.A1 = H_in;
        p.lda0 = p.lda1 = ld_in;
        p.ksplitA = F;
        p.B0 = p.B1 = i == 0 ? Ws : Wn;
        p.ldb0 = p.ldb1 = h;
        p.ksplitB = F;
        p.C = i == 0 ? H_out : Z;
        p.ldc = i == 0 ? ld_out : ldz;
        p.no_relu = i == 1;
        if (c) {
            // Z stays fp32 for the aggregation; the self half is kept in
            // bf16 (and in fp32 only when an aggregation reads it)
            p.hA0 = p.hA1 = c->Hin;
            p.hlda0 = p.hlda1 = c->ld_hin;
            p.hB0 = p.hB1 = i == 0 ? c->Ws : c->Wn;
            p.hldb0 = p.hldb1 = h;
            if (i == 0) {
                p.hC = c->Hout;
                p.ldhc = c->ld_hout;
                p.c_from = c->hout_fp32 ? 0 : h;
            }
        }
        b.p[i] = p;
    }
    GCN_HIP(launch_gemm(b, A_MK, B_KN, EPI_BIAS_RELU, first ? ROLE_FWD_IN : ROLE_FWD, bf16, s),
            fn);
    // with copies the neighbour half goes to the bf16 copy only (no
    // aggregation reads a narrow layer's output: the next layer transforms
    // before it aggregates)
    if (c && c->hout_fp32) {
        set_error("%s: a narrow layer's fp32 output is not kept with bf16 copies", fn);
        return GCN_E_INTERNAL;
    }
    return do_aggregate(fn, g, false, h, Z, ldz, H_out + h, ld_out, sp, ws, s,
                        AGG_MEAN_BIAS_RELU, nullptr, c ? c->Hout + h : nullptr,
                        c ? c->ld_hout : 0);
}

// Backward of a narrow layer: T = A D^-1 G_neigh (also for the first
// layer), G_in as in the paper order, and dW_neigh = H_in^T T.
int do_layer_bwd_narrow(const char* fn, const gcn_dgraph* g, int32_t F, int32_t h,
                        const float* G, int64_t ldg, const float* H_in, int64_t ld_in,
                        float* Ws, float* Wn, const OptimArgs& oa, const OptState& st_self,
                        const OptState& st_neigh, float* G_in, int64_t ldgi,
                        float* dWs_out, float* dWn_out, bool bf16, const ScratchPlan& sp,
                        void* ws, hipStream_t s, const LayerCopies* c = nullptr,
                        bool first = false, SgdList* defer = nullptr, int region = 0) {
    const int32_t n = g->n;
    float* T = fptr(ws, sp.T);
    const int64_t ldt = ldg <= sp.ld_max ? ldg : r4(h);
    GCN_TRY(do_aggregate(fn, g, true, h, G + h, ldg, T, ldt, sp, ws, s, AGG_SUM, nullptr,
                         c ? c->T : nullptr, c ? c->ldt : 0));
    if (G_in) {
        GemmBatch b;
        std::memset(&b, 0, sizeof(b));
        b.nprob = 1;
        GemmProblem p = gp_zero();
        p.M = n;
        p.N = F;
        p.K = 2 * h;
        p.A0 = G;
        p.lda0 = ldg;
        p.A1 = T;
        p.lda1 = ldt;
        p.ksplitA = h;
        p.B0 = Ws;
        p.ldb0 = h;
        p.B1 = Wn;
        p.ldb1 = h;
        p.ksplitB = h;
        p.mask = H_in;
        p.ldmask = ld_in;
        p.C = G_in;
        p.ldc = ldgi;
        if (c) {
            p.hA0 = c->G;
            p.hlda0 = c->ldg;
            p.hA1 = c->T;
            p.hlda1 = c->ldt;
            p.hB0 = c->Ws;
            p.hB1 = c->Wn;
            p.hldb0 = p.hldb1 = h;
            p.hC = c->Gin;
            p.ldhc = c->ldgi;
            p.c_from = c->gin_fp32_from;
            p.hmask = c->Hin;
            p.ldhmask = c->ld_hin;
        }
        b.p[0] = p;
        GCN_HIP(launch_gemm(b, A_MK, B_NK, EPI_MASK, ROLE_DX, bf16, s), fn);
    }
    GemmBatch b;
    std::memset(&b, 0, sizeof(b));
    b.nprob = 2;
    float* part0 = part_region(ws, sp, region);
    float* part1 = part0 + sp.gemm_part_floats;
    const int tm = (first && !bf16) ? 32 : 128;   // as in the paper order
    b.tbm = tm == 32 ? 32 : 0;
    b.p[0] = dw_problem(n, F, false, h, H_in, ld_in, G, ldg, part0, 2, tm);
    b.p[1] = dw_problem(n, F, false, h, H_in, ld_in, T, ldt, part1, 2, tm);
    if (c) {
        for (int i = 0; i < 2; ++i) {
            b.p[i].hA0 = b.p[i].hA1 = c->Hin;
            b.p[i].hlda0 = b.p[i].hlda1 = c->ld_hin;
            b.p[i].hB0 = b.p[i].hB1 = i == 0 ? c->G : c->T;
            b.p[i].hldb0 = b.p[i].hldb1 = i == 0 ? c->ldg : c->ldt;
        }
    }
    GCN_HIP(launch_gemm(b, A_KM, B_KN, EPI_PARTIAL, first ? ROLE_DW_IN : ROLE_DW, bf16, s), fn);
    SgdProblem q[2] = {
        with_state(sgd_problem(b.p[0], F, h, Ws, nullptr, dWs_out, nullptr), st_self),
        with_state(sgd_problem(b.p[1], F, h, Wn, nullptr, dWn_out, nullptr), st_neigh)};
    GCN_HIP(sgd_now_or_later(q, 2, oa, defer, s), fn);
    return GCN_OK;
}

bool narrow_layer(const gcn_model_desc* d, int32_t F) {
    return d->order == GCN_ORDER_NARROW && F > d->h;
}

// bf16 copies of the step's product operands (precision GCN_PREC_BF16, h a
// multiple of 8): byte offsets into the workspace, ld in elements. A
// paper-order layer's AH is then kept in bf16 only (pub.AH, pub.ld_AH); a
// narrow layer's region keeps holding the fp32 H W_neigh it aggregates.
struct CopyLayout {
    bool on;
    int64_t X, ld_x;                                  // [n x f_in]
    int64_t Ws[GCN_MAX_LAYERS], Wn[GCN_MAX_LAYERS];   // [F_l x h], ld h
    int64_t Wc, ld_wc;                                // [2h x C]
    int64_t H[GCN_MAX_LAYERS];                        // [n x 2h], ld ld_H
    int64_t G[GCN_MAX_LAYERS];                        // ping-pong like the fp32 G
    int64_t T;                                        // [n x h], ld ld_H
    int64_t dZ, ld_dz;                                // [n x C]
};

bool step_copies(const gcn_model_desc* d) {
    return d->precision == GCN_PREC_BF16 && d->h % 8 == 0;
}

// Whether layer l's fp32 output is read by an aggregation: the next layer's,
// when that layer aggregates before it transforms. With bf16 copies nothing
// else reads it (products and ReLU masks read the bf16 copy).
bool output_aggregated(const gcn_model_desc* d, int l) {
    return l + 1 < d->L && !narrow_layer(d, 2 * d->h);
}

// Whether the fp32 gradient of layer l's output is aggregated (its
// neighbour half): by layer l's backward when it computes T, i.e. above the
// first layer, or at any layer that transforms first.
bool gradient_aggregated(const gcn_model_desc* d, int l) {
    return l > 0 || narrow_layer(d, d->f_in);
}

struct StepLayout {
    gcn_ws_layout pub;
    ScratchPlan sp;
    CopyLayout cp;
    int64_t H32[GCN_MAX_LAYERS];   // the fp32 H regions (pub.H reports -1 where unwritten)
};

int plan_step(const gcn_dgraph* g, const gcn_model_desc* d, StepLayout* out) {
    const int64_t n = g->n;
    std::memset(&out->pub, 0, sizeof(out->pub));
    for (int i = 0; i < GCN_MAX_LAYERS; ++i)
        out->pub.AH[i] = out->pub.H[i] = out->pub.G[i] = out->pub.ld_AH[i] = -1;
    int64_t off = 0;
    auto take = [&](int64_t bytes) {
        int64_t o = off;
        off = round_up(off + std::max<int64_t>(bytes, 1), kAlign);
        return o;
    };
    const int64_t ldH = r4(2 * (int64_t)d->h);
    const int64_t ldC = r4(d->C);
    const bool copies = step_copies(d);
    CopyLayout& cp = out->cp;
    std::memset(&cp, 0, sizeof(cp));
    cp.on = copies;
    out->pub.ah_bytes = copies ? 2 : 4;
    for (int i = 0; i < GCN_MAX_LAYERS; ++i) out->pub.H16[i] = out->pub.G16[i] = -1;
    for (int l = 0; l < d->L; ++l) {
        const int64_t F = l == 0 ? d->f_in : 2 * (int64_t)d->h;
        const bool h16 = copies && !narrow_layer(d, (int32_t)F);   // AH in bf16
        out->pub.ld_AH[l] = h16 ? r8(F) : r4(F);
        out->pub.AH[l] = take((h16 ? 2 : 4) * n * out->pub.ld_AH[l]);
        out->H32[l] = take(4 * n * ldH);
        out->pub.H[l] = (copies && !output_aggregated(d, l)) ? -1 : out->H32[l];
    }
    out->pub.ld_H = ldH;
    out->pub.logits = take(4 * n * ldC);
    out->pub.dlogits = take(4 * n * ldC);
    out->pub.ld_C = ldC;
    const int64_t g0 = take(4 * n * ldH), g1 = take(4 * n * ldH);
    // G[l] is the masked gradient of layer l's output; layers alternate
    for (int l = 0; l < d->L; ++l) out->pub.G[l] = ((d->L - 1 - l) % 2 == 0) ? g0 : g1;
    if (copies) {
        const int64_t h = d->h;
        cp.ld_x = r8(d->f_in);
        cp.X = take(2 * n * cp.ld_x);
        for (int l = 0; l < d->L; ++l) {
            const int64_t F = l == 0 ? d->f_in : 2 * h;
            cp.Ws[l] = take(2 * F * h);
            cp.Wn[l] = take(2 * F * h);
        }
        cp.ld_wc = r8(d->C);
        cp.Wc = take(2 * 2 * h * cp.ld_wc);
        for (int l = 0; l < d->L; ++l) cp.H[l] = take(2 * n * ldH);
        const int64_t h0 = take(2 * n * ldH), h1 = take(2 * n * ldH);
        for (int l = 0; l < d->L; ++l) cp.G[l] = ((d->L - 1 - l) % 2 == 0) ? h0 : h1;
        for (int l = 0; l < d->L; ++l) {
            out->pub.H16[l] = cp.H[l];
            out->pub.G16[l] = cp.G[l];
        }
        cp.T = take(2 * n * ldH);
        cp.ld_dz = r8(d->C);
        cp.dZ = take(2 * n * cp.ld_dz);
    }
    const int64_t W = std::max<int64_t>({(int64_t)d->f_in, 2 * (int64_t)d->h, (int64_t)d->C});
    out->sp = plan_scratch(n, g->naux, W, d->L + 1);
    out->pub.scratch = off;
    out->pub.scratch_bytes = out->sp.total;
    out->pub.status = out->pub.scratch + out->sp.status;
    out->pub.total_bytes = off + out->sp.total;
    return GCN_OK;
}

int check_desc(const char* fn, const gcn_model_desc* d) {
    GCN_CHECK_ARG(d != nullptr, "%s: model descriptor is NULL", fn);
    GCN_CHECK_ARG(d->L >= 1 && d->L <= GCN_MAX_LAYERS, "%s: L=%d outside [1, %d]",
                  fn, d->L, GCN_MAX_LAYERS);
    GCN_CHECK_ARG(d->f_in >= 1, "%s: f_in < 1", fn);
    GCN_CHECK_ARG(d->h >= 4 && d->h % 4 == 0, "%s: h=%d must be a positive multiple of 4", fn, d->h);
    GCN_CHECK_ARG(d->C >= 1, "%s: C < 1", fn);
    if (d->C > 64 * kMaxLossVPL) {
        set_error("%s: C=%d above the %d classes of the loss kernel", fn, d->C, 64 * kMaxLossVPL);
        return GCN_E_UNSUPPORTED;
    }
    GCN_CHECK_ARG(d->loss == GCN_LOSS_SOFTMAX_CE || d->loss == GCN_LOSS_SIGMOID_BCE,
                  "%s: unknown loss %d", fn, d->loss);
    GCN_CHECK_ARG(d->ld_x >= d->f_in && d->ld_x % 4 == 0,
                  "%s: ld_x=%lld must be >= f_in and a multiple of 4", fn, (long long)d->ld_x);
    GCN_CHECK_ARG(d->order == GCN_ORDER_PAPER || d->order == GCN_ORDER_NARROW,
                  "%s: unknown order %d", fn, d->order);
    if (d->order == GCN_ORDER_NARROW && d->has_bias) {
        set_error("%s: the narrow-side order is built without biases", fn);
        return GCN_E_UNSUPPORTED;
    }
    return check_precision(fn, d->precision);
}

}  // namespace

extern "C" {

int gcn_graph_upload(const void* host_image, size_t bytes, void* dev_buf,
                     gcn_dgraph* out, gcn_stream_t stream) {
    gcn_dgraph tmp;
    int rc = gcn_graph_describe(host_image, bytes, dev_buf, &tmp);
    if (rc) return rc;
    ImageHeader h;
    std::memcpy(&h, host_image, sizeof(h));
    // all `bytes`: the image and what the caller placed after it (a sampled
    // pipeline job's vertex ids)
    GCN_HIP(hipMemcpyAsync(dev_buf, host_image, bytes, hipMemcpyHostToDevice,
                           (hipStream_t)stream),
            "gcn_graph_upload");
    *out = tmp;
    return GCN_OK;
}

int gcn_scratch_bytes(const gcn_dgraph* g, int32_t n, int32_t max_width, size_t* bytes) {
    GCN_CHECK_ARG(bytes != nullptr, "gcn_scratch_bytes: bytes is NULL");
    GCN_CHECK_ARG(max_width >= 1, "gcn_scratch_bytes: max_width < 1");
    if (g) GCN_TRY(check_graph("gcn_scratch_bytes", g));
    const ScratchPlan sp = g ? plan_scratch(g->n, g->naux, max_width)
                             : plan_scratch(std::max(n, 0), 0, max_width);
    *bytes = (size_t)sp.total;
    return GCN_OK;
}

int gcn_aggregate(const gcn_dgraph* g, int32_t mode, int32_t F, const float* X,
                  int64_t ldx, float* Y, int64_t ldy, void* ws, size_t ws_bytes,
                  gcn_stream_t stream) {
    const char* fn = "gcn_aggregate";
    GCN_TRY(check_graph(fn, g));
    GCN_CHECK_ARG(mode == GCN_AGG_MEAN || mode == GCN_AGG_TRANSPOSED, "%s: unknown mode", fn);
    GCN_CHECK_ARG(F >= 1, "%s: F < 1", fn);
    GCN_TRY(check_mat(fn, "X", X, g->n, F, ldx));
    GCN_TRY(check_mat(fn, "Y", Y, g->n, F, ldy));
    GCN_CHECK_ARG(g->n == 0 || X != Y, "%s: X and Y must not overlap", fn);
    const ScratchPlan sp = plan_scratch(g->n, g->naux, F);
    GCN_TRY(check_ws(fn, ws, ws_bytes, sp.total));
    return do_aggregate(fn, g, mode == GCN_AGG_TRANSPOSED, F, X, ldx, Y, ldy, sp, ws,
                        (hipStream_t)stream);
}

int gcn_aggregate_noalloc(const gcn_dgraph* g, int32_t mode, int32_t F, const float* X,
                          int64_t ldx, float* Y, int64_t ldy, gcn_stream_t stream) {
    const char* fn = "gcn_aggregate_noalloc";
    GCN_TRY(check_graph(fn, g));
    GCN_CHECK_ARG(mode == GCN_AGG_MEAN || mode == GCN_AGG_TRANSPOSED, "%s: unknown mode", fn);
    GCN_CHECK_ARG(F >= 1, "%s: F < 1", fn);
    GCN_TRY(check_mat(fn, "X", X, g->n, F, ldx));
    GCN_TRY(check_mat(fn, "Y", Y, g->n, F, ldy));
    GCN_CHECK_ARG(g->n == 0 || X != Y, "%s: X and Y must not overlap", fn);
    // the aggregation reads only the pair-sum region, which leads the plan
    // after the status word and is written before it is read
    const ScratchPlan sp = plan_scratch(g->n, g->naux, F);
    const int64_t need = sp.T;
    GCN_CHECK_ARG(need <= kAggStaticBytes,
                  "%s: %lld scratch bytes needed (naux %d, F %d) "
                  "exceed the fixed %lld; use gcn_aggregate with a workspace",
                  fn, (long long)need, g->naux, F, (long long)kAggStaticBytes);
    void* ws = nullptr;
    GCN_TRY(static_scratch(fn, &ws));
    return do_aggregate(fn, g, mode == GCN_AGG_TRANSPOSED, F, X, ldx, Y, ldy, sp, ws,
                        (hipStream_t)stream);
}

int gcn_layer_fwd(const gcn_dgraph* g, int32_t F, int32_t h, const float* H_in,
                  int64_t ld_in, const float* W_self, const float* W_neigh,
                  const float* bias, float* AH, int64_t ld_ah, float* H_out,
                  int64_t ld_out, int32_t precision, void* ws, size_t ws_bytes,
                  gcn_stream_t stream) {
    const char* fn = "gcn_layer_fwd";
    GCN_TRY(check_graph(fn, g));
    GCN_CHECK_ARG(F >= 1, "%s: F < 1", fn);
    GCN_CHECK_ARG(h >= 4 && h % 4 == 0, "%s: h=%d must be a positive multiple of 4", fn, h);
    GCN_TRY(check_precision(fn, precision));
    const int64_t n = g->n;
    GCN_TRY(check_mat(fn, "H_in", H_in, n, F, ld_in));
    GCN_TRY(check_mat(fn, "AH", AH, n, F, ld_ah));
    GCN_TRY(check_mat(fn, "H_out", H_out, n, 2 * (int64_t)h, ld_out));
    GCN_TRY(check_mat(fn, "W_self", W_self, F, h, h));
    GCN_TRY(check_mat(fn, "W_neigh", W_neigh, F, h, h));
    if (bias) GCN_TRY(check_vec(fn, "bias", bias, 2 * (int64_t)h));
    const ScratchPlan sp = plan_scratch(n, g->naux, std::max(F, 2 * h));
    GCN_TRY(check_ws(fn, ws, ws_bytes, sp.total));
    return do_layer_fwd(fn, g, F, h, H_in, ld_in, W_self, W_neigh, bias, AH, ld_ah,
                        H_out, ld_out, precision == GCN_PREC_BF16, sp, ws,
                        (hipStream_t)stream);
}

int gcn_classifier_fwd(int32_t n, int32_t K, int32_t C, const float* H, int64_t ldh,
                       const float* W_cls, const float* b_cls, float* logits,
                       int64_t ldz, int32_t precision, void* ws, size_t ws_bytes,
                       gcn_stream_t stream) {
    const char* fn = "gcn_classifier_fwd";
    GCN_CHECK_ARG(n >= 0 && K >= 1 && C >= 1, "%s: bad sizes", fn);
    GCN_TRY(check_precision(fn, precision));
    GCN_TRY(check_mat(fn, "H", H, n, K, ldh));
    GCN_TRY(check_vec(fn, "W_cls", W_cls, (int64_t)K * C));
    if (b_cls) GCN_TRY(check_vec(fn, "b_cls", b_cls, C));
    GCN_TRY(check_mat(fn, "logits", logits, n, C, ldz));
    const ScratchPlan sp = plan_scratch(n, 0, std::max(K, C));
    GCN_TRY(check_ws(fn, ws, ws_bytes, sp.total));
    return do_classifier_fwd(fn, n, K, C, H, ldh, W_cls, b_cls, logits, ldz,
                             precision == GCN_PREC_BF16, sp, ws, (hipStream_t)stream, true,
                             nullptr);
}

int gcn_loss(int32_t n, int32_t C, int32_t kind, const float* logits, int64_t ldz,
             const void* labels, float* dlogits, int64_t ldd, float* loss_out, void* ws,
             size_t ws_bytes, gcn_stream_t stream) {
    const char* fn = "gcn_loss";
    GCN_CHECK_ARG(n >= 0 && C >= 1, "%s: bad sizes", fn);
    GCN_CHECK_ARG(kind == GCN_LOSS_SOFTMAX_CE || kind == GCN_LOSS_SIGMOID_BCE,
                  "%s: unknown loss %d", fn, kind);
    if (C > 64 * kMaxLossVPL) {
        set_error("%s: C=%d above the %d classes of the loss kernel", fn, C, 64 * kMaxLossVPL);
        return GCN_E_UNSUPPORTED;
    }
    GCN_TRY(check_mat(fn, "logits", logits, n, C, ldz));
    GCN_TRY(check_mat(fn, "dlogits", dlogits, n, C, ldd));
    GCN_CHECK_ARG(n == 0 || labels != nullptr, "%s: labels is NULL", fn);
    GCN_CHECK_ARG(kind != GCN_LOSS_SOFTMAX_CE || ((uintptr_t)labels & 3) == 0,
                  "%s: int32 labels not 4-byte aligned", fn);
    GCN_CHECK_ARG(logits != dlogits || ldz == ldd, "%s: in-place loss needs ldz == ldd", fn);
    GCN_TRY(check_vec(fn, "loss_out", loss_out, 1));
    const ScratchPlan sp = plan_scratch(n, 0, C);
    GCN_TRY(check_ws(fn, ws, ws_bytes, sp.total));
    GCN_HIP(launch_loss(n, C, kind, logits, ldz, labels, dlogits, ldd, fptr(ws, sp.rowloss),
                        iptr(ws, sp.rowflag), iptr(ws, sp.status), loss_out,
                        (hipStream_t)stream),
            fn);
    return GCN_OK;
}

int gcn_status_check(const void* status, gcn_stream_t stream) {
    const char* fn = "gcn_status_check";
    GCN_CHECK_ARG(status != nullptr && ((uintptr_t)status & 3) == 0,
                  "%s: status word NULL or not 4-byte aligned", fn);
    GCN_HIP(hipStreamSynchronize((hipStream_t)stream), fn);
    int32_t w = 0;
    GCN_HIP(hipMemcpy(&w, status, sizeof(w), hipMemcpyDeviceToHost), fn);
    if (w & 1) {
        set_error("%s: a label is invalid (softmax: class outside [0, C); multi-label: a "
                  "byte other than 0 or 1); the loss and gradients of that call are wrong", fn);
        return GCN_E_INVALID_ARG;
    }
    if (w & 2) {
        set_error("%s: the loss is not finite (inf or NaN in the logits or the inputs)", fn);
        return GCN_E_NONFINITE;
    }
    return GCN_OK;
}

int gcn_classifier_bwd(int32_t n, int32_t K, int32_t C, const float* dZ, int64_t ldd,
                       const float* H, int64_t ldh, float* W_cls, float* b_cls, float lr,
                       float* G_out, int64_t ldg, float* dW_cls_out, float* db_cls_out,
                       int32_t precision, void* ws, size_t ws_bytes, gcn_stream_t stream) {
    const char* fn = "gcn_classifier_bwd";
    GCN_CHECK_ARG(n >= 0 && K >= 1 && C >= 1, "%s: bad sizes", fn);
    GCN_TRY(check_precision(fn, precision));
    GCN_TRY(check_mat(fn, "dZ", dZ, n, C, ldd));
    GCN_TRY(check_mat(fn, "H", H, n, K, ldh));
    GCN_TRY(check_vec(fn, "W_cls", W_cls, (int64_t)K * C));
    if (b_cls) GCN_TRY(check_vec(fn, "b_cls", b_cls, C));
    if (G_out) GCN_TRY(check_mat(fn, "G_out", G_out, n, K, ldg));
    if (dW_cls_out) GCN_TRY(check_vec(fn, "dW_cls_out", dW_cls_out, (int64_t)K * C));
    if (db_cls_out) GCN_TRY(check_vec(fn, "db_cls_out", db_cls_out, C));
    const ScratchPlan sp = plan_scratch(n, 0, std::max(K, C));
    GCN_TRY(check_ws(fn, ws, ws_bytes, sp.total));
    return do_classifier_bwd(fn, n, K, C, dZ, ldd, H, ldh, W_cls, b_cls, sgd_args(lr),
                             OptState{}, G_out, ldg, dW_cls_out, db_cls_out,
                             precision == GCN_PREC_BF16, sp, ws, (hipStream_t)stream);
}

int gcn_layer_bwd(const gcn_dgraph* g, int32_t F, int32_t h, const float* G, int64_t ldg,
                  const float* H_in, int64_t ld_in, const float* AH, int64_t ld_ah,
                  float* W_self, float* W_neigh, float* bias, float lr, float* G_in,
                  int64_t ldgi, float* dW_self_out, float* dW_neigh_out, float* db_out,
                  int32_t precision, void* ws, size_t ws_bytes, gcn_stream_t stream) {
    const char* fn = "gcn_layer_bwd";
    GCN_TRY(check_graph(fn, g));
    GCN_CHECK_ARG(F >= 1, "%s: F < 1", fn);
    GCN_CHECK_ARG(h >= 4 && h % 4 == 0, "%s: h=%d must be a positive multiple of 4", fn, h);
    GCN_TRY(check_precision(fn, precision));
    const int64_t n = g->n;
    GCN_TRY(check_mat(fn, "G", G, n, 2 * (int64_t)h, ldg));
    GCN_TRY(check_mat(fn, "H_in", H_in, n, F, ld_in));
    GCN_TRY(check_mat(fn, "AH", AH, n, F, ld_ah));
    GCN_TRY(check_mat(fn, "W_self", W_self, F, h, h));
    GCN_TRY(check_mat(fn, "W_neigh", W_neigh, F, h, h));
    if (bias) GCN_TRY(check_vec(fn, "bias", bias, 2 * (int64_t)h));
    if (G_in) GCN_TRY(check_mat(fn, "G_in", G_in, n, F, ldgi));
    if (dW_self_out) GCN_TRY(check_vec(fn, "dW_self_out", dW_self_out, (int64_t)F * h));
    if (dW_neigh_out) GCN_TRY(check_vec(fn, "dW_neigh_out", dW_neigh_out, (int64_t)F * h));
    if (db_out) GCN_TRY(check_vec(fn, "db_out", db_out, 2 * (int64_t)h));
    GCN_CHECK_ARG(db_out == nullptr || bias != nullptr, "%s: db_out without bias", fn);
    const ScratchPlan sp = plan_scratch(n, g->naux, std::max(F, 2 * h));
    GCN_TRY(check_ws(fn, ws, ws_bytes, sp.total));
    return do_layer_bwd(fn, g, F, h, G, ldg, H_in, ld_in, AH, ld_ah, W_self, W_neigh, bias,
                        sgd_args(lr), OptState{}, OptState{}, G_in, ldgi, dW_self_out,
                        dW_neigh_out, db_out, precision == GCN_PREC_BF16, sp, ws,
                        (hipStream_t)stream);
}

int gcn_workspace_layout(const gcn_dgraph* g, const gcn_model_desc* desc,
                         gcn_ws_layout* out) {
    const char* fn = "gcn_workspace_layout";
    GCN_TRY(check_graph(fn, g));
    GCN_TRY(check_desc(fn, desc));
    GCN_CHECK_ARG(out != nullptr, "%s: out is NULL", fn);
    StepLayout sl;
    GCN_TRY(plan_step(g, desc, &sl));
    *out = sl.pub;
    return GCN_OK;
}

int gcn_workspace_bytes(const gcn_dgraph* g, const gcn_model_desc* desc, size_t* bytes) {
    gcn_ws_layout l;
    GCN_TRY(gcn_workspace_layout(g, desc, &l));
    GCN_CHECK_ARG(bytes != nullptr, "gcn_workspace_bytes: bytes is NULL");
    *bytes = (size_t)l.total_bytes;
    return GCN_OK;
}

}  // extern "C"

namespace {

// The state buffers an optimiser needs for every weight (and bias) of the
// model: shaped like the weights, non-NULL.
int check_state(const char* fn, const char* what, const gcn_model_desc* d,
                const gcn_params* st) {
    GCN_CHECK_ARG(st != nullptr, "%s: %s is NULL", fn, what);
    const int32_t h = d->h, C = d->C;
    for (int l = 0; l < d->L; ++l) {
        const int64_t F = l == 0 ? d->f_in : 2 * (int64_t)h;
        GCN_TRY(check_vec(fn, what, st->W_self[l], F * h));
        GCN_TRY(check_vec(fn, what, st->W_neigh[l], F * h));
        if (d->has_bias) GCN_TRY(check_vec(fn, what, st->b[l], 2 * (int64_t)h));
    }
    GCN_TRY(check_vec(fn, what, st->W_cls, 2 * (int64_t)h * C));
    if (d->has_bias) GCN_TRY(check_vec(fn, what, st->b_cls, C));
    return GCN_OK;
}

// Optimiser state of layer l's self (half 0) or neighbour (half 1) weight,
// with the matching half of its bias.
OptState layer_state(const gcn_model_desc* d, const gcn_params* s1, const gcn_params* s2,
                     int l, int half) {
    OptState st;
    const int64_t boff = half ? d->h : 0;
    if (s1) {
        st.s1 = half ? s1->W_neigh[l] : s1->W_self[l];
        st.s1b = d->has_bias ? s1->b[l] + boff : nullptr;
    }
    if (s2) {
        st.s2 = half ? s2->W_neigh[l] : s2->W_self[l];
        st.s2b = d->has_bias ? s2->b[l] + boff : nullptr;
    }
    return st;
}

// The training step; or, with infer_logits set, its forward pass alone
// finished into the caller's logits (inference: no loss, no update).
int train_step_impl(const char* fn, const gcn_dgraph* g, const gcn_model_desc* d,
                    const gcn_params* P, const float* X, const void* labels,
                    const OptimArgs& oa, const gcn_params* st1, const gcn_params* st2,
                    float* loss_out, const gcn_params* grads, void* ws, size_t ws_bytes,
                    gcn_stream_t stream, float* infer_logits = nullptr,
                    int64_t ld_infer = 0) {
    GCN_TRY(check_graph(fn, g));
    GCN_TRY(check_desc(fn, d));
    GCN_CHECK_ARG(P != nullptr, "%s: params is NULL", fn);
    const int64_t n = g->n;
    const int32_t h = d->h, C = d->C, L = d->L;
    const bool infer = infer_logits != nullptr || ld_infer != 0;
    GCN_TRY(check_mat(fn, "X", X, n, d->f_in, d->ld_x));
    if (infer) {
        GCN_TRY(check_mat(fn, "logits", infer_logits, n, C, ld_infer));
    } else {
        GCN_CHECK_ARG(n == 0 || labels != nullptr, "%s: labels is NULL", fn);
        GCN_TRY(check_vec(fn, "loss_out", loss_out, 1));
    }
    for (int l = 0; l < L; ++l) {
        const int64_t F = l == 0 ? d->f_in : 2 * (int64_t)h;
        GCN_TRY(check_mat(fn, "W_self[l]", P->W_self[l], F, h, h));
        GCN_TRY(check_mat(fn, "W_neigh[l]", P->W_neigh[l], F, h, h));
        if (d->has_bias) GCN_TRY(check_vec(fn, "b[l]", P->b[l], 2 * (int64_t)h));
        if (grads) {
            if (grads->W_self[l]) GCN_TRY(check_vec(fn, "grads W_self[l]", grads->W_self[l], F * h));
            if (grads->W_neigh[l]) GCN_TRY(check_vec(fn, "grads W_neigh[l]", grads->W_neigh[l], F * h));
            if (grads->b[l]) {
                GCN_CHECK_ARG(d->has_bias, "%s: bias gradient requested without biases", fn);
                GCN_TRY(check_vec(fn, "grads b[l]", grads->b[l], 2 * (int64_t)h));
            }
        }
    }
    GCN_TRY(check_vec(fn, "W_cls", P->W_cls, 2 * (int64_t)h * C));
    if (d->has_bias) GCN_TRY(check_vec(fn, "b_cls", P->b_cls, C));
    if (grads) {
        if (grads->W_cls) GCN_TRY(check_vec(fn, "grads W_cls", grads->W_cls, 2 * (int64_t)h * C));
        if (grads->b_cls) {
            GCN_CHECK_ARG(d->has_bias, "%s: bias gradient requested without biases", fn);
            GCN_TRY(check_vec(fn, "grads b_cls", grads->b_cls, C));
        }
    }
    StepLayout sl;
    GCN_TRY(plan_step(g, d, &sl));
    GCN_TRY(check_ws(fn, ws, ws_bytes, sl.pub.total_bytes));

    hipStream_t s = (hipStream_t)stream;
    const bool bf16 = d->precision == GCN_PREC_BF16;
    void* scratch = static_cast<char*>(ws) + sl.pub.scratch;
    const ScratchPlan& sp = sl.sp;
    const CopyLayout& cp = sl.cp;
    const int64_t ldH = sl.pub.ld_H, ldC = sl.pub.ld_C;
    auto act = [&](int64_t off) { return fptr(ws, off); };
    auto h16 = [&](int64_t off) { return hptr(ws, off); };
    // With copies, the region of AH holds bf16 values that only the products
    // read; the fp32 pointers handed along for it are never dereferenced.
    if (cp.on) {
        ConvJob jobs[kMaxConvJobs];
        int nj = 0;
        jobs[nj++] = ConvJob{X, d->ld_x, h16(cp.X), cp.ld_x, (int32_t)n, d->f_in};
        for (int l = 0; l < L; ++l) {
            const int32_t F = l == 0 ? d->f_in : 2 * h;
            jobs[nj++] = ConvJob{P->W_self[l], h, h16(cp.Ws[l]), h, F, h};
            jobs[nj++] = ConvJob{P->W_neigh[l], h, h16(cp.Wn[l]), h, F, h};
        }
        jobs[nj++] = ConvJob{P->W_cls, C, h16(cp.Wc), cp.ld_wc, 2 * h, C};
        GCN_HIP(launch_to_bf16(jobs, nj, s), fn);
    }
    auto layer_copies = [&](int l) {
        LayerCopies c{};
        c.Hin = l == 0 ? h16(cp.X) : h16(cp.H[l - 1]);
        c.ld_hin = l == 0 ? cp.ld_x : ldH;
        c.AH = h16(sl.pub.AH[l]);
        c.ld_ah = sl.pub.ld_AH[l];
        c.Ws = h16(cp.Ws[l]);
        c.Wn = h16(cp.Wn[l]);
        c.Hout = h16(cp.H[l]);
        c.ld_hout = ldH;
        c.hout_fp32 = output_aggregated(d, l);
        c.G = h16(cp.G[l]);
        c.ldg = ldH;
        c.T = h16(cp.T);
        c.ldt = ldH;
        c.Gin = l > 0 ? h16(cp.G[l - 1]) : nullptr;
        c.ldgi = ldH;
        // the fp32 aggregation of the layer below reads only the neighbour
        // half of its gradient, and only where that layer aggregates it
        c.gin_fp32_from = l > 0 && gradient_aggregated(d, l - 1) ? h : 2 * h;
        return c;
    };

    // forward (Eq. 1, every layer)
    const float* Hprev = X;
    int64_t ldprev = d->ld_x;
    for (int l = 0; l < L; ++l) {
        const int32_t F = l == 0 ? d->f_in : 2 * h;
        const LayerCopies lc = layer_copies(l);
        if (narrow_layer(d, F)) {
            GCN_TRY(do_layer_fwd_narrow(fn, g, F, h, Hprev, ldprev, P->W_self[l], P->W_neigh[l],
                                        act(sl.pub.AH[l]), sl.pub.ld_AH[l], act(sl.H32[l]),
                                        ldH, bf16, sp, scratch, s, cp.on ? &lc : nullptr, l == 0));
        } else {
            GCN_TRY(do_layer_fwd(fn, g, F, h, Hprev, ldprev, P->W_self[l], P->W_neigh[l],
                                 d->has_bias ? P->b[l] : nullptr, act(sl.pub.AH[l]),
                                 sl.pub.ld_AH[l], act(sl.H32[l]), ldH, bf16, sp, scratch, s,
                                 cp.on ? &lc : nullptr, l == 0));
        }
        Hprev = act(sl.H32[l]);
        ldprev = ldH;
    }
    const float* bcls = d->has_bias ? P->b_cls : nullptr;
    if (infer) {
        // inference ends with the logits, slices summed with the bias here
        if (n > 0)
            GCN_TRY(do_classifier_fwd(fn, (int32_t)n, 2 * h, C, Hprev, ldH, P->W_cls, bcls,
                                      infer_logits, ld_infer, bf16, sp, scratch, s, true, nullptr,
                                      cp.on ? h16(cp.H[L - 1]) : nullptr, ldH,
                                      cp.on ? h16(cp.Wc) : nullptr, cp.ld_wc));
        return GCN_OK;
    }
    // classifier + loss
    float* Z = act(sl.pub.logits);
    float* dZ = act(sl.pub.dlogits);
    Logits lg;
    GCN_TRY(do_classifier_fwd(fn, (int32_t)n, 2 * h, C, Hprev, ldH, P->W_cls, bcls, Z, ldC,
                              bf16, sp, scratch, s, false, &lg,
                              cp.on ? h16(cp.H[L - 1]) : nullptr, ldH,
                              cp.on ? h16(cp.Wc) : nullptr, cp.ld_wc));
    // split logits are summed (with the bias) inside the loss kernel
    GCN_HIP(launch_loss_parts((int32_t)n, C, d->loss, lg.part, lg.stride, lg.splits, lg.ldp,
                              lg.splits > 1 ? bcls : nullptr, Z, ldC, labels, dZ, ldC,
                              fptr(scratch, sp.rowloss), iptr(scratch, sp.rowflag),
                              iptr(scratch, sp.status), loss_out, s,
                              cp.on ? h16(cp.dZ) : nullptr, cp.ld_dz),
            fn);
    // backward (classifier, then Eq. 2a-2c layer by layer); every weight's
    // input gradient is formed before the one launch that updates them all
    SgdList updates;
    float* Gcur = act(sl.pub.G[L - 1]);
    OptState cst;
    if (st1) {
        cst.s1 = st1->W_cls;
        cst.s1b = d->has_bias ? st1->b_cls : nullptr;
    }
    if (st2) {
        cst.s2 = st2->W_cls;
        cst.s2b = d->has_bias ? st2->b_cls : nullptr;
    }
    const ClsCopies cc{cp.on ? h16(cp.H[L - 1]) : nullptr, ldH,
                       cp.on ? h16(cp.Wc) : nullptr, cp.ld_wc,
                       cp.on ? h16(cp.dZ) : nullptr, cp.ld_dz,
                       cp.on ? h16(cp.G[L - 1]) : nullptr, ldH,
                       gradient_aggregated(d, L - 1) ? h : 2 * h};
    GCN_TRY(do_classifier_bwd(fn, (int32_t)n, 2 * h, C, dZ, ldC, Hprev, ldH, P->W_cls,
                              d->has_bias ? P->b_cls : nullptr, oa, cst, Gcur, ldH,
                              grads ? grads->W_cls : nullptr,
                              grads ? grads->b_cls : nullptr, bf16, sp, scratch, s,
                              cp.on ? &cc : nullptr, &updates, L));
    for (int l = L - 1; l >= 0; --l) {
        const int32_t F = l == 0 ? d->f_in : 2 * h;
        const float* Hin = l == 0 ? X : act(sl.H32[l - 1]);
        const int64_t ldin = l == 0 ? d->ld_x : ldH;
        float* Gnext = l > 0 ? act(sl.pub.G[l - 1]) : nullptr;
        const LayerCopies lc = layer_copies(l);
        if (narrow_layer(d, F)) {
            GCN_TRY(do_layer_bwd_narrow(fn, g, F, h, Gcur, ldH, Hin, ldin, P->W_self[l],
                                        P->W_neigh[l], oa, layer_state(d, st1, st2, l, 0),
                                        layer_state(d, st1, st2, l, 1), Gnext, ldH,
                                        grads ? grads->W_self[l] : nullptr,
                                        grads ? grads->W_neigh[l] : nullptr, bf16, sp, scratch,
                                        s, cp.on ? &lc : nullptr, l == 0, &updates, l));
            Gcur = Gnext;
            continue;
        }
        GCN_TRY(do_layer_bwd(fn, g, F, h, Gcur, ldH, Hin, ldin, act(sl.pub.AH[l]),
                             sl.pub.ld_AH[l], P->W_self[l], P->W_neigh[l],
                             d->has_bias ? P->b[l] : nullptr, oa,
                             layer_state(d, st1, st2, l, 0), layer_state(d, st1, st2, l, 1),
                             Gnext, ldH, grads ? grads->W_self[l] : nullptr,
                             grads ? grads->W_neigh[l] : nullptr,
                             grads ? grads->b[l] : nullptr, bf16, sp, scratch, s,
                             cp.on ? &lc : nullptr, l == 0, &updates, l));
        Gcur = Gnext;
    }
    GCN_HIP(launch_sgd_reduce(updates.p, updates.n, oa, s), fn);
    return GCN_OK;
}

}  // namespace

extern "C" {

int gcn_train_step(const gcn_dgraph* g, const gcn_model_desc* d, const gcn_params* P,
                   const float* X, const void* labels, float lr, float* loss_out,
                   const gcn_params* grads, void* ws, size_t ws_bytes,
                   gcn_stream_t stream) {
    return train_step_impl("gcn_train_step", g, d, P, X, labels, sgd_args(lr), nullptr,
                           nullptr, loss_out, grads, ws, ws_bytes, stream);
}

int gcn_infer(const gcn_dgraph* g, const gcn_model_desc* d, const gcn_params* P,
              const float* X, float* logits, int64_t ld_logits, void* ws, size_t ws_bytes,
              gcn_stream_t stream) {
    GCN_CHECK_ARG(ld_logits > 0, "gcn_infer: ld_logits must be positive");
    return train_step_impl("gcn_infer", g, d, P, X, nullptr, sgd_args(0.f), nullptr, nullptr,
                           nullptr, nullptr, ws, ws_bytes, stream, logits, ld_logits);
}

int gcn_train_step_optim(const gcn_dgraph* g, const gcn_model_desc* d, const gcn_params* P,
                         const float* X, const void* labels, const gcn_optim* opt,
                         const gcn_params* state1, const gcn_params* state2,
                         float* loss_out, const gcn_params* grads, void* ws,
                         size_t ws_bytes, gcn_stream_t stream) {
    const char* fn = "gcn_train_step_optim";
    GCN_CHECK_ARG(opt != nullptr, "%s: opt is NULL", fn);
    GCN_TRY(check_desc(fn, d));
    GCN_CHECK_ARG(std::isfinite(opt->lr), "%s: lr is not finite", fn);
    OptimArgs oa = sgd_args(opt->lr);
    const gcn_params* s1 = nullptr;
    const gcn_params* s2 = nullptr;
    switch (opt->kind) {
        case GCN_OPT_SGD:
            break;
        case GCN_OPT_MOMENTUM:
            GCN_CHECK_ARG(opt->momentum >= 0.f && opt->momentum < 1.f,
                          "%s: momentum %g outside [0, 1)", fn, (double)opt->momentum);
            GCN_TRY(check_state(fn, "state1", d, state1));
            oa.kind = OPT_MOMENTUM;
            oa.mu = opt->momentum;
            s1 = state1;
            break;
        case GCN_OPT_ADAM: {
            GCN_CHECK_ARG(opt->beta1 >= 0.f && opt->beta1 < 1.f && opt->beta2 >= 0.f &&
                              opt->beta2 < 1.f,
                          "%s: beta1 %g / beta2 %g outside [0, 1)", fn, (double)opt->beta1,
                          (double)opt->beta2);
            GCN_CHECK_ARG(opt->eps > 0.f && std::isfinite(opt->eps), "%s: eps must be > 0",
                          fn);
            GCN_CHECK_ARG(opt->step >= 1, "%s: step %d < 1", fn, opt->step);
            GCN_TRY(check_state(fn, "state1", d, state1));
            GCN_TRY(check_state(fn, "state2", d, state2));
            oa.kind = OPT_ADAM;
            oa.b1 = opt->beta1;
            oa.b2 = opt->beta2;
            oa.eps = opt->eps;
            oa.c1 = (float)(1.0 / (1.0 - std::pow((double)opt->beta1, (double)opt->step)));
            oa.c2 = (float)(1.0 / (1.0 - std::pow((double)opt->beta2, (double)opt->step)));
            s1 = state1;
            s2 = state2;
            break;
        }
        default:
            set_error("%s: unknown optimiser kind %d", fn, opt->kind);
            return GCN_E_INVALID_ARG;
    }
    return train_step_impl(fn, g, d, P, X, labels, oa, s1, s2, loss_out, grads, ws, ws_bytes,
                           stream);
}

}  // extern "C"
