// Feature aggregation on G_s^# (Section 4.2): pair sums (step 1), list sums
// (step 2) and the degree scaling (step 3, fused). The pair sums of all
// rounds are formed in one launch, each from its expansion into original
// rows (a list like any other), so no launch waits on an earlier round.
//
// Work decomposition (gfx950, 64-lane wavefronts): a group of GL lanes
// (16, 32 or 64, chosen from the feature width) owns one pair sum or one list
// segment and sweeps the feature row in float4 chunks, NCH chunks per lane,
// so every neighbour-row gather is a coalesced run of GL*16 bytes. The
// group loads up to GL neighbour ids at once (one per lane) and broadcasts
// them lane by lane (readlane for a full wavefront, a width-GL shuffle
// otherwise). Lists longer than the segment length are split on the host;
// their segments write partial sums to scratch slots that a second pass adds
// in slot order, so the result is deterministic and no row serialises a
// whole wavefront for thousands of neighbours.
// Wide rows (F >= 512) are cut into 8 column slices and workgroup b works on
// slice b % 8, which is also the XCD it runs on: each XCD then gathers only
// its slice of every feature row, so its 4 MB L2 holds that slice of the
// whole matrix instead of every XCD streaming all of it.
#include "kernels.h"
#include "prof.h"

namespace gcn {
namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ const float* row_of(const RowSource& s, int c) {
    return c < s.n ? s.X + (int64_t)c * s.ldx
                   : s.aux + (int64_t)(c - s.n) * s.ldaux;
}

__device__ __forceinline__ float4 ld4(const float* p) {
    return *reinterpret_cast<const float4*>(p);
}

__device__ __forceinline__ void st4(float* p, float4 v) {
    *reinterpret_cast<float4*>(p) = v;
}

// stores the first `valid` elements of v (valid >= 1)
__device__ __forceinline__ void st4_masked(float* p, float4 v, int valid) {
    if (valid >= 4) {
        st4(p, v);
        return;
    }
    p[0] = v.x;
    if (valid > 1) p[1] = v.y;
    if (valid > 2) p[2] = v.z;
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// bf16 (nearest even) of the first `valid` elements of v (valid >= 1)
__device__ __forceinline__ void st4h_masked(__bf16* p, float4 v, int valid) {
    if (valid >= 4) {
        bf16x4 h;
        h[0] = (__bf16)v.x;
        h[1] = (__bf16)v.y;
        h[2] = (__bf16)v.z;
        h[3] = (__bf16)v.w;
        *reinterpret_cast<bf16x4*>(p) = h;
        return;
    }
    p[0] = (__bf16)v.x;
    if (valid > 1) p[1] = (__bf16)v.y;
    if (valid > 2) p[2] = (__bf16)v.z;
}

// A finished row chunk goes to Yh as bf16 when Yh is set, else to Y.
__device__ __forceinline__ void put_row(float* Y, int64_t ldy, __bf16* Yh, int64_t ldyh, int row,
                                        int c, float4 v, int valid) {
    if (Yh)
        st4h_masked(Yh + (int64_t)row * ldyh + c, v, valid);
    else
        st4_masked(Y + (int64_t)row * ldy + c, v, valid);
}

__device__ __forceinline__ void fma4(float4& acc, float s, float4 v) {
    acc.x = fmaf(s, v.x, acc.x);
    acc.y = fmaf(s, v.y, acc.y);
    acc.z = fmaf(s, v.z, acc.z);
    acc.w = fmaf(s, v.w, acc.w);
}

__device__ __forceinline__ void add4(float4& acc, float4 v) {
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
}

template <int GL>
__device__ __forceinline__ int bcast_i(int v, int t) {
    if constexpr (GL == 64) {
        return __builtin_amdgcn_readlane(v, t);
    } else {
        return __shfl(v, t, GL);
    }
}

template <int GL>
__device__ __forceinline__ float bcast_f(float v, int t) {
    return __int_as_float(bcast_i<GL>(__float_as_int(v), t));
}

// Column slice and group index of this thread: workgroup b covers slice
// b % nsl; the group index is made wave-uniform when the group is a whole
// wavefront.
struct Slice {
    int c4_begin, c4_end;   // float4 columns [begin, end)
};

template <int GL>
__device__ __forceinline__ int group_index(int nsl) {
    int g = (int)(blockIdx.x / nsl) * (kBlock / GL) + (int)threadIdx.x / GL;
    if constexpr (GL == 64) g = __builtin_amdgcn_readfirstlane(g);
    return g;
}

__device__ __forceinline__ Slice slice_of(int nsl, int slice_f4, int nf4) {
    const int sl = (int)(blockIdx.x % nsl);
    const int b = sl * slice_f4;
    return {b, min(nf4, b + slice_f4)};
}

// What a finished list sum becomes (AggEpi): the sum itself, its mean
// over the original degree, or max(mean + bias, 0) (the neighbour branch
// of Eq. 1 when the transform runs before the aggregation).
template <int EPI>
__device__ __forceinline__ float4 finish_row(float4 v, int row, int c4,
                                             const float* __restrict__ inv_deg,
                                             const float* __restrict__ bias, int F) {
    if constexpr (EPI != AGG_SUM) {
        const float sc = inv_deg[row];
        v = make_float4(v.x * sc, v.y * sc, v.z * sc, v.w * sc);
    }
    if constexpr (EPI == AGG_MEAN_BIAS_RELU) {
        if (bias) {
            const int c = 4 * c4;
            v.x += bias[c];
            if (c + 1 < F) v.y += bias[c + 1];
            if (c + 2 < F) v.z += bias[c + 2];
            if (c + 3 < F) v.w += bias[c + 3];
        }
        // max(x, 0) keeping a NaN, as the GEMM epilogues do
        auto relu = [](float x) { return x <= 0.f ? 0.f : x; };
        v = make_float4(relu(v.x), relu(v.y), relu(v.z), relu(v.w));
    }
    return v;
}

// One group per segment (row, begin, end, slot) of the work list. PAIRS
// marks the pair-sum launches (same code; a kernel name of their own so
// per-kernel profiles and counters separate the two passes).
template <int GL, int NCH, bool PRE, int EPI, bool PAIRS>
__global__ __launch_bounds__(kBlock) void list_sums_kernel(
    const int4* __restrict__ seg, int nseg, const int32_t* __restrict__ col,
    RowSource src, const float* __restrict__ inv_deg, const float* __restrict__ bias,
    float* __restrict__ Y, int64_t ldy, float* __restrict__ partial, int64_t ldp, int F, int nsl,
    int slice_f4, __bf16* __restrict__ Yh, int64_t ldyh) {
    const int lane = (int)threadIdx.x % GL;
    const int sidx = group_index<GL>(nsl);
    if (sidx >= nseg) return;
    const int4 sg = seg[sidx];
    const int row = sg.x, b = sg.y, e = sg.z, slot = sg.w;
    const Slice sl = slice_of(nsl, slice_f4, (F + 3) >> 2);
    const int nf4 = sl.c4_end;
    for (int base = sl.c4_begin; base < nf4; base += GL * NCH) {
        float4 acc[NCH];
#pragma unroll
        for (int j = 0; j < NCH; ++j) acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int i0 = b; i0 < e; i0 += GL) {
            const int cnt = min(GL, e - i0);
            int my_c = 0;
            float my_s = 1.0f;
            if (lane < cnt) {
                my_c = col[i0 + lane];
                if (PRE && my_c < src.n) my_s = inv_deg[my_c];
            }
            int t = 0;
            // four neighbours in flight per step
            for (; t + 4 <= cnt; t += 4) {
                const float* r[4];
                float s[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    r[u] = row_of(src, bcast_i<GL>(my_c, t + u));
                    s[u] = PRE ? bcast_f<GL>(my_s, t + u) : 1.0f;
                }
#pragma unroll
                for (int j = 0; j < NCH; ++j) {
                    const int c4 = base + lane + j * GL;
                    if (c4 < nf4) {
                        float4 v[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u) v[u] = ld4(r[u] + 4 * c4);
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            if (PRE) fma4(acc[j], s[u], v[u]);
                            else add4(acc[j], v[u]);
                        }
                    }
                }
            }
            for (; t < cnt; ++t) {
                const float* r = row_of(src, bcast_i<GL>(my_c, t));
                const float s = PRE ? bcast_f<GL>(my_s, t) : 1.0f;
#pragma unroll
                for (int j = 0; j < NCH; ++j) {
                    const int c4 = base + lane + j * GL;
                    if (c4 < nf4) {
                        float4 v = ld4(r + 4 * c4);
                        if (PRE) fma4(acc[j], s, v);
                        else add4(acc[j], v);
                    }
                }
            }
        }
        if (slot < 0) {
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
                const int c4 = base + lane + j * GL;
                if (c4 < nf4)
                    put_row(Y, ldy, Yh, ldyh, row, 4 * c4,
                            finish_row<EPI>(acc[j], row, c4, inv_deg, bias, F), F - 4 * c4);
            }
        } else {
            float* out = partial + (int64_t)slot * ldp;
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
                const int c4 = base + lane + j * GL;
                if (c4 < nf4) st4(out + 4 * c4, acc[j]);
            }
        }
    }
}

// One group per split list: add its slots in order, finish, store.
template <int GL, int NCH, int EPI>
__global__ __launch_bounds__(kBlock) void fixup_kernel(
    const int4* __restrict__ longrows, int nlong,
    const float* __restrict__ partial, int64_t ldp,
    const float* __restrict__ inv_deg, const float* __restrict__ bias, float* __restrict__ Y,
    int64_t ldy, int F, int nsl, int slice_f4, __bf16* __restrict__ Yh, int64_t ldyh) {
    const int lane = (int)threadIdx.x % GL;
    const int li = group_index<GL>(nsl);
    if (li >= nlong) return;
    const int4 lr = longrows[li];
    const int row = lr.x, first = lr.y, ns = lr.z;
    const Slice sl = slice_of(nsl, slice_f4, (F + 3) >> 2);
    const int nf4 = sl.c4_end;
    for (int base = sl.c4_begin; base < nf4; base += GL * NCH) {
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            const int c4 = base + lane + j * GL;
            if (c4 < nf4) {
                // eight slots in flight, added in slot order
                const float* src = partial + (int64_t)first * ldp + 4 * c4;
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                int sI = 0;
                for (; sI + 8 <= ns; sI += 8) {
                    float4 v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) v[u] = ld4(src + (int64_t)(sI + u) * ldp);
#pragma unroll
                    for (int u = 0; u < 8; ++u) add4(acc, v[u]);
                }
                for (; sI < ns; ++sI) add4(acc, ld4(src + (int64_t)sI * ldp));
                put_row(Y, ldy, Yh, ldyh, row, 4 * c4,
                        finish_row<EPI>(acc, row, c4, inv_deg, bias, F), F - 4 * c4);
            }
        }
    }
}

struct Shape {
    int gl, nch;      // lanes per group, float4 per lane per pass
    int nsl;          // column slices (8: one per XCD)
    int slice_f4;     // float4 columns per slice
};

Shape lanes_for(int f4) {
    if (f4 <= 16) return {16, 1, 1, f4};
    if (f4 <= 32) return {32, 1, 1, f4};
    if (f4 <= 64) return {64, 1, 1, f4};
    if (f4 <= 128) return {64, 2, 1, f4};
    if (f4 <= 192) return {64, 3, 1, f4};
    return {64, 4, 1, f4};
}

Shape pick_shape(int F) {
    const int nf4 = (F + 3) / 4;
    if (nf4 < 128) return lanes_for(nf4);
    const int slice = (nf4 + 7) / 8;
    Shape sh = lanes_for(slice);
    sh.nsl = 8;
    sh.slice_f4 = slice;
    return sh;
}

int blocks_for(int groups, const Shape& sh) {
    const int per = kBlock / sh.gl;
    return ((groups + per - 1) / per) * sh.nsl;
}

#define GCN_SHAPES(X) \
    X(16, 1) X(32, 1) X(64, 1) X(64, 2) X(64, 3) X(64, 4)

}  // namespace

hipError_t launch_pair_sums(const gcn_dgraph* g, RowSource src, bool prescale,
                            float* aux, int64_t ldaux, int32_t F, hipStream_t s) {
    if (g->naux <= 0 || F <= 0) return hipSuccess;
    const Shape sh = pick_shape(F);
    const int4* seg = reinterpret_cast<const int4*>(g->exp_seg);
    const dim3 grid(blocks_for(g->naux, sh)), block(kBlock);
    const double e = (double)g->exp_nnz, k = (double)g->naux;
    // one gather per expansion entry, its id, one write per pair sum
    ProfScope prof(s, K_PAIR_SUMS, e * F * (prescale ? 2.0 : 1.0), 4.0 * F * e + 4.0 * e + 4.0 * F * k);
#define GCN_LAUNCH_PAIR(GL_, NCH_)                                                          \
    if (sh.gl == GL_ && sh.nch == NCH_) {                                                   \
        if (prescale)                                                                       \
            list_sums_kernel<GL_, NCH_, true, AGG_SUM, true><<<grid, block, 0, s>>>(        \
                seg, g->naux, g->exp_col, src, g->inv_deg, nullptr, aux, ldaux, nullptr, 0, \
                F, sh.nsl, sh.slice_f4, nullptr, 0);                                        \
        else                                                                                \
            list_sums_kernel<GL_, NCH_, false, AGG_SUM, true><<<grid, block, 0, s>>>(       \
                seg, g->naux, g->exp_col, src, g->inv_deg, nullptr, aux, ldaux, nullptr, 0, \
                F, sh.nsl, sh.slice_f4, nullptr, 0);                                        \
        return hipGetLastError();                                                           \
    }
    GCN_SHAPES(GCN_LAUNCH_PAIR)
#undef GCN_LAUNCH_PAIR
    return hipErrorInvalidValue;
}

hipError_t launch_list_sums(const gcn_dgraph* g, RowSource src, bool prescale, AggEpi epi,
                            const float* bias, float* Y, int64_t ldy, float* partial,
                            int64_t ldp, int32_t F, hipStream_t s, __bf16* Yh, int64_t ldyh) {
    if (g->n <= 0 || F <= 0) return hipSuccess;
    if (prescale && epi != AGG_SUM) return hipErrorInvalidValue;
    const Shape sh = pick_shape(F);
    const int4* seg = reinterpret_cast<const int4*>(g->seg);
    const int4* lr = reinterpret_cast<const int4*>(g->longrows);
    const dim3 block(kBlock);
    const dim3 grid(blocks_for(g->nseg, sh));
    const dim3 gfix(blocks_for(g->nlong, sh));
    const double nnz = (double)g->nnz, n = (double)g->n;
    {
        // algorithmic: one gather per list entry, its id, one write per row
        ProfScope prof(s, K_LIST_SUMS,
                       nnz * F * (prescale ? 2.0 : 1.0) + (epi != AGG_SUM ? n * F : 0.0),
                       4.0 * F * nnz + 4.0 * nnz + (Yh ? 2.0 : 4.0) * F * n);
#define GCN_LAUNCH_LIST(GL_, NCH_)                                                           \
        if (sh.gl == GL_ && sh.nch == NCH_) {                                                \
            if (prescale)                                                                    \
                list_sums_kernel<GL_, NCH_, true, AGG_SUM, false><<<grid, block, 0, s>>>(    \
                    seg, g->nseg, g->col, src, g->inv_deg, nullptr, Y, ldy, partial, ldp, F, \
                    sh.nsl, sh.slice_f4, Yh, ldyh);                                          \
            else if (epi == AGG_MEAN)                                                        \
                list_sums_kernel<GL_, NCH_, false, AGG_MEAN, false><<<grid, block, 0, s>>>(  \
                    seg, g->nseg, g->col, src, g->inv_deg, nullptr, Y, ldy, partial, ldp, F, \
                    sh.nsl, sh.slice_f4, Yh, ldyh);                                          \
            else                                                                             \
                list_sums_kernel<GL_, NCH_, false, AGG_MEAN_BIAS_RELU, false>                \
                    <<<grid, block, 0, s>>>(seg, g->nseg, g->col, src, g->inv_deg, bias, Y,  \
                                            ldy, partial, ldp, F, sh.nsl, sh.slice_f4, Yh,   \
                                            ldyh);                                           \
        } else
        GCN_SHAPES(GCN_LAUNCH_LIST) { return hipErrorInvalidValue; }
#undef GCN_LAUNCH_LIST
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (g->nlong == 0) return hipSuccess;
    ProfScope prof(s, K_LIST_FIXUP, (double)g->nslots * F,
                   4.0 * F * g->nslots + (Yh ? 2.0 : 4.0) * F * g->nlong);
#define GCN_LAUNCH_FIX(GL_, NCH_)                                                             \
    if (sh.gl == GL_ && sh.nch == NCH_) {                                                     \
        if (epi == AGG_SUM)                                                                   \
            fixup_kernel<GL_, NCH_, AGG_SUM><<<gfix, block, 0, s>>>(                          \
                lr, g->nlong, partial, ldp, g->inv_deg, nullptr, Y, ldy, F, sh.nsl, sh.slice_f4, \
                Yh, ldyh);                                                                    \
        else if (epi == AGG_MEAN)                                                             \
            fixup_kernel<GL_, NCH_, AGG_MEAN><<<gfix, block, 0, s>>>(                         \
                lr, g->nlong, partial, ldp, g->inv_deg, nullptr, Y, ldy, F, sh.nsl, sh.slice_f4, \
                Yh, ldyh);                                                                    \
        else                                                                                  \
            fixup_kernel<GL_, NCH_, AGG_MEAN_BIAS_RELU><<<gfix, block, 0, s>>>(               \
                lr, g->nlong, partial, ldp, g->inv_deg, bias, Y, ldy, F, sh.nsl, sh.slice_f4,    \
                Yh, ldyh);                                                                    \
    } else
    GCN_SHAPES(GCN_LAUNCH_FIX) { return hipErrorInvalidValue; }
#undef GCN_LAUNCH_FIX
    return hipGetLastError();
}

}  // namespace gcn
