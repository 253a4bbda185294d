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
// otherwise). Lists longer than the piece length are split on the host into
// pieces that one workgroup of kBinGroups groups runs side by side (the
// image's bins): the groups holding later pieces of a row leave their sums
// in LDS and the group holding its first piece adds them in group order,
// so the result is deterministic, one launch finishes every row, and no row
// serialises one group for thousands of neighbours.
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

// Adds entries [b, e) of a list to acc, for the float4 columns
// base + lane + j * GL (j < NCH) below nf4.
template <int GL, int NCH, bool PRE>
__device__ __forceinline__ void add_piece(float4 (&acc)[NCH], const int32_t* __restrict__ col,
                                          int b, int e, const RowSource& src,
                                          const float* __restrict__ inv_deg, int base, int nf4,
                                          int lane) {
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
}

// Float4 columns per hub workgroup of T threads (T / hub_cols(T) neighbour
// rows in flight per step, four steps per batch).
constexpr int hub_cols(int T) { return T >= 1024 ? 8 : 4; }

// A hub's list (one row of more than kBinGroups pieces), for float4 columns
// [cs * SW, cs * SW + SW): thread t takes column cs * SW + t % SW of
// neighbours t / SW, t / SW + NSUB, ... in list order (four in flight, the
// next four ids fetched meanwhile); a tree over LDS then adds the NSUB sums
// of each column in a fixed order, and the first NSUB-th of the threads
// finishes and stores the row. The hub's workgroups split its columns, so
// no sum crosses a workgroup.
template <int T, bool PRE, int EPI>
__device__ __forceinline__ void hub_row(int h, int cs, const int4* __restrict__ seg,
                                        const int32_t* __restrict__ bins,
                                        const int32_t* __restrict__ col, const RowSource& src,
                                        const float* __restrict__ inv_deg,
                                        const float* __restrict__ bias, float* __restrict__ Y,
                                        int64_t ldy, int F, __bf16* __restrict__ Yh,
                                        int64_t ldyh, float4* red) {
    constexpr int SW = hub_cols(T), NSUB = T / SW;
    const int t = (int)threadIdx.x, sub = t / SW;
    const int s0 = bins[h], s1 = bins[h + 1];
    const int4 f0 = seg[s0];
    const int row = f0.x, E = seg[s1 - 1].z;
    const int nf4 = (F + 3) >> 2;
    const int c4 = cs * SW + t % SW;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c4 < nf4) {
        auto id = [&](int i) { return i < E ? col[i] : -1; };
        int c[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) c[u] = id(f0.y + sub + u * NSUB);
        for (int i = f0.y + sub; i < E; i += 4 * NSUB) {
            int nx[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) nx[u] = id(i + (4 + u) * NSUB);
            float4 v[4];
            float sc[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                sc[u] = 1.0f;
                if (c[u] >= 0) {
                    v[u] = ld4(row_of(src, c[u]) + 4 * c4);
                    if (PRE && c[u] < src.n) sc[u] = inv_deg[c[u]];
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (c[u] >= 0) {
                    if (PRE) fma4(acc, sc[u], v[u]);
                    else add4(acc, v[u]);
                }
                c[u] = nx[u];
            }
        }
    }
    red[t] = acc;
    __syncthreads();
    for (int st = NSUB / 2; st > 0; st >>= 1) {
        if (sub < st) {
            float4 a = red[t];
            add4(a, red[t + st * SW]);
            red[t] = a;
        }
        __syncthreads();
    }
    if (sub == 0 && c4 < nf4)
        put_row(Y, ldy, Yh, ldyh, row, 4 * c4, finish_row<EPI>(red[t], row, c4, inv_deg, bias, F),
                F - 4 * c4);
}

// Pair sums (Section 4.2 step 1): one group per expansion list
// (k, begin, end, -1), stored as aux row k.
template <int GL, int NCH, bool PRE>
__global__ __launch_bounds__(kBlock) void pair_sums_kernel(
    const int4* __restrict__ seg, int nseg, const int32_t* __restrict__ col, RowSource src,
    const float* __restrict__ inv_deg, float* __restrict__ aux, int64_t ldaux, int F, int nsl,
    int slice_f4) {
    const int lane = (int)threadIdx.x % GL;
    const int sidx = group_index<GL>(nsl);
    if (sidx >= nseg) return;
    const int4 sg = seg[sidx];
    const Slice sl = slice_of(nsl, slice_f4, (F + 3) >> 2);
    const int nf4 = sl.c4_end;
    for (int base = sl.c4_begin; base < nf4; base += GL * NCH) {
        float4 acc[NCH];
#pragma unroll
        for (int j = 0; j < NCH; ++j) acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        add_piece<GL, NCH, PRE>(acc, col, sg.y, sg.z, src, inv_deg, base, nf4, lane);
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            const int c4 = base + lane + j * GL;
            if (c4 < nf4) st4_masked(aux + (int64_t)sg.x * ldaux + 4 * c4, acc[j], F - 4 * c4);
        }
    }
}

// List sums (step 2, with step 3 fused). The first hub_blocks workgroups
// take the nhub hubs, hub_slices column ranges each (hub_row); the others
// take one (bin, column slice) each, with kBinGroups groups: group g takes
// piece g of the bin, and a group whose piece starts its row (lead = the
// row's piece count) finishes that row, after adding, for a split row, the
// sums that the next lead - 1 groups leave in LDS, in group order.
template <int GL, int NCH, bool PRE, int EPI>
__global__ __launch_bounds__(kBinGroups * GL) void list_sums_kernel(
    const int4* __restrict__ seg, const int32_t* __restrict__ bins, int nmulti, int nhub,
    int hub_slices, int hub_blocks, const int32_t* __restrict__ col, RowSource src,
    const float* __restrict__ inv_deg, const float* __restrict__ bias, float* __restrict__ Y,
    int64_t ldy, int F, int nsl, int slice_f4, __bf16* __restrict__ Yh, int64_t ldyh) {
    constexpr int G = kBinGroups, T = G * GL;
    // sums of groups 1..G-1 (group 0 always starts a row), or a hub's T sums
    constexpr int kRed = (G - 1) * NCH * GL > T ? (G - 1) * NCH * GL : T;
    __shared__ float4 red[kRed];
    if ((int)blockIdx.x < hub_blocks) {
        // block b runs on XCD b % 8; (hub, slice) pairs are dealt to the
        // XCDs in contiguous runs, so neighbouring slices, which share
        // cache lines, share an L2
        const int b = (int)blockIdx.x;
        const int q = (b % 8) * (hub_blocks / 8) + b / 8;
        const int h = q / hub_slices;
        if (h < nhub)
            hub_row<T, PRE, EPI>(h, q % hub_slices, seg, bins, col, src, inv_deg, bias, Y, ldy,
                                 F, Yh, ldyh, red);
        return;
    }
    // hub_blocks is a multiple of 8, so slice b % nsl still runs on XCD b % 8
    const int b = (int)blockIdx.x - hub_blocks;
    const int lane = (int)threadIdx.x % GL;
    int grp = (int)threadIdx.x / GL;
    if constexpr (GL == 64) grp = __builtin_amdgcn_readfirstlane(grp);
    const int bin = nhub + b / nsl;
    const int s0 = bins[bin], s1 = bins[bin + 1];
    const bool multi = bin < nmulti;   // the same for the whole workgroup
    const bool has = s0 + grp < s1;
    const int4 f = has ? seg[s0 + grp] : make_int4(0, 0, 0, 0);
    const int row = f.x, lead = f.w;
    const int sb = (b % nsl) * slice_f4;
    const int nf4 = min((F + 3) >> 2, sb + slice_f4);
    for (int base = sb; base < nf4; base += GL * NCH) {
        float4 acc[NCH];
#pragma unroll
        for (int j = 0; j < NCH; ++j) acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (has) add_piece<GL, NCH, PRE>(acc, col, f.y, f.z, src, inv_deg, base, nf4, lane);
        if (multi) {
            if (has && lead == 0 && grp > 0) {
#pragma unroll
                for (int j = 0; j < NCH; ++j) red[((grp - 1) * NCH + j) * GL + lane] = acc[j];
            }
            __syncthreads();
            if (lead > 1) {
                const int m = min(lead, G - grp);
                for (int q = grp + 1; q < grp + m; ++q) {
#pragma unroll
                    for (int j = 0; j < NCH; ++j) add4(acc[j], red[((q - 1) * NCH + j) * GL + lane]);
                }
            }
        }
        if (lead > 0) {
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
                const int c4 = base + lane + j * GL;
                if (c4 < nf4)
                    put_row(Y, ldy, Yh, ldyh, row, 4 * c4,
                            finish_row<EPI>(acc[j], row, c4, inv_deg, bias, F), F - 4 * c4);
            }
        }
        // the next pass rewrites red
        if (multi && base + GL * NCH < nf4) __syncthreads();
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
#define GCN_LAUNCH_PAIR(GL_, NCH_)                                                         \
    if (sh.gl == GL_ && sh.nch == NCH_) {                                                  \
        if (prescale)                                                                      \
            pair_sums_kernel<GL_, NCH_, true><<<grid, block, 0, s>>>(                      \
                seg, g->naux, g->exp_col, src, g->inv_deg, aux, ldaux, F, sh.nsl, sh.slice_f4); \
        else                                                                               \
            pair_sums_kernel<GL_, NCH_, false><<<grid, block, 0, s>>>(                     \
                seg, g->naux, g->exp_col, src, g->inv_deg, aux, ldaux, F, sh.nsl, sh.slice_f4); \
        return hipGetLastError();                                                          \
    }
    GCN_SHAPES(GCN_LAUNCH_PAIR)
#undef GCN_LAUNCH_PAIR
    return hipErrorInvalidValue;
}

hipError_t launch_list_sums(const gcn_dgraph* g, RowSource src, bool prescale, AggEpi epi,
                            const float* bias, float* Y, int64_t ldy, int32_t F, hipStream_t s,
                            __bf16* Yh, int64_t ldyh) {
    if (g->n <= 0 || F <= 0) return hipSuccess;
    if (prescale && epi != AGG_SUM) return hipErrorInvalidValue;
    const Shape sh = pick_shape(F);
    const int4* seg = reinterpret_cast<const int4*>(g->seg);
    const int T = kBinGroups * sh.gl;
    const int hub_slices = ((F + 3) / 4 + hub_cols(T) - 1) / hub_cols(T);
    const int64_t hub_blocks = ((int64_t)g->nhub * hub_slices + 7) / 8 * 8;
    const int64_t blocks = hub_blocks + (int64_t)(g->nbins - g->nhub) * sh.nsl;
    if (blocks > INT32_MAX) return hipErrorInvalidValue;
    const dim3 block(T), grid((unsigned)blocks);
    const double nnz = (double)g->nnz, n = (double)g->n;
    // algorithmic: one gather per list entry, its id, one write per row
    ProfScope prof(s, K_LIST_SUMS,
                   nnz * F * (prescale ? 2.0 : 1.0) + (epi != AGG_SUM ? n * F : 0.0),
                   4.0 * F * nnz + 4.0 * nnz + (Yh ? 2.0 : 4.0) * F * n);
#define GCN_LAUNCH_LIST(GL_, NCH_)                                                          \
    if (sh.gl == GL_ && sh.nch == NCH_) {                                                   \
        if (prescale)                                                                       \
            list_sums_kernel<GL_, NCH_, true, AGG_SUM><<<grid, block, 0, s>>>(              \
                seg, g->bins, g->nmulti, g->nhub, hub_slices, (int)hub_blocks, g->col, src, \
                g->inv_deg, nullptr, Y, ldy, F,                                             \
                sh.nsl, sh.slice_f4, Yh, ldyh);                                             \
        else if (epi == AGG_MEAN)                                                           \
            list_sums_kernel<GL_, NCH_, false, AGG_MEAN><<<grid, block, 0, s>>>(            \
                seg, g->bins, g->nmulti, g->nhub, hub_slices, (int)hub_blocks, g->col, src, \
                g->inv_deg, nullptr, Y, ldy, F,                                             \
                sh.nsl, sh.slice_f4, Yh, ldyh);                                             \
        else                                                                                \
            list_sums_kernel<GL_, NCH_, false, AGG_MEAN_BIAS_RELU><<<grid, block, 0, s>>>(  \
                seg, g->bins, g->nmulti, g->nhub, hub_slices, (int)hub_blocks, g->col, src, \
                g->inv_deg, bias, Y, ldy, F,                                                \
                sh.nsl, sh.slice_f4, Yh, ldyh);                                             \
        return hipGetLastError();                                                           \
    }
    GCN_SHAPES(GCN_LAUNCH_LIST)
#undef GCN_LAUNCH_LIST
    return hipErrorInvalidValue;
}

}  // namespace gcn
