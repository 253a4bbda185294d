// Dense products of the layer (Eq. 1 transforms, Eq. 2 gradients) on the
// gfx950 matrix cores: v_mfma_f32_32x32x2_f32, fp32 in and out.
//
// Tile: 128 x 128 per 256-thread workgroup (one workgroup per CU: LDS holds
// two 64-deep K steps of both operands), four wavefronts in a 2 x 2 grid, each
// owning 64 x 64 = 2 x 2 MFMA 32x32 accumulators.
// LDS layout follows HBM: an operand whose rows are contiguous along K
// (A_MK, B_NK) is kept [row][k] and its fragments are read 4 K values at a
// time with 128-bit LDS reads; a K-major operand (A_KM, B_KN) is kept [k][col]
// and read 32 consecutive floats per half-wave. Both fill LDS with 128-bit
// stores, no transposition. Within a group of 8 K values, MFMA step j of lane
// half g takes k = 4 g + j (a fixed permutation of K, the same for A and B).
// Global loads for the next K step are issued before the current step's MFMAs
// and written to the other LDS buffer after them (one barrier per step); LDS
// fragments of the next group are read before the current group's MFMAs.
// Ragged M / N / K edges are zero-filled at LDS-store time. Epilogues fuse
// what the layer needs next: bias + ReLU + placement into one half of the
// concatenated output (forward), the ReLU mask of the previous layer (input
// gradient), or a split-K slice (weight gradient, summed later in fixed
// order). Tiles are renumbered so consecutive tiles (sharing A rows or a K
// range) land on the same XCD, whose L2 then serves their common operand.
#include <algorithm>
#include <cstring>
#include <type_traits>

#include "kernels.h"
#include "prof.h"

namespace gcn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int kThreads = 256;
constexpr int kXcds = 8;
constexpr int kQuads = BK * BM / 4 / kThreads;   // float4 loads per operand per step
constexpr int kRowStride = BK + 4;               // [row][k] layout, floats
constexpr int kColStride = BM + 4;               // [k][col] layout, floats
constexpr int kOperandFloats = (BM * kRowStride > BK * kColStride) ? BM * kRowStride
                                                                   : BK * kColStride;

__device__ __forceinline__ float4 ld4(const float* p) {
    return *reinterpret_cast<const float4*>(p);
}

// max(x, 0) that keeps a NaN (as IEEE maximum does), so a non-finite input
// reaches the loss instead of vanishing in a ReLU
__device__ __forceinline__ float relu(float x) { return x <= 0.f ? 0.f : x; }

// Whole K steps [kbeg, kbeg + nfull * BK) of a K-concatenated operand load
// from one per-step base plus fixed per-thread offsets when the
// concatenation point lies past them (a one-part operand has it at K), or
// on a K-step boundary between parts of equal leading dimension (kbeg is a
// multiple of BK).
__device__ __forceinline__ bool concat_fast(int ksplit, int kbeg, int nfull, int64_t ld1,
                                            int64_t ld0) {
    return ksplit >= kbeg + nfull * BK || (ksplit % BK == 0 && ld1 == ld0);
}

__device__ __forceinline__ void zero_from(float4& v, int valid) {
    // keep the first `valid` elements (valid may be <= 0 or >= 4)
    if (valid < 4) v.w = 0.f;
    if (valid < 3) v.z = 0.f;
    if (valid < 2) v.y = 0.f;
    if (valid < 1) v.x = 0.f;
}

// Operand loads are split in two halves so that prefetching never waits:
// the load half only issues memory reads and records how many of the four
// elements are valid; the store half, run during the MFMA work of the
// current K step, zero-fills the invalid tail and writes LDS. Vector loads
// are branchless (an empty quad reads the operand's first 16 bytes instead)
// so that a whole K step is one basic block the scheduler can interleave.
struct Quad {
    float4 v;
    int valid;   // elements [0, valid) are real; the rest become 0
    int one;     // element index that is an implicit 1, or -1
};

__device__ __forceinline__ float4 finish(const Quad& q) {
    float4 v = q.v;
    zero_from(v, q.valid);
    if (q.one == 0) v.x = 1.f;
    if (q.one == 1) v.y = 1.f;
    if (q.one == 2) v.z = 1.f;
    if (q.one == 3) v.w = 1.f;
    return v;
}

template <bool VEC>
__device__ __forceinline__ void issue(Quad& q, const float* p, const float* safe, int valid) {
    q.valid = valid;
    if constexpr (VEC) {
        q.v = ld4(valid > 0 ? p : safe);
    } else {
        q.v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (valid > 0) q.v.x = p[0];
        if (valid > 1) q.v.y = p[1];
        if (valid > 2) q.v.z = p[2];
        if (valid > 3) q.v.w = p[3];
    }
}

// Per-thread view of one operand quad: which row / column it covers.
struct RowQuad {      // row-contiguous operand: row r, K offset kofs
    const float* p0;  // row r of the first K-concatenated part
    const float* p1;  // row r of the second part
    bool live;        // r inside the operand
};

struct ColQuad {      // K-major operand: columns c..c+3 of K row kofs + k0
    int c;
};

// Output tile of a workgroup. XCD-aware renumbering: workgroup b runs on
// XCD b % 8, and each XCD gets a contiguous range of logical tiles.
struct TileInfo {
    int pi, split, m0, n0, kbeg, kend, nk;
};

template <int TBM = BM, int TBN = BN>
__device__ __forceinline__ TileInfo decode_tile(const GemmBatch& batch) {
    const int T = batch.total_tiles;
    const int bid = blockIdx.x;
    const int xcd = bid % kXcds, slot = bid / kXcds;
    const int per = T / kXcds, rem = T % kXcds;
    const int tile = xcd * per + min(xcd, rem) + slot;
    TileInfo ti;
    ti.pi = (batch.nprob > 1 && tile >= batch.p[1].tile_begin) ? 1 : 0;
    const GemmProblem& P = batch.p[ti.pi];
    int local = tile - P.tile_begin;
    const int per_split = P.tiles_m * P.tiles_n;
    ti.split = local / per_split;
    local -= ti.split * per_split;
    ti.m0 = (local / P.tiles_n) * TBM;
    ti.n0 = (local % P.tiles_n) * TBN;
    ti.kbeg = ti.split * P.kchunk;
    ti.kend = min(P.K, ti.kbeg + P.kchunk);
    ti.nk = ti.kend > ti.kbeg ? (ti.kend - ti.kbeg + BK - 1) / BK : 0;
    return ti;
}

__device__ __forceinline__ bf16x4 to_bf16(float a, float b, float c, float d) {
    bf16x4 r;
    r[0] = (__bf16)a;
    r[1] = (__bf16)b;
    r[2] = (__bf16)c;
    r[3] = (__bf16)d;
    return r;
}

// Epilogue of a wavefront's block of MB x NB accumulators of 32 x 32.
// The MFMAs take the B fragment as their first operand, so they produce the
// transposed block: accumulator element r of lane l is C[i][j] of its
// 32 x 32 block with i = l % 32 and j = (r % 4) + 8 (r / 4) + 4 (l / 32).
// Every lane thus holds four runs of four consecutive columns of one row,
// stored (and masked) with 16-byte accesses where the row is aligned.
template <Epilogue EP, int MB = 2, int NB = 2>
__device__ __forceinline__ void store_tile(const GemmProblem& P, int split, int mw, int nw,
                                           int half, int l32, const floatx16 (&acc)[MB][NB]) {
    float* C = P.C;
    if constexpr (EP == EPI_PARTIAL) C += (int64_t)split * P.part_stride;
    const bool cvec = ((reinterpret_cast<uintptr_t>(C) | (uintptr_t)(P.ldc * 4)) & 15) == 0;
    bool mvec = false;
    if constexpr (EP == EPI_MASK)
        mvec = ((reinterpret_cast<uintptr_t>(P.mask) | (uintptr_t)(P.ldmask * 4)) & 15) == 0;
#pragma unroll
    for (int bi = 0; bi < MB; ++bi) {
        const int m = mw + bi * 32 + l32;
        if (m >= P.M) continue;
        float* crow = C + (int64_t)m * P.ldc;
#pragma unroll
        for (int bj = 0; bj < NB; ++bj) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = nw + bj * 32 + 8 * g + 4 * half;
                if (n >= P.N) continue;
                const bool whole = n + 4 <= P.N;
                float v[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) v[t] = acc[bi][bj][4 * g + t];
                if constexpr (EP == EPI_BIAS_RELU || EP == EPI_BIAS) {
                    if (P.bias) {
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            if (n + t < P.N) v[t] += P.bias[n + t];
                    }
                    if constexpr (EP == EPI_BIAS_RELU) {
                        if (!P.no_relu) {
#pragma unroll
                            for (int t = 0; t < 4; ++t) v[t] = relu(v[t]);
                        }
                    }
                } else if constexpr (EP == EPI_MASK) {
                    const float* mp = P.mask + (int64_t)m * P.ldmask + n;
                    float h[4];
                    if (whole && mvec) {
                        const float4 q = ld4(mp);
                        h[0] = q.x, h[1] = q.y, h[2] = q.z, h[3] = q.w;
                    } else {
#pragma unroll
                        for (int t = 0; t < 4; ++t) h[t] = n + t < P.N ? mp[t] : 0.f;
                    }
#pragma unroll
                    for (int t = 0; t < 4; ++t) v[t] = h[t] > 0.f ? v[t] : 0.f;
                }
                if (whole && cvec) {
                    *reinterpret_cast<float4*>(crow + n) = make_float4(v[0], v[1], v[2], v[3]);
                } else {
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        if (n + t < P.N) crow[n + t] = v[t];
                }
            }
        }
    }
}

// Epilogue through LDS: the wavefront's 64 x (32 NB) block goes to `stage`
// (its own 32 x (32 NB + 4) floats of the freed operand buffers) 32 rows at
// a time, and is read back so that each load and store instruction covers
// whole row runs of 32 NB floats (8 NB lanes per row) instead of 32 rows x
// 32 bytes. HC: also the bf16 copy. The caller has synchronised the
// workgroup.
template <Epilogue EP, bool HC, int NB = 2>
__device__ __forceinline__ void store_tile_lds(const GemmProblem& P, int split, int mw, int nw,
                                               int half, int l32, int lane, float* stage,
                                               const floatx16 (&acc)[2][NB]) {
    constexpr int kSS = 32 * NB + 4;   // staged row stride, floats
    constexpr int kLPR = 8 * NB;       // lanes per staged row
    constexpr int kRPP = 64 / kLPR;    // rows per read-back pass
    constexpr int kPass = 32 / kRPP;
    float* C = P.C;
    if constexpr (EP == EPI_PARTIAL) C += (int64_t)split * P.part_stride;
    const bool cvec = ((reinterpret_cast<uintptr_t>(C) | (uintptr_t)(P.ldc * 4)) & 15) == 0;
    const bool mvec =
        EP == EPI_MASK &&
        ((reinterpret_cast<uintptr_t>(P.mask) | (uintptr_t)(P.ldmask * 4)) & 15) == 0;
    const int c = 4 * (lane % kLPR);   // this lane's four columns of the block
    const int n = nw + c;
    const bool whole = n + 4 <= P.N;
    float bv[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (EP == EPI_BIAS_RELU || EP == EPI_BIAS) {
        if (P.bias) {
#pragma unroll
            for (int t = 0; t < 4; ++t) bv[t] = n + t < P.N ? P.bias[n + t] : 0.f;
        }
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
        // lane (l32, half): row l32, columns 32 bj + 8 g + 4 half .. + 3
#pragma unroll
        for (int bj = 0; bj < NB; ++bj)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<float4*>(&stage[l32 * kSS + 32 * bj + 8 * g + 4 * half]) =
                    make_float4(acc[bi][bj][4 * g], acc[bi][bj][4 * g + 1],
                                acc[bi][bj][4 * g + 2], acc[bi][bj][4 * g + 3]);
        __syncthreads();
        // lane l: rows l / kLPR + kRPP k of the 32, columns c .. c + 3
        float v[kPass][4];
        float mk[kPass][4];
#pragma unroll
        for (int k = 0; k < kPass; ++k) {
            const int r = lane / kLPR + kRPP * k;
            const float4 q = *reinterpret_cast<const float4*>(&stage[r * kSS + c]);
            v[k][0] = q.x, v[k][1] = q.y, v[k][2] = q.z, v[k][3] = q.w;
            if constexpr (EP == EPI_MASK && HC) {
                if (P.hmask) {
                    // only the sign is used: for the non-negative activations
                    // a mask reads, bf16(x) > 0 exactly when x > 2^-134
                    const int m = mw + 32 * bi + r;
                    const __bf16* mp = P.hmask + (int64_t)m * P.ldhmask + n;
                    if (m < P.M && whole) {
                        const bf16x4 h = *reinterpret_cast<const bf16x4*>(mp);
#pragma unroll
                        for (int t = 0; t < 4; ++t) mk[k][t] = (float)h[t];
                    } else {
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            mk[k][t] = (m < P.M && n + t < P.N) ? (float)mp[t] : 0.f;
                    }
                    continue;
                }
            }
            if constexpr (EP == EPI_MASK) {
                const int m = mw + 32 * bi + r;
                const float* mp = P.mask + (int64_t)m * P.ldmask + n;
                if (m < P.M && whole && mvec) {
                    const float4 h = ld4(mp);
                    mk[k][0] = h.x, mk[k][1] = h.y, mk[k][2] = h.z, mk[k][3] = h.w;
                } else {
#pragma unroll
                    for (int t = 0; t < 4; ++t) mk[k][t] = (m < P.M && n + t < P.N) ? mp[t] : 0.f;
                }
            }
        }
        __syncthreads();   // the stage is rewritten by the next pass
#pragma unroll
        for (int k = 0; k < kPass; ++k) {
            const int m = mw + 32 * bi + lane / kLPR + kRPP * k;
            if (m >= P.M || n >= P.N) continue;
            float* w = v[k];
            if constexpr (EP == EPI_BIAS_RELU || EP == EPI_BIAS) {
                if (P.bias) {
#pragma unroll
                    for (int t = 0; t < 4; ++t) w[t] += bv[t];
                }
                if constexpr (EP == EPI_BIAS_RELU) {
                    if (!P.no_relu) {
#pragma unroll
                        for (int t = 0; t < 4; ++t) w[t] = relu(w[t]);
                    }
                }
            } else if constexpr (EP == EPI_MASK) {
#pragma unroll
                for (int t = 0; t < 4; ++t) w[t] = mk[k][t] > 0.f ? w[t] : 0.f;
            }
            if (!HC || !P.hC || n >= P.c_from) {
                float* crow = C + (int64_t)m * P.ldc;
                if (whole && cvec) {
                    *reinterpret_cast<float4*>(crow + n) = make_float4(w[0], w[1], w[2], w[3]);
                } else {
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        if (n + t < P.N) crow[n + t] = w[t];
                }
            }
            if constexpr (HC) {
                if (P.hC) {
                    __bf16* hrow = P.hC + (int64_t)m * P.ldhc + n;
                    if (whole) {
                        *reinterpret_cast<bf16x4*>(hrow) = to_bf16(w[0], w[1], w[2], w[3]);
                    } else {
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            if (n + t < P.N) hrow[t] = (__bf16)w[t];
                    }
                }
            }
        }
    }
}

// A rows are always 16-byte aligned (checked on the host); BVEC selects
// float4 or element loads for B (the classifier weight has any width C).
// Tile shape: the four wavefronts form a WM x (4 / WM) grid and each owns
// MB x NB accumulators of 32 x 32, so the tile is (32 MB WM) x (32 NB 4/WM):
// 128 x 128 by default, 128 x 64 where the launch planner finds that it
// spreads the tiles more evenly over the CUs, 32 x 128 (one row of
// wavefronts, one accumulator each) for the weight gradients of the
// classifier (M its input width, N its class count) and of the first layer
// (M = f_in): less padding of M and fewer K slices to sum, and 64 x 128 for
// the classifier's logits (N = C): twice the row tiles of 128 x 128, so
// half the K slices (launch_gemm).
template <ALayout AL, BLayout BL, Epilogue EP, bool BVEC, GemmRole ROLE, bool HALF = false,
          int MB = 2, int NB = 2, int WM = 2>
__global__ __launch_bounds__(kThreads, 2) void gemm_kernel(GemmBatch batch) {
    static_assert(WM == 1 || WM == 2 || WM == 4, "four wavefronts per workgroup");
    constexpr int WN = 4 / WM;
    constexpr int TBM = 32 * MB * WM, TBN = 32 * NB * WN;
    static_assert(TBM <= BM && TBN <= BN, "operand buffers are sized for 128 x 128");
    static_assert(!HALF || (MB == 2 && NB == 2 && WM == 2), "half-row mode is for 128 x 128 tiles");
    // float4 quads per operand and K step, and the K-major layout of each
    // operand: quads per K row, K rows covered per quad index, LDS stride
    constexpr int kQA = BK * TBM / 4 / kThreads, kQB = BK * TBN / 4 / kThreads;
    constexpr int kQRA = TBM / 4, kQRB = TBN / 4;
    constexpr int kKStepA = kThreads / kQRA, kKStepB = kThreads / kQRB;
    constexpr int kColStrideA = TBM + 4, kColStrideB = TBN + 4;
    static_assert(kQA * kKStepA == BK && kQB * kKStepB == BK, "K-major quads cover BK rows");
    // operand buffers: [buffer][A | B]; 128-row tiles keep both at the
    // 128 x 128 size (two workgroups per CU), a 32-row tile sizes each for
    // its own operand
    constexpr int kSA = TBM == BM ? kOperandFloats
                                  : (AL == A_MK ? TBM * kRowStride : BK * kColStrideA);
    constexpr int kSB = TBM == BM ? kOperandFloats
                                  : (BL == B_NK ? TBN * kRowStride : BK * kColStrideB);
    __shared__ __attribute__((aligned(16))) float smem[2 * (kSA + kSB)];
    auto sA = [&](int buf) -> float* { return smem + buf * (kSA + kSB); };
    auto sB = [&](int buf) -> float* { return smem + buf * (kSA + kSB) + kSA; };

    const TileInfo ti = decode_tile<TBM, TBN>(batch);
    const GemmProblem& P = batch.p[ti.pi];
    const int split = ti.split, m0 = ti.m0, n0 = ti.n0;
    const int kbeg = ti.kbeg, kend = ti.kend, nk = ti.nk;

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int half = lane >> 5, l32 = lane & 31;
    // HALF (every row of the product within the tile's first 64): both
    // wavefront rows work on rows 0-63, each on two of the four K groups
    // of every step; their sums are added before the epilogue
    const int g0 = HALF ? 2 * wm : 0;   // this wavefront's first K group

    // operand descriptors, fixed for the whole K loop
    const float* const A0 = P.A0;
    const float* const B0 = P.B0;
    const int M = P.M, N = P.N;
    const int Areal = M - P.ones_row;   // rows of A backed by memory
    const bool ones = P.ones_row != 0;
    const int ksplitA = P.ksplitA, ksplitB = P.ksplitB;
    const int64_t lda0 = P.lda0, ldb0 = P.ldb0;

    // Thread t moves kQA / kQB float4 of A / B per K step:
    //   row-contiguous: row t / (BK/4) + q * (256 / (BK/4)), k = 4 (t % (BK/4))
    //   K-major:        k row t / kQR + kKStep q, column 4 (t % kQR)
    constexpr int kPerRow = BK / 4, kRowStep = kThreads / kPerRow;
    const int rk = 4 * (t % kPerRow);   // K offset of a row-contiguous quad
    const int krA = t / kQRA;           // K row of a K-major A quad (+ kKStepA q)
    const int krB = t / kQRB;           // K row of a K-major B quad (+ kKStepB q)
    RowQuad arow[kQA], brow[kQB];
    ColQuad acol, bcol;
    acol.c = m0 + 4 * (t % kQRA);
    bcol.c = n0 + 4 * (t % kQRB);
#pragma unroll
    for (int q = 0; q < kQA; ++q) {
        if constexpr (AL == A_MK) {
            const int r = m0 + t / kPerRow + kRowStep * q;
            arow[q].live = r < M;
            const int rr = arow[q].live ? r : 0;
            arow[q].p0 = A0 + (int64_t)rr * lda0;
            arow[q].p1 = P.A1 + (int64_t)rr * P.lda1;
        }
    }
#pragma unroll
    for (int q = 0; q < kQB; ++q) {
        if constexpr (BL == B_NK) {
            const int r = n0 + t / kPerRow + kRowStep * q;
            brow[q].live = r < N;
            const int rr = brow[q].live ? r : 0;
            brow[q].p0 = B0 + (int64_t)rr * ldb0;
            brow[q].p1 = P.B1 + (int64_t)rr * P.ldb1;
        }
    }

    // two register sets: set s holds the K steps kt with kt % 2 == s
    Quad ra[2][kQA], rb[2][kQB];
    auto gload_a = [&](int set, int k0, int q) {
        Quad& r = ra[set][q];
        if constexpr (AL == A_MK) {
            const int k = k0 + rk;
            const float* p = k < ksplitA ? arow[q].p0 + k : arow[q].p1 + (k - ksplitA);
            r.one = -1;
            issue<true>(r, p, A0, (arow[q].live && k < kend) ? kend - k : 0);
        } else {
            const int k = k0 + krA + kKStepA * q;
            const int c = acol.c;
            const bool krow = k < kend;
            r.one = (ones && krow && Areal - c >= 0 && Areal - c < 4) ? Areal - c : -1;
            issue<true>(r, A0 + (int64_t)k * lda0 + c, A0, (krow && c < Areal) ? Areal - c : 0);
        }
    };
    auto gload_b = [&](int set, int k0, int q) {
        Quad& r = rb[set][q];
        if constexpr (BL == B_NK) {
            const int k = k0 + rk;
            const float* p = k < ksplitB ? brow[q].p0 + k : brow[q].p1 + (k - ksplitB);
            r.one = -1;
            issue<BVEC>(r, p, B0, (brow[q].live && k < kend) ? kend - k : 0);
        } else {
            const int k = k0 + krB + kKStepB * q;
            const int c = bcol.c;
            const bool krow = k < kend;
            r.one = -1;
            issue<BVEC>(r, B0 + (int64_t)k * ldb0 + c, B0, (krow && c < N) ? N - c : 0);
        }
    };
    // LDS placement of quad q (row-contiguous: [row][k]; K-major: [k][col])
    auto a_slot = [&](int q) {
        return AL == A_MK ? (t / kPerRow + kRowStep * q) * kRowStride + rk
                          : (krA + kKStepA * q) * kColStrideA + 4 * (t % kQRA);
    };
    auto b_slot = [&](int q) {
        return BL == B_NK ? (t / kPerRow + kRowStep * q) * kRowStride + rk
                          : (krB + kKStepB * q) * kColStrideB + 4 * (t % kQRB);
    };
    auto sstore = [&](int buf, int set) {
        constexpr int kQM = kQA > kQB ? kQA : kQB;
#pragma unroll
        for (int q = 0; q < kQM; ++q) {
            if (q < kQA) *reinterpret_cast<float4*>(&sA(buf)[a_slot(q)]) = finish(ra[set][q]);
            if (q < kQB) *reinterpret_cast<float4*>(&sB(buf)[b_slot(q)]) = finish(rb[set][q]);
        }
    };

    floatx16 acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragments of one group of 8 K values: element j feeds MFMA step j
    float4 fa[2][MB], fb[2][NB];
    auto frag = [&](const float* As, const float* Bs, int sg, int fslot) {
        const int kb = 8 * sg + 4 * half;
        constexpr int kFM = MB > NB ? MB : NB;
#pragma unroll
        for (int i = 0; i < kFM; ++i) {
            if (i < MB) {
                const int m = (HALF ? 0 : wm * 32 * MB) + i * 32 + l32;
                if constexpr (AL == A_MK) {
                    fa[fslot][i] = *reinterpret_cast<const float4*>(&As[m * kRowStride + kb]);
                } else {
                    fa[fslot][i] = make_float4(As[(kb + 0) * kColStrideA + m], As[(kb + 1) * kColStrideA + m],
                                               As[(kb + 2) * kColStrideA + m], As[(kb + 3) * kColStrideA + m]);
                }
            }
            if (i < NB) {
                const int nn = wn * 32 * NB + i * 32 + l32;
                if constexpr (BL == B_NK) {
                    fb[fslot][i] = *reinterpret_cast<const float4*>(&Bs[nn * kRowStride + kb]);
                } else {
                    fb[fslot][i] = make_float4(Bs[(kb + 0) * kColStrideB + nn], Bs[(kb + 1) * kColStrideB + nn],
                                               Bs[(kb + 2) * kColStrideB + nn], Bs[(kb + 3) * kColStrideB + nn]);
                }
            }
        }
    };
    auto elem = [](const float4& v, int j) {
        return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
    };
    auto mfma_group = [&](int fslot) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                const float a = elem(fa[fslot][i], j);
#pragma unroll
                for (int jj = 0; jj < NB; ++jj) {
                    // B first: the accumulators hold the transposed blocks (store_tile)
                    acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(elem(fb[fslot][jj], j), a,
                                                                      acc[i][jj], 0, 0, 0);
                }
            }
        }
    };
    // interleave of global loads (or LDS stores) with the MFMAs of a group:
    // kLoads of them per K step, kPer MFMAs after each, kRest at the end
    constexpr int kMfmas = 4 * MB * NB, kLoads = kQA + kQB;
    constexpr int kPer = kMfmas / kLoads > 0 ? kMfmas / kLoads : 1;
    constexpr int kRest = kMfmas > kPer * kLoads ? kMfmas - kPer * kLoads : 0;
    constexpr int kDsFirst = (MB == 2 && NB == 2) ? 8 : 2 * (MB + NB);

    // Fast steps (as in the bf16 kernel below): operand rows / K-major
    // column quads outside the operand are clamped into it, since they only
    // feed outputs the epilogue drops; in a tile with vector loads, no
    // appended row of ones and the K concatenation point on a K-step
    // boundary between parts of equal leading dimension, a whole K step
    // loads from a uniform per-step base plus fixed per-thread offsets and
    // stores without masking.
    const int nfull = (kend - kbeg) / BK;
    const bool fast_tile = BVEC && !(ones && Areal >= m0 && Areal < m0 + TBM) &&
                           (AL == A_KM || concat_fast(ksplitA, kbeg, nfull, P.lda1, lda0)) &&
                           (BL == B_KN || concat_fast(ksplitB, kbeg, nfull, P.ldb1, ldb0));
    int64_t oa[kQA], ob[kQB];
#pragma unroll
    for (int q = 0; q < kQA; ++q) {
        if constexpr (AL == A_MK) {
            const int r = m0 + t / kPerRow + kRowStep * q;
            oa[q] = (int64_t)(r < M ? r : 0) * lda0 + rk;
        } else {
            oa[q] = (int64_t)(krA + kKStepA * q) * lda0 + (acol.c < Areal ? acol.c : 0);
        }
    }
#pragma unroll
    for (int q = 0; q < kQB; ++q) {
        if constexpr (BL == B_NK) {
            const int r = n0 + t / kPerRow + kRowStep * q;
            ob[q] = (int64_t)(r < N ? r : 0) * ldb0 + rk;
        } else {
            ob[q] = (int64_t)(krB + kKStepB * q) * ldb0 + (bcol.c < N ? bcol.c : 0);
        }
    }
    // per-step operand bases, uniform across the workgroup (computed once
    // per K step, outside the per-quad loads)
    const float* const A1 = P.A1;
    const float* const B1 = P.B1;
    auto step_base_a = [&](int k0) -> const float* {
        if constexpr (AL == A_MK)
            return k0 >= ksplitA ? A1 + (k0 - ksplitA) : A0 + k0;
        else
            return A0 + (int64_t)k0 * lda0;
    };
    auto step_base_b = [&](int k0) -> const float* {
        if constexpr (BL == B_NK)
            return k0 >= ksplitB ? B1 + (k0 - ksplitB) : B0 + k0;
        else
            return B0 + (int64_t)k0 * ldb0;
    };
    // the whole step's loads and stores of both operands, quad q of A then
    // quad q of B
    constexpr int kQMax = kQA > kQB ? kQA : kQB;
    auto gload_full = [&](int set, const float* sa, const float* sb) {
#pragma unroll
        for (int q = 0; q < kQMax; ++q) {
            if (q < kQA) ra[set][q].v = ld4(sa + oa[q]);
            if (q < kQB) rb[set][q].v = ld4(sb + ob[q]);
        }
    };
    auto gload = [&](int set, int k0) {
#pragma unroll
        for (int q = 0; q < kQMax; ++q) {
            if (q < kQA) gload_a(set, k0, q);
            if (q < kQB) gload_b(set, k0, q);
        }
    };
    auto sstore_full = [&](int buf, int set) {
#pragma unroll
        for (int q = 0; q < kQMax; ++q) {
            if (q < kQA) *reinterpret_cast<float4*>(&sA(buf)[a_slot(q)]) = ra[set][q].v;
            if (q < kQB) *reinterpret_cast<float4*>(&sB(buf)[b_slot(q)]) = rb[set][q].v;
        }
    };
    // quads of a set filled by whole-step loads, for a masked store
    auto mark_full = [&](int set) {
#pragma unroll
        for (int q = 0; q < kQA; ++q) {
            ra[set][q].valid = 4;
            ra[set][q].one = -1;
        }
#pragma unroll
        for (int q = 0; q < kQB; ++q) {
            rb[set][q].valid = 4;
            rb[set][q].one = -1;
        }
    };

    static_assert(BK / 8 == 4, "the K step is laid out as four groups of 8");
    // One K step. LDS buffer kt % 2 holds step kt; register set (kt + 1) % 2
    // holds step kt + 1 and step kt + 2 is loaded into set kt % 2 meanwhile,
    // so every global load has two K steps of MFMA work to arrive. FULL:
    // steps kt + 1 and kt + 2 are whole steps of a fast tile.
    auto kstep = [&](int kt, int set, auto FULL) {
        const int buf = kt & 1;
        const float* As = sA(buf);
        const float* Bs = sB(buf);
        const int kload = kbeg + (kt + 2) * BK;   // past kend near the end: empty quads
        // group 0: next group's fragments, the global loads of step kt + 2
        frag(As, Bs, 1, 1);
        const float* const sa = step_base_a(kload);
        const float* const sb = step_base_b(kload);
        if constexpr (FULL)
            gload_full(set, sa, sb);
        else
            gload(set, kload);
        mfma_group(0);
        __builtin_amdgcn_sched_group_barrier(0x100, kDsFirst, 0);      // DS reads first
#pragma unroll
        for (int q = 0; q < kLoads; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);     // one global load
            __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);  // kPer MFMAs
        }
        if constexpr (kRest > 0) __builtin_amdgcn_sched_group_barrier(0x008, kRest, 0);
        __builtin_amdgcn_sched_barrier(0);
        // group 1
        frag(As, Bs, 2, 0);
        mfma_group(1);
        __builtin_amdgcn_sched_barrier(0);
        // group 2: step kt + 1 goes from its register set into the other
        // buffer, whose last reader (step kt - 1) finished before the
        // previous barrier
        frag(As, Bs, 3, 1);
        const bool more = FULL || kt + 1 < nk;
        if (more) {
            if constexpr (FULL)
                sstore_full(buf ^ 1, set ^ 1);
            else
                sstore(buf ^ 1, set ^ 1);
        }
        mfma_group(0);
        __builtin_amdgcn_sched_group_barrier(0x100, kDsFirst, 0);      // DS reads first
#pragma unroll
        for (int q = 0; q < kLoads; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);     // one LDS store
            __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);  // kPer MFMAs
        }
        if constexpr (kRest > 0) __builtin_amdgcn_sched_group_barrier(0x008, kRest, 0);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        // group 3: its fragments are already in registers, so the next
        // step's first LDS reads are hidden behind these MFMAs
        if (more) frag(sA(buf ^ 1), sB(buf ^ 1), 0, 0);
        mfma_group(1);
        __builtin_amdgcn_sched_barrier(0);
    };
    // HALF: the wavefront's two groups of the step; loads and stores are
    // interleaved with them as above
    auto kstep_half = [&](int kt, int set, auto FULL) __attribute__((always_inline)) {
        const int buf = kt & 1;
        const float* As = sA(buf);
        const float* Bs = sB(buf);
        const int kload = kbeg + (kt + 2) * BK;
        frag(As, Bs, g0 + 1, 1);
        const float* const sa = step_base_a(kload);
        const float* const sb = step_base_b(kload);
        if constexpr (FULL)
            gload_full(set, sa, sb);
        else
            gload(set, kload);
        mfma_group(0);
        __builtin_amdgcn_sched_group_barrier(0x100, kDsFirst, 0);
#pragma unroll
        for (int q = 0; q < kLoads; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        const bool more = FULL || kt + 1 < nk;
        if (more) {
            if constexpr (FULL)
                sstore_full(buf ^ 1, set ^ 1);
            else
                sstore(buf ^ 1, set ^ 1);
        }
        mfma_group(1);
#pragma unroll
        for (int q = 0; q < kLoads; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, kPer, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        if (more) frag(sA(buf ^ 1), sB(buf ^ 1), g0, 0);
    };
    auto step = [&](int kt, int set, auto FULL) __attribute__((always_inline)) {
        if constexpr (HALF)
            kstep_half(kt, set, FULL);
        else
            kstep(kt, set, FULL);
    };
    using Full = std::true_type;
    using Masked = std::false_type;
    const bool fast_start = fast_tile && nfull >= 2;
    if (fast_start) {
        gload_full(0, step_base_a(kbeg), step_base_b(kbeg));
        gload_full(1, step_base_a(kbeg + BK), step_base_b(kbeg + BK));
        sstore_full(0, 0);
    } else if (nk > 0) {
        gload(0, kbeg);
        gload(1, kbeg + BK);
        sstore(0, 0);
    }
    if (nk > 0) {
        __syncthreads();
        frag(sA(0), sB(0), g0, 0);
    }
    int kt = 0;
    if (fast_start) {
        for (; kt + 3 < nfull; kt += 2) {
            step(kt, 0, Full{});
            step(kt + 1, 1, Full{});
        }
        mark_full(0);
        mark_full(1);
    }
    for (; kt + 1 < nk; kt += 2) {
        step(kt, 0, Masked{});
        step(kt + 1, 1, Masked{});
    }
    if (kt < nk) step(kt, 0, Masked{});

    if constexpr (HALF) {
        // the second wavefront row's sums join the first's (fixed order);
        // its own rows (64-127) lie outside the product and store nothing
        __syncthreads();
        float* red = smem;
        auto at = [&](int i, int j, int r) { return ((wn * 4 + i * 2 + j) * 16 + r) * 64 + lane; };
        static_assert(!HALF || MB * NB == 4, "half-row reduction layout");
        if (wm == 1) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) red[at(i, j, r)] = acc[i][j][r];
        }
        __syncthreads();
        if (wm == 0) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[i][j][r] += red[at(i, j, r)];
        }
    }
    store_tile<EP, MB, NB>(P, split, m0 + wm * 32 * MB, n0 + wn * 32 * NB, half, l32, acc);
}

// ------------------------------------------------------------ bf16 variant
// The same products with bf16 operands and fp32 accumulation
// (v_mfma_f32_32x32x16_bf16). Operands stay fp32 in HBM; they are rounded
// to bf16 (round to nearest even, v_cvt_pk_bf16_f32) when written to LDS,
// which then always holds [row][k] with K contiguous, so every fragment is
// one 128-bit LDS read of 8 consecutive K values for one row. A K-major
// operand is transposed on the way: a thread loads four consecutive K rows
// of the same four columns and writes four 4-element K runs. Tiling and
// epilogues are those of the fp32 kernel; an MFMA step covers 16 K values,
// so a K step of 32 is two MFMA steps. Global loads run two K steps ahead
// (two register sets) to cover memory latency behind the shorter MFMA work.
constexpr int kHStride = BK + 8;   // bf16 per LDS row: 80 bytes, conflict-free 128-bit reads

template <ALayout AL, BLayout BL, Epilogue EP, bool BVEC, GemmRole ROLE>
__global__ __launch_bounds__(kThreads, 2) void gemm_bf16_kernel(GemmBatch batch) {
    // [buffer][A | B] operand tiles, [row][k]
    __shared__ __attribute__((aligned(16))) __bf16 hs[2][2][BM * kHStride];

    const TileInfo ti = decode_tile(batch);
    const GemmProblem& P = batch.p[ti.pi];
    const int split = ti.split, m0 = ti.m0, n0 = ti.n0;
    const int kbeg = ti.kbeg, kend = ti.kend, nk = ti.nk;

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int half = lane >> 5, l32 = lane & 31;

    const float* const A0 = P.A0;
    const float* const B0 = P.B0;
    const int M = P.M, N = P.N;
    const int Areal = M - P.ones_row;
    const bool ones = P.ones_row != 0;
    const int ksplitA = P.ksplitA, ksplitB = P.ksplitB;
    const int64_t lda0 = P.lda0, ldb0 = P.ldb0;

    // Thread t moves kQuads float4 per operand and K step:
    //   row-contiguous: row t / 8 + 32 q, K offset 4 (t % 8)
    //   K-major:        K row 4 (t / 32) + q, columns 4 (t % 32) .. + 3
    constexpr int kPerRow = BK / 4, kRowStep = kThreads / kPerRow;
    static_assert(kQuads == 4 && kThreads / 32 * 4 == BK, "K-major quads cover 4 K rows");
    const int rk = 4 * (t % kPerRow);
    const int kq = 4 * (t >> 5);
    const int ac = m0 + 4 * (t & 31), bc = n0 + 4 * (t & 31);
    RowQuad arow[kQuads], brow[kQuads];
#pragma unroll
    for (int q = 0; q < kQuads; ++q) {
        if constexpr (AL == A_MK) {
            const int r = m0 + t / kPerRow + kRowStep * q;
            arow[q].live = r < M;
            const int rr = arow[q].live ? r : 0;
            arow[q].p0 = A0 + (int64_t)rr * lda0;
            arow[q].p1 = P.A1 + (int64_t)rr * P.lda1;
        }
        if constexpr (BL == B_NK) {
            const int r = n0 + t / kPerRow + kRowStep * q;
            brow[q].live = r < N;
            const int rr = brow[q].live ? r : 0;
            brow[q].p0 = B0 + (int64_t)rr * ldb0;
            brow[q].p1 = P.B1 + (int64_t)rr * P.ldb1;
        }
    }

    // Fast steps. Outside the operand, a row (or a K-major column quad)
    // only feeds outputs that the epilogue drops, so its loads are clamped
    // to row 0 (column 0) instead of masked. In a tile with vector loads, no
    // appended row of ones, and the K concatenation point on a K-step
    // boundary between parts of equal leading dimension, every whole K step
    // then needs no per-element work besides the bf16 conversion; the last
    // (partial) steps and every other tile take the masked path.
    const int nfull = (kend - kbeg) / BK;   // whole K steps of this split
    const bool fast_tile = BVEC && !(ones && Areal >= m0 && Areal < m0 + BM) &&
                           (AL == A_KM || concat_fast(ksplitA, kbeg, nfull, P.lda1, lda0)) &&
                           (BL == B_KN || concat_fast(ksplitB, kbeg, nfull, P.ldb1, ldb0));
    // Fast loads address element (row, k) of an operand as a base pointer
    // that depends only on the K step (uniform: scalar registers) plus a
    // per-thread offset fixed for the whole loop. Both parts of a
    // K-concatenated operand then share the offsets, which needs equal
    // leading dimensions (part of the fast-tile condition).
    int64_t oa[kQuads], ob[kQuads];
#pragma unroll
    for (int q = 0; q < kQuads; ++q) {
        if constexpr (AL == A_MK) {
            const int r = m0 + t / kPerRow + kRowStep * q;
            oa[q] = (int64_t)(r < M ? r : 0) * lda0 + rk;
        } else {
            oa[q] = (int64_t)(kq + q) * lda0 + (ac < Areal ? ac : 0);
        }
        if constexpr (BL == B_NK) {
            const int r = n0 + t / kPerRow + kRowStep * q;
            ob[q] = (int64_t)(r < N ? r : 0) * ldb0 + rk;
        } else {
            ob[q] = (int64_t)(kq + q) * ldb0 + (bc < N ? bc : 0);
        }
    }

    Quad ra[2][kQuads], rb[2][kQuads];
    auto gload_full = [&](int set, int k0) {
        const float* sa;
        const float* sb;
        if constexpr (AL == A_MK)
            sa = k0 >= ksplitA ? P.A1 + (k0 - ksplitA) : A0 + k0;
        else
            sa = A0 + (int64_t)k0 * lda0;
        if constexpr (BL == B_NK)
            sb = k0 >= ksplitB ? P.B1 + (k0 - ksplitB) : B0 + k0;
        else
            sb = B0 + (int64_t)k0 * ldb0;
#pragma unroll
        for (int q = 0; q < kQuads; ++q) {
            ra[set][q].v = ld4(sa + oa[q]);
            rb[set][q].v = ld4(sb + ob[q]);
        }
    };
    // quads loaded whole, to be stored by the masked path
    auto mark_full = [&](int set) {
#pragma unroll
        for (int q = 0; q < kQuads; ++q) {
            ra[set][q].valid = rb[set][q].valid = 4;
            ra[set][q].one = rb[set][q].one = -1;
        }
    };
    auto gload_masked = [&](int set, int k0) {
#pragma unroll
        for (int q = 0; q < kQuads; ++q) {
            Quad& a = ra[set][q];
            if constexpr (AL == A_MK) {
                const int k = k0 + rk;
                const float* p = k < ksplitA ? arow[q].p0 + k : arow[q].p1 + (k - ksplitA);
                a.one = -1;
                issue<true>(a, p, A0, (arow[q].live && k < kend) ? kend - k : 0);
            } else {
                const int k = k0 + kq + q;
                const bool krow = k < kend;
                a.one = (ones && krow && Areal - ac >= 0 && Areal - ac < 4) ? Areal - ac : -1;
                issue<true>(a, A0 + (int64_t)k * lda0 + ac, A0, (krow && ac < Areal) ? Areal - ac : 0);
            }
            Quad& b = rb[set][q];
            if constexpr (BL == B_NK) {
                const int k = k0 + rk;
                const float* p = k < ksplitB ? brow[q].p0 + k : brow[q].p1 + (k - ksplitB);
                b.one = -1;
                issue<BVEC>(b, p, B0, (brow[q].live && k < kend) ? kend - k : 0);
            } else {
                const int k = k0 + kq + q;
                b.one = -1;
                issue<BVEC>(b, B0 + (int64_t)k * ldb0 + bc, B0, (k < kend && bc < N) ? N - bc : 0);
            }
        }
    };
    // one operand's quads into LDS tile S ([row][k]); `full`: no masking
    auto sstore_op = [&](__bf16* S, const Quad (&r)[kQuads], bool kmajor, bool full) {
        float4 v[kQuads];
#pragma unroll
        for (int q = 0; q < kQuads; ++q) v[q] = full ? r[q].v : finish(r[q]);
        if (!kmajor) {
#pragma unroll
            for (int q = 0; q < kQuads; ++q)
                *reinterpret_cast<bf16x4*>(&S[(t / kPerRow + kRowStep * q) * kHStride + rk]) =
                    to_bf16(v[q].x, v[q].y, v[q].z, v[q].w);
        } else {
            const int c = 4 * (t & 31);
            *reinterpret_cast<bf16x4*>(&S[(c + 0) * kHStride + kq]) = to_bf16(v[0].x, v[1].x, v[2].x, v[3].x);
            *reinterpret_cast<bf16x4*>(&S[(c + 1) * kHStride + kq]) = to_bf16(v[0].y, v[1].y, v[2].y, v[3].y);
            *reinterpret_cast<bf16x4*>(&S[(c + 2) * kHStride + kq]) = to_bf16(v[0].z, v[1].z, v[2].z, v[3].z);
            *reinterpret_cast<bf16x4*>(&S[(c + 3) * kHStride + kq]) = to_bf16(v[0].w, v[1].w, v[2].w, v[3].w);
        }
    };
    auto sstore = [&](int buf, int set, bool full) {
        sstore_op(hs[buf][0], ra[set], AL == A_KM, full);
        sstore_op(hs[buf][1], rb[set], BL == B_KN, full);
    };

    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragments of MFMA step ks (K values 16 ks .. 16 ks + 15 of the K step):
    // lane half g holds K values 8 g .. 8 g + 7 of its row
    bf16x8 fa[2][2], fb[2][2];
    auto frag = [&](int buf, int ks, int fslot) {
        const __bf16* As = hs[buf][0];
        const __bf16* Bs = hs[buf][1];
        const int kb = 16 * ks + 8 * half;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            fa[fslot][i] = *reinterpret_cast<const bf16x8*>(&As[(wm * 64 + i * 32 + l32) * kHStride + kb]);
            fb[fslot][i] = *reinterpret_cast<const bf16x8*>(&Bs[(wn * 64 + i * 32 + l32) * kHStride + kb]);
        }
    };
    auto mfma = [&](int fslot) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[fslot][j], fa[fslot][i],
                                                                    acc[i][j], 0, 0, 0);
    };

    // LDS buffer kt % 2 holds K step kt; register set (kt + 1) % 2 holds
    // step kt + 1, and step kt + 2 is loaded into set kt % 2 meanwhile.
    // FULL: steps kt + 1 and kt + 2 are whole steps of a fast tile.
    auto kstep = [&](int kt, int set, auto FULL) {
        const int buf = kt & 1;
        if constexpr (FULL)
            gload_full(set, kbeg + (kt + 2) * BK);
        else
            gload_masked(set, kbeg + (kt + 2) * BK);   // past kend: empty quads
        frag(buf, 1, 1);
        mfma(0);
        mfma(1);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (FULL) {
            sstore(buf ^ 1, set ^ 1, true);
            __syncthreads();
            frag(buf ^ 1, 0, 0);
        } else {
            if (kt + 1 < nk) sstore(buf ^ 1, set ^ 1, false);
            __syncthreads();
            if (kt + 1 < nk) frag(buf ^ 1, 0, 0);
        }
    };
    using Full = std::true_type;
    using Masked = std::false_type;
    const bool fast_start = fast_tile && nfull >= 2;
    if (fast_start) {
        gload_full(0, kbeg);
        gload_full(1, kbeg + BK);
        sstore(0, 0, true);
    } else if (nk > 0) {
        gload_masked(0, kbeg);
        gload_masked(1, kbeg + BK);
        sstore(0, 0, false);
    }
    if (nk > 0) {
        __syncthreads();
        frag(0, 0, 0);
    }
    int kt = 0;
    if (fast_start) {
        for (; kt + 3 < nfull; kt += 2) {
            kstep(kt, 0, Full{});
            kstep(kt + 1, 1, Full{});
        }
        mark_full(0);
        mark_full(1);
    }
    for (; kt + 1 < nk; kt += 2) {
        kstep(kt, 0, Masked{});
        kstep(kt + 1, 1, Masked{});
    }
    if (kt < nk) kstep(kt, 0, Masked{});

    store_tile<EP>(P, split, m0 + wm * 64, n0 + wn * 64, half, l32, acc);
}

// ------------------------------------------------------------ bf16 copies
// The bf16 products when every operand already has a bf16 copy in HBM
// (written by the kernel that produced it): half the operand bytes of the
// kernel above and no per-element work between the loads and LDS. LDS keeps
// each operand in its HBM orientation. K-contiguous operands are [row][k]
// (stride 40 bf16, 80 bytes), a fragment being one 128-bit read. K-major
// operands are [k][col] (stride 144 bf16, 288 bytes) and their fragments
// come from two transposing reads (ds_read_b64_tr_b16): each group of 16
// lanes names a 4 x 16 block (lane j: k row j / 4, columns 4 (j % 4) ..
// + 3) and lane i receives column i of it, four consecutive K values. Tile,
// K step, tile order, split-K and epilogues are those of the kernels above,
// and the MFMAs take the same K values in the same order, so every product
// equals that of the fp32-operand bf16 kernel bit for bit.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

constexpr int kRS16 = BK + 8;    // [row][k] stride, bf16
constexpr int kKS16 = BM + 16;   // [k][col] stride, bf16
constexpr int kOp16 = (BM * kRS16 > BK * kKS16) ? BM * kRS16 : BK * kKS16;
constexpr int kQ16 = BK * BM / 8 / kThreads;   // 16-byte chunks per operand per thread

// Eight bf16 of one operand row (or K-major row) and how many are real.
struct HChunk {
    u32x4 v;
    int valid;   // elements [0, valid) are real; the rest become 0
    int one;     // element that is an implicit 1.0, or -1
};

__device__ __forceinline__ u32x4 finish16(const HChunk& q) {
    u32x4 v = q.v;
    // word w holds elements 2w (low half) and 2w + 1 (high half)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const unsigned keep = q.valid >= 2 * w + 2 ? 0xffffffffu
                              : q.valid == 2 * w + 1 ? 0x0000ffffu : 0u;
        v[w] &= keep;
        if (q.one >= 0 && (q.one >> 1) == w)
            v[w] |= (q.one & 1) ? 0x3f800000u : 0x00003f80u;   // bf16 1.0
    }
    return v;
}

__device__ __forceinline__ u32x4 ld16(const __bf16* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

template <ALayout AL, BLayout BL, Epilogue EP, GemmRole ROLE, int NB = 2>
__global__ __launch_bounds__(kThreads, 2) void gemm_h16_kernel(GemmBatch batch) {
    // tile 128 x (64 NB): each wavefront of the 2 x 2 grid owns 2 x NB
    // accumulators of 32 x 32
    constexpr int TBN = 64 * NB;
    // [buffer][A | B] operand tiles
    __shared__ __attribute__((aligned(16))) __bf16 hs[2][2][kOp16];

    const TileInfo ti = decode_tile<BM, TBN>(batch);
    const GemmProblem& P = batch.p[ti.pi];
    const int split = ti.split, m0 = ti.m0, n0 = ti.n0;
    const int kbeg = ti.kbeg, kend = ti.kend, nk = ti.nk;

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int half = lane >> 5, l32 = lane & 31;
    const int i16 = lane & 15, sub = (lane >> 4) & 1;

    const __bf16* const A0 = P.hA0;
    const __bf16* const B0 = P.hB0;
    const int M = P.M, N = P.N;
    const int Areal = M - P.ones_row;
    const bool ones = P.ones_row != 0;
    const int ksplitA = P.ksplitA, ksplitB = P.ksplitB;
    const int64_t lda0 = P.hlda0, ldb0 = P.hldb0;

    // Thread t moves kQ16 (A) / kQB chunks (B) of 8 bf16 per K step:
    //   K-contiguous: row t / 4 + 64 q, K offset 8 (t % 4)
    //   K-major:      K row t / kCPK + kKStep q, columns 8 (t % kCPK) .. + 7
    //                 (kCPK = 16 chunks per 128 columns, 8 per 64 for B)
    constexpr int kCPR = BK / 8, kRowStep = kThreads / kCPR;
    constexpr int kCPK = BM / 8, kKStep = kThreads / kCPK;
    constexpr int kQB = BK * TBN / 8 / kThreads;
    constexpr int kCPKB = TBN / 8, kKStepB = kThreads / kCPKB;
    static_assert(kQ16 * kRowStep == BM && kQ16 * kKStep == BK, "chunks cover the tile");
    static_assert(kQB * kRowStep == TBN && kQB * kKStepB == BK, "chunks cover the B tile");
    const int rk = 8 * (t % kCPR);
    const int kq = t / kCPK, kqB = t / kCPKB;
    const int ac = m0 + 8 * (t % kCPK), bc = n0 + 8 * (t % kCPKB);
    int sofs_a[kQ16], sofs_b[kQB];   // LDS element offsets of the chunks
#pragma unroll
    for (int q = 0; q < kQ16; ++q)
        sofs_a[q] = AL == A_MK ? (t / kCPR + kRowStep * q) * kRS16 + rk
                               : (kq + kKStep * q) * kKS16 + 8 * (t % kCPK);
#pragma unroll
    for (int q = 0; q < kQB; ++q)
        sofs_b[q] = BL == B_NK ? (t / kCPR + kRowStep * q) * kRS16 + rk
                               : (kqB + kKStepB * q) * kKS16 + 8 * (t % kCPKB);

    // Fast tiles: no appended row of ones here and the K concatenation
    // point on a K-step boundary between parts of equal leading dimension;
    // whole K steps then load from a per-step base plus fixed per-thread
    // offsets (rows / columns outside the operand clamped into it: they
    // only feed outputs the epilogue drops).
    const int nfull = (kend - kbeg) / BK;
    const bool fast_tile = !(ones && Areal >= m0 && Areal < m0 + BM) &&
                           (AL == A_KM || concat_fast(ksplitA, kbeg, nfull, P.hlda1, lda0)) &&
                           (BL == B_KN || concat_fast(ksplitB, kbeg, nfull, P.hldb1, ldb0));
    int64_t oa[kQ16], ob[kQB];
#pragma unroll
    for (int q = 0; q < kQ16; ++q) {
        if constexpr (AL == A_MK) {
            const int r = m0 + t / kCPR + kRowStep * q;
            oa[q] = (int64_t)(r < M ? r : 0) * lda0 + rk;
        } else {
            oa[q] = (int64_t)(kq + kKStep * q) * lda0 + (ac < Areal ? ac : 0);
        }
    }
#pragma unroll
    for (int q = 0; q < kQB; ++q) {
        if constexpr (BL == B_NK) {
            const int r = n0 + t / kCPR + kRowStep * q;
            ob[q] = (int64_t)(r < N ? r : 0) * ldb0 + rk;
        } else {
            ob[q] = (int64_t)(kqB + kKStepB * q) * ldb0 + (bc < N ? bc : 0);
        }
    }

    HChunk ra[2][kQ16], rb[2][kQB];
    auto gload_full = [&](int set, int k0) {
        const __bf16* sa;
        const __bf16* sb;
        if constexpr (AL == A_MK)
            sa = k0 >= ksplitA ? P.hA1 + (k0 - ksplitA) : A0 + k0;
        else
            sa = A0 + (int64_t)k0 * lda0;
        if constexpr (BL == B_NK)
            sb = k0 >= ksplitB ? P.hB1 + (k0 - ksplitB) : B0 + k0;
        else
            sb = B0 + (int64_t)k0 * ldb0;
#pragma unroll
        for (int q = 0; q < kQ16; ++q) {
            ra[set][q].v = ld16(sa + oa[q]);
            if (q < kQB) rb[set][q].v = ld16(sb + ob[q]);
        }
    };
    auto mark_full = [&](int set) {
#pragma unroll
        for (int q = 0; q < kQ16; ++q) {
            ra[set][q].valid = 8;
            ra[set][q].one = -1;
        }
#pragma unroll
        for (int q = 0; q < kQB; ++q) {
            rb[set][q].valid = 8;
            rb[set][q].one = -1;
        }
    };
    // a K-contiguous chunk (row r, K offset k) of a possibly concatenated operand
    auto row_chunk = [&](HChunk& c, const __bf16* p0, const __bf16* p1, int64_t ld0, int64_t ld1,
                         int ksplit, int r, int rows, int k) {
        const bool live = r < rows && k < kend;
        c.valid = live ? min(8, kend - k) : 0;
        c.one = -1;
        const __bf16* p = k < ksplit ? p0 + (int64_t)r * ld0 + k
                                     : p1 + (int64_t)r * ld1 + (k - ksplit);
        c.v = ld16(live ? p : p0);
    };
    auto gload_masked = [&](int set, int k0) {
#pragma unroll
        for (int q = 0; q < kQ16; ++q) {
            HChunk& a = ra[set][q];
            if constexpr (AL == A_MK) {
                row_chunk(a, A0, P.hA1, lda0, P.hlda1, ksplitA, m0 + t / kCPR + kRowStep * q, M,
                          k0 + rk);
            } else {
                const int k = k0 + kq + kKStep * q;
                const bool krow = k < kend;
                a.valid = (krow && ac < Areal) ? min(8, Areal - ac) : 0;
                a.one = (ones && krow && Areal - ac >= 0 && Areal - ac < 8) ? Areal - ac : -1;
                a.v = ld16(a.valid > 0 ? A0 + (int64_t)k * lda0 + ac : A0);
            }
            if (q >= kQB) continue;
            HChunk& b = rb[set][q];
            if constexpr (BL == B_NK) {
                row_chunk(b, B0, P.hB1, ldb0, P.hldb1, ksplitB, n0 + t / kCPR + kRowStep * q, N,
                          k0 + rk);
            } else {
                const int k = k0 + kqB + kKStepB * q;
                b.valid = (k < kend && bc < N) ? min(8, N - bc) : 0;
                b.one = -1;
                b.v = ld16(b.valid > 0 ? B0 + (int64_t)k * ldb0 + bc : B0);
            }
        }
    };
    auto sstore = [&](int buf, int set, bool full) {
        __bf16* As = hs[buf][0];
        __bf16* Bs = hs[buf][1];
#pragma unroll
        for (int q = 0; q < kQ16; ++q) {
            *reinterpret_cast<u32x4*>(&As[sofs_a[q]]) = full ? ra[set][q].v : finish16(ra[set][q]);
            if (q < kQB)
                *reinterpret_cast<u32x4*>(&Bs[sofs_b[q]]) =
                    full ? rb[set][q].v : finish16(rb[set][q]);
        }
    };

    floatx16 acc[2][NB];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragment of MFMA step ks for the 32 rows (columns) from `base`: lane
    // half g holds K values 16 ks + 8 g .. + 7 of row (column) base + l32
    auto frag_op = [&](const __bf16* S, bool kmajor, int base, int ks) -> bf16x8 {
        if (!kmajor)
            return *reinterpret_cast<const bf16x8*>(&S[(base + l32) * kRS16 + 16 * ks + 8 * half]);
        typedef __attribute__((address_space(3))) s16x4* lds_s16x4;
        const int k0 = 16 * ks + 8 * half + (i16 >> 2);
        const int c = base + 16 * sub + 4 * (i16 & 3);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(S + k0 * kKS16 + c));
        const s16x4 hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(S + (k0 + 4) * kKS16 + c));
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    bf16x8 fa[2][2], fb[2][NB];
    auto frag = [&](int buf, int ks, int fslot) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            fa[fslot][i] = frag_op(hs[buf][0], AL == A_KM, wm * 64 + i * 32, ks);
            if (i < NB) fb[fslot][i] = frag_op(hs[buf][1], BL == B_KN, wn * 32 * NB + i * 32, ks);
        }
    };
    auto mfma = [&](int fslot) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[fslot][j], fa[fslot][i],
                                                                    acc[i][j], 0, 0, 0);
    };

    // LDS buffer kt % 2 holds K step kt; register set (kt + 1) % 2 holds
    // step kt + 1, and step kt + 2 is loaded into set kt % 2 meanwhile.
    auto kstep = [&](int kt, int set, auto FULL) {
        const int buf = kt & 1;
        if constexpr (FULL)
            gload_full(set, kbeg + (kt + 2) * BK);
        else
            gload_masked(set, kbeg + (kt + 2) * BK);   // past kend: empty chunks
        frag(buf, 1, 1);
        mfma(0);
        mfma(1);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (FULL) {
            sstore(buf ^ 1, set ^ 1, true);
            __syncthreads();
            frag(buf ^ 1, 0, 0);
        } else {
            if (kt + 1 < nk) sstore(buf ^ 1, set ^ 1, false);
            __syncthreads();
            if (kt + 1 < nk) frag(buf ^ 1, 0, 0);
        }
    };
    using Full = std::true_type;
    using Masked = std::false_type;
    const bool fast_start = fast_tile && nfull >= 2;
    if (fast_start) {
        gload_full(0, kbeg);
        gload_full(1, kbeg + BK);
        sstore(0, 0, true);
    } else if (nk > 0) {
        gload_masked(0, kbeg);
        gload_masked(1, kbeg + BK);
        sstore(0, 0, false);
    }
    if (nk > 0) {
        __syncthreads();
        frag(0, 0, 0);
    }
    int kt = 0;
    if (fast_start) {
        for (; kt + 3 < nfull; kt += 2) {
            kstep(kt, 0, Full{});
            kstep(kt + 1, 1, Full{});
        }
        mark_full(0);
        mark_full(1);
    }
    for (; kt + 1 < nk; kt += 2) {
        kstep(kt, 0, Masked{});
        kstep(kt + 1, 1, Masked{});
    }
    if (kt < nk) kstep(kt, 0, Masked{});

    __syncthreads();   // every fragment read done: the operand buffers become the stage
    constexpr int kStage = 2 * 2 * kOp16 / 2 / 4;   // floats per wavefront
    static_assert(kStage >= 32 * (32 * NB + 4), "a 32 x 32 NB block fits each wavefront's share");
    float* stage = reinterpret_cast<float*>(&hs[0][0][0]) + wave * kStage;
    store_tile_lds<EP, EP == EPI_BIAS_RELU || EP == EPI_MASK, NB>(
        P, split, m0 + wm * 64, n0 + wn * 32 * NB, half, l32, lane, stage, acc);
}

// ------------------------------------------------------------ staged bf16
// The bf16 copies products of launches whose every K step is whole (K and
// the K concatenation points multiples of 32, no appended row of ones),
// with both operands K-contiguous (A [m][k], B [n][k]: the input
// gradients). The operands go from HBM straight into LDS
// (global_load_lds_dwordx4: each wavefront instruction moves 1 KB, 16 bytes
// per lane, to consecutive LDS addresses), kH16Stages K steps in flight, so
// no register staging limits how far ahead the loads run; three stages of
// 16 KB leave room for three workgroups per CU. Each stage holds both
// operands as [row][k] (64-byte rows), unpadded, the four 16-byte chunks
// of row r at positions chunk ^ ((r / 4) % 4), so that the 128-bit fragment
// reads of 16 consecutive rows meet no bank conflicts. The loads of a
// stage land before a workgroup barrier that follows a wait on this
// wavefront's own outstanding loads. Tile, tile order, the MFMAs and the
// order they take the K values are those of the copies kernel above, so
// the products equal its bit for bit; rows outside the operands are clamped
// into them (they only feed outputs the epilogue drops).
constexpr int kH16Stages = 3;

template <Epilogue EP, GemmRole ROLE, int NB = 2>
__global__ __launch_bounds__(kThreads, 2) void gemm_h16s_kernel(GemmBatch batch) {
    constexpr int TBN = 64 * NB;
    constexpr int kS = kH16Stages;
    constexpr int kABytes = BM * BK * 2;               // 8 KB
    constexpr int kBBytes = TBN * BK * 2;              // 4 KB per NB
    constexpr int kStageBytes = kABytes + kBBytes;
    constexpr int kAInst = kABytes / 1024 / 4;         // A loads per wavefront and stage
    constexpr int kBInst = kBBytes / 1024 / 4;         // B loads per wavefront and stage
    constexpr int kLoads = kAInst + kBInst;
    static_assert(kAInst * 4096 == kABytes && kBInst * 4096 == kBBytes, "whole loads");
    constexpr int kEpiFloats = 4 * 32 * (32 * NB + 4);
    static_assert(kEpiFloats * 4 <= kS * kStageBytes, "the epilogue stage fits");
    __shared__ __attribute__((aligned(1024))) char lds[kS * kStageBytes];
    typedef __attribute__((address_space(3))) void lds_void;

    const TileInfo ti = decode_tile<BM, TBN>(batch);
    const GemmProblem& P = batch.p[ti.pi];
    const int split = ti.split, m0 = ti.m0, n0 = ti.n0;
    const int kbeg = ti.kbeg, nk = ti.nk;

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int half = lane >> 5, l32 = lane & 31;
    const int M = P.M, N = P.N;

    // Per-lane source offsets (elements), fixed for the whole K loop: load i
    // of this wavefront covers rows 16 (kAInst wave + i) + lane / 4 of A (and
    // likewise of B), LDS slot lane % 4 of the row receiving chunk
    // (lane % 4) ^ ((row / 4) % 4)
    int64_t oa[kAInst], ob[kBInst];
#pragma unroll
    for (int i = 0; i < kAInst; ++i) {
        const int r = 16 * (kAInst * wave + i) + (lane >> 2);
        const int c = (lane & 3) ^ ((r >> 2) & 3);
        oa[i] = (int64_t)min(m0 + r, M - 1) * P.hlda0 + 8 * c;
    }
#pragma unroll
    for (int i = 0; i < kBInst; ++i) {
        const int r = 16 * (kBInst * wave + i) + (lane >> 2);
        const int c = (lane & 3) ^ ((r >> 2) & 3);
        ob[i] = (int64_t)min(n0 + r, N - 1) * P.hldb0 + 8 * c;
    }
    auto stage_a = [&](int buf) { return lds + buf * kStageBytes; };
    auto stage_b = [&](int buf) { return lds + buf * kStageBytes + kABytes; };
    // loads of K step kt into buffer kt % kS (uniform base per step)
    auto issue = [&](int kt) {
        const int k0 = kbeg + kt * BK;
        const __bf16* sa = k0 >= P.ksplitA ? P.hA1 + (k0 - P.ksplitA) : P.hA0 + k0;
        const __bf16* sb = k0 >= P.ksplitB ? P.hB1 + (k0 - P.ksplitB) : P.hB0 + k0;
        char* da = stage_a(kt % kS);
        char* db = stage_b(kt % kS);
#pragma unroll
        for (int i = 0; i < kAInst; ++i)
            __builtin_amdgcn_global_load_lds((const void*)(sa + oa[i]),
                                             (lds_void*)(da + 1024 * (kAInst * wave + i)), 16, 0,
                                             0);
#pragma unroll
        for (int i = 0; i < kBInst; ++i)
            __builtin_amdgcn_global_load_lds((const void*)(sb + ob[i]),
                                             (lds_void*)(db + 1024 * (kBInst * wave + i)), 16, 0,
                                             0);
    };

    floatx16 acc[2][NB];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // fragment of MFMA step ks: lane half g holds K values 16 ks + 8 g .. + 7
    // of row base + l32
    auto frag_rk = [&](const char* S, int base, int ks) -> bf16x8 {
        const int r = base + l32, c = 2 * ks + half;
        return *reinterpret_cast<const bf16x8*>(S + 64 * r + 16 * (c ^ ((r >> 2) & 3)));
    };
    bf16x8 fa[2][2], fb[2][NB];
    auto compute = [&](int buf) {
        const char* As = stage_a(buf);
        const char* Bs = stage_b(buf);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int i = 0; i < 2; ++i) fa[ks][i] = frag_rk(As, wm * 64 + i * 32, ks);
#pragma unroll
            for (int j = 0; j < NB; ++j) fb[ks][j] = frag_rk(Bs, wn * 32 * NB + j * 32, ks);
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[ks][j], fa[ks][i],
                                                                        acc[i][j], 0, 0, 0);
    };
    // s_waitcnt vmcnt(n), no wait on the other counters (gfx9 encoding)
#define GCN_WAIT_VM(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 15) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))
    // workgroup barrier without the memory fence of __syncthreads (which
    // would wait for every load in flight); the empty asm statements keep
    // the compiler from moving LDS accesses across it
    auto stage_barrier = [] {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };

#pragma unroll
    for (int s0 = 0; s0 < kS - 1; ++s0)
        if (s0 < nk) issue(s0);
    int kt = 0;
    // steady state: step kt lands while steps kt + 1 .. kt + kS - 2 stay in
    // flight; buffer (kt + kS - 1) % kS was last read in step kt - 1, which
    // every wavefront finished before this step's barrier
    for (; kt + kS - 1 < nk; ++kt) {
        GCN_WAIT_VM((kS - 2) * kLoads);
        stage_barrier();
        issue(kt + kS - 1);
        compute(kt % kS);
    }
    // the last steps: everything issued has landed after one wait
    if (kt < nk) {
        GCN_WAIT_VM(0);
        stage_barrier();
        for (; kt < nk; ++kt) compute(kt % kS);
    }
#undef GCN_WAIT_VM
    __syncthreads();   // every fragment read done: the stages become the epilogue stage
    float* stage = reinterpret_cast<float*>(lds) + wave * (kEpiFloats / 4);
    store_tile_lds<EP, EP == EPI_BIAS_RELU || EP == EPI_MASK, NB>(
        P, split, m0 + wm * 64, n0 + wn * 32 * NB, half, l32, lane, stage, acc);
}

// Rounding of fp32 matrices to bf16 copies: one thread per 8 output
// elements of one row, jobs laid end to end (fewer than 2^31 chunks).
struct ConvBatch {
    ConvJob job[kMaxConvJobs];
    int32_t first[kMaxConvJobs + 1];   // first chunk of each job
    int32_t njobs;
};

__global__ __launch_bounds__(256) void to_bf16_kernel(ConvBatch b) {
    const int idx = (int)(blockIdx.x * 256 + threadIdx.x);
    if (idx >= b.first[b.njobs]) return;
    int j = 0;
    while (idx >= b.first[j + 1]) ++j;
    const ConvJob& J = b.job[j];
    const int per_row = (int)(J.ldd >> 3);
    const int local = idx - b.first[j];
    const int r = local / per_row;
    const int c0 = (local - r * per_row) * 8;
    const float* src = J.src + (int64_t)r * J.lds + c0;
    float f[8];
    if (c0 + 8 <= J.cols && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
        const float4 x = ld4(src), y = ld4(src + 4);
        f[0] = x.x, f[1] = x.y, f[2] = x.z, f[3] = x.w;
        f[4] = y.x, f[5] = y.y, f[6] = y.z, f[7] = y.w;
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = c0 + e < J.cols ? src[e] : 0.f;
    }
    bf16x8 out;
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = (__bf16)f[e];
    *reinterpret_cast<bf16x8*>(J.dst + (int64_t)r * J.ldd + c0) = out;
}

// sum_j src[j * stride], j ascending; eight loads in flight at a time
__device__ __forceinline__ float sum_slices(const float* src, int64_t stride, int splits) {
    float d = 0.f;
    int j = 0;
    for (; j + 8 <= splits; j += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = src[(int64_t)(j + u) * stride];
#pragma unroll
        for (int u = 0; u < 8; ++u) d += v[u];
    }
    for (; j < splits; ++j) d += src[(int64_t)j * stride];
    return d;
}

// One weight's update from its summed gradient d (and its state slot i).
template <int KIND>
__device__ __forceinline__ float opt_update(float w, float d, float* s1, float* s2, int64_t i,
                                            const OptimArgs& o) {
    if constexpr (KIND == OPT_SGD) {
        return fmaf(-o.lr, d, w);
    } else if constexpr (KIND == OPT_MOMENTUM) {
        const float u = fmaf(o.mu, s1[i], d);
        s1[i] = u;
        return fmaf(-o.lr, u, w);
    } else {
        const float m = o.b1 * s1[i] + (1.0f - o.b1) * d;
        const float v = o.b2 * s2[i] + (1.0f - o.b2) * (d * d);
        s1[i] = m;
        s2[i] = v;
        return w - o.lr * (m * o.c1) / (sqrtf(v * o.c2) + o.eps);
    }
}

// The weights of one launch laid end to end: problem i covers elements
// [end[i - 1], end[i]) (end[-1] = 0).
struct SgdBatch {
    SgdProblem p[kMaxSgdProblems];
    int64_t end[kMaxSgdProblems];
    int32_t n;
};

template <int KIND>
__global__ __launch_bounds__(256) void sgd_reduce_kernel(SgdBatch b, OptimArgs o) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= b.end[b.n - 1]) return;
    int i = 0;
    while (idx >= b.end[i]) ++i;
    const SgdProblem& p = b.p[i];
    const int64_t e = idx - (i > 0 ? b.end[i - 1] : 0);
    const int m = (int)(e / p.N), nn = (int)(e % p.N);
    const float* src = p.part + (int64_t)m * p.ldp + nn;
    const float d = sum_slices(src, p.part_stride, p.splits);
    if (m < p.Mw) {
        const int64_t w = (int64_t)m * p.N + nn;
        p.W[w] = opt_update<KIND>(p.W[w], d, p.s1, p.s2, w, o);
        if (p.dW_out) p.dW_out[w] = d;
    } else {
        p.b[nn] = opt_update<KIND>(p.b[nn], d, p.s1b, p.s2b, nn, o);
        if (p.db_out) p.db_out[nn] = d;
    }
}

__global__ __launch_bounds__(256) void splitk_finish_kernel(
    const float* __restrict__ part, int64_t part_stride, int64_t ldp, int splits, int M,
    int N, const float* __restrict__ bias, float* __restrict__ C, int64_t ldc) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)M * N) return;
    const int m = (int)(idx / N), nn = (int)(idx % N);
    float d = sum_slices(part + (int64_t)m * ldp + nn, part_stride, splits);
    if (bias) d += bias[nn];
    C[(int64_t)m * ldc + nn] = d;
}

}  // namespace

hipError_t launch_splitk_finish(const float* part, int64_t part_stride, int64_t ldp,
                                int32_t splits, int32_t M, int32_t N, const float* bias,
                                float* C, int64_t ldc, hipStream_t s) {
    const int64_t total = (int64_t)M * N;
    if (total == 0) return hipSuccess;
    ProfScope prof(s, K_SPLITK_FINISH, (double)total * splits,
                   4.0 * (double)total * (splits + 1));
    splitk_finish_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s>>>(
        part, part_stride, ldp, splits, M, N, bias, C, ldc);
    return hipGetLastError();
}

void gemm_split_plan(int32_t M, int32_t N, int32_t K, int32_t nprob, int32_t* splits,
                     int32_t* kchunk) {
    gemm_split_plan_tiles((int64_t)((M + BM - 1) / BM) * ((N + BN - 1) / BN) * std::max(nprob, 1),
                          K, splits, kchunk);
}

void gemm_split_plan_tiles(int64_t tiles, int32_t K, int32_t* splits, int32_t* kchunk) {
    // Two workgroups fit per CU: pick the smallest split whose tile count
    // fills the 512 resident slots of the 256 CUs to >= 90 %, keeping >= 2 K
    // steps per split and at most 512 slices in all (the scratch bound of the
    // partial sums).
    constexpr int64_t kSlots = 512;
    const int64_t smax = std::max<int64_t>(1, std::min<int64_t>(32, K / (2 * BK)));
    int64_t best = 1;
    double best_eff = -1.0;
    for (int64_t s = 1; s <= smax; ++s) {
        const int64_t total = tiles * s;
        if (s > 1 && total > kSlots) break;
        const double eff = (double)total / (double)(((total + kSlots - 1) / kSlots) * kSlots);
        if (eff >= 0.9) {
            best = s;
            break;
        }
        if (eff > best_eff + 1e-9) {
            best_eff = eff;
            best = s;
        }
    }
    const int64_t kc = (K + best - 1) / best;
    const int64_t chunk = std::max<int64_t>(BK, (kc + BK - 1) / BK * BK);
    *kchunk = (int32_t)chunk;
    *splits = K > 0 ? (int32_t)((K + chunk - 1) / chunk) : 1;
}

// Tile shape of a one-pass (not split-K) fp32 launch: 128 x 128, or
// 128 x 64 when that spreads the work more evenly over the CUs. The tiles
// are handed out in waves over the 256 CUs (two resident per CU), so a CU
// computes ceil(tiles / 256) tiles in all; the shape with the smaller
// ceil(tiles / 256) x tile area finishes first, the narrower tile charged
// 5 % for its extra operand traffic per flop, and a launch that leaves a
// CU with a single tile charged 30 % (nothing overlaps its start and end).
// yelp10k's 10,000 x 1,024 outputs: 632 tiles of 128 x 128 (3 per CU,
// 2.47 on average) or 1,264 of 128 x 64 (5 per CU, 4.94 on average).
// The bf16 copies kernel charges its narrow tile 22 % instead (two MFMAs
// per three fragment reads against four per four, on a kernel whose LDS
// reads already pace it; fitted to yelp10k's launches), so there it only
// pays where 128 x 128 tiles leave CUs idle.
bool gemm_narrow_tiles(const GemmBatch& b, double narrow_eff) {
    constexpr int64_t kCUs = 256;
    int64_t t2 = 0, t1 = 0;
    for (int i = 0; i < b.nprob; ++i) {
        const GemmProblem& p = b.p[i];
        if (p.M <= 0 || p.N <= 0) continue;
        const int64_t tm = (p.M + 127) / 128;
        t2 += tm * ((p.N + 127) / 128);
        t1 += tm * ((p.N + 63) / 64);
    }
    if (t2 == 0) return false;
    auto cost = [&](int64_t tiles, double area, double eff) {
        const int64_t per_cu = (tiles + kCUs - 1) / kCUs;
        return per_cu * area / eff * (tiles <= kCUs ? 1.3 : 1.0);
    };
    return cost(t1, 128.0 * 64.0, narrow_eff) < cost(t2, 128.0 * 128.0, 1.0);
}

hipError_t launch_gemm(GemmBatch& b, ALayout al, BLayout bl, Epilogue ep, GemmRole role,
                       bool bf16, hipStream_t s) {
    // 32 x 128 or 64 x 128 tiles where the caller asks for them (fp32: the
    // weight gradients of the classifier and the first layer, the
    // classifier's logits); else 128 x 64 tiles where they spread better:
    // fp32 kernel, one pass over K, row-contiguous A
    if (b.tbm != 0 && b.tbm != BM && b.tbm != 32 && b.tbm != 64) return hipErrorInvalidValue;
    const bool small = !bf16 && b.tbm == 32;
    const bool mid = !bf16 && b.tbm == 64;
    if (small && role != ROLE_CLS_DW && role != ROLE_DW_IN) return hipErrorInvalidValue;
    if (mid && role != ROLE_CLS_FWD) return hipErrorInvalidValue;
    // bf16 with operand copies in every problem: the copies kernel
    bool copies = bf16;
    for (int i = 0; i < b.nprob; ++i) copies = copies && b.p[i].hA0 && b.p[i].hB0;
    const bool nb1 = !small && !mid && (!bf16 || copies) && ep != EPI_PARTIAL && al == A_MK &&
                     gemm_narrow_tiles(b, bf16 ? 0.78 : 0.95);
    const int tbm = small ? 32 : mid ? 64 : BM;
    const int tbn = nb1 ? 64 : BN;
    int total = 0;
    for (int i = 0; i < b.nprob; ++i) {
        GemmProblem& p = b.p[i];
        p.tiles_m = (p.M + tbm - 1) / tbm;
        p.tiles_n = (p.N + tbn - 1) / tbn;
        if (ep != EPI_PARTIAL) {
            p.splits = 1;
            p.kchunk = std::max(BK, (p.K + BK - 1) / BK * BK);
        } else if (p.splits < 1 || p.kchunk < 1) {
            return hipErrorInvalidValue;
        }
        p.tile_begin = total;
        auto aligned = [](const float* q, int64_t ld) {
            return q == nullptr || (((uintptr_t)q & 15) == 0 && (ld & 3) == 0);
        };
        p.a_vec = aligned(p.A0, p.lda0) && aligned(p.A1, p.lda1);
        p.b_vec = aligned(p.B0, p.ldb0) && aligned(p.B1, p.ldb1);
        if (p.M > 0 && p.N > 0) total += p.tiles_m * p.tiles_n * p.splits;
    }
    b.total_tiles = total;
    if (total == 0) return hipSuccess;
    const dim3 grid(total), block(kThreads);
    double flops = 0, bytes = 0;
    for (int i = 0; i < b.nprob; ++i) {
        const GemmProblem& p = b.p[i];
        const double M = p.M, N = p.N, K = p.K;
        flops += 2.0 * M * N * K;
        bytes += 4.0 * (M * K + K * N + M * N) + (ep == EPI_MASK ? 4.0 * M * N : 0.0);
    }
    static const int kKinds[] = {K_GEMM_FWD, K_GEMM_CLS, K_GEMM_DX, K_GEMM_CLS_DX,
                                 K_GEMM_DW, K_GEMM_CLS_DW, K_GEMM_FWD_IN, K_GEMM_DW_IN};
    static const int kKinds16[] = {K_GEMM_FWD_BF16, K_GEMM_CLS_BF16, K_GEMM_DX_BF16,
                                   K_GEMM_CLS_DX_BF16, K_GEMM_DW_BF16, K_GEMM_CLS_DW_BF16,
                                   K_GEMM_FWD_IN_BF16, K_GEMM_DW_IN_BF16};
    if (copies) {
        auto ok16 = [](const __bf16* q, int64_t ld) {
            return q == nullptr || (((uintptr_t)q & 15) == 0 && (ld & 7) == 0);
        };
        for (int i = 0; i < b.nprob; ++i) {
            const GemmProblem& p = b.p[i];
            const bool catA = al == A_MK && p.ksplitA < p.K;
            const bool catB = bl == B_NK && p.ksplitB < p.K;
            if ((p.hC && p.c_from % 4) || (!p.C && !(p.hC && p.c_from >= p.N)) ||
                (p.hmask && (((uintptr_t)p.hmask & 7) || (p.ldhmask & 3))) ||
                !ok16(p.hA0, p.hlda0) || !ok16(p.hB0, p.hldb0) ||
                (catA && (!p.hA1 || !ok16(p.hA1, p.hlda1) || p.ksplitA % 8)) ||
                (catB && (!p.hB1 || !ok16(p.hB1, p.hldb1) || p.ksplitB % 8)) ||
                (p.hC && (((uintptr_t)p.hC & 7) || (p.ldhc & 3))))
                return hipErrorInvalidValue;
        }
        // operands are read as bf16
        bytes = 0;
        for (int i = 0; i < b.nprob; ++i) {
            const GemmProblem& p = b.p[i];
            const double M = p.M, N = p.N, K = p.K;
            const double n32 = p.hC ? std::max(0.0, N - p.c_from) : N;   // fp32 columns
            bytes += 2.0 * (M * K + K * N) + 4.0 * M * n32 +
                     (ep == EPI_MASK ? (p.hmask ? 2.0 : 4.0) * M * N : 0.0) +
                     (p.hC ? 2.0 * M * N : 0.0);
        }
    }
    // the staged copies kernel: every K step whole in every problem, B as
    // [n][k] (with B as [k][n] its transposing reads made the forward
    // products slower than the kernel above on every workload measured)
    bool staged = copies && al == A_MK && bl == B_NK && ep != EPI_PARTIAL;
    for (int i = 0; i < b.nprob && staged; ++i) {
        const GemmProblem& p = b.p[i];
        staged = p.ones_row == 0 && p.K % BK == 0 &&
                 (p.ksplitA >= p.K || (p.ksplitA % BK == 0 && p.hlda1 == p.hlda0)) &&
                 (p.ksplitB >= p.K || (p.ksplitB % BK == 0 && p.hldb1 == p.hldb0));
    }
    const int kind = bf16 ? kKinds16[role] : kKinds[role];
    ProfScope prof(s, kind, flops, bytes);
    bool bvec = true;
    for (int i = 0; i < b.nprob; ++i) {
        if (!copies && !b.p[i].a_vec) return hipErrorInvalidValue;   // A rows must be aligned
        bvec = bvec && b.p[i].b_vec;
    }
    bool half_m = true;   // every problem's rows fit the first half of a tile
    for (int i = 0; i < b.nprob; ++i) half_m = half_m && b.p[i].M <= BM / 2;
#define GCN_GEMM_CASE(AL_, BL_, EP_, ROLE_)                                          \
    if (al == AL_ && bl == BL_ && ep == EP_ && role == ROLE_) {                       \
        constexpr bool kNarrowOk = EP_ != EPI_PARTIAL && AL_ == A_MK;                 \
        constexpr bool kSmallOk = ROLE_ == ROLE_CLS_DW || ROLE_ == ROLE_DW_IN;      \
        constexpr bool kMidOk = ROLE_ == ROLE_CLS_FWD;                               \
        if (copies) {                                                                \
            if (staged) {                                                            \
                if constexpr (kNarrowOk && BL_ == B_NK) {                            \
                    if (nb1)                                                         \
                        gemm_h16s_kernel<EP_, ROLE_, 1><<<grid, block, 0, s>>>(b);    \
                    else                                                             \
                        gemm_h16s_kernel<EP_, ROLE_, 2><<<grid, block, 0, s>>>(b);    \
                }                                                                    \
            } else if (nb1) {                                                        \
                if constexpr (kNarrowOk)                                             \
                    gemm_h16_kernel<AL_, BL_, EP_, ROLE_, 1><<<grid, block, 0, s>>>(b);\
            } else {                                                                 \
                gemm_h16_kernel<AL_, BL_, EP_, ROLE_><<<grid, block, 0, s>>>(b);      \
            }                                                                        \
        } else if (bf16 && bvec)                                                       \
            gemm_bf16_kernel<AL_, BL_, EP_, true, ROLE_><<<grid, block, 0, s>>>(b);   \
        else if (bf16)                                                               \
            gemm_bf16_kernel<AL_, BL_, EP_, false, ROLE_><<<grid, block, 0, s>>>(b);  \
        else if (small) {                                                            \
            if constexpr (kSmallOk) {                                                \
                if (bvec)                                                            \
                    gemm_kernel<AL_, BL_, EP_, true, ROLE_, false, 1, 1, 1>           \
                        <<<grid, block, 0, s>>>(b);                                  \
                else                                                                 \
                    gemm_kernel<AL_, BL_, EP_, false, ROLE_, false, 1, 1, 1>          \
                        <<<grid, block, 0, s>>>(b);                                  \
            }                                                                        \
        } else if (mid) {                                                            \
            if constexpr (kMidOk) {                                                  \
                if (bvec)                                                            \
                    gemm_kernel<AL_, BL_, EP_, true, ROLE_, false, 1, 2, 2>           \
                        <<<grid, block, 0, s>>>(b);                                  \
                else                                                                 \
                    gemm_kernel<AL_, BL_, EP_, false, ROLE_, false, 1, 2, 2>          \
                        <<<grid, block, 0, s>>>(b);                                  \
            }                                                                        \
        } else if (bvec && half_m && EP_ == EPI_PARTIAL && AL_ == A_KM)                 \
            gemm_kernel<AL_, BL_, EP_, true, ROLE_, true><<<grid, block, 0, s>>>(b);  \
        else if (nb1) {                                                              \
            if constexpr (kNarrowOk) {                                               \
                if (bvec)                                                            \
                    gemm_kernel<AL_, BL_, EP_, true, ROLE_, false, 2, 1>              \
                        <<<grid, block, 0, s>>>(b);                                  \
                else                                                                 \
                    gemm_kernel<AL_, BL_, EP_, false, ROLE_, false, 2, 1>             \
                        <<<grid, block, 0, s>>>(b);                                  \
            }                                                                        \
        } else if (bvec)                                                             \
            gemm_kernel<AL_, BL_, EP_, true, ROLE_><<<grid, block, 0, s>>>(b);        \
        else                                                                         \
            gemm_kernel<AL_, BL_, EP_, false, ROLE_><<<grid, block, 0, s>>>(b);       \
        return hipGetLastError();                                                    \
    }
    GCN_GEMM_CASE(A_MK, B_KN, EPI_BIAS_RELU, ROLE_FWD)
    GCN_GEMM_CASE(A_MK, B_KN, EPI_BIAS_RELU, ROLE_FWD_IN)
    GCN_GEMM_CASE(A_MK, B_KN, EPI_BIAS, ROLE_CLS_FWD)
    GCN_GEMM_CASE(A_MK, B_KN, EPI_PARTIAL, ROLE_CLS_FWD)
    GCN_GEMM_CASE(A_MK, B_NK, EPI_MASK, ROLE_DX)
    GCN_GEMM_CASE(A_MK, B_NK, EPI_MASK, ROLE_CLS_DX)
    GCN_GEMM_CASE(A_KM, B_KN, EPI_PARTIAL, ROLE_DW)
    GCN_GEMM_CASE(A_KM, B_KN, EPI_PARTIAL, ROLE_DW_IN)
    GCN_GEMM_CASE(A_KM, B_KN, EPI_PARTIAL, ROLE_CLS_DW)
#undef GCN_GEMM_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_to_bf16(const ConvJob* jobs, int njobs, hipStream_t s) {
    if (njobs < 0 || njobs > kMaxConvJobs) return hipErrorInvalidValue;
    ConvBatch b;
    std::memset(&b, 0, sizeof(b));
    b.njobs = njobs;
    b.first[0] = 0;
    double elems = 0;
    for (int j = 0; j < njobs; ++j) {
        const ConvJob& J = jobs[j];
        if (J.rows < 0 || J.cols < 0 || J.ldd < 8 || (J.ldd & 7) || J.ldd < J.cols ||
            ((uintptr_t)J.dst & 15) || (J.rows > 0 && (!J.src || !J.dst || J.lds < J.cols)))
            return hipErrorInvalidValue;
        b.job[j] = J;
        const int64_t next = (int64_t)b.first[j] + (int64_t)J.rows * (J.ldd / 8);
        if (next >= (int64_t)1 << 31) return hipErrorInvalidValue;
        b.first[j + 1] = (int32_t)next;
        elems += (double)J.rows * J.cols;
    }
    const int64_t total = b.first[njobs];
    if (total == 0) return hipSuccess;
    ProfScope prof(s, K_TO_BF16, elems, 6.0 * elems);
    to_bf16_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s>>>(b);
    return hipGetLastError();
}

hipError_t launch_sgd_reduce(const SgdProblem* p, int nprob, const OptimArgs& o,
                             hipStream_t s) {
    if (nprob <= 0) return hipSuccess;
    if (nprob > kMaxSgdProblems) return hipErrorInvalidValue;
    SgdBatch batch;
    std::memset(&batch, 0, sizeof(batch));
    int64_t total = 0;
    for (int i = 0; i < nprob; ++i) {
        batch.p[i] = p[i];
        total += (int64_t)(p[i].Mw + (p[i].b ? 1 : 0)) * p[i].N;
        batch.end[i] = total;
    }
    batch.n = nprob;
    if (total == 0) return hipSuccess;
    const int64_t blocks = (total + 255) / 256;
    double flops = 0, bytes = 0;
    // state words read and written per weight: momentum 1, Adam 2
    const double state = o.kind == OPT_ADAM ? 2.0 : o.kind == OPT_MOMENTUM ? 1.0 : 0.0;
    for (int i = 0; i < nprob; ++i) {
        const double cells = (double)(p[i].Mw + (p[i].b ? 1 : 0)) * p[i].N;
        flops += cells * (p[i].splits + 1.0 + 4.0 * state);
        bytes += 4.0 * cells * (p[i].splits + 2.0 + 2.0 * state);
    }
    ProfScope prof(s, K_SGD, flops, bytes);
    const dim3 grid((unsigned)blocks), block(256);
    if (o.kind == OPT_ADAM)
        sgd_reduce_kernel<OPT_ADAM><<<grid, block, 0, s>>>(batch, o);
    else if (o.kind == OPT_MOMENTUM)
        sgd_reduce_kernel<OPT_MOMENTUM><<<grid, block, 0, s>>>(batch, o);
    else
        sgd_reduce_kernel<OPT_SGD><<<grid, block, 0, s>>>(batch, o);
    return hipGetLastError();
}

}  // namespace gcn
