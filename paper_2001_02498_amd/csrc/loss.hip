// Classifier loss and its gradient w.r.t. the logits (Section 2.1: softmax
// with cross-entropy, whose gradient is a subtraction; the multi-label
// workloads use a sigmoid with binary cross-entropy). One wavefront per
// vertex row, the row's logits in registers (summed from the classifier's
// split-K slices when it was split, which also writes the logits); per-row
// losses are then summed by a single workgroup in a fixed order, so the
// scalar loss is bitwise reproducible. A row whose label is invalid (a class
// outside [0, C), a multi-label byte other than 0 or 1) is flagged; the
// summing workgroup folds the flags and a non-finite mean into one status
// word (bit 0: invalid label, bit 1: non-finite loss), written every call.
#include "kernels.h"
#include "prof.h"

namespace gcn {
namespace {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
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

// One wavefront per row; lane l holds logits l, l+64, ... (VPL per lane).
// The logits are the sum of `splits` split-K slices (one slice: the logits
// themselves) plus the optional bias; they are written to z_out (if it
// differs from the slices) and kept in registers for the loss.
template <int VPL, bool BCE>
__global__ __launch_bounds__(256) void loss_kernel(
    int n, int C, const float* __restrict__ part, int64_t stride, int splits, int64_t ldp,
    const float* __restrict__ bias, float* z_out, int64_t ldz, const void* __restrict__ labels,
    float* __restrict__ dz, int64_t ldd, float* __restrict__ rowloss, int32_t* __restrict__ rowflag,
    __bf16* __restrict__ dzh, int64_t lddh) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= n) return;
    const bool write_z = z_out != part;
    float v[VPL];
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int c = lane + 64 * i;
        v[i] = 0.f;
        if (c < C) {
            v[i] = sum_slices(part + (int64_t)row * ldp + c, stride, splits);
            if (bias) v[i] += bias[c];
            if (write_z) z_out[(int64_t)row * ldz + c] = v[i];
        }
    }
    float* dr = dz + (int64_t)row * ldd;
    __bf16* drh = dzh ? dzh + (int64_t)row * lddh : nullptr;
    if constexpr (!BCE) {
        const int y = static_cast<const int32_t*>(labels)[row];
        float m = -INFINITY;
#pragma unroll
        for (int i = 0; i < VPL; ++i)
            if (lane + 64 * i < C) m = fmaxf(m, v[i]);
        m = wave_max(m);
        float ssum = 0.f;
#pragma unroll
        for (int i = 0; i < VPL; ++i)
            if (lane + 64 * i < C) ssum += expf(v[i] - m);
        ssum = wave_sum(ssum);
        float zy = 0.f;
#pragma unroll
        for (int i = 0; i < VPL; ++i)
            if (lane + 64 * i == y) zy = v[i];
        zy = wave_sum(zy);   // exactly one lane holds z_y (none: label out of range)
        const float inv_s = 1.0f / ssum, inv_n = 1.0f / (float)n;
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            const int c = lane + 64 * i;
            if (c < C) {
                const float d = (expf(v[i] - m) * inv_s - (c == y ? 1.0f : 0.0f)) * inv_n;
                dr[c] = d;
                if (drh) drh[c] = (__bf16)d;
            }
        }
        if (lane == 0) {
            rowloss[row] = (m + logf(ssum)) - zy;
            if (rowflag) rowflag[row] = (y < 0 || y >= C) ? 1 : 0;
        }
    } else {
        const uint8_t* yr = static_cast<const uint8_t*>(labels) + (int64_t)row * C;
        const float scale = 1.0f / ((float)n * (float)C);
        float acc = 0.f;
        bool bad = false;
#pragma unroll
        for (int i = 0; i < VPL; ++i) {
            const int c = lane + 64 * i;
            if (c < C) {
                const float z = v[i];
                const uint8_t yb = yr[c];
                bad = bad || yb > 1;
                const float y = yb ? 1.0f : 0.0f;
                acc += fmaxf(z, 0.f) - z * y + log1pf(expf(-fabsf(z)));
                const float d = (1.0f / (1.0f + expf(-z)) - y) * scale;
                dr[c] = d;
                if (drh) drh[c] = (__bf16)d;
            }
        }
        acc = wave_sum(acc);
        const bool any_bad = __ballot(bad) != 0;
        if (lane == 0) {
            rowloss[row] = acc;
            if (rowflag) rowflag[row] = any_bad ? 1 : 0;
        }
    }
}

// Fixed-order reduction: thread t sums rows t, t+256, ...; then a tree.
__global__ __launch_bounds__(256) void mean_kernel(int n, const float* __restrict__ rowloss,
                                                   const int32_t* __restrict__ rowflag,
                                                   float denom, float* __restrict__ out,
                                                   int32_t* __restrict__ status) {
    __shared__ float part[256];
    __shared__ int flags[256];
    // thread t sums rows t, t+256, ... in order (and ORs their flags), eight
    // rows in flight
    float s = 0.f;
    int f = 0;
    int i = threadIdx.x;
    for (; i + 7 * 256 < n; i += 8 * 256) {
        float v[8];
        int g[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            v[u] = rowloss[i + u * 256];
            g[u] = rowflag ? rowflag[i + u * 256] : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            s += v[u];
            f |= g[u];
        }
    }
    for (; i < n; i += 256) {
        s += rowloss[i];
        f |= rowflag ? rowflag[i] : 0;
    }
    part[threadIdx.x] = s;
    flags[threadIdx.x] = f;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w) {
            part[threadIdx.x] += part[threadIdx.x + w];
            flags[threadIdx.x] |= flags[threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const float loss = part[0] / denom;
        out[0] = loss;
        if (status) status[0] = (flags[0] ? 1 : 0) | (isfinite(loss) ? 0 : 2);
    }
}

}  // namespace

hipError_t launch_loss_parts(int32_t n, int32_t C, int32_t kind, const float* part,
                             int64_t stride, int32_t splits, int64_t ldp, const float* bias,
                             float* z_out, int64_t ldz, const void* labels, float* dz,
                             int64_t ldd, float* rowloss, int32_t* rowflag, int32_t* status,
                             float* loss_out, hipStream_t s, __bf16* dzh, int64_t lddh) {
    if (C > 64 * kMaxLossVPL) return hipErrorInvalidValue;
    if (n > 0) {
        const dim3 grid((n + 3) / 4), block(256);
        ProfScope prof(s, K_LOSS_ROWS, (double)n * C * (8.0 + splits),
                       4.0 * (double)n * C * (splits + 2.0) + (dzh ? 2.0 : 0.0) * n * C +
                           4.0 * n);
        const int vpl = (C + 63) / 64;
#define GCN_LOSS_CASE(V_)                                                                 \
        if (vpl <= V_) {                                                                  \
            if (kind == GCN_LOSS_SOFTMAX_CE)                                              \
                loss_kernel<V_, false><<<grid, block, 0, s>>>(n, C, part, stride, splits, \
                    ldp, bias, z_out, ldz, labels, dz, ldd, rowloss, rowflag, dzh, lddh);         \
            else                                                                          \
                loss_kernel<V_, true><<<grid, block, 0, s>>>(n, C, part, stride, splits,  \
                    ldp, bias, z_out, ldz, labels, dz, ldd, rowloss, rowflag, dzh, lddh);         \
        } else
        GCN_LOSS_CASE(1) GCN_LOSS_CASE(2) GCN_LOSS_CASE(4) GCN_LOSS_CASE(8) {
            return hipErrorInvalidValue;
        }
#undef GCN_LOSS_CASE
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const float denom = kind == GCN_LOSS_SOFTMAX_CE ? (float)n : (float)n * (float)C;
    ProfScope prof(s, K_LOSS_MEAN, (double)n, 4.0 * n);
    mean_kernel<<<dim3(1), dim3(256), 0, s>>>(n, rowloss, rowflag, denom > 0 ? denom : 1.0f,
                                              loss_out, status);
    return hipGetLastError();
}

hipError_t launch_loss(int32_t n, int32_t C, int32_t kind, const float* z, int64_t ldz,
                       const void* labels, float* dz, int64_t ldd, float* rowloss,
                       int32_t* rowflag, int32_t* status, float* loss_out, hipStream_t s) {
    return launch_loss_parts(n, C, kind, z, 0, 1, ldz, nullptr, const_cast<float*>(z), ldz,
                             labels, dz, ldd, rowloss, rowflag, status, loss_out, s);
}

}  // namespace gcn
