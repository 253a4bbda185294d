// Classifier loss and its gradient w.r.t. the logits (Section 2.1: softmax
// with cross-entropy, whose gradient is a subtraction; the multi-label
// workloads use a sigmoid with binary cross-entropy). One wavefront per
// vertex row; per-row losses are then summed by a single workgroup in a
// fixed order, so the scalar loss is bitwise reproducible.
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

__global__ __launch_bounds__(256) void softmax_ce_kernel(
    int n, int C, const float* __restrict__ z, int64_t ldz,
    const int32_t* __restrict__ labels, float* __restrict__ dz, int64_t ldd,
    float* __restrict__ rowloss) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= n) return;
    const float* zr = z + (int64_t)row * ldz;
    float m = -INFINITY;
    for (int c = lane; c < C; c += 64) m = fmaxf(m, zr[c]);
    m = wave_max(m);
    float s = 0.f;
    for (int c = lane; c < C; c += 64) s += expf(zr[c] - m);
    s = wave_sum(s);
    const int y = labels[row];
    const bool y_ok = y >= 0 && y < C;
    const float zy = y_ok ? zr[y] : 0.f;
    const float inv_s = 1.0f / s;
    const float inv_n = 1.0f / (float)n;
    float* dr = dz + (int64_t)row * ldd;
    for (int c = lane; c < C; c += 64) {
        const float p = expf(zr[c] - m) * inv_s;
        dr[c] = (p - (c == y ? 1.0f : 0.0f)) * inv_n;
    }
    if (lane == 0) rowloss[row] = (m + logf(s)) - zy;
}

__global__ __launch_bounds__(256) void sigmoid_bce_kernel(
    int n, int C, const float* __restrict__ z, int64_t ldz,
    const uint8_t* __restrict__ labels, float* __restrict__ dz, int64_t ldd,
    float* __restrict__ rowloss) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= n) return;
    const float* zr = z + (int64_t)row * ldz;
    const uint8_t* yr = labels + (int64_t)row * C;
    float* dr = dz + (int64_t)row * ldd;
    const float scale = 1.0f / ((float)n * (float)C);
    float acc = 0.f;
    for (int c = lane; c < C; c += 64) {
        const float v = zr[c];
        const float y = yr[c] ? 1.0f : 0.0f;
        acc += fmaxf(v, 0.f) - v * y + log1pf(expf(-fabsf(v)));
        const float sig = 1.0f / (1.0f + expf(-v));
        dr[c] = (sig - y) * scale;
    }
    acc = wave_sum(acc);
    if (lane == 0) rowloss[row] = acc;
}

// Fixed-order reduction: thread t sums rows t, t+256, ...; then a tree.
__global__ __launch_bounds__(256) void mean_kernel(int n, const float* __restrict__ rowloss,
                                                   float denom, float* __restrict__ out) {
    __shared__ float part[256];
    float s = 0.f;
    for (int i = threadIdx.x; i < n; i += 256) s += rowloss[i];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = part[0] / denom;
}

}  // namespace

hipError_t launch_loss(int32_t n, int32_t C, int32_t kind, const float* z,
                       int64_t ldz, const void* labels, float* dz, int64_t ldd,
                       float* rowloss, float* loss_out, hipStream_t s) {
    if (n > 0) {
        const dim3 grid((n + 3) / 4), block(256);
        ProfScope prof(s, K_LOSS_ROWS, 8.0 * n * C, 8.0 * n * C + 4.0 * n);
        if (kind == GCN_LOSS_SOFTMAX_CE)
            softmax_ce_kernel<<<grid, block, 0, s>>>(
                n, C, z, ldz, static_cast<const int32_t*>(labels), dz, ldd, rowloss);
        else
            sigmoid_bce_kernel<<<grid, block, 0, s>>>(
                n, C, z, ldz, static_cast<const uint8_t*>(labels), dz, ldd, rowloss);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const float denom = kind == GCN_LOSS_SOFTMAX_CE ? (float)n : (float)n * (float)C;
    ProfScope prof(s, K_LOSS_MEAN, (double)n, 4.0 * n);
    mean_kernel<<<dim3(1), dim3(256), 0, s>>>(n, rowloss, denom > 0 ? denom : 1.0f, loss_out);
    return hipGetLastError();
}

}  // namespace gcn
