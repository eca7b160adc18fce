// Loss against the ground truth (mean softmax cross-entropy over the target
// rows, fused forward and gradient), the SGD step, and small helpers of the
// training step.  Reductions run in a fixed order (no atomics).
#include "internal.h"

namespace gnn {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// One wavefront per target row.
__global__ void __launch_bounds__(kThreads) softmax_ce_kernel(const float *__restrict__ z, int64_t b, int64_t c,
                                                               const int64_t *__restrict__ labels,
                                                               const int64_t *__restrict__ targets,
                                                               float *__restrict__ g, float *__restrict__ row_loss) {
    const int lane = threadIdx.x & 63;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6);
    if (i >= b) return;
    const float *zi = z + i * c;
    float mx = -INFINITY;
    for (int64_t k = lane; k < c; k += 64) mx = fmaxf(mx, zi[k]);
    mx = wave_max(mx);
    float s = 0.f;
    for (int64_t k = lane; k < c; k += 64) s += expf(zi[k] - mx);
    s = wave_sum(s);
    const float lse = mx + logf(s);
    const int64_t y = labels[targets ? targets[i] : i];
    const float inv_b = 1.f / static_cast<float>(b);
    for (int64_t k = lane; k < c; k += 64) {
        const float p = expf(zi[k] - lse);
        g[i * c + k] = (p - (k == y ? 1.f : 0.f)) * inv_b;
    }
    if (lane == 0) row_loss[i] = lse - zi[y];
}

// Single block: loss = (sum of row losses) / b in a fixed order.
__global__ void __launch_bounds__(kThreads) loss_reduce_kernel(const float *__restrict__ row_loss, int64_t b,
                                                                float *__restrict__ loss) {
    __shared__ float sh[kThreads / 64];
    float s = 0.f;
    for (int64_t i = threadIdx.x; i < b; i += kThreads) s += row_loss[i];
    s = wave_sum(s);
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int w = 0; w < kThreads / 64; ++w) t += sh[w];
        *loss = b > 0 ? t / static_cast<float>(b) : 0.f;
    }
}

__global__ void zero_words_kernel(uint32_t *p, int64_t n) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[i] = 0u;
}

__global__ void sgd_kernel(float *__restrict__ w, const float *__restrict__ dw, int64_t n, float lr) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        w[i] = w[i] - lr * dw[i];
}

}  // namespace

size_t softmax_ce_ws_bytes(int64_t b) { return round_up(static_cast<size_t>(b > 0 ? b : 1) * 4, 256); }

gnn_status launch_softmax_ce(const float *logits, int64_t b, int64_t c, const int64_t *labels,
                             const int64_t *targets, float *g_out, float *loss_out, void *ws, hipStream_t s) {
    float *row_loss = static_cast<float *>(ws);
    if (b > 0) {
        softmax_ce_kernel<<<static_cast<unsigned>(ceil_div(b, kThreads / 64)), kThreads, 0, s>>>(
            logits, b, c, labels, targets, g_out, row_loss);
        GNN_LAUNCHED("softmax_ce");
    }
    loss_reduce_kernel<<<1, kThreads, 0, s>>>(row_loss, b, loss_out);
    GNN_LAUNCHED("loss_reduce");
    return GNN_OK;
}

gnn_status launch_fill_zero(void *p, size_t bytes, hipStream_t s) {
    const int64_t words = static_cast<int64_t>(bytes / 4);
    if (words == 0) return GNN_OK;
    int64_t blocks = ceil_div(words, 256);
    if (blocks > 65536) blocks = 65536;
    zero_words_kernel<<<static_cast<unsigned>(blocks), 256, 0, s>>>(static_cast<uint32_t *>(p), words);
    GNN_LAUNCHED("fill_zero");
    return GNN_OK;
}

gnn_status launch_sgd(float *w, const float *dw, int64_t n, float lr, hipStream_t s) {
    if (n == 0) return GNN_OK;
    int64_t blocks = ceil_div(n, 256);
    if (blocks > 65536) blocks = 65536;
    sgd_kernel<<<static_cast<unsigned>(blocks), 256, 0, s>>>(w, dw, n, lr);
    GNN_LAUNCHED("sgd");
    return GNN_OK;
}

}  // namespace gnn
