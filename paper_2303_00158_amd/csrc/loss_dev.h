// Device side of the loss (see loss_sgd.hip): mean softmax cross-entropy
// over the target rows, as jobs.  The per-row work (gradient and row loss)
// and the fixed-order reduction of the row losses are separate jobs, so the
// training step can run the reduction alongside its last kernel.
#pragma once

#include "internal.h"

namespace gnn {
namespace loss {

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

// One wavefront per target row: g = (softmax(z) - onehot(y)) / b and the
// row loss logsumexp(z) - z_y.
struct SoftmaxJob {
    const float *z;
    int64_t b, c;
    const int64_t *labels, *targets;
    float *g, *row_loss;
    __device__ void run(int64_t blk, int64_t) const {
        const int lane = threadIdx.x & 63;
        const int64_t i = blk * (kThreads / 64) + (threadIdx.x >> 6);
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
};

// Run by one whole workgroup: (sum of the b row losses) / b in a fixed order.
__device__ __forceinline__ float reduce_row_losses(const float *row_loss, int64_t b) {
    __shared__ float sh[kThreads / 64];
    float s = 0.f;
    for (int64_t i = threadIdx.x; i < b; i += kThreads) s += row_loss[i];
    s = wave_sum(s);
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = s;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) t += sh[w];
    return b > 0 ? t / static_cast<float>(b) : 0.f;
}

// Workgroup 0 only.
struct LossReduceJob {
    const float *row_loss;
    int64_t b;
    float *loss;
    __device__ void run(int64_t blk, int64_t) const {
        if (blk != 0) return;
        const float v = reduce_row_losses(row_loss, b);
        if (threadIdx.x == 0) *loss = v;
    }
};

// End of a training step (workgroup 0 only): the loss from the row losses,
// the step's sampled edges (sum of the blocks' nnz counters) and its device
// error flags (OR of the blocks' counts[3]), written to `error` by the first
// step of a call and ORed into it by the later ones.
struct TailJob {
    const int64_t *counts[GNN_MAX_LAYERS];
    int num_blocks;
    const float *row_loss;
    int64_t b;
    float *loss, *loss_out;
    int64_t *edges, *edges_out;
    int64_t *error;
    int accumulate;
    __device__ void run(int64_t blk, int64_t) const {
        if (blk != 0) return;
        const float v = reduce_row_losses(row_loss, b);
        if (threadIdx.x == 0) {
            int64_t e = 0, err = 0;
            for (int h = 0; h < num_blocks; ++h) {
                e += counts[h][2];
                err |= counts[h][3];
            }
            *error = accumulate ? (*error | err) : err;
            *edges = e;
            if (edges_out) *edges_out = e;
            *loss = v;
            if (loss_out) *loss_out = v;
        }
    }
};

}  // namespace loss
}  // namespace gnn
