// Loss against the ground truth (mean softmax cross-entropy over the target
// rows, fused forward and gradient), the SGD step, and small helpers of the
// training step.  Reductions run in a fixed order (no atomics).
#include "jobs.h"
#include "loss_dev.h"

namespace gnn {

namespace {

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
    if (b > 0)
        GNN_TRY(launch_job(loss::SoftmaxJob{logits, b, c, labels, targets, g_out, row_loss},
                           static_cast<unsigned>(ceil_div(b, loss::kThreads / 64)), s, "softmax_ce"));
    return launch_job(loss::LossReduceJob{row_loss, b, loss_out}, 1, s, "loss_reduce");
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
