// Update gradients (equation 2's backward) on the matrix-core engine; the
// job types are in gemm_bwd_dev.h.
#include <algorithm>
#include <type_traits>

#include "gemm_bwd_dev.h"
#include "jobs.h"

namespace gnn {

namespace {

// wt[n][k] = bf16(w[k][n]): one thread per element, writes coalesced.
__global__ void __launch_bounds__(256) shadow_sync_kernel(const float *__restrict__ w, int64_t K, int64_t n,
                                                          uint16_t *__restrict__ wt) {
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < K * n;
         t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t j = t / K, k = t - j * K;
        wt[t] = f32_to_bf16(w[k * n + j]);
    }
}

}  // namespace

size_t update_bwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt) {
    const gbwd::DwPlan p = gbwd::plan_dw(k, n_out, cap_m, gemm_dt == GNN_BF16);
    size_t bytes = round_up(gbwd::dw_part_bytes(p, k, n_out), 256);
    if (gbwd::wide_bwd_shape(k, n_out, gemm_dt))
        bytes = std::max(bytes, static_cast<size_t>(gbwd::plan_wide_bwd(k, n_out, cap_m).ws_bytes));
    return bytes;
}

gnn_status launch_shadow_sync(const float *w, int64_t K, int64_t n, uint16_t *wt, hipStream_t s) {
    if (K * n == 0) return GNN_OK;
    const unsigned grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(K * n, 256), 1 << 16));
    shadow_sync_kernel<<<grid, 256, 0, s>>>(w, K, n, wt);
    GNN_LAUNCHED("shadow_sync");
    return GNN_OK;
}

gnn_status launch_update_bwd_gemms(const gbwd::Args &a, const gbwd::Plan &p, hipStream_t s) {
    if (p.wide) return gbwd::launch_wide_bwd_gemms(a, s);
    GNN_CHECK(p.pa.map.blocks() <= kMaxGrid && p.pw.map.blocks() <= kMaxGrid, GNN_ESIZE,
              "update_bwd: too many tiles for one launch");
    // The common variants (64 x 64 tiles, vector activations and dA, the
    // activation type of the precision mode) share one launch; the input
    // gradient reads W, which only the later reduction job updates.
    const bool act_matches = a.adt == (p.bf ? GNN_BF16 : GNN_F32);
    if (p.din_grid && p.pa.tile == 64 && p.pw.tile == 64 && p.vec_o && p.vec_a && act_matches) {
        gnn_status st = GNN_OK;
        auto go = [&](auto din, auto dwj) {
            st = launch_job2(din, p.din_grid, dwj, p.dw_grid, s, "update_dinput+dweight");
        };
        if (p.bf) {
            if (p.vec_g)
                go(gbwd::dinput_job<true, 64, true, true>(a, p), gbwd::dweight_job<true, 64, uint16_t, true, true>(a, p));
            else
                go(gbwd::dinput_job<true, 64, false, true>(a, p),
                   gbwd::dweight_job<true, 64, uint16_t, true, false>(a, p));
        } else {
            if (p.vec_g)
                go(gbwd::dinput_job<false, 64, true, true>(a, p), gbwd::dweight_job<false, 64, float, true, true>(a, p));
            else
                go(gbwd::dinput_job<false, 64, false, true>(a, p),
                   gbwd::dweight_job<false, 64, float, true, false>(a, p));
        }
        return st;
    }
    gnn_status st = GNN_OK;
    if (p.din_grid) gbwd::with_dinput_job(a, p, [&](auto job) { st = launch_job(job, p.din_grid, s, "update_dinput"); });
    GNN_TRY(st);
    gbwd::with_dweight_job(a, p, [&](auto job) { st = launch_job(job, p.dw_grid, s, "update_dweight"); });
    return st;
}

gnn_status launch_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt, float *dw,
                             float *db, float *d_a, void *ws, float *w_upd, float *b_upd, uint16_t *wt_upd, float lr,
                             hipStream_t s) {
    if (n_out == 0) return GNN_OK;
    const gbwd::Args a{a_self, a_nbr, adt, k_each, m_dev, cap_m, w, g, n_out, gemm_dt, dw, db, d_a,
                       static_cast<float *>(ws), w_upd, b_upd, wt_upd, lr};
    const gbwd::Plan p = gbwd::plan(a);
    GNN_TRY(launch_update_bwd_gemms(a, p, s));
    gnn_status st = GNN_OK;
    gbwd::with_reduce_job(a, p, [&](auto job) { st = launch_job(job, p.red_grid, s, "update_dw_reduce"); });
    return st;
}

}  // namespace gnn
