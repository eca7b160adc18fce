// Update gradients on the matrix-core engine of gemm_engine.h:
//   input     dA = G W^T                  (layers above the first)
//   weights   dW = A^T G, db = colsum(G)  (optionally followed by SGD)
#include "gemm_engine.h"

namespace gnn {

namespace {

using namespace gemm;

// ---------------------------------------------------------------------------
// input gradient: d_a = g W^T   (M x K; reduction over n_out)
// ---------------------------------------------------------------------------
template <bool BF16, int BM, int BN, bool V>
__global__ void __launch_bounds__(kThreads) update_dinput_kernel(const float *__restrict__ g,
                                                                  const float *__restrict__ w, const int64_t *m_dev,
                                                                  int64_t cap_m, int64_t K, int64_t n_out,
                                                                  float *__restrict__ d_a, float *part,
                                                                  int *tickets) {
    __shared__ __attribute__((aligned(16))) char lds[lds_bytes<BM, BN>()];
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * BM;
    const int64_t col0 = static_cast<int64_t>(blockIdx.y) * BN;
    if (row0 >= M) return;
    int64_t r_beg, r_end;
    split_range<Cfg<BF16>::BK>(n_out, gridDim.z, blockIdx.z, &r_beg, &r_end);
    SrcRows<BF16, BM, float, V> sp{g, nullptr, n_out, n_out, M, n_out, row0, {}};
    SrcRows<BF16, BN, float, V> sq{w, nullptr, n_out, n_out, K, n_out, col0, {}};
    Acc<BM, BN> acc;
    run_tile<BF16>(acc, sp, sq, r_beg, r_end, lds, [](const auto &, int64_t, bool) {});
    const int tile = blockIdx.y * gridDim.x + blockIdx.x;
    if (!reduce_splits(acc, part, tickets, tile, gridDim.x * gridDim.y, gridDim.z, blockIdx.z)) return;
    store_tile(acc, lds, d_a, K, row0, col0, M, K, [](int64_t, float v) { return v; });
}

// ---------------------------------------------------------------------------
// weight gradient: dW = A^T g over the rows (split over blockIdx.z), db from
// the k-tile-0 workgroups, optional SGD on the final values.
// ---------------------------------------------------------------------------
template <bool BF16, int BM, int BN, class TA, bool VA, bool VG>
__global__ void __launch_bounds__(kThreads) update_dweight_kernel(
    const TA *__restrict__ a_self, const TA *__restrict__ a_nbr, int64_t k_each, const float *__restrict__ g,
    const int64_t *m_dev, int64_t cap_m, int64_t n_out, float *__restrict__ dw,
    float *__restrict__ db, float *w_upd, float *b_upd, float lr, float *part, float *dbpart, int *tickets) {
    using SQ = SrcCols<BF16, BN, float, VG>;
    __shared__ __attribute__((aligned(16))) char lds[lds_bytes<BM, BN>()];
    __shared__ float cs[SQ::RPP][BN];
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * BM;  // over K
    const int64_t col0 = static_cast<int64_t>(blockIdx.y) * BN;  // over n_out
    const int nsplit = gridDim.z, split = blockIdx.z;
    int64_t r_beg, r_end;
    split_range<Cfg<BF16>::BK>(M, nsplit, split, &r_beg, &r_end);
    SrcCols<BF16, BM, TA, VA> sp{a_self, a_nbr, k_each, k_each, K, r_end, row0, {}};
    SQ sq{g, nullptr, n_out, n_out, n_out, r_end, col0, {}};
    const bool do_db = db != nullptr && blockIdx.x == 0;
    float4 colsum = make_float4(0.f, 0.f, 0.f, 0.f);
    Acc<BM, BN> acc;
    run_tile<BF16>(acc, sp, sq, r_beg, r_end, lds, [&](const SQ &src, int64_t r0, bool tail) {
        if (do_db) src.add_colsum(colsum, r0, tail);
    });
    if (do_db) {
        // fold the threads that share a column group, in order
        const int rr = threadIdx.x / SQ::TPR, tt = (threadIdx.x % SQ::TPR) * 4;
        cs[rr][tt + 0] = colsum.x;
        cs[rr][tt + 1] = colsum.y;
        cs[rr][tt + 2] = colsum.z;
        cs[rr][tt + 3] = colsum.w;
        __syncthreads();
        if (threadIdx.x < BN) {
            float s = 0.f;
            for (int k = 0; k < SQ::RPP; ++k) s += cs[k][threadIdx.x];
            dbpart[(static_cast<int64_t>(split) * gridDim.y + blockIdx.y) * BN + threadIdx.x] = s;
        }
    }
    const int tile = blockIdx.y * gridDim.x + blockIdx.x;
    if (!reduce_splits(acc, part, tickets, tile, gridDim.x * gridDim.y, nsplit, split)) return;
#pragma unroll
    for (int i = 0; i < Acc<BM, BN>::WI; ++i)
#pragma unroll
        for (int j = 0; j < Acc<BM, BN>::WJ; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t k = row0 + acc_row<BM, BN>(i, q), n = col0 + acc_col<BM, BN>(j);
                if (k < K && n < n_out) {
                    const float v = acc.c[i][j][q];
                    dw[k * n_out + n] = v;
                    if (w_upd) w_upd[k * n_out + n] -= lr * v;
                }
            }
    if (do_db && threadIdx.x < BN) {
        const int64_t n = col0 + threadIdx.x;
        if (n < n_out) {
            float s = 0.f;
            for (int s2 = 0; s2 < nsplit; ++s2)
                s += dbpart[(static_cast<int64_t>(s2) * gridDim.y + blockIdx.y) * BN + threadIdx.x];
            db[n] = s;
            if (b_upd) b_upd[n] -= lr * s;
        }
    }
}

}  // namespace

using gemm::kTicketBytes;

size_t update_bwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt) {
    const bool bf = gemm_dt == GNN_BF16;
    const Plan pw = plan_dw(k, n_out, cap_m, bf);
    const Plan pa = plan_fwd(cap_m, k, n_out, bf);
    return 2 * kTicketBytes + round_up(part_bytes(pw), 256) + round_up(dbpart_bytes(pw, n_out), 256) +
           round_up(part_bytes(pa), 256);
}

gnn_status launch_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt, float *dw,
                             float *db, float *d_a, void *ws, float *w_upd, float *b_upd, float lr, hipStream_t s) {
    if (n_out == 0) return GNN_OK;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const bool bf = gemm_dt == GNN_BF16;
    const Plan pw = plan_dw(K, n_out, cap_m, bf);
    const Plan pa = plan_fwd(cap_m, K, n_out, bf);
    Carver c(ws);
    int *tick_w = c.ptr<int>(c.take(kTicketBytes));
    int *tick_a = c.ptr<int>(c.take(kTicketBytes));
    float *part_w = c.ptr<float>(c.take(part_bytes(pw)));
    float *dbpart = c.ptr<float>(c.take(dbpart_bytes(pw, n_out)));
    float *part_a = c.ptr<float>(c.take(part_bytes(pa)));
    const size_t asz = dtype_size(adt);
    const bool vec_a = (k_each % 4 == 0) && aligned(a_self, 4 * asz) && (!a_nbr || aligned(a_nbr, 4 * asz));
    const bool vec_g = (n_out % 4 == 0) && aligned(g, 16) && aligned(w, 16);
    // input gradient first: it reads W before an optional fused SGD changes it
    if (d_a && cap_m > 0) {
#define DA(BFV, T, V) \
    update_dinput_kernel<BFV, T, T, V><<<pa.grid, kThreads, 0, s>>>(g, w, m_dev, cap_m, K, n_out, d_a, part_a, tick_a)
#define DA_V(BFV, T)                 \
    do {                             \
        if (vec_g) DA(BFV, T, true);  \
        else DA(BFV, T, false);       \
    } while (0)
        if (bf) {
            if (pa.tile == 128) DA_V(true, 128); else DA_V(true, 64);
        } else {
            if (pa.tile == 128) DA_V(false, 128); else DA_V(false, 64);
        }
#undef DA_V
#undef DA
        GNN_LAUNCHED("update_dinput");
    }
#define DW(BFV, T, TA, VA, VG)                                                                                  \
    update_dweight_kernel<BFV, T, T, TA, VA, VG><<<pw.grid, kThreads, 0, s>>>(                                 \
        static_cast<const TA *>(a_self), static_cast<const TA *>(a_nbr), k_each, g, m_dev, cap_m, n_out, dw, db, \
        w_upd, b_upd, lr, part_w, dbpart, tick_w)
#define DW_V(BFV, T, TA)                              \
    do {                                              \
        if (vec_a && vec_g) DW(BFV, T, TA, true, true);      \
        else if (vec_a) DW(BFV, T, TA, true, false);         \
        else if (vec_g) DW(BFV, T, TA, false, true);         \
        else DW(BFV, T, TA, false, false);                   \
    } while (0)
#define DW_T(BFV, TA)            \
    do {                         \
        if (pw.tile == 128)      \
            DW_V(BFV, 128, TA);  \
        else                     \
            DW_V(BFV, 64, TA);   \
    } while (0)
    if (bf) {
        if (adt == GNN_BF16) DW_T(true, uint16_t); else DW_T(true, float);
    } else {
        if (adt == GNN_BF16) DW_T(false, uint16_t); else DW_T(false, float);
    }
#undef DW_T
#undef DW_V
#undef DW
    GNN_LAUNCHED("update_dweight");
    return GNN_OK;
}

}  // namespace gnn
