// Forward update (equation 2): Z = [A_self || A_nbr] W + b with the ReLU
// and narrowing epilogue, on the matrix-core engine of gemm_engine.h.
#include "gemm_engine.h"

namespace gnn {

namespace {

using namespace gemm;

// ---------------------------------------------------------------------------
// forward: out = act([self || nbr] W + b)
// ---------------------------------------------------------------------------
template <bool BF16, int BM, int BN, class TA, class TO, bool VA, bool VW>
__global__ void __launch_bounds__(kThreads) update_fwd_kernel(const TA *__restrict__ a_self,
                                                               const TA *__restrict__ a_nbr, int64_t k_each,
                                                               const int64_t *m_dev, int64_t cap_m,
                                                               const float *__restrict__ w,
                                                               const float *__restrict__ bias, int64_t n_out,
                                                               int relu, TO *__restrict__ out, float *part,
                                                               int *tickets) {
    __shared__ __attribute__((aligned(16))) char lds[lds_bytes<BM, BN>()];
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * BM;
    const int64_t col0 = static_cast<int64_t>(blockIdx.y) * BN;
    if (row0 >= M) return;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    int64_t r_beg, r_end;
    split_range<Cfg<BF16>::BK>(K, gridDim.z, blockIdx.z, &r_beg, &r_end);
    SrcRows<BF16, BM, TA, VA> sp{a_self, a_nbr, k_each, k_each, M, K, row0, {}};
    SrcCols<BF16, BN, float, VW> sq{w, nullptr, n_out, n_out, n_out, r_end, col0, {}};
    Acc<BM, BN> acc;
    run_tile<BF16>(acc, sp, sq, r_beg, r_end, lds, [](const auto &, int64_t, bool) {});
    const int tile = blockIdx.y * gridDim.x + blockIdx.x;
    if (!reduce_splits(acc, part, tickets, tile, gridDim.x * gridDim.y, gridDim.z, blockIdx.z)) return;
    store_tile(acc, lds, out, n_out, row0, col0, M, n_out, [&](int64_t n, float v) {
        float z = v + (bias ? bias[n] : 0.f);
        if (relu && !(z > 0.f)) z = 0.f;
        return z;
    });
}

}  // namespace

using gemm::kTicketBytes;

size_t update_fwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt) {
    const Plan p = plan_fwd(cap_m, n_out, k, gemm_dt == GNN_BF16);
    return kTicketBytes + round_up(part_bytes(p), 256);
}

gnn_status launch_update_fwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *bias, int64_t n_out, int relu, int gemm_dt,
                             void *out, int odt, void *ws, hipStream_t s) {
    if (cap_m == 0 || n_out == 0) return GNN_OK;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const bool bf = gemm_dt == GNN_BF16;
    Plan p = plan_fwd(cap_m, n_out, K, bf);
    if (ws == nullptr) {
        p.nsplit = 1;
        p.grid.z = 1;
    }
    int *tickets = static_cast<int *>(ws);
    float *part = ws ? reinterpret_cast<float *>(static_cast<char *>(ws) + kTicketBytes) : nullptr;
    const size_t asz = dtype_size(adt);
    const bool vec_a = (k_each % 4 == 0) && aligned(a_self, 4 * asz) && (!a_nbr || aligned(a_nbr, 4 * asz));
    const bool vec_w = (n_out % 4 == 0) && aligned(w, 16);
#define FWD(BFV, T, TA, TO, VA, VW)                                                                                 \
    update_fwd_kernel<BFV, T, T, TA, TO, VA, VW><<<p.grid, kThreads, 0, s>>>(                                      \
        static_cast<const TA *>(a_self), static_cast<const TA *>(a_nbr), k_each, m_dev, cap_m, w, bias, n_out, relu, \
        static_cast<TO *>(out), part, tickets)
#define FWD_V(BFV, T, TA, TO)                              \
    do {                                                   \
        if (vec_a && vec_w) FWD(BFV, T, TA, TO, true, true);      \
        else if (vec_a) FWD(BFV, T, TA, TO, true, false);         \
        else if (vec_w) FWD(BFV, T, TA, TO, false, true);         \
        else FWD(BFV, T, TA, TO, false, false);                   \
    } while (0)
#define FWD_T(BFV, TA, TO)            \
    do {                              \
        if (p.tile == 128)            \
            FWD_V(BFV, 128, TA, TO);  \
        else                          \
            FWD_V(BFV, 64, TA, TO);   \
    } while (0)
    if (bf) {
        if (adt == GNN_BF16 && odt == GNN_BF16) FWD_T(true, uint16_t, uint16_t);
        else if (adt == GNN_BF16 && odt == GNN_F32) FWD_T(true, uint16_t, float);
        else if (adt == GNN_F32 && odt == GNN_BF16) FWD_T(true, float, uint16_t);
        else FWD_T(true, float, float);
    } else {
        if (adt == GNN_BF16 && odt == GNN_BF16) FWD_T(false, uint16_t, uint16_t);
        else if (adt == GNN_BF16 && odt == GNN_F32) FWD_T(false, uint16_t, float);
        else if (adt == GNN_F32 && odt == GNN_BF16) FWD_T(false, float, uint16_t);
        else FWD_T(false, float, float);
    }
#undef FWD_T
#undef FWD_V
#undef FWD
    GNN_LAUNCHED("update_fwd");
    return GNN_OK;
}

}  // namespace gnn
