// Update gradients on the matrix-core engine of gemm_engine.h:
//   input     dA = G W^T                  (layers above the first)
//   weights   dW = A^T G, db = colsum(G)  (optionally followed by SGD)
//
// dA reduces over n_out only and runs unsplit.  dW reduces over the
// mini-batch rows, so the rows are split across workgroups: each split
// writes its dW tile (and, from the first row tile, its db columns) as a
// row-major fp32 partial, and dw_reduce_kernel sums the partials in split
// order and applies SGD to W and b with the final values.
#include "gemm_engine.h"

namespace gnn {

namespace {

using namespace gemm;

// ---------------------------------------------------------------------------
// input gradient: d_a = g W^T   (M x K; reduction over n_out)
// ---------------------------------------------------------------------------
template <bool BF16, int TILE, bool V, bool VO>
__global__ void __launch_bounds__(kThreads) update_dinput_kernel(const float *__restrict__ g,
                                                                  const float *__restrict__ w, const int64_t *m_dev,
                                                                  int64_t cap_m, int64_t K, int64_t n_out,
                                                                  float *__restrict__ d_a, TileMap map) {
    constexpr int D = depth<TILE>();
    __shared__ __attribute__((aligned(16))) char lds[lds_bytes<TILE, TILE>()];
    int64_t tx, ty;
    map.tile_of(blockIdx.x, &tx, &ty);
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t row0 = tx * TILE, col0 = ty * TILE;
    if (tx >= map.mt || row0 >= M) return;
    SrcRows<BF16, TILE, float, V, D> sp{g, nullptr, n_out, n_out, M, n_out, row0, {}};
    SrcRows<BF16, TILE, float, V, D> sq{w, nullptr, n_out, n_out, K, n_out, col0, {}};
    Acc<TILE, TILE> acc;
    run_tile<BF16, D>(acc, sp, sq, 0, n_out, lds, [](const auto &, int, int64_t, bool) {});
    const int64_t gc = col0 + TileOut<TILE, TILE>::col();
    emit_tile(acc, lds, [&](int, int r, int, float4 v) {
        const int64_t gr = row0 + r;
        if (gr < M) store4_masked<VO>(d_a, gr * K, gc, K, v);
    });
}

// ---------------------------------------------------------------------------
// weight gradient partials: part[split][k][n] = sum over this split's rows
// of A[row][k] g[row][n]; part[split][K][n] = sum of g[row][n] (db).
// ---------------------------------------------------------------------------
template <bool BF16, int TILE, class TA, bool VA, bool VG>
__global__ void __launch_bounds__(kThreads) update_dweight_kernel(const TA *__restrict__ a_self,
                                                                   const TA *__restrict__ a_nbr, int64_t k_each,
                                                                   const float *__restrict__ g, const int64_t *m_dev,
                                                                   int64_t cap_m, int64_t n_out, int want_db,
                                                                   float *__restrict__ part, SplitMap map,
                                                                   int64_t k_tiles) {
    constexpr int D = depth<TILE>();
    using SQ = SrcCols<BF16, TILE, float, VG, D>;
    __shared__ __attribute__((aligned(16))) char lds[lds_bytes<TILE, TILE>()];
    __shared__ float cs[SQ::RPP][TILE];
    int split;
    int64_t tile;
    map.of(blockIdx.x, &split, &tile);
    if (split >= map.nsplit) return;
    const int64_t tk = tile % k_tiles, tn = tile / k_tiles;
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const int64_t row0 = tk * TILE;  // over K
    const int64_t col0 = tn * TILE;  // over n_out
    const int nsplit = map.nsplit;
    int64_t r_beg, r_end;
    split_range<Cfg<BF16>::BK>(M, nsplit, split, &r_beg, &r_end);
    SrcCols<BF16, TILE, TA, VA, D> sp{a_self, a_nbr, k_each, k_each, K, r_end, row0, {}};
    SQ sq{g, nullptr, n_out, n_out, n_out, r_end, col0, {}};
    const bool do_db = want_db && tk == 0;
    float4 colsum = make_float4(0.f, 0.f, 0.f, 0.f);
    Acc<TILE, TILE> acc;
    run_tile<BF16, D>(acc, sp, sq, r_beg, r_end, lds, [&](const SQ &src, int s, int64_t r0, bool tail) {
        if (do_db) src.add_colsum(s, colsum, r0, tail);
    });
    const int64_t ldp = part_ld(n_out);
    float *pp = part + static_cast<int64_t>(split) * (K + 1) * ldp;
    if (do_db) {
        // fold the threads that share a column group, in order
        const int rr = threadIdx.x / SQ::TPR, tt = (threadIdx.x % SQ::TPR) * 4;
        cs[rr][tt + 0] = colsum.x;
        cs[rr][tt + 1] = colsum.y;
        cs[rr][tt + 2] = colsum.z;
        cs[rr][tt + 3] = colsum.w;
        __syncthreads();
        if (threadIdx.x < TILE && col0 + threadIdx.x < ldp) {
            float sum = 0.f;
            for (int k = 0; k < SQ::RPP; ++k) sum += cs[k][threadIdx.x];
            pp[K * ldp + col0 + threadIdx.x] = sum;
        }
    }
    const int64_t gc = col0 + TileOut<TILE, TILE>::col();
    emit_tile(acc, lds, [&](int, int r, int, float4 v) {
        const int64_t k = row0 + r;
        if (k < K && gc < ldp) *reinterpret_cast<float4 *>(pp + k * ldp + gc) = v;
    });
}

// dw = sum over splits of the partials (db from row K); then, when w_upd /
// b_upd are given, w_upd -= lr * dw and b_upd -= lr * db.  The values an
// update reads are loaded before the partials, so each thread waits once.
template <bool VO>
__global__ void __launch_bounds__(256) dw_reduce_kernel(const float *__restrict__ part, int nsplit, int64_t K,
                                                        int64_t n_out, float *__restrict__ dw,
                                                        float *__restrict__ db, float *__restrict__ w_upd,
                                                        float *__restrict__ b_upd, uint16_t *__restrict__ wt_upd,
                                                        float lr) {
    const int64_t ldp = part_ld(n_out), chunks = ldp / 4;
    const int64_t rows = K + (db ? 1 : 0);
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < rows * chunks;
         t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = t / chunks, c = (t % chunks) * 4;
        const bool brow = r == K;
        const int64_t base = brow ? 0 : r * n_out;
        float *upd = brow ? b_upd : w_upd;
        const float4 old = upd ? load4_clamped<VO>(upd, base, c, n_out) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 s = sum_splits(part + r * ldp + c, (K + 1) * ldp, nsplit);
        store4_masked<VO>(brow ? db : dw, base, c, n_out, s);
        if (upd) {
            const float4 nw = make_float4(old.x - lr * s.x, old.y - lr * s.y, old.z - lr * s.z, old.w - lr * s.w);
            store4_masked<VO>(upd, base, c, n_out, nw);
            if (wt_upd && !brow) {
                const float v[4] = {nw.x, nw.y, nw.z, nw.w};
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (c + e < n_out) wt_upd[(c + e) * K + r] = f32_to_bf16(v[e]);
            }
        }
    }
}

// wt[n][k] = bf16(w[k][n]): one thread per element, writes coalesced.
__global__ void __launch_bounds__(256) shadow_sync_kernel(const float *__restrict__ w, int64_t K, int64_t n,
                                                          uint16_t *__restrict__ wt) {
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < K * n;
         t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t j = t / K, k = t - j * K;
        wt[t] = f32_to_bf16(w[k * n + j]);
    }
}

struct DwPlan {
    int tile, nsplit;
    int64_t k_tiles;
    SplitMap map;
};

DwPlan plan_dw(int64_t K, int64_t n_out, int64_t cap_m, bool bf16) {
    DwPlan p;
    p.tile = pick_tile(K, n_out);
    p.k_tiles = ceil_div(K, p.tile);
    const int64_t tiles = p.k_tiles * ceil_div(n_out, p.tile);
    const int64_t nch = std::max<int64_t>(ceil_div(cap_m, bk_of(bf16)), 1);
    p.nsplit = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>({ceil_div(512, tiles), 64, nch})));
    p.map = SplitMap{tiles, p.nsplit};
    return p;
}

struct DinPlan {
    int tile;
    TileMap map;
};

DinPlan plan_dinput(int64_t cap_m, int64_t K) {
    DinPlan p;
    p.tile = pick_tile(cap_m, K);
    p.map = TileMap{ceil_div(std::max<int64_t>(cap_m, 1), p.tile), ceil_div(K, p.tile)};
    return p;
}

size_t dw_part_bytes(const DwPlan &p, int64_t K, int64_t n_out) {
    return static_cast<size_t>(p.nsplit) * (K + 1) * part_ld(n_out) * 4;
}

}  // namespace

size_t update_bwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt) {
    return round_up(dw_part_bytes(plan_dw(k, n_out, cap_m, gemm_dt == GNN_BF16), k, n_out), 256);
}

gnn_status launch_shadow_sync(const float *w, int64_t K, int64_t n, uint16_t *wt, hipStream_t s) {
    if (K * n == 0) return GNN_OK;
    const unsigned grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(K * n, 256), 1 << 16));
    shadow_sync_kernel<<<grid, 256, 0, s>>>(w, K, n, wt);
    GNN_LAUNCHED("shadow_sync");
    return GNN_OK;
}

gnn_status launch_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt, float *dw,
                             float *db, float *d_a, void *ws, float *w_upd, float *b_upd, uint16_t *wt_upd, float lr,
                             hipStream_t s) {
    if (n_out == 0) return GNN_OK;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const bool bf = gemm_dt == GNN_BF16;
    const DwPlan pw = plan_dw(K, n_out, cap_m, bf);
    float *part = static_cast<float *>(ws);
    const size_t asz = dtype_size(adt);
    const bool vec_a = (k_each % 4 == 0) && aligned(a_self, 4 * asz) && (!a_nbr || aligned(a_nbr, 4 * asz));
    const bool vec_g = (n_out % 4 == 0) && aligned(g, 16) && aligned(w, 16);
    // input gradient first: it reads W before an optional SGD changes it
    if (d_a && cap_m > 0) {
        const DinPlan pa = plan_dinput(cap_m, K);
        GNN_CHECK(pa.map.blocks() <= kMaxGrid, GNN_ESIZE, "update_bwd: cap_m exceeds the grid limit");
        const bool vec_o = (K % 4 == 0) && aligned(d_a, 16);
        const dim3 grid(static_cast<unsigned>(pa.map.blocks()));
#define DA(BFV, T, V, VO) \
    update_dinput_kernel<BFV, T, V, VO><<<grid, kThreads, 0, s>>>(g, w, m_dev, cap_m, K, n_out, d_a, pa.map)
#define DA_V(BFV, T)                                     \
    do {                                                 \
        if (vec_g && vec_o) DA(BFV, T, true, true);      \
        else if (vec_g) DA(BFV, T, true, false);         \
        else if (vec_o) DA(BFV, T, false, true);         \
        else DA(BFV, T, false, false);                   \
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
    GNN_CHECK(pw.map.blocks() <= kMaxGrid, GNN_ESIZE, "update_bwd: too many weight-gradient tiles");
    const dim3 grid(static_cast<unsigned>(pw.map.blocks()));
    const int want_db = db != nullptr;
#define DW(BFV, T, TA, VA, VG)                                                                                  \
    update_dweight_kernel<BFV, T, TA, VA, VG><<<grid, kThreads, 0, s>>>(                                       \
        static_cast<const TA *>(a_self), static_cast<const TA *>(a_nbr), k_each, g, m_dev, cap_m, n_out, want_db, \
        part, pw.map, pw.k_tiles)
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
    const bool vec_r = (n_out % 4 == 0) && aligned(dw, 16) && aligned(db, 16) && aligned(w_upd, 16) &&
                       aligned(b_upd, 16);
    const int64_t work = (K + 1) * (part_ld(n_out) / 4);
    const unsigned rgrid = static_cast<unsigned>(std::min<int64_t>(ceil_div(work, 256), 1 << 20));
    if (vec_r)
        dw_reduce_kernel<true><<<rgrid, 256, 0, s>>>(part, pw.nsplit, K, n_out, dw, db, w_upd, b_upd, wt_upd, lr);
    else
        dw_reduce_kernel<false><<<rgrid, 256, 0, s>>>(part, pw.nsplit, K, n_out, dw, db, w_upd, b_upd, wt_upd, lr);
    GNN_LAUNCHED("update_dw_reduce");
    return GNN_OK;
}

}  // namespace gnn
