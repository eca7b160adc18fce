// Forward update (equation 2): Z = [A_self || A_nbr] W + b with the ReLU
// and narrowing epilogue, on the matrix-core engine of gemm_engine.h.
//
// The whole reduction of a tile normally runs in one workgroup.  Only when
// the output has few tiles and K is long is the reduction split; the
// partial tiles then go to the workspace and fwd_reduce_kernel finishes
// them (sum in split order, bias, ReLU, narrowing).
#include "gemm_engine.h"

namespace gnn {

namespace {

using namespace gemm;

// Where the W operand comes from.
enum WSrc {
    kWCols = 0,     // fp32 W (K x n_out), element loads (n_out not a multiple of 4)
    kWColsVec = 1,  // fp32 W, 16-byte loads
    kWtBf16 = 2,    // bf16 shadow W^T (n_out x K), 8-byte loads, no transpose
};

template <bool BF16, int TILE, int WS, int D> struct WOperand;
template <bool BF16, int TILE, int D> struct WOperand<BF16, TILE, kWCols, D> {
    using type = SrcCols<BF16, TILE, float, false, D>;
    __device__ static type make(const float *w, const uint16_t *, int64_t K, int64_t n_out, int64_t r_end,
                                int64_t col0) {
        return type{w, nullptr, n_out, n_out, n_out, r_end, col0, {}};
    }
};
template <bool BF16, int TILE, int D> struct WOperand<BF16, TILE, kWColsVec, D> {
    using type = SrcCols<BF16, TILE, float, true, D>;
    __device__ static type make(const float *w, const uint16_t *, int64_t K, int64_t n_out, int64_t r_end,
                                int64_t col0) {
        return type{w, nullptr, n_out, n_out, n_out, r_end, col0, {}};
    }
};
template <int TILE, int D> struct WOperand<true, TILE, kWtBf16, D> {
    using type = SrcRows<true, TILE, uint16_t, true, D>;
    __device__ static type make(const float *, const uint16_t *wt, int64_t K, int64_t n_out, int64_t,
                                int64_t col0) {
        return type{wt, nullptr, K, K, n_out, K, col0, {}};
    }
};

template <bool BF16, int TILE, class TA, class TO, bool VA, int WS, bool VO>
__global__ void __launch_bounds__(kThreads) update_fwd_kernel(const TA *__restrict__ a_self,
                                                               const TA *__restrict__ a_nbr, int64_t k_each,
                                                               const int64_t *m_dev, int64_t cap_m,
                                                               const float *__restrict__ w,
                                                               const uint16_t *__restrict__ wt,
                                                               const float *__restrict__ bias, int64_t n_out,
                                                               int relu, TO *__restrict__ out,
                                                               float *__restrict__ part, TileMap map) {
    constexpr int D = depth<TILE>();
    __shared__ __attribute__((aligned(16))) char lds[lds_bytes<TILE, TILE>()];
    int64_t tx, ty;
    map.tile_of(blockIdx.x, &tx, &ty);
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t row0 = tx * TILE, col0 = ty * TILE;
    if (tx >= map.mt || row0 >= M) return;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    int64_t r_beg, r_end;
    split_range<Cfg<BF16>::BK>(K, gridDim.z, blockIdx.z, &r_beg, &r_end);
    SrcRows<BF16, TILE, TA, VA, D> sp{a_self, a_nbr, k_each, k_each, M, K, row0, {}};
    auto sq = WOperand<BF16, TILE, WS, D>::make(w, wt, K, n_out, r_end, col0);
    Acc<TILE, TILE> acc;
    run_tile<BF16, D>(acc, sp, sq, r_beg, r_end, lds, [](const auto &, int, int64_t, bool) {});
    const int64_t gc = col0 + TileOut<TILE, TILE>::col();
    if (gridDim.z > 1) {
        const int64_t ldp = part_ld(n_out);
        float *pp = part + static_cast<int64_t>(blockIdx.z) * cap_m * ldp;
        emit_tile(acc, lds, [&](int, int r, int, float4 v) {
            const int64_t gr = row0 + r;
            if (gr < M && gc < ldp) *reinterpret_cast<float4 *>(pp + gr * ldp + gc) = v;
        });
        return;
    }
    const float4 b4 = bias ? load4_clamped<VO>(bias, 0, gc, n_out) : make_float4(0.f, 0.f, 0.f, 0.f);
    emit_tile(acc, lds, [&](int, int r, int, float4 v) {
        const int64_t gr = row0 + r;
        if (gr < M) store4_masked<VO>(out, gr * n_out, gc, n_out, bias_act(v, b4, relu));
    });
}

// out[r] = act(sum over splits of part[s][r] + b) for the rows below M.
template <class TO, bool VO>
__global__ void __launch_bounds__(256) fwd_reduce_kernel(const float *__restrict__ part, int nsplit,
                                                         const int64_t *m_dev, int64_t cap_m, int64_t n_out,
                                                         const float *__restrict__ bias, int relu,
                                                         TO *__restrict__ out) {
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t ldp = part_ld(n_out), chunks = ldp / 4;
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; t < M * chunks;
         t += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t r = t / chunks, c = (t % chunks) * 4;
        const float4 b4 = bias ? load4_clamped<VO>(bias, 0, c, n_out) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 s = sum_splits(part + r * ldp + c, cap_m * ldp, nsplit);
        store4_masked<VO>(out, r * n_out, c, n_out, bias_act(s, b4, relu));
    }
}

struct FwdPlan {
    int tile, nsplit;
    TileMap map;
};

FwdPlan plan_fwd(int64_t cap_m, int64_t n_out, int64_t K, bool bf16) {
    FwdPlan p;
    p.tile = pick_tile(cap_m, n_out);
    p.map = TileMap{ceil_div(std::max<int64_t>(cap_m, 1), p.tile), ceil_div(n_out, p.tile)};
    const int64_t tiles = p.map.mt * p.map.nt;
    const int64_t nch = ceil_div(K, bk_of(bf16));
    // split only long reductions over few tiles, at least 8 chunks a split
    int64_t s = 1;
    if (tiles < 128 && nch >= 16) s = std::min<int64_t>({nch / 8, ceil_div(256, tiles), 16});
    p.nsplit = static_cast<int>(s);
    return p;
}

size_t part_bytes(const FwdPlan &p, int64_t cap_m, int64_t n_out) {
    return p.nsplit > 1 ? static_cast<size_t>(p.nsplit) * cap_m * part_ld(n_out) * 4 : 0;
}

// Launch-time dispatch over the kernel's template parameters.
struct FwdLaunch {
    const void *a_self, *a_nbr;
    int64_t k_each;
    const int64_t *m_dev;
    int64_t cap_m;
    const float *w;
    const uint16_t *wt;
    const float *bias;
    int64_t n_out;
    int relu;
    void *out;
    float *part;
    TileMap map;
    dim3 grid;
    hipStream_t s;
};

template <bool BF16, int T, class TA, class TO, bool VA, int WS>
void fwd_launch(const FwdLaunch &L, bool vec_o) {
    const TA *as = static_cast<const TA *>(L.a_self), *an = static_cast<const TA *>(L.a_nbr);
    TO *o = static_cast<TO *>(L.out);
    if (vec_o)
        update_fwd_kernel<BF16, T, TA, TO, VA, WS, true><<<L.grid, kThreads, 0, L.s>>>(
            as, an, L.k_each, L.m_dev, L.cap_m, L.w, L.wt, L.bias, L.n_out, L.relu, o, L.part, L.map);
    else
        update_fwd_kernel<BF16, T, TA, TO, VA, WS, false><<<L.grid, kThreads, 0, L.s>>>(
            as, an, L.k_each, L.m_dev, L.cap_m, L.w, L.wt, L.bias, L.n_out, L.relu, o, L.part, L.map);
}

template <bool BF16, int T, class TA, class TO, bool VA>
void fwd_by_wsrc(const FwdLaunch &L, int wsrc, bool vec_o) {
    if constexpr (BF16) {
        if (wsrc == kWtBf16) return fwd_launch<BF16, T, TA, TO, VA, kWtBf16>(L, vec_o);
    }
    if (wsrc == kWColsVec) fwd_launch<BF16, T, TA, TO, VA, kWColsVec>(L, vec_o);
    else fwd_launch<BF16, T, TA, TO, VA, kWCols>(L, vec_o);
}

template <bool BF16, class TA, class TO>
void fwd_by_tile(const FwdLaunch &L, int tile, bool vec_a, int wsrc, bool vec_o) {
    if (tile == 128) {
        if (vec_a) fwd_by_wsrc<BF16, 128, TA, TO, true>(L, wsrc, vec_o);
        else fwd_by_wsrc<BF16, 128, TA, TO, false>(L, wsrc, vec_o);
    } else {
        if (vec_a) fwd_by_wsrc<BF16, 64, TA, TO, true>(L, wsrc, vec_o);
        else fwd_by_wsrc<BF16, 64, TA, TO, false>(L, wsrc, vec_o);
    }
}

}  // namespace

size_t update_fwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt) {
    const FwdPlan p = plan_fwd(cap_m, n_out, k, gemm_dt == GNN_BF16);
    size_t bytes = round_up(part_bytes(p, cap_m, n_out), 256);
    // layers the wide kernel may take (its split's partial tiles)
    if (gemm_dt == GNN_BF16 && k >= 512 && n_out >= 512 && n_out % 8 == 0 && k % 128 == 0)
        bytes = std::max(bytes, wide_fwd_ws_bytes(n_out, cap_m));
    return bytes;
}

gnn_status launch_update_fwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const uint16_t *wt, const float *bias, int64_t n_out,
                             int relu, int gemm_dt, void *out, int odt, void *ws, hipStream_t s) {
    if (cap_m == 0 || n_out == 0) return GNN_OK;
    // A hidden bf16 layer whose bf16 W^T is given and fits the register
    // tiles: the fused layer kernel in A-load mode (W^T fragments in
    // registers, A rows staged through LDS, no reduction split).  GCN's
    // single A operand is its "aggregation part".
    if (gemm_dt == GNN_BF16 && wt && adt == GNN_BF16 && odt == GNN_BF16 && relu) {
        const int kind = a_nbr ? GNN_AGG_SAGE_MEAN : GNN_AGG_GCN_SYM;
        const void *agg = a_nbr ? a_nbr : a_self;
        if (fused_layer_ok(kind, GNN_BF16, k_each, n_out, cap_m, 1, false, a_self, wt, agg)) {
            gnn_block b{};
            b.cap_dst = cap_m;
            b.counts = const_cast<int64_t *>(m_dev);
            return launch_fused_update(&b, kind, a_nbr ? a_self : nullptr, agg, k_each, wt, bias, n_out, out, false,
                                       nullptr, nullptr, nullptr, 0, s);
        }
    }
    // Wide layers (K and n_out of 512 and more) are bound by the matrix
    // cores: 256 x 256 tiles with operands copied straight to LDS.
    if (wide_fwd_ok(a_self, a_nbr, adt, k_each, cap_m, n_out, wt, gemm_dt, out))
        return launch_wide_fwd(a_self, a_nbr, k_each, m_dev, cap_m, wt, bias, n_out, relu, out, odt, ws, s);
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const bool bf = gemm_dt == GNN_BF16;
    FwdPlan p = plan_fwd(cap_m, n_out, K, bf);
    if (ws == nullptr) p.nsplit = 1;
    GNN_CHECK(p.map.blocks() <= kMaxGrid, GNN_ESIZE, "update_fwd: cap_m exceeds the grid limit");
    float *part = static_cast<float *>(ws);
    const dim3 grid(static_cast<unsigned>(p.map.blocks()), 1, static_cast<unsigned>(p.nsplit));
    const size_t asz = dtype_size(adt), osz = dtype_size(odt);
    const bool vec_a = (k_each % 4 == 0) && aligned(a_self, 4 * asz) && (!a_nbr || aligned(a_nbr, 4 * asz));
    const bool use_wt = bf && wt != nullptr && K % 4 == 0 && aligned(wt, 8);
    const int wsrc = use_wt ? kWtBf16 : ((n_out % 4 == 0) && aligned(w, 16) ? kWColsVec : kWCols);
    const bool vec_o = (n_out % 4 == 0) && aligned(out, 4 * osz) && aligned(bias, 16);
    const FwdLaunch L{static_cast<const void *>(a_self), a_nbr, k_each, m_dev, cap_m, w, wt, bias, n_out, relu, out,
                      part, p.map, grid, s};
    if (bf) {
        if (adt == GNN_BF16 && odt == GNN_BF16) fwd_by_tile<true, uint16_t, uint16_t>(L, p.tile, vec_a, wsrc, vec_o);
        else if (adt == GNN_BF16 && odt == GNN_F32) fwd_by_tile<true, uint16_t, float>(L, p.tile, vec_a, wsrc, vec_o);
        else if (adt == GNN_F32 && odt == GNN_BF16) fwd_by_tile<true, float, uint16_t>(L, p.tile, vec_a, wsrc, vec_o);
        else fwd_by_tile<true, float, float>(L, p.tile, vec_a, wsrc, vec_o);
    } else {
        if (adt == GNN_BF16 && odt == GNN_BF16) fwd_by_tile<false, uint16_t, uint16_t>(L, p.tile, vec_a, wsrc, vec_o);
        else if (adt == GNN_BF16 && odt == GNN_F32) fwd_by_tile<false, uint16_t, float>(L, p.tile, vec_a, wsrc, vec_o);
        else if (adt == GNN_F32 && odt == GNN_BF16) fwd_by_tile<false, float, uint16_t>(L, p.tile, vec_a, wsrc, vec_o);
        else fwd_by_tile<false, float, float>(L, p.tile, vec_a, wsrc, vec_o);
    }
    GNN_LAUNCHED("update_fwd");
    if (p.nsplit > 1) {
        const int64_t work = cap_m * (part_ld(n_out) / 4);
        const unsigned rgrid = static_cast<unsigned>(std::min<int64_t>(ceil_div(work, 256), 1 << 20));
        if (odt == GNN_BF16) {
            if (vec_o)
                fwd_reduce_kernel<uint16_t, true><<<rgrid, 256, 0, s>>>(part, p.nsplit, m_dev, cap_m, n_out, bias,
                                                                         relu, static_cast<uint16_t *>(out));
            else
                fwd_reduce_kernel<uint16_t, false><<<rgrid, 256, 0, s>>>(part, p.nsplit, m_dev, cap_m, n_out, bias,
                                                                          relu, static_cast<uint16_t *>(out));
        } else {
            if (vec_o)
                fwd_reduce_kernel<float, true><<<rgrid, 256, 0, s>>>(part, p.nsplit, m_dev, cap_m, n_out, bias, relu,
                                                                      static_cast<float *>(out));
            else
                fwd_reduce_kernel<float, false><<<rgrid, 256, 0, s>>>(part, p.nsplit, m_dev, cap_m, n_out, bias,
                                                                       relu, static_cast<float *>(out));
        }
        GNN_LAUNCHED("update_fwd_reduce");
    }
    return GNN_OK;
}

}  // namespace gnn
