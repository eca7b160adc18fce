// Device side of the update gradients (see gemm_bwd.hip) as jobs:
//   input     dA = G W^T                  (layers above the first)
//   weights   dW = A^T G, db = colsum(G)  (optionally followed by SGD)
//
// dA reduces over n_out only and runs unsplit.  dW reduces over the
// mini-batch rows, so the rows are split across workgroups: each split
// writes its dW tile (and, from the first row tile, its db columns) as a
// row-major fp32 partial, and the reduction job sums the partials in split
// order and applies SGD to W and b (and refreshes the bf16 shadow of W).
#pragma once

#include <type_traits>

#include "gemm_engine.h"

namespace gnn {
namespace gbwd {

using namespace gemm;

// One layer's update backward.
struct Args {
    const void *a_self, *a_nbr;  // A = [a_self || a_nbr], adt
    int adt;
    int64_t k_each;
    const int64_t *m_dev;
    int64_t cap_m;
    const float *w, *g;
    int64_t n_out;
    int gemm_dt;
    float *dw, *db, *d_a;
    float *part;                 // workspace: dW partials
    float *w_upd, *b_upd;        // SGD targets, or null
    uint16_t *wt_upd;            // bf16 shadow of w_upd, or null
    float lr;
    int64_t K() const { return a_nbr ? 2 * k_each : k_each; }
};

// ---------------------------------------------------------------------------
// input gradient: d_a = g W^T   (M x K; reduction over n_out)
// ---------------------------------------------------------------------------
template <bool BF16, int TILE, bool V, bool VO>
struct DinputJob {
    const float *g, *w;
    const int64_t *m_dev;
    int64_t cap_m, K, n_out;
    float *d_a;
    TileMap map;
    __device__ void run(int64_t blk, int64_t) const {
        constexpr int D = depth<TILE>();
        __shared__ __attribute__((aligned(16))) char lds[lds_bytes<TILE, TILE>()];
        int64_t tx, ty;
        map.tile_of(blk, &tx, &ty);
        const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
        const int64_t row0 = tx * TILE, col0 = ty * TILE;
        if (tx >= map.mt || row0 >= M) return;
        SrcRows<BF16, TILE, float, V, D> sp{g, nullptr, n_out, n_out, M, n_out, row0, {}};
        SrcRows<BF16, TILE, float, V, D> sq{w, nullptr, n_out, n_out, K, n_out, col0, {}};
        Acc<TILE, TILE> acc;
        run_tile<BF16, D>(acc, sp, sq, 0, n_out, lds, [](const auto &, int, int64_t, bool) {});
        const int64_t gc = col0 + TileOut<TILE, TILE>::col();
        float *out = d_a;
        const int64_t ld = K;
        emit_tile(acc, lds, [&](int, int r, int, float4 v) {
            const int64_t gr = row0 + r;
            if (gr < M) store4_masked<VO>(out, gr * ld, gc, ld, v);
        });
    }
};

// ---------------------------------------------------------------------------
// weight gradient partials: part[split][k][n] = sum over this split's rows
// of A[row][k] g[row][n]; part[split][K][n] = sum of g[row][n] (db).
// ---------------------------------------------------------------------------
template <bool BF16, int TILE, class TA, bool VA, bool VG>
struct DweightJob {
    const TA *a_self, *a_nbr;
    int64_t k_each;
    const float *g;
    const int64_t *m_dev;
    int64_t cap_m, n_out;
    int want_db;
    float *part;
    SplitMap map;
    int64_t k_tiles;
    static constexpr int D = depth<TILE>();
    using SP = SrcCols<BF16, TILE, TA, VA, D>;
    using SQ = SrcCols<BF16, TILE, float, VG, D>;
    static constexpr int kLdsBytes = lds_bytes<TILE, TILE>();
    using ColSums = float[SQ::RPP][TILE];
    // One workgroup's tile between its first loads (begin) and its partial
    // stores (finish), so that another job can run in between.
    struct Tile {
        SP sp;
        SQ sq;
        int split;
        int64_t K, row0, col0, r_beg, r_end;
        bool do_db;
    };
    __device__ bool begin(int64_t blk, Tile &t) const {
        int64_t tile;
        map.of(blk, &t.split, &tile);
        if (t.split >= map.nsplit) return false;
        const int64_t tk = tile % k_tiles, tn = tile / k_tiles;
        const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
        t.K = a_nbr ? 2 * k_each : k_each;
        t.row0 = tk * TILE;  // over K
        t.col0 = tn * TILE;  // over n_out
        split_range<Cfg<BF16>::BK>(M, map.nsplit, t.split, &t.r_beg, &t.r_end);
        t.sp = SP{a_self, a_nbr, k_each, k_each, t.K, t.r_end, t.row0, {}};
        t.sq = SQ{g, nullptr, n_out, n_out, n_out, t.r_end, t.col0, {}};
        t.do_db = want_db && tk == 0;
        if (t.r_beg < t.r_end) tile_prefetch<BF16, D>(t.sp, t.sq, t.r_beg);
        return true;
    }
    __device__ void run(int64_t blk, int64_t) const {
        __shared__ __attribute__((aligned(16))) char lds[kLdsBytes];
        __shared__ ColSums cs;
        Tile t;
        if (begin(blk, t)) finish(t, lds, cs);
    }
    __device__ void finish(Tile &t, char *lds, ColSums &cs) const {
        const int64_t K = t.K, col0 = t.col0, row0 = t.row0;
        const bool do_db = t.do_db;
        float4 colsum = make_float4(0.f, 0.f, 0.f, 0.f);
        Acc<TILE, TILE> acc;
        zero_acc(acc);
        if (t.r_beg < t.r_end)
            tile_rest<BF16, D>(acc, t.sp, t.sq, t.r_beg, t.r_end, lds, [&](const SQ &src, int s, int64_t r0, bool tail) {
                if (do_db) src.add_colsum(s, colsum, r0, tail);
            });
        const int64_t ldp = part_ld(n_out);
        float *pp = part + static_cast<int64_t>(t.split) * (K + 1) * ldp;
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
};

// Lanes that share one output float4 of the split reduction: one per 16
// splits (up to 64 splits; a lane's 16 loads are one round trip).
__host__ __device__ inline int reduce_lanes(int nsplit) { return nsplit > 32 ? 4 : nsplit > 16 ? 2 : 1; }

// dw = sum over splits of the partials (db from row K); then, when w_upd /
// b_upd are given, w_upd -= lr * dw and b_upd -= lr * db, and wt_upd (if
// given) = bf16(w_upd^T).  The splits are summed in blocks of 16, each in
// split order by its own lane, and the blocks' sums are added in block
// order by the first lane (a fixed order, so results are reproducible).
// The values an update reads are loaded before the partials, so each
// thread waits once.
template <bool VO>
struct DwReduceJob {
    const float *part;
    int nsplit;
    int64_t K, n_out;
    float *dw, *db, *w_upd, *b_upd;
    uint16_t *wt_upd;
    float lr;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t ldp = part_ld(n_out), chunks = ldp / 4;
        const int64_t rows = K + (db ? 1 : 0);
        const int G = reduce_lanes(nsplit);  // divides 64: a group's lanes share a wavefront
        const int64_t stride = (K + 1) * ldp;
        for (int64_t t = blk * 256 + threadIdx.x; t < rows * chunks * G; t += nblk * 256) {
            const int64_t item = t / G;
            const int j = static_cast<int>(t % G);
            const int64_t r = item / chunks, c = (item % chunks) * 4;
            const bool brow = r == K;
            const int64_t base = brow ? 0 : r * n_out;
            float *upd = brow ? b_upd : w_upd;
            const float4 old =
                (upd && j == 0) ? load4_clamped<VO>(upd, base, c, n_out) : make_float4(0.f, 0.f, 0.f, 0.f);
            const int s0 = 16 * j;
            float4 s = nsplit > s0 ? sum_splits(part + r * ldp + c + s0 * stride, stride, min(16, nsplit - s0))
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
            if (G > 1) {
                const int lane0 = (threadIdx.x & 63) - j;
                float4 tot = make_float4(__shfl(s.x, lane0, 64), __shfl(s.y, lane0, 64), __shfl(s.z, lane0, 64),
                                         __shfl(s.w, lane0, 64));
                for (int k = 1; k < G; ++k) {
                    tot.x += __shfl(s.x, lane0 + k, 64);
                    tot.y += __shfl(s.y, lane0 + k, 64);
                    tot.z += __shfl(s.z, lane0 + k, 64);
                    tot.w += __shfl(s.w, lane0 + k, 64);
                }
                s = tot;
            }
            if (j != 0) continue;
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
};

// ---------------------------------------------------------------------------
// plans
// ---------------------------------------------------------------------------
struct DwPlan {
    int tile, nsplit;
    int64_t k_tiles;
    SplitMap map;
};

inline DwPlan plan_dw(int64_t K, int64_t n_out, int64_t cap_m, bool bf16) {
    DwPlan p;
    // Wide layers (K and n_out both >= 512) take 128 x 128 tiles, which read
    // half the operand bytes per flop of 64 x 64 ones, and split the rows
    // over up to 2,048 workgroups: with 512, a 1536 x 1024 dW has 2 splits
    // and each workgroup walks half of all rows alone (3-6x slower at
    // 26k-131k rows).  Narrow layers split over up to 1,024 workgroups: a
    // first layer of 200 x 256 then has 64 splits of at most 2 row chunks
    // each, the shape the two-layer step's folded layer-1 job (which takes
    // the same splits) is built for.
    const bool wide = K >= 512 && n_out >= 512;
    p.tile = wide ? 128 : pick_tile(K, n_out);
    p.k_tiles = ceil_div(K, p.tile);
    const int64_t tiles = p.k_tiles * ceil_div(n_out, p.tile);
    const int64_t nch = std::max<int64_t>(ceil_div(cap_m, bk_of(bf16)), 1);
    const int64_t target = wide ? 2048 : 1024;
    p.nsplit = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>({ceil_div(target, tiles), 64, nch})));
    p.map = SplitMap{tiles, p.nsplit};
    return p;
}

struct DinPlan {
    int tile;
    TileMap map;
};

inline DinPlan plan_dinput(int64_t cap_m, int64_t K) {
    DinPlan p;
    p.tile = pick_tile(cap_m, K);
    p.map = TileMap{ceil_div(std::max<int64_t>(cap_m, 1), p.tile), ceil_div(K, p.tile)};
    return p;
}

inline size_t dw_part_bytes(const DwPlan &p, int64_t K, int64_t n_out) {
    return static_cast<size_t>(p.nsplit) * (K + 1) * part_ld(n_out) * 4;
}

// Wide layers on the matrix-core tiles of gemm_wide_bwd.hip: 256 x 256
// tiles, dW split over the rows into as many splits as fill the CUs in one
// wave; the workspace holds the partials, then the bf16 copies of W and G
// that dA reads.
struct WideBwdPlan {
    int64_t k_tiles, tiles;
    int64_t nsplit;     // dW alone
    int64_t nsplit_da;  // dW sharing its launch with dA
    int64_t part_bytes, ws_bytes;
};
WideBwdPlan plan_wide_bwd(int64_t K, int64_t n_out, int64_t cap_m);
// Shapes the wide path may take (the workspace is sized for them) ...
bool wide_bwd_shape(int64_t K, int64_t n_out, int gemm_dt);
// ... and calls it takes: bf16 activations, a K tile in one half of
// [a_self || a_nbr], 32-bit buffer offsets, aligned operands.
bool wide_bwd_ok(const Args &a);
// dA (when a.d_a is given) and the dW partials; the caller runs the
// reduction job with the plan's split count.
gnn_status launch_wide_bwd_gemms(const Args &a, hipStream_t s);

// Everything the launch-time dispatch needs.
struct Plan {
    bool bf, vec_a, vec_g, vec_o, vec_r, wide;
    DinPlan pa;
    DwPlan pw;
    unsigned din_grid, dw_grid, red_grid;
};

inline Plan plan(const Args &a) {
    Plan p;
    const int64_t K = a.K();
    p.bf = a.gemm_dt == GNN_BF16;
    const size_t asz = dtype_size(a.adt);
    p.vec_a = (a.k_each % 4 == 0) && aligned(a.a_self, 4 * asz) && (!a.a_nbr || aligned(a.a_nbr, 4 * asz));
    p.vec_g = (a.n_out % 4 == 0) && aligned(a.g, 16) && aligned(a.w, 16);
    p.vec_o = (K % 4 == 0) && aligned(a.d_a, 16);
    p.vec_r = (a.n_out % 4 == 0) && aligned(a.dw, 16) && aligned(a.db, 16) && aligned(a.w_upd, 16) &&
              aligned(a.b_upd, 16);
    p.pa = plan_dinput(a.cap_m, K);
    p.pw = plan_dw(K, a.n_out, a.cap_m, p.bf);
    p.wide = wide_bwd_ok(a);
    if (p.wide) {
        const WideBwdPlan w = plan_wide_bwd(K, a.n_out, a.cap_m);
        p.pw.nsplit = static_cast<int>(a.d_a ? w.nsplit_da : w.nsplit);
    }
    p.din_grid = (a.d_a && a.cap_m > 0) ? static_cast<unsigned>(p.pa.map.blocks()) : 0;
    p.dw_grid = static_cast<unsigned>(p.pw.map.blocks());
    const int64_t work = (K + 1) * (part_ld(a.n_out) / 4) * reduce_lanes(p.pw.nsplit);
    p.red_grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(work, 256), 1 << 20));
    return p;
}

// ---------------------------------------------------------------------------
// launch-time dispatch: f(job) with the job of the matching variant
// ---------------------------------------------------------------------------
template <class T> struct TypeTag {
    using type = T;
};
template <bool BF16, int T, bool V, bool VO>
DinputJob<BF16, T, V, VO> dinput_job(const Args &a, const Plan &p) {
    return {a.g, a.w, a.m_dev, a.cap_m, a.K(), a.n_out, a.d_a, p.pa.map};
}

template <class F> void with_dinput_job(const Args &a, const Plan &p, F &&f) {
    auto by_vec = [&](auto bf_tag, auto tile_tag) {
        constexpr bool BF = decltype(bf_tag)::value;
        constexpr int T = decltype(tile_tag)::value;
        if (p.vec_g && p.vec_o) f(dinput_job<BF, T, true, true>(a, p));
        else if (p.vec_g) f(dinput_job<BF, T, true, false>(a, p));
        else if (p.vec_o) f(dinput_job<BF, T, false, true>(a, p));
        else f(dinput_job<BF, T, false, false>(a, p));
    };
    using B1 = std::true_type;
    using B0 = std::false_type;
    using T128 = std::integral_constant<int, 128>;
    using T64 = std::integral_constant<int, 64>;
    if (p.bf) {
        if (p.pa.tile == 128) by_vec(B1{}, T128{}); else by_vec(B1{}, T64{});
    } else {
        if (p.pa.tile == 128) by_vec(B0{}, T128{}); else by_vec(B0{}, T64{});
    }
}

template <bool BF16, int T, class TA, bool VA, bool VG>
DweightJob<BF16, T, TA, VA, VG> dweight_job(const Args &a, const Plan &p) {
    return {static_cast<const TA *>(a.a_self), static_cast<const TA *>(a.a_nbr), a.k_each, a.g, a.m_dev, a.cap_m,
            a.n_out, a.db != nullptr, a.part, p.pw.map, p.pw.k_tiles};
}

template <class F> void with_dweight_job(const Args &a, const Plan &p, F &&f) {
    auto by_vec = [&](auto bf_tag, auto tile_tag, auto ta_tag) {
        constexpr bool BF = decltype(bf_tag)::value;
        constexpr int T = decltype(tile_tag)::value;
        using TA = typename decltype(ta_tag)::type;
        if (p.vec_a && p.vec_g) f(dweight_job<BF, T, TA, true, true>(a, p));
        else if (p.vec_a) f(dweight_job<BF, T, TA, true, false>(a, p));
        else if (p.vec_g) f(dweight_job<BF, T, TA, false, true>(a, p));
        else f(dweight_job<BF, T, TA, false, false>(a, p));
    };
    auto by_type = [&](auto bf_tag, auto tile_tag) {
        if (a.adt == GNN_BF16) by_vec(bf_tag, tile_tag, TypeTag<uint16_t>{});
        else by_vec(bf_tag, tile_tag, TypeTag<float>{});
    };
    using B1 = std::true_type;
    using B0 = std::false_type;
    using T128 = std::integral_constant<int, 128>;
    using T64 = std::integral_constant<int, 64>;
    if (p.bf) {
        if (p.pw.tile == 128) by_type(B1{}, T128{}); else by_type(B1{}, T64{});
    } else {
        if (p.pw.tile == 128) by_type(B0{}, T128{}); else by_type(B0{}, T64{});
    }
}

template <class F> void with_reduce_job(const Args &a, const Plan &p, F &&f) {
    const int64_t K = a.K();
    if (p.vec_r)
        f(DwReduceJob<true>{a.part, p.pw.nsplit, K, a.n_out, a.dw, a.db, a.w_upd, a.b_upd, a.wt_upd, a.lr});
    else
        f(DwReduceJob<false>{a.part, p.pw.nsplit, K, a.n_out, a.dw, a.db, a.w_upd, a.b_upd, a.wt_upd, a.lr});
}

}  // namespace gbwd

// Host side (gemm_bwd.hip).
// The two GEMMs of a layer's update backward (dA when a.d_a is given, and
// the dW partials), in one launch when their variants allow it.
gnn_status launch_update_bwd_gemms(const gbwd::Args &a, const gbwd::Plan &p, hipStream_t s);

}  // namespace gnn
