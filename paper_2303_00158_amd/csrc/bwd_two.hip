// Host side of the folded two-layer backward (bwd_pull_dev.h) and the
// gnn_two_layer_bwd entry point's launches.
#include "bwd_pull_dev.h"
#include "jobs.h"

namespace gnn {

TwoBwdPlan plan_two_bwd(int kind, const gnn_block &b2, const void *x_self, const void *m1, int64_t f0,
                        const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1, const void *agg2,
                        const int32_t *arg2, const float *d_a2, const float *g2, int64_t n_out, const float *w1, float *dw1, float *db1,
                        float *part1, float *w1_upd, float *b1_upd, uint16_t *wt1_upd, const float *w2, float *dw2,
                        float *db2, float *part2, float *w2_upd, float *b2_upd, uint16_t *wt2_upd, float lr) {
    TwoBwdPlan t{};
    const bool sage = kind != GNN_AGG_GCN_SYM;  // A = [h_self || aggregation]
    t.a2 = gbwd::Args{sage ? static_cast<const void *>(h1) : agg2, sage ? agg2 : nullptr, GNN_BF16, f1, b2.counts,
                      b2.cap_dst, w2, g2, n_out, GNN_BF16, dw2, db2, nullptr, part2, w2_upd, b2_upd, wt2_upd, lr};
    t.a1 = gbwd::Args{sage ? x_self : m1, sage ? m1 : nullptr, GNN_BF16, f0, m1_rows, cap_m1, w1, nullptr, f1,
                      GNN_BF16, dw1, db1, nullptr, part1, w1_upd, b1_upd, wt1_upd, lr};
    t.p2 = gbwd::plan(t.a2);
    t.p1 = gbwd::plan(t.a1);
    t.gemm_ok = t.p2.bf && t.p1.bf && t.p2.pw.tile == 64 && t.p1.pw.tile == 64 && t.p2.vec_a && t.p1.vec_a &&
                t.p2.pw.map.blocks() <= kMaxGrid && t.p1.pw.map.blocks() <= kMaxGrid;
    // The folded job repeats the aggregation backward's arithmetic when that
    // walks each row's edges in one sequence (S == 1) and takes all of K in
    // one workgroup; its split plan is the dW GEMM's.
    int C, S;
    agg::split_row(f1, &C, &S);
    t.pm = gbwd::SplitMap{ceil_div(f1, 64), t.p1.pw.nsplit};
    t.b2 = b2;
    t.arg2 = arg2;
    t.d_a2 = d_a2;
    t.h1 = h1;
    t.grid = static_cast<unsigned>(std::max<int64_t>(t.pm.blocks(), t.p2.dw_grid));
    t.pull = (kind != GNN_AGG_SAGE_MAX || (arg2 && aligned(arg2, 16))) && t.gemm_ok && S == 1 && f1 % 4 == 0 && t.a1.K() <= gbwd::kPullMaxK && b2.cscptr != nullptr &&
             b2.cscrow != nullptr && (sage || b2.src_norm != nullptr) && cap_m1 <= b2.cap_src &&
             aligned(d_a2, 16) && aligned(h1, 8) && t.pm.blocks() <= kMaxGrid;
    return t;
}

gnn_status launch_two_bwd_partials(const TwoBwdPlan &t, int kind, hipStream_t s) {
    gnn_status st = GNN_OK;
    auto go = [&](auto kind_tag, auto dwj) {
        constexpr int KIND = decltype(kind_tag)::value;
        const gbwd::DweightPullJob<KIND, true, decltype(dwj)> j{
            static_cast<const uint16_t *>(t.a1.a_self), static_cast<const uint16_t *>(t.a1.a_nbr), t.a1.k_each,
            t.a1.m_dev, t.a1.cap_m, t.b2, t.d_a2, t.h1, t.a1.n_out, t.a1.db != nullptr, t.a1.part, t.pm, dwj,
            static_cast<int64_t>(t.p2.dw_grid), t.arg2};
        st = launch_job(j, t.grid, s, "update_dweight_l2+update_dweight_pull_l1");
    };
    auto by_kind = [&](auto dwj) {
        if (kind == GNN_AGG_SAGE_MAX) go(std::integral_constant<int, GNN_AGG_SAGE_MAX>{}, dwj);
        else if (kind == GNN_AGG_SAGE_MEAN) go(std::integral_constant<int, GNN_AGG_SAGE_MEAN>{}, dwj);
        else go(std::integral_constant<int, GNN_AGG_GCN_SYM>{}, dwj);
    };
    if (t.p2.vec_g) by_kind(gbwd::dweight_job<true, 64, uint16_t, true, true>(t.a2, t.p2));
    else by_kind(gbwd::dweight_job<true, 64, uint16_t, true, false>(t.a2, t.p2));
    return st;
}

size_t two_bwd_ws_bytes(int kind, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_m1, int64_t cap_m2) {
    const bool sage = kind != GNN_AGG_GCN_SYM;
    const int64_t k1 = sage ? 2 * f0 : f0, k2 = sage ? 2 * f1 : f1;
    const gbwd::DwPlan p1 = gbwd::plan_dw(k1, f1, cap_m1, true), p2 = gbwd::plan_dw(k2, n_out, cap_m2, true);
    return round_up(gbwd::dw_part_bytes(p1, k1, f1), 256) + gbwd::dw_part_bytes(p2, k2, n_out);
}

gnn_status launch_two_bwd(const gnn_block *b2, int kind, const void *x_self, const void *m1, int64_t f0,
                          const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1, const void *agg2,
                          const int32_t *arg2, const float *d_a2, const float *g2, int64_t n_out, float *dw1,
                          float *db1, float *dw2, float *db2, void *ws, hipStream_t s) {
    const bool sage = kind != GNN_AGG_GCN_SYM;
    const int64_t k1 = sage ? 2 * f0 : f0;
    const gbwd::DwPlan q1 = gbwd::plan_dw(k1, f1, cap_m1, true);
    float *part1 = static_cast<float *>(ws);
    float *part2 = reinterpret_cast<float *>(static_cast<char *>(ws) + round_up(gbwd::dw_part_bytes(q1, k1, f1), 256));
    const TwoBwdPlan t = plan_two_bwd(kind, *b2, x_self, m1, f0, m1_rows, cap_m1, h1, f1, agg2, arg2, d_a2, g2, n_out,
                                      nullptr, dw1, db1, part1, nullptr, nullptr, nullptr, nullptr, dw2, db2, part2,
                                      nullptr, nullptr, nullptr, 0.f);
    if (!t.pull)
        return fail(GNN_EUNSUPPORTED, "gnn_two_layer_bwd: these shapes or alignments do not take the folded backward");
    GNN_TRY(launch_two_bwd_partials(t, kind, s));
    gnn_status st = GNN_OK;
    gbwd::with_reduce_job(t.a1, t.p1, [&](auto r1) {
        gbwd::with_reduce_job(t.a2, t.p2, [&](auto r2) {
            st = launch_jobs(s, "dw_reduce_l1+dw_reduce_l2", role(r1, t.p1.red_grid), role(r2, t.p2.red_grid));
        });
    });
    return st;
}

}  // namespace gnn
