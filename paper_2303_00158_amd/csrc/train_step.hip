// One training iteration composed from the kernels: sample L blocks, gather
// X', L forward layers, loss, backward in reverse order (no input gradient
// below the first layer), SGD.  The host never waits: counts produced on the
// device are read by later kernels.
//
// The step has two stages with separate workspaces: prepare (sampling and the
// gather of X') and compute (the rest).  A caller can run the prepare stage
// of the next step on a second stream while the compute stage of this one
// runs, which hides the feature loading from a host-resident table (two-stage
// feature prefetching, Section IV-B).
//
// Everything runs on the caller's stream.  The block transposes (CSC), which
// only the backward pass reads, cost no launch of their own: their phases
// (csc_dev.h) ride along with the sampling launches of later hops, and the
// last sort with layer 1's aggregation, which the prepare stage computes
// because it needs no weights.
#include <algorithm>
#include <type_traits>

#include "aggregate_dev.h"
#include "bwd_pull_dev.h"
#include "csc_dev.h"
#include "gather_dev.h"
#include "gemm_bwd_dev.h"
#include "internal.h"
#include "jobs.h"
#include "loss_dev.h"
#include "sampler_dev.h"

namespace gnn {

namespace {

int64_t k_of(const gnn_model *m, int l) {  // reduction width of layer l (1-based)
    const int64_t f = m->dims[l - 1];
    return m->kind == GNN_AGG_GCN_SYM ? f : 2 * f;
}

}  // namespace

gnn_status step_layout(const gnn_model *m, int64_t graph_n, int64_t batch, gnn_step_layout *o) {
    const int L = m->num_layers;
    *o = gnn_step_layout{};
    const int act = m->precision;
    const size_t asz = dtype_size(act);
    // prepare part: sampler state, blocks, transposes, X'
    Carver c(nullptr);
    int64_t cap_dst = batch;
    size_t hop_max = 0;
    for (int h = 0; h < L; ++h) {
        const int64_t k = m->fanouts[h];
        o->cap_dst[h] = cap_dst;
        o->cap_nnz[h] = cap_dst * k;
        o->cap_src[h] = std::min<int64_t>(cap_dst + cap_dst * k, std::max<int64_t>(graph_n, cap_dst));
        hop_max = std::max(hop_max, sampler_hop_bytes(graph_n, cap_dst, static_cast<int32_t>(k)));
        cap_dst = o->cap_src[h];
    }
    // the shared part and two hop scratch regions: consecutive hops overlap
    // (relabel of one hop runs with the prepare of the next)
    const size_t samp = sampler_shared_bytes(graph_n) + 2 * hop_max;
    o->sampler_ws = c.take(samp);
    o->sampler_ws_bytes = samp;
    for (int h = 0; h < L; ++h) {
        o->blk_counts[h] = c.take(4 * 8);
        o->blk_src_ids[h] = c.take(static_cast<size_t>(o->cap_src[h]) * 8);
        o->blk_rowptr[h] = c.take(static_cast<size_t>(o->cap_dst[h] + 1) * 8);
        o->blk_col[h] = c.take(static_cast<size_t>(std::max<int64_t>(o->cap_nnz[h], 1)) * 4);
        if (h < L - 1) {
            o->blk_cscptr[h] = c.take(static_cast<size_t>(o->cap_src[h] + 1) * 8);
            o->blk_cscrow[h] = c.take(static_cast<size_t>(std::max<int64_t>(o->cap_nnz[h], 1)) * 4);
        }
        if (m->kind == GNN_AGG_GCN_SYM) o->blk_src_norm[h] = c.take(static_cast<size_t>(o->cap_src[h]) * 4);
        if (h < L - 1) o->blk_csc_ws[h] = c.take(block_csc_ws_bytes(o->cap_src[h], o->cap_nnz[h]));
    }
    o->x0 = c.take(static_cast<size_t>(o->cap_src[L - 1]) * m->dims[0] * asz);
    // layer 1's aggregation: computed in the prepare stage (it needs no
    // weights), so it lives with the prepare buffers
    o->agg[1] = c.take(static_cast<size_t>(o->cap_dst[L - 1]) * m->dims[0] * asz);
    o->prep_bytes = round_up(c.off, 256);
    // compute part: activations, gradients, GEMM and loss scratch, outputs
    Carver d(nullptr);
    size_t bwd = 0, fwd = 0;
    for (int l = 1; l <= L; ++l) {
        const int hb = L - l;
        const int64_t rows = o->cap_dst[hb];
        if (l >= 2) o->agg[l] = d.take(static_cast<size_t>(rows) * m->dims[l - 1] * asz);
        o->h[l] = d.take(static_cast<size_t>(rows) * m->dims[l] * (l < L ? asz : 4));
        o->grad[l] = d.take(static_cast<size_t>(rows) * m->dims[l] * 4);
        if (l >= 2) o->d_a[l] = d.take(static_cast<size_t>(rows) * k_of(m, l) * 4);
        if (l >= 2 && m->kind == GNN_AGG_SAGE_MAX)
            o->argmax[l] = d.take(static_cast<size_t>(rows) * m->dims[l - 1] * 4);
        fwd = std::max(fwd, update_fwd_ws_bytes(k_of(m, l), m->dims[l], rows, m->precision));
        // every layer its own region: the two-layer backward reduces layer
        // 2's partials while layer 1's are being written
        bwd += update_bwd_ws_bytes(k_of(m, l), m->dims[l], rows, m->precision);
    }
    o->fwd_ws = d.take(fwd);
    o->fwd_ws_bytes = fwd;
    o->bwd_ws = d.take(bwd);
    o->bwd_ws_bytes = bwd;
    o->loss_ws_bytes = softmax_ce_ws_bytes(batch);
    o->loss_ws = d.take(o->loss_ws_bytes);
    o->edges = d.take(8);
    o->error = d.take(8);
    o->loss = d.take(4);
    o->compute_bytes = round_up(d.off, 256);
    o->total_bytes = o->prep_bytes + o->compute_bytes;
    return GNN_OK;
}

static gnn_block block_view(const gnn_step_layout &o, int h, char *base) {
    gnn_block b{};
    b.cap_dst = o.cap_dst[h];
    b.cap_src = o.cap_src[h];
    b.cap_nnz = o.cap_nnz[h];
    b.counts = reinterpret_cast<int64_t *>(base + o.blk_counts[h]);
    b.src_ids = reinterpret_cast<int64_t *>(base + o.blk_src_ids[h]);
    b.rowptr = reinterpret_cast<int64_t *>(base + o.blk_rowptr[h]);
    b.col = reinterpret_cast<int32_t *>(base + o.blk_col[h]);
    b.cscptr = o.blk_cscptr[h] ? reinterpret_cast<int64_t *>(base + o.blk_cscptr[h]) : nullptr;
    b.cscrow = o.blk_cscrow[h] ? reinterpret_cast<int32_t *>(base + o.blk_cscrow[h]) : nullptr;
    b.src_norm = o.blk_src_norm[h] ? reinterpret_cast<float *>(base + o.blk_src_norm[h]) : nullptr;
    return b;
}

namespace {

void block_views(const gnn_model *m, const gnn_step_layout &o, char *prep, gnn_block *blk) {
    for (int h = 0; h < m->num_layers; ++h) blk[h] = block_view(o, h, prep);
}

// The feature loading fuses into layer 1's sum aggregations for an fp32
// table in device memory feeding bf16 layers (the aggregation reads the
// table rows it sums, and X' is gathered only for the destination rows,
// which the update and the backward read); a host table is read once over
// the link into X', and so is every table of the max aggregator.
bool fused_loading(const gnn_model *m, const gnn_graph *g, bool host_table, int tdt, int act) {
    return m->kind != GNN_AGG_SAGE_MAX && !host_table && tdt == GNN_F32 && act == GNN_BF16 && g->n <= INT32_MAX;
}

// Sampling of all hops, the gather of X' and layer 1's aggregation (which
// needs no weights) into a prepare workspace, with the transposes of blocks
// 1 .. L-1 (0-based hops 0 .. L-2).  Launches, for hop h >= 1 (relabel(h)
// also counts the columns of block h's transpose):
//   A_h = relabel(h-1) + prepare(h) + place(h-2)
//   B_h = emit(h) + scan(h-1) + sort(h-2)   (no sort role for h < 2)
//   F   = relabel(L-1) + gather + place(L-2)
//   G   = sort(L-2) + aggregation of layer 1 (the input layer's block, X')
gnn_status run_prepare(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table, int tdt,
                       bool host_table, int64_t row_stride, const int64_t *targets, uint64_t seed, uint64_t step,
                       char *prep, const gnn_step_layout &o, hipStream_t s) {
    const int L = m->num_layers;
    const int act = m->precision;
    gnn_block blk[GNN_MAX_LAYERS];
    block_views(m, o, prep, blk);
    csc::Args ca[GNN_MAX_LAYERS] = {};
    csc::Grids cg[GNN_MAX_LAYERS] = {};
    for (int h = 0; h + 1 < L; ++h) {
        ca[h] = csc_args(&blk[h], prep + o.blk_csc_ws[h], o.cap_src[h], o.cap_nnz[h]);
        cg[h] = csc_grids(ca[h]);
    }
    auto place = [&](int h) { return role(csc::PlaceJob{ca[h >= 0 ? h : 0]}, h >= 0 ? cg[h].place : 0u); };
    auto scan = [&](int h) { return role(csc::ScanJob{ca[h >= 0 ? h : 0]}, h >= 0 ? cg[h].scan : 0u); };
    auto sort = [&](int h) { return role(csc::SortJob{ca[h >= 0 ? h : 0]}, h >= 0 ? cg[h].sort : 0u); };

    // hop 1 around the targets, then outwards; hop h's relabel only needs
    // hop h's sources, like hop h+1's prepare
    char *shared = prep + o.sampler_ws;
    size_t hop_max = 0;
    for (int h = 0; h < L; ++h)
        hop_max = std::max(hop_max, sampler_hop_bytes(g->n, o.cap_dst[h], m->fanouts[h]));
    samp::HopPlan plan[GNN_MAX_LAYERS];
    for (int h = 0; h < L; ++h) {
        const int64_t *dst = h == 0 ? targets : blk[h - 1].src_ids;
        const int64_t *n_dst = h == 0 ? nullptr : blk[h - 1].counts + 1;
        void *scratch = shared + sampler_shared_bytes(g->n) + (h % 2) * hop_max;
        plan[h] = plan_hop(g, m->kind == GNN_AGG_GCN_SYM ? gcn_norm : nullptr, dst, n_dst, m->fanouts[h], seed, step,
                           h + 1, &blk[h], shared, scratch, h + 1 < L ? &ca[h] : nullptr);
    }
    GNN_TRY(launch_hop_prepare(plan[0], s));
    GNN_TRY(launch_hop_emit(plan[0], s));
    for (int h = 1; h < L; ++h) {
        gnn_status st = GNN_OK;
        samp::with_prepare_job(plan[h], [&](auto job) {
            st = launch_jobs(s, "hop_relabel+prepare+csc_place", role(samp::RelabelJob{plan[h - 1].a},
                                                                       plan[h - 1].relabel_grid),
                             role(job, plan[h].prep_grid), place(h - 2));
        });
        GNN_TRY(st);
        if (h >= 2)
            GNN_TRY(launch_jobs(s, "hop_emit+csc_scan+csc_sort", role(samp::EmitJob{plan[h].a}, plan[h].emit_grid),
                                scan(h - 1), sort(h - 2)));
        else
            GNN_TRY(launch_jobs(s, "hop_emit+csc_scan", role(samp::EmitJob{plan[h].a}, plan[h].emit_grid),
                                scan(h - 1)));
    }
    // feature loading (rows of the input layer's sources) with the last
    // hop's relabel
    const gnn_block &b0 = blk[L - 1];
    const bool fuse = fused_loading(m, g, host_table, tdt, act);
    // X': all sources of the input layer's block, or its destination rows
    // (counts[0]) when the aggregation reads the table itself
    const gath::Args ga{table, row_stride, b0.src_ids, b0.counts + (fuse ? 0 : 1), fuse ? b0.cap_dst : b0.cap_src,
                        m->dims[0], prep + o.x0};
    const unsigned ggrid = gath::grid_for(ga.cap, m->dims[0], gath::vec_ok(ga, tdt, act), host_table);
    gnn_status st = GNN_OK;
    const bool ok = gath::with_job(ga, tdt, act, [&](auto job) {
        st = launch_jobs(s, "hop_relabel+gather+csc_place",
                         role(samp::RelabelJob{plan[L - 1].a}, plan[L - 1].relabel_grid), role(job, ggrid),
                         place(L - 2));
    });
    GNN_CHECK(ok, GNN_EUNSUPPORTED, "train_step: table dtype %d cannot feed precision %d", tdt, act);
    GNN_TRY(st);
    if (fuse) {
        agg::with_fwd_table_job(&b0, m->kind, plan[L - 1].a.gpad, plan[L - 1].a.k, gcn_norm,
                                static_cast<const float *>(table), row_stride,
                                reinterpret_cast<const uint16_t *>(prep + o.x0), m->dims[0],
                                reinterpret_cast<uint16_t *>(prep + o.agg[1]), [&](auto aj) {
            st = launch_jobs(s, "csc_sort+aggregate_l1_from_table", sort(L - 2), role(aj, agg::row_grid(b0.cap_dst)));
        });
        return st;
    }
    // (layer 1's argmax is not kept: no aggregation backward below layer 2)
    agg::with_fwd_kind_job(&b0, m->kind, prep + o.x0, act, m->dims[0], prep + o.agg[1], act, nullptr, [&](auto aj) {
        st = launch_jobs(s, "csc_sort+aggregate_l1", sort(L - 2), role(aj, agg::row_grid(b0.cap_dst)));
    });
    return st;
}

// Workgroups of a group's host-table gather, all copies together.  Reads of
// host memory have microsecond latencies; with many in flight they hold up
// the device-memory traffic of the compute stage running beside them (its
// kernels ran up to 100x slower under a 256-workgroup gather).  64
// workgroups still keep the host link near its rate: measured on the
// 30M-vertex host-table workload, 64 -> 0.97 ms per step, 32 -> 0.97,
// 16 -> 1.36 (link-starved), 256 -> 1.13.
constexpr int kHostGroupGrid = 64;

// The prepare stages of G (2 .. kMaxCopies) steps at once: the same
// launches as run_prepare, each carrying one copy of every role per step
// (Multi), so a group of steps pays the launch and latency chain of the
// sampler once.  Step c of the group has targets targets + c * batch, step
// number first_step + c and prepare workspace preps[c]; the transposes are
// complete when the last launch ends.
gnn_status run_prepare_group(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                             int tdt, bool host_table, int64_t row_stride, const int64_t *targets, int64_t batch,
                             uint64_t seed, uint64_t first_step, int G, void *const *preps,
                             const gnn_step_layout &o, hipStream_t s) {
    const int L = m->num_layers;
    const int act = m->precision;
    gnn_block blk[kMaxCopies][GNN_MAX_LAYERS];
    csc::Args ca[kMaxCopies][GNN_MAX_LAYERS] = {};
    csc::Grids cg[GNN_MAX_LAYERS] = {};
    samp::HopPlan plan[kMaxCopies][GNN_MAX_LAYERS];
    size_t hop_max = 0;
    for (int h = 0; h < L; ++h)
        hop_max = std::max(hop_max, sampler_hop_bytes(g->n, o.cap_dst[h], m->fanouts[h]));
    for (int c = 0; c < G; ++c) {
        char *prep = static_cast<char *>(preps[c]);
        block_views(m, o, prep, blk[c]);
        for (int h = 0; h + 1 < L; ++h) {
            ca[c][h] = csc_args(&blk[c][h], prep + o.blk_csc_ws[h], o.cap_src[h], o.cap_nnz[h]);
            cg[h] = csc_grids(ca[c][h]);
        }
        char *shared = prep + o.sampler_ws;
        for (int h = 0; h < L; ++h) {
            const int64_t *dst = h == 0 ? targets + c * batch : blk[c][h - 1].src_ids;
            const int64_t *n_dst = h == 0 ? nullptr : blk[c][h - 1].counts + 1;
            void *scratch = shared + sampler_shared_bytes(g->n) + (h % 2) * hop_max;
            plan[c][h] = plan_hop(g, m->kind == GNN_AGG_GCN_SYM ? gcn_norm : nullptr, dst, n_dst, m->fanouts[h],
                                  seed, first_step + static_cast<uint64_t>(c), h + 1, &blk[c][h], shared, scratch,
                                  h + 1 < L ? &ca[c][h] : nullptr);
        }
    }
    auto place = [&](int h) {
        return multi_role([&](int c) { return csc::PlaceJob{ca[c][h >= 0 ? h : 0]}; }, G, h >= 0 ? cg[h].place : 0u);
    };
    auto scan = [&](int h) {
        return multi_role([&](int c) { return csc::ScanJob{ca[c][h >= 0 ? h : 0]}; }, G, h >= 0 ? cg[h].scan : 0u);
    };
    auto sort = [&](int h) {
        return multi_role([&](int c) { return csc::SortJob{ca[c][h >= 0 ? h : 0]}; }, G, h >= 0 ? cg[h].sort : 0u);
    };
    auto relabel = [&](int h) {
        return multi_role([&](int c) { return samp::RelabelJob{plan[c][h].a}; }, G, plan[0][h].relabel_grid);
    };
    auto emit = [&](int h) {
        return multi_role([&](int c) { return samp::EmitJob{plan[c][h].a}; }, G, plan[0][h].emit_grid);
    };
    gnn_status st = GNN_OK;
    samp::with_prepare_job(plan[0][0], [&](auto job) {
        using J = decltype(job);
        st = launch_jobs(s, "hop_prepare", multi_role([&](int c) { return J{plan[c][0].a}; }, G,
                                                       plan[0][0].prep_grid));
    });
    GNN_TRY(st);
    GNN_TRY(launch_jobs(s, "hop_emit", emit(0)));
    for (int h = 1; h < L; ++h) {
        samp::with_prepare_job(plan[0][h], [&](auto job) {
            using J = decltype(job);
            st = launch_jobs(s, "hop_relabel+prepare+csc_place", relabel(h - 1),
                             multi_role([&](int c) { return J{plan[c][h].a}; }, G, plan[0][h].prep_grid),
                             place(h - 2));
        });
        GNN_TRY(st);
        if (h >= 2) GNN_TRY(launch_jobs(s, "hop_emit+csc_scan+csc_sort", emit(h), scan(h - 1), sort(h - 2)));
        else GNN_TRY(launch_jobs(s, "hop_emit+csc_scan", emit(h), scan(h - 1)));
    }
    const bool fuse = fused_loading(m, g, host_table, tdt, act);
    gath::Args ga[kMaxCopies];
    for (int c = 0; c < G; ++c) {
        const gnn_block &b0 = blk[c][L - 1];
        ga[c] = gath::Args{table, row_stride, b0.src_ids, b0.counts + (fuse ? 0 : 1), fuse ? b0.cap_dst : b0.cap_src,
                           m->dims[0], static_cast<char *>(preps[c]) + o.x0};
    }
    // A host table's rows come over the host link, which a few hundred
    // workgroups in total already saturate: the copies share that budget, so
    // the rest of the GPU stays free for the compute stage running beside.
    unsigned ggrid = gath::grid_for(ga[0].cap, m->dims[0], gath::vec_ok(ga[0], tdt, act), host_table);
    if (host_table) ggrid = std::max(1u, std::min(ggrid, static_cast<unsigned>(kHostGroupGrid / G)));
    bool same = true;
    const bool ok = gath::with_job(ga[0], tdt, act, [&](auto job) {
        using J = decltype(job);
        J js[kMaxCopies];
        for (int c = 0; c < G; ++c)
            gath::with_job(ga[c], tdt, act, [&](auto jc) {
                if constexpr (std::is_same<decltype(jc), J>::value) js[c] = jc;
                else same = false;
            });
        if (same)
            st = launch_jobs(s, "hop_relabel+gather+csc_place", relabel(L - 1),
                             multi_role([&](int c) { return js[c]; }, G, ggrid), place(L - 2));
    });
    GNN_CHECK(ok, GNN_EUNSUPPORTED, "train_step: table dtype %d cannot feed precision %d", tdt, act);
    GNN_CHECK(same, GNN_EINVAL, "train_step: prepare workspaces differ in alignment");
    GNN_TRY(st);
    // last: the sort of block L-2 and layer 1's aggregation
    if (fuse) {
        auto tjob = [&](int c, auto &&f) {
            agg::with_fwd_table_job(&blk[c][L - 1], m->kind, plan[c][L - 1].a.gpad, plan[c][L - 1].a.k, gcn_norm,
                                    static_cast<const float *>(table), row_stride,
                                    reinterpret_cast<const uint16_t *>(static_cast<char *>(preps[c]) + o.x0),
                                    m->dims[0], reinterpret_cast<uint16_t *>(static_cast<char *>(preps[c]) + o.agg[1]),
                                    f);
        };
        tjob(0, [&](auto aj) {
            using J = decltype(aj);
            J js[kMaxCopies];
            for (int c = 0; c < G; ++c)
                tjob(c, [&](auto jc) {
                    if constexpr (std::is_same<decltype(jc), J>::value) js[c] = jc;
                    else same = false;
                });
            if (same)
                st = launch_jobs(s, "csc_sort+aggregate_l1_from_table", sort(L - 2),
                                 multi_role([&](int c) { return js[c]; }, G, agg::row_grid(blk[0][L - 1].cap_dst)));
        });
        GNN_CHECK(same, GNN_EINVAL, "train_step: prepare workspaces differ in alignment");
        return st;
    }
    agg::with_fwd_kind_job(&blk[0][L - 1], m->kind, static_cast<char *>(preps[0]) + o.x0, act, m->dims[0],
                           static_cast<char *>(preps[0]) + o.agg[1], act, nullptr, [&](auto aj) {
        using J = decltype(aj);
        J js[kMaxCopies];
        for (int c = 0; c < G; ++c)
            agg::with_fwd_kind_job(&blk[c][L - 1], m->kind, static_cast<char *>(preps[c]) + o.x0, act, m->dims[0],
                                   static_cast<char *>(preps[c]) + o.agg[1], act, nullptr, [&](auto jc) {
                if constexpr (std::is_same<decltype(jc), J>::value) js[c] = jc;
                else same = false;
            });
        if (same)
            st = launch_jobs(s, "csc_sort+aggregate_l1", sort(L - 2),
                             multi_role([&](int c) { return js[c]; }, G, agg::row_grid(blk[0][L - 1].cap_dst)));
    });
    GNN_CHECK(same, GNN_EINVAL, "train_step: prepare workspaces differ in alignment");
    return st;
}

namespace {

// Layer l's region of the update-backward workspace inside the compute
// workspace comp (layers in order, as step_layout carves them).
float *bwd_region(const gnn_model *m, const gnn_step_layout &o, char *comp, int l) {
    size_t off = o.bwd_ws;
    for (int j = 1; j < l; ++j)
        off += update_bwd_ws_bytes(k_of(m, j), m->dims[j], o.cap_dst[m->num_layers - j], m->precision);
    return reinterpret_cast<float *>(comp + off);
}

// The backward of a two-layer step whose forward was one launch that also
// produced layer 2's input gradient dA^2: three launches.
//   1. layer 2's dW partials, and the aggregation backward through the last
//      block (dLoss/dZ^1, with the ReLU mask of H^1);
//   2. layer 1's dW partials, and layer 2's reduction with SGD on W^2, b^2
//      and its bf16 shadow (nothing else in launch 2 reads them);
//   3. layer 1's reduction with SGD, and the end of the step.
// Both layers' partials are live in launch 2, so each has its own region.
struct TwoBwd {
    TwoBwdPlan q;  // both layers' dW (q.pull: layer 2's aggregation backward folded into layer 1's)
    agg::BwdJob<GNN_AGG_SAGE_MEAN, uint16_t, true> sage_bwd;  // else G^1 through memory
    agg::BwdJob<GNN_AGG_GCN_SYM, uint16_t, true> gcn_bwd;
    agg::BwdMaxJob<uint16_t, true> max_bwd;  // (the max aggregator's, through its argmax table)
    bool ok;
};

TwoBwd two_layer_bwd_plan(const gnn_model *m, const gnn_block *blk, const void *x0, const void *m1, char *comp,
                          const gnn_step_layout &o, float lr) {
    TwoBwd t{};
    const int64_t f0 = m->dims[0], f1 = m->dims[1];
    const gnn_block &b2 = blk[0], &b1 = blk[1];
    const uint16_t *h1 = reinterpret_cast<const uint16_t *>(comp + o.h[1]);
    float *d_a2 = reinterpret_cast<float *>(comp + o.d_a[2]);
    float *g1 = reinterpret_cast<float *>(comp + o.grad[1]);
    const int32_t *arg2 = m->kind == GNN_AGG_SAGE_MAX ? reinterpret_cast<const int32_t *>(comp + o.argmax[2]) : nullptr;
    t.q = plan_two_bwd(m->kind, b2, x0, m1, f0, b1.counts, b1.cap_dst, h1, f1, comp + o.agg[2], arg2, d_a2,
                       reinterpret_cast<const float *>(comp + o.grad[2]), m->dims[2], m->w[0], m->dw[0], m->db[0],
                       bwd_region(m, o, comp, 1), m->w[0], m->b[0], m->wt[0], m->w[1], m->dw[1], m->db[1],
                       bwd_region(m, o, comp, 2), m->w[1], m->b[1], m->wt[1], lr);
    t.q.a1.g = g1;  // the unfused path's G^1
    int C, S;
    agg::split_row(f1, &C, &S);
    t.sage_bwd = {b2, d_a2, f1, C, S, h1, g1};
    t.gcn_bwd = {b2, d_a2, f1, C, S, h1, g1};
    t.max_bwd = {b2, arg2, d_a2, f1, C, S, h1, g1};
    const TwoBwdPlan &q = t.q;
    t.ok = m->precision == GNN_BF16 && q.gemm_ok && f1 % 4 == 0 && aligned(d_a2, 16) && aligned(g1, 16) &&
           aligned(h1, 8) && aligned(arg2, 16) &&
           reinterpret_cast<char *>(q.a2.part) + gbwd::dw_part_bytes(q.p2.pw, q.a2.K(), m->dims[2]) <=
               comp + o.bwd_ws + o.bwd_ws_bytes &&
           reinterpret_cast<char *>(q.a1.part) + gbwd::dw_part_bytes(q.p1.pw, q.a1.K(), f1) <=
               reinterpret_cast<char *>(q.a2.part);
    return t;
}

template <bool VG>
gbwd::DweightJob<true, 64, uint16_t, true, VG> dweight64(const gbwd::Args &a, const gbwd::Plan &p) {
    return gbwd::dweight_job<true, 64, uint16_t, true, VG>(a, p);
}

gnn_status two_layer_bwd(const gnn_model *m, const TwoBwd &t, unsigned bwd_grid, const loss::TailJob &tail,
                         hipStream_t s) {
    const TwoBwdPlan &q = t.q;
    gnn_status st = GNN_OK;
    if (q.pull) {
        // both layers' dW partials (G^1 pulled through the transpose), then
        // both reductions with SGD and the end of the step
        GNN_TRY(launch_two_bwd_partials(q, m->kind, s));
        gbwd::with_reduce_job(q.a1, q.p1, [&](auto r1) {
            gbwd::with_reduce_job(q.a2, q.p2, [&](auto r2) {
                st = launch_jobs(s, "dw_reduce_l1+dw_reduce_l2+step_tail", role(r1, q.p1.red_grid),
                                 role(r2, q.p2.red_grid), role(tail, 1u));
            });
        });
        return st;
    }
    auto first = [&](auto dwj) {
        if (m->kind == GNN_AGG_SAGE_MAX)
            st = launch_job2(dwj, q.p2.dw_grid, t.max_bwd, bwd_grid, s, "update_dweight_l2+aggregate_bwd_max");
        else if (m->kind == GNN_AGG_SAGE_MEAN)
            st = launch_job2(dwj, q.p2.dw_grid, t.sage_bwd, bwd_grid, s, "update_dweight_l2+aggregate_bwd");
        else
            st = launch_job2(dwj, q.p2.dw_grid, t.gcn_bwd, bwd_grid, s, "update_dweight_l2+aggregate_bwd");
    };
    if (q.p2.vec_g) first(dweight64<true>(q.a2, q.p2));
    else first(dweight64<false>(q.a2, q.p2));
    GNN_TRY(st);
    auto second = [&](auto dwj) {
        gbwd::with_reduce_job(q.a2, q.p2, [&](auto rj) {
            st = launch_job2(dwj, q.p1.dw_grid, rj, q.p2.red_grid, s, "update_dweight_l1+dw_reduce_l2");
        });
    };
    if (q.p1.vec_g) second(dweight64<true>(q.a1, q.p1));
    else second(dweight64<false>(q.a1, q.p1));
    GNN_TRY(st);
    gbwd::with_reduce_job(q.a1, q.p1, [&](auto rj) {
        st = launch_job2(rj, q.p1.red_grid, tail, 1, s, "update_dw_reduce+step_tail");
    });
    return st;
}

}  // namespace

// Forward, loss, backward and SGD from a prepared workspace (blocks, their
// transposes, X' and layer 1's aggregation).  The targets are the first rows
// of hop 1's sources (destinations come first).
// first: the step opens a call (its tail writes the error word; later steps
// of the call OR into it).
gnn_status run_compute(const gnn_model *m, const int64_t *labels, int64_t batch, float lr, float *loss_dev,
                       int64_t *edges_dev, char *prep, char *comp, const gnn_step_layout &o, bool first,
                       hipStream_t s) {
    const int L = m->num_layers;
    const int act = m->precision;
    gnn_block blk[GNN_MAX_LAYERS];
    block_views(m, o, prep, blk);
    const void *x0 = prep + o.x0;

    // aggregation output of layer l (layer 1's was made by the prepare stage)
    auto agg_of = [&](int l) { return l == 1 ? prep + o.agg[1] : comp + o.agg[l]; };

    // forward: one fused launch per layer where the shapes allow it (the
    // last one with the loss in its epilogue; layer 1 only multiplies, its
    // aggregation is done), else aggregation and update as separate launches
    float *row_loss = reinterpret_cast<float *>(comp + o.loss_ws);
    float *g_last = reinterpret_cast<float *>(comp + o.grad[L]);
    bool loss_done = false;
    const bool sage = m->kind != GNN_AGG_GCN_SYM;  // A = [h_self || aggregation]
    const bool maxagg = m->kind == GNN_AGG_SAGE_MAX;
    auto argmax_of = [&](int l) { return reinterpret_cast<int32_t *>(comp + o.argmax[l]); };
    // a two-layer model at a small mini-batch: both layers in one launch
    // (layer 1's rows computed where the last layer reads them; with the
    // max aggregator it also writes layer 2's argmax table); the fused layer
    // kernel implements the sum aggregations only
    TwoBwd tb{};
    bool two = L == 2 && two_layer_ok(m->kind, m->precision, m->dims[0], m->dims[1], m->dims[2], blk[0].cap_dst,
                                      m->fanouts[0], x0, agg_of(1), m->wt[0], m->wt[1], comp + o.h[1],
                                      comp + o.agg[2], maxagg ? argmax_of(2) : nullptr);
    if (two) {
        tb = two_layer_bwd_plan(m, blk, x0, agg_of(1), comp, o, lr);
        two = tb.ok;
    }
    if (two) {
        GNN_TRY(launch_two_layer(&blk[0], m->kind, m->fanouts[0], x0, agg_of(1), m->dims[0], m->wt[0], m->b[0],
                                 m->dims[1], comp + o.h[1], m->wt[1], m->b[1], m->dims[2], comp + o.agg[2],
                                 reinterpret_cast<float *>(comp + o.h[2]), labels, g_last, row_loss, batch,
                                 reinterpret_cast<float *>(comp + o.d_a[2]), maxagg ? argmax_of(2) : nullptr, s));
        loss_done = true;
    }
    for (int l = 1; l <= L && !two; ++l) {
        const gnn_block &b = blk[L - l];
        const void *hin = (l == 1) ? x0 : static_cast<const void *>(comp + o.h[l - 1]);
        void *agg = agg_of(l);
        const int64_t f_in = m->dims[l - 1];
        const int32_t maxdeg = l == 1 ? 1 : m->fanouts[L - l];
        if (!maxagg && (l > 1 || l == L) && fused_layer_ok(m->kind, m->precision, f_in, m->dims[l], b.cap_dst, maxdeg, l == L,
                                                 hin, m->wt[l - 1], agg)) {
            if (l == 1)  // a one-layer model: the prepared aggregation, with the loss
                GNN_TRY(launch_fused_update(&b, m->kind, sage ? hin : nullptr, agg, f_in, m->wt[0], m->b[0],
                                            m->dims[1], comp + o.h[1], true, labels, g_last, row_loss, batch, s));
            else
                GNN_TRY(launch_fused_layer(&b, m->kind, maxdeg, hin, f_in, m->wt[l - 1], m->b[l - 1], m->dims[l],
                                           agg, comp + o.h[l], l == L, labels, g_last, row_loss, batch, s));
            loss_done = l == L;
            continue;
        }
        // (a hidden layer 1 with a bf16 W^T that fits takes the fused
        // kernel in A-load mode inside launch_update_fwd)
        if (l > 1 && maxagg) GNN_TRY(launch_aggregate_fwd_max(&b, hin, act, f_in, agg, act, argmax_of(l), s));
        else if (l > 1) GNN_TRY(launch_aggregate_fwd(&b, m->kind, hin, act, f_in, agg, act, s));
        GNN_TRY(launch_update_fwd(sage ? hin : agg, sage ? agg : nullptr, act, f_in, b.counts, b.cap_dst, m->w[l - 1],
                                  m->wt[l - 1], m->b[l - 1], m->dims[l], l < L, m->precision, comp + o.h[l],
                                  l < L ? act : GNN_F32, comp + o.fwd_ws, s));
    }
    // loss on the targets (unless fused into the last layer): gradient and
    // row losses now, the mean with the last kernel of the step
    if (!loss_done)
        GNN_TRY(launch_job(loss::SoftmaxJob{reinterpret_cast<const float *>(comp + o.h[L]), batch, m->dims[L], labels,
                                            blk[0].src_ids, g_last, row_loss},
                           static_cast<unsigned>(ceil_div(batch, loss::kThreads / 64)), s, "softmax_ce"));
    // backward (reads the transposes).  Per layer: the dA and dW GEMMs in
    // one launch, then the dW reduction (with SGD on W^l, b^l and the
    // shadow) in one launch with the aggregation backward of the layer, or
    // with the end of the step for layer 1.  Every later step reads only
    // lower layers' weights.
    loss::TailJob tail{};
    for (int h = 0; h < L; ++h) tail.counts[h] = blk[h].counts;
    tail.num_blocks = L;
    tail.row_loss = row_loss;
    tail.b = batch;
    tail.loss = reinterpret_cast<float *>(comp + o.loss);
    tail.loss_out = loss_dev;
    tail.edges = reinterpret_cast<int64_t *>(comp + o.edges);
    tail.edges_out = edges_dev;
    tail.error = reinterpret_cast<int64_t *>(comp + o.error);
    tail.accumulate = first ? 0 : 1;
    if (two) return two_layer_bwd(m, tb, agg::row_grid(blk[0].cap_src), tail, s);
    for (int l = L; l >= 1; --l) {
        const gnn_block &b = blk[L - l];
        const void *hin = (l == 1) ? x0 : static_cast<const void *>(comp + o.h[l - 1]);
        const void *agg_out = agg_of(l);
        const int64_t f_in = m->dims[l - 1];
        float *d_a = l > 1 ? reinterpret_cast<float *>(comp + o.d_a[l]) : nullptr;
        const gbwd::Args a{sage ? hin : agg_out, sage ? agg_out : nullptr, act, f_in, b.counts, b.cap_dst,
                           m->w[l - 1], reinterpret_cast<const float *>(comp + o.grad[l]), m->dims[l], m->precision,
                           m->dw[l - 1], m->db[l - 1], d_a, reinterpret_cast<float *>(comp + o.bwd_ws), m->w[l - 1],
                           m->b[l - 1], m->wt[l - 1], lr};
        const gbwd::Plan p = gbwd::plan(a);
        GNN_TRY(launch_update_bwd_gemms(a, p, s));
        gnn_status st = GNN_OK;
        if (l > 1) {
            float *d_src = reinterpret_cast<float *>(comp + o.grad[l - 1]);
            auto pair = [&](auto aj) {
                gbwd::with_reduce_job(a, p, [&](auto rj) {
                    st = launch_job2(rj, p.red_grid, aj, agg::row_grid(b.cap_src), s, "update_dw_reduce+aggregate_bwd");
                });
            };
            if (maxagg) agg::with_bwd_max_job(&b, argmax_of(l), d_a, f_in, hin, act, d_src, pair);
            else agg::with_bwd_job(&b, m->kind, d_a, f_in, hin, act, d_src, pair);
        } else {
            gbwd::with_reduce_job(a, p, [&](auto rj) {
                st = launch_job2(rj, p.red_grid, tail, 1, s, "update_dw_reduce+step_tail");
            });
        }
        GNN_TRY(st);
    }
    return GNN_OK;
}

}  // namespace

// The whole step on one stream.
gnn_status run_train_step(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                          int tdt, bool host_table, int64_t row_stride, const int64_t *labels,
                          const int64_t *targets, int64_t batch, uint64_t seed, uint64_t step, float lr,
                          float *loss_dev, int64_t *edges_dev, void *ws, hipStream_t s) {
    gnn_step_layout o;
    GNN_TRY(step_layout(m, g->n, batch, &o));
    char *prep = static_cast<char *>(ws);
    char *comp = prep + o.prep_bytes;
    GNN_TRY(run_prepare(m, g, gcn_norm, table, tdt, host_table, row_stride, targets, seed, step, prep, o, s));
    return run_compute(m, labels, batch, lr, loss_dev, edges_dev, prep, comp, o, true, s);
}

gnn_status run_step_prepare(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                            int tdt, bool host_table, int64_t row_stride, const int64_t *targets, int64_t batch,
                            uint64_t seed, uint64_t step, void *prep_ws, hipStream_t s) {
    gnn_step_layout o;
    GNN_TRY(step_layout(m, g->n, batch, &o));
    return run_prepare(m, g, gcn_norm, table, tdt, host_table, row_stride, targets, seed, step,
                       static_cast<char *>(prep_ws), o, s);
}

gnn_status run_step_compute(const gnn_model *m, int64_t graph_n, const int64_t *labels, int64_t batch, float lr,
                            float *loss_dev, int64_t *edges_dev, void *prep_ws, void *comp_ws, hipStream_t s,
                            bool first) {
    gnn_step_layout o;
    GNN_TRY(step_layout(m, graph_n, batch, &o));
    return run_compute(m, labels, batch, lr, loss_dev, edges_dev, static_cast<char *>(prep_ws),
                       static_cast<char *>(comp_ws), o, first, s);
}

namespace {

// Events of one pipelined call, destroyed on every exit path (a pending
// event's resources are released once it completes).
struct EventSet {
    hipEvent_t e[8] = {};
    int n = 0;
    gnn_status make(int count) {
        for (; n < count; ++n) GNN_HIP(hipEventCreateWithFlags(&e[n], hipEventDisableTiming));
        return GNN_OK;
    }
    ~EventSet() {
        for (int i = 0; i < n; ++i) (void)hipEventDestroy(e[i]);
    }
};

}  // namespace

// `steps` training steps in groups of G = max(1, n_prep / 2): the prepare
// stages of group q+1 run on ps while the computes of group q run on s.
// Group q uses slots (q % 2) * G .. (q % 2) * G + G - 1.  The streams meet
// once per group: a group's computes wait for all its prepares
// (prepared[q % 2]), and a group's prepares wait for the computes that last
// read its slots, those of group q-2 (consumed[q % 2]).  The first prepares
// wait for the work already on s.  Host-side stream events are costly
// relative to a launch, so grouping keeps them to about one per step.
gnn_status run_train_steps(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table, int tdt,
                           bool host_table, int64_t row_stride, const int64_t *labels, const int64_t *targets,
                           int64_t batch, uint64_t seed, uint64_t first_step, int64_t steps, float lr,
                           float *loss_dev, int64_t *edges_dev, void *const *prep_ws, int n_prep, void *comp_ws,
                           hipStream_t s, hipStream_t ps) {
    if (steps == 0) return GNN_OK;
    const int G = std::min(kMaxCopies, std::max(1, n_prep / 2));
    const int64_t groups = ceil_div(steps, G);
    EventSet ev;
    GNN_TRY(ev.make(5));
    hipEvent_t prepared[2] = {ev.e[0], ev.e[1]}, consumed[2] = {ev.e[2], ev.e[3]}, start = ev.e[4];
    GNN_HIP(hipEventRecord(start, s));
    GNN_HIP(hipStreamWaitEvent(ps, start, 0));
    auto prepare_group = [&](int64_t q) -> gnn_status {
        const int half = static_cast<int>(q % 2);
        if (q >= 2) GNN_HIP(hipStreamWaitEvent(ps, consumed[half], 0));
        const int64_t i0 = q * G;
        const int gq = static_cast<int>(std::min<int64_t>(G, steps - i0));
        if (gq == 1) {
            GNN_TRY(run_step_prepare(m, g, gcn_norm, table, tdt, host_table, row_stride, targets + i0 * batch, batch,
                                     seed, first_step + static_cast<uint64_t>(i0), prep_ws[half * G], ps));
        } else {
            gnn_step_layout o;
            GNN_TRY(step_layout(m, g->n, batch, &o));
            GNN_TRY(run_prepare_group(m, g, gcn_norm, table, tdt, host_table, row_stride, targets + i0 * batch,
                                      batch, seed, first_step + static_cast<uint64_t>(i0), gq, prep_ws + half * G, o,
                                      ps));
        }
        GNN_HIP(hipEventRecord(prepared[half], ps));
        return GNN_OK;
    };
    GNN_TRY(prepare_group(0));
    for (int64_t q = 0; q < groups; ++q) {
        if (q + 1 < groups) GNN_TRY(prepare_group(q + 1));
        const int half = static_cast<int>(q % 2);
        GNN_HIP(hipStreamWaitEvent(s, prepared[half], 0));
        for (int j = 0; j < G && q * G + j < steps; ++j) {
            const int64_t i = q * G + j;
            GNN_TRY(run_step_compute(m, g->n, labels, batch, lr, loss_dev ? loss_dev + i : nullptr,
                                     edges_dev ? edges_dev + i : nullptr, prep_ws[half * G + j], comp_ws, s, i == 0));
        }
        GNN_HIP(hipEventRecord(consumed[half], s));
    }
    return GNN_OK;
}

}  // namespace gnn
