// Neighbour aggregation over a sampled block, forward (pull over the block
// CSR) and backward (pull over its transpose, no atomics): the mean and GCN
// sums, and GraphSAGE's max aggregator with its argmax table.
//
// Work split: one wavefront per output row.  A row of f elements is cut into
// C = ceil(f / 4) chunks of 4; when C <= 32 the wavefront is divided into
// S = 64 / C slots that walk different edges of the row at once (f = 100:
// two slots of 25 lanes), and the slot partial sums are folded with lane
// shuffles at the end.  Up to 64 neighbour indices and weights of the row are
// held one per lane and broadcast with shuffles.  Sums are fp32.
#include "aggregate_dev.h"
#include "jobs.h"

namespace gnn {

gnn_status launch_aggregate_fwd(const gnn_block *b, int kind, const void *h, int hdt, int64_t f, void *out, int odt,
                                hipStream_t s) {
    if (b->cap_dst == 0 || f == 0) return GNN_OK;
    gnn_status st = GNN_OK;
    const bool ok = agg::with_fwd_job(b, kind, h, hdt, f, out, odt, [&](auto job) {
        st = launch_job(job, agg::row_grid(b->cap_dst), s, "aggregate_fwd");
    });
    if (!ok) return fail(GNN_EUNSUPPORTED, "aggregate_fwd: unsupported dtypes %d -> %d", hdt, odt);
    return st;
}

gnn_status launch_aggregate_bwd(const gnn_block *b, int kind, const float *d_a, int64_t f, const void *h_below,
                                int hbdt, float *d_src, hipStream_t s) {
    if (b->cap_src == 0 || f == 0) return GNN_OK;
    gnn_status st = GNN_OK;
    agg::with_bwd_job(b, kind, d_a, f, h_below, hbdt, d_src, [&](auto job) {
        st = launch_job(job, agg::row_grid(b->cap_src), s, "aggregate_bwd");
    });
    return st;
}

gnn_status launch_aggregate_fwd_max(const gnn_block *b, const void *h, int hdt, int64_t f, void *out, int odt,
                                    int32_t *argmax, hipStream_t s) {
    if (b->cap_dst == 0 || f == 0) return GNN_OK;
    gnn_status st = GNN_OK;
    const bool ok = agg::with_fwd_max_job(b, h, hdt, f, out, odt, argmax, [&](auto job) {
        st = launch_job(job, agg::row_grid(b->cap_dst), s, "aggregate_fwd_max");
    });
    if (!ok) return fail(GNN_EUNSUPPORTED, "aggregate_fwd_max: unsupported dtypes %d -> %d", hdt, odt);
    return st;
}

gnn_status launch_aggregate_bwd_max(const gnn_block *b, const int32_t *argmax, const float *d_a, int64_t f,
                                    const void *h_below, int hbdt, float *d_src, hipStream_t s) {
    if (b->cap_src == 0 || f == 0) return GNN_OK;
    gnn_status st = GNN_OK;
    agg::with_bwd_max_job(b, argmax, d_a, f, h_below, hbdt, d_src, [&](auto job) {
        st = launch_job(job, agg::row_grid(b->cap_src), s, "aggregate_bwd_max");
    });
    return st;
}

}  // namespace gnn
