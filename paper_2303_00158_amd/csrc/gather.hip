// Feature loader: X' = X[ids] with an optional narrowing to bf16 (the job
// types are in gather_dev.h).
#include "gather_dev.h"
#include "jobs.h"

namespace gnn {

gnn_status launch_gather(const void *table, int tdt, int64_t dim, int64_t row_stride, const int64_t *ids,
                         const int64_t *n_ids_dev, int64_t cap_ids, void *out, int odt, bool host, hipStream_t s) {
    if (cap_ids == 0 || dim == 0) return GNN_OK;
    const gath::Args a{table, row_stride, ids, n_ids_dev, cap_ids, dim, out};
    const unsigned grid = gath::grid_for(cap_ids, dim, gath::vec_ok(a, tdt, odt), host);
    gnn_status st = GNN_OK;
    const bool ok = gath::with_job(a, tdt, odt, [&](auto job) { st = launch_job(job, grid, s, "gather"); });
    if (!ok) return fail(GNN_EUNSUPPORTED, "gather: unsupported dtype pair %d -> %d", tdt, odt);
    return st;
}

}  // namespace gnn
