// extern "C" entry points: host-side validation, then the launchers.
#include <algorithm>
#include <cstdarg>
#include <cstdio>

#include "csc_dev.h"
#include "internal.h"

namespace gnn {

// ---------------------------------------------------------------------------
// errors: one message per host thread
// ---------------------------------------------------------------------------
static thread_local char g_err[512];

gnn_status fail(gnn_status code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_err[0] = '\0'; }

gnn_status launch_status(const char *what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(GNN_EHIP, "%s: kernel launch failed: %s", what, hipGetErrorString(e));
    return GNN_OK;
}

gnn_status launch_gcn_norm(const gnn_graph *g, float *nrm, hipStream_t s);
gnn_status step_layout(const gnn_model *m, int64_t graph_n, int64_t batch, gnn_step_layout *o);
gnn_status run_train_step(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table, int tdt,
                          bool host_table, int64_t row_stride, const int64_t *labels, const int64_t *targets,
                          int64_t batch, uint64_t seed, uint64_t step, float lr, float *loss_dev, int64_t *edges_dev,
                          void *ws, hipStream_t s);
gnn_status run_step_prepare(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                            int tdt, bool host_table, int64_t row_stride, const int64_t *targets, int64_t batch,
                            uint64_t seed, uint64_t step, void *prep_ws, hipStream_t s);
gnn_status run_step_compute(const gnn_model *m, int64_t graph_n, const int64_t *labels, int64_t batch, float lr,
                            float *loss_dev, int64_t *edges_dev, void *prep_ws, void *comp_ws, hipStream_t s,
                            bool first = true);
gnn_status run_train_steps(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table, int tdt,
                           bool host_table, int64_t row_stride, const int64_t *labels, const int64_t *targets,
                           int64_t batch, uint64_t seed, uint64_t first_step, int64_t steps, float lr,
                           float *loss_dev, int64_t *edges_dev, void *const *prep_ws, int n_prep, void *comp_ws,
                           hipStream_t s, hipStream_t ps);

namespace {

bool act_dtype(int dt) { return dt == GNN_F32 || dt == GNN_BF16; }
bool dim_ok(int64_t f) { return f >= 1 && f <= GNN_MAX_DIM; }

gnn_status check_graph(const gnn_graph *g, const char *who) {
    GNN_CHECK(g, GNN_EINVAL, "%s: graph is NULL", who);
    GNN_CHECK(g->n >= 0 && g->nnz >= 0, GNN_EINVAL, "%s: negative graph size", who);
    GNN_CHECK(g->n < (1ll << 31), GNN_EUNSUPPORTED, "%s: graphs above 2^31 - 1 vertices are not supported", who);
    GNN_CHECK(g->rowptr && (g->col || g->nnz == 0), GNN_EINVAL, "%s: graph arrays are NULL", who);
    GNN_CHECK(aligned(g->rowptr, 8) && aligned(g->col, 8), GNN_EINVAL, "%s: graph arrays must be 8-byte aligned",
              who);
    return GNN_OK;
}

// Pinned host memory is addressed through its device mapping.
gnn_status device_view(const void *p, int loc, const void **out, const char *who) {
    if (loc == GNN_LOC_DEVICE) {
        *out = p;
        return GNN_OK;
    }
    void *d = nullptr;
    hipError_t e = hipHostGetDevicePointer(&d, const_cast<void *>(p), 0);
    if (e != hipSuccess || d == nullptr) {
        (void)hipGetLastError();
        return fail(GNN_EINVAL, "%s: table is not pinned host memory mapped for the device (%s)", who,
                    hipGetErrorString(e));
    }
    *out = d;
    return GNN_OK;
}

gnn_status check_model(const gnn_model *m, const char *who) {
    GNN_CHECK(m, GNN_EINVAL, "%s: model is NULL", who);
    GNN_CHECK(m->num_layers >= 1 && m->num_layers <= GNN_MAX_LAYERS, GNN_EINVAL, "%s: num_layers must be in [1, %d]",
              who, GNN_MAX_LAYERS);
    GNN_CHECK(m->kind == GNN_AGG_SAGE_MEAN || m->kind == GNN_AGG_GCN_SYM || m->kind == GNN_AGG_SAGE_MAX, GNN_EINVAL,
              "%s: unknown aggregation %d", who, m->kind);
    GNN_CHECK(act_dtype(m->precision), GNN_EUNSUPPORTED, "%s: precision must be GNN_F32 or GNN_BF16", who);
    for (int l = 0; l <= m->num_layers; ++l)
        GNN_CHECK(dim_ok(m->dims[l]), GNN_EINVAL, "%s: dims[%d] = %d out of [1, %d]", who, l, m->dims[l], GNN_MAX_DIM);
    for (int h = 0; h < m->num_layers; ++h)
        GNN_CHECK(m->fanouts[h] >= 1 && m->fanouts[h] <= GNN_MAX_FANOUT, GNN_EINVAL,
                  "%s: fanouts[%d] = %d out of [1, %d]", who, h, m->fanouts[h], GNN_MAX_FANOUT);
    return GNN_OK;
}

gnn_status check_model_buffers(const gnn_model *m, const char *who) {
    for (int l = 0; l < m->num_layers; ++l) {
        GNN_CHECK(m->w[l] && m->b[l] && m->dw[l] && m->db[l], GNN_EINVAL, "%s: layer %d weight buffers are NULL", who,
                  l + 1);
        GNN_CHECK(aligned(m->w[l], 16) && aligned(m->dw[l], 16) && aligned(m->b[l], 4) && aligned(m->db[l], 4),
                  GNN_EINVAL, "%s: weights must be 16-byte aligned", who);
        GNN_CHECK(!m->wt[l] || (m->precision == GNN_BF16 && aligned(m->wt[l], 8)), GNN_EINVAL,
                  "%s: layer %d shadow must be 8-byte aligned and needs a GNN_BF16 model", who, l + 1);
    }
    return GNN_OK;
}

}  // namespace

gnn_status check_block(const gnn_block *b, bool need_csc, bool need_norm, const char *who) {
    GNN_CHECK(b, GNN_EINVAL, "%s: block is NULL", who);
    GNN_CHECK(b->cap_dst >= 0 && b->cap_src >= 0 && b->cap_nnz >= 0, GNN_EINVAL, "%s: negative block capacity", who);
    GNN_CHECK(b->cap_src < (1ll << 31) && b->cap_nnz < (1ll << 31), GNN_EUNSUPPORTED,
              "%s: block capacities above 2^31 - 1 are not supported", who);
    GNN_CHECK(b->counts && b->src_ids && b->rowptr && (b->col || b->cap_nnz == 0), GNN_EINVAL,
              "%s: block arrays are NULL", who);
    GNN_CHECK(aligned(b->counts, 8) && aligned(b->src_ids, 8) && aligned(b->rowptr, 8) && aligned(b->col, 4),
              GNN_EINVAL, "%s: misaligned block arrays", who);
    if (need_csc)
        GNN_CHECK(b->cscptr && (b->cscrow || b->cap_nnz == 0) && aligned(b->cscptr, 8) && aligned(b->cscrow, 4),
                  GNN_EINVAL, "%s: the block transpose (cscptr/cscrow) is required", who);
    if (need_norm)
        GNN_CHECK(b->src_norm && aligned(b->src_norm, 4), GNN_EINVAL, "%s: GCN needs block->src_norm", who);
    return GNN_OK;
}

// Host validation shared by the update-backward entry points; *ws_need is
// the scratch the call needs.
gnn_status check_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                            int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt,
                            const float *dw, const float *db, const float *d_a, size_t *ws_need, const char *who) {
    GNN_CHECK(act_dtype(adt) && act_dtype(gemm_dt), GNN_EUNSUPPORTED, "%s: dtypes must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(k_each) && dim_ok(n_out), GNN_EINVAL, "%s: k_each / n_out out of [1, %d]", who, GNN_MAX_DIM);
    GNN_CHECK(cap_m >= 0 && cap_m < (1ll << 40), GNN_EINVAL, "%s: bad cap_m", who);
    GNN_CHECK((a_self || cap_m == 0) && w && (g || cap_m == 0) && dw, GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(a_self, dtype_size(adt)) && aligned(a_nbr, dtype_size(adt)) && aligned(w, 4) && aligned(g, 4) &&
                  aligned(dw, 4) && aligned(db, 4) && aligned(d_a, 4) && aligned(m_dev, 8),
              GNN_EINVAL, "%s: misaligned data", who);
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    *ws_need = update_bwd_ws_bytes(K, n_out, cap_m, gemm_dt);
    return GNN_OK;
}

}  // namespace gnn

using namespace gnn;

extern "C" {

const char *gnn_last_error(void) { return g_err; }

int32_t gnn_abi_version(void) { return GNN_ABI_VERSION; }

gnn_status gnn_gcn_norm(const gnn_graph *g, float *nrm_out, gnn_stream s) {
    clear_error();
    GNN_TRY(check_graph(g, "gnn_gcn_norm"));
    GNN_CHECK(nrm_out || g->n == 0, GNN_EINVAL, "gnn_gcn_norm: nrm_out is NULL");
    return launch_gcn_norm(g, nrm_out, stream_of(s));
}

gnn_status gnn_block_bounds(int64_t graph_n, int64_t cap_dst, int32_t fanout, int64_t *cap_src, int64_t *cap_nnz) {
    clear_error();
    GNN_CHECK(cap_src && cap_nnz, GNN_EINVAL, "gnn_block_bounds: output pointers are NULL");
    GNN_CHECK(graph_n >= 0 && cap_dst >= 0, GNN_EINVAL, "gnn_block_bounds: negative size");
    GNN_CHECK(fanout >= 1 && fanout <= GNN_MAX_FANOUT, GNN_EINVAL, "gnn_block_bounds: fanout %d out of [1, %d]",
              fanout, GNN_MAX_FANOUT);
    GNN_CHECK(cap_dst <= (1ll << 40), GNN_ESIZE, "gnn_block_bounds: cap_dst too large");
    *cap_nnz = cap_dst * fanout;
    *cap_src = std::min<int64_t>(cap_dst + *cap_nnz, std::max(graph_n, cap_dst));
    return GNN_OK;
}

gnn_status gnn_sampler_workspace_size(int64_t graph_n, int64_t cap_dst, int32_t fanout, size_t *bytes) {
    clear_error();
    GNN_CHECK(bytes, GNN_EINVAL, "gnn_sampler_workspace_size: bytes is NULL");
    GNN_CHECK(graph_n >= 0 && cap_dst >= 0, GNN_EINVAL, "gnn_sampler_workspace_size: negative size");
    GNN_CHECK(fanout >= 1 && fanout <= GNN_MAX_FANOUT, GNN_EINVAL, "gnn_sampler_workspace_size: bad fanout %d",
              fanout);
    *bytes = sampler_ws_bytes(graph_n, cap_dst, fanout);
    return GNN_OK;
}

gnn_status gnn_sampler_workspace_init(void *ws, size_t ws_bytes, int64_t graph_n, gnn_stream s) {
    clear_error();
    GNN_CHECK(ws && aligned(ws, 256), GNN_EINVAL, "gnn_sampler_workspace_init: ws must be non-NULL, 256-byte aligned");
    GNN_CHECK(graph_n >= 0 && graph_n < (1ll << 31), GNN_EINVAL, "gnn_sampler_workspace_init: bad graph size");
    GNN_CHECK(ws_bytes >= sampler_ws_bytes(graph_n, 1, 1), GNN_ESIZE, "gnn_sampler_workspace_init: workspace too small");
    return launch_sampler_ws_init(ws, graph_n, stream_of(s));
}

gnn_status gnn_build_block(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids,
                           const int64_t *n_dst_dev, int32_t fanout, uint64_t seed, uint64_t step, int32_t hop,
                           int32_t want_csc, gnn_block *out, void *ws, size_t ws_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_build_block";
    GNN_TRY(check_graph(g, who));
    GNN_CHECK(fanout >= 1 && fanout <= GNN_MAX_FANOUT, GNN_EINVAL, "%s: fanout %d out of [1, %d]", who, fanout,
              GNN_MAX_FANOUT);
    GNN_TRY(check_block(out, want_csc != 0, false, who));
    GNN_CHECK(dst_ids || out->cap_dst == 0, GNN_EINVAL, "%s: dst_ids is NULL", who);
    GNN_CHECK(aligned(dst_ids, 8) && aligned(n_dst_dev, 8), GNN_EINVAL, "%s: misaligned dst arrays", who);
    int64_t need_src, need_nnz;
    GNN_TRY(gnn_block_bounds(g->n, out->cap_dst, fanout, &need_src, &need_nnz));
    GNN_CHECK(out->cap_src >= need_src && out->cap_nnz >= need_nnz, GNN_ESIZE,
              "%s: block capacities (src %lld, nnz %lld) below the bounds (src %lld, nnz %lld)", who,
              (long long)out->cap_src, (long long)out->cap_nnz, (long long)need_src, (long long)need_nnz);
    GNN_CHECK((gcn_norm == nullptr) == (out->src_norm == nullptr), GNN_EINVAL,
              "%s: gcn_norm and out->src_norm must be given together", who);
    GNN_CHECK(ws && aligned(ws, 256), GNN_EINVAL, "%s: ws must be non-NULL and 256-byte aligned", who);
    const size_t need = sampler_ws_bytes(g->n, out->cap_dst, fanout);
    GNN_CHECK(ws_bytes >= need, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, ws_bytes, need);
    csc::Args ca{};
    if (want_csc)
        ca = csc_args(out, sampler_csc_ws(ws, g->n, out->cap_dst, fanout), src_bound(g->n, out->cap_dst, fanout),
                      out->cap_dst * fanout);
    GNN_TRY(launch_build_block(g, gcn_norm, dst_ids, n_dst_dev, fanout, seed, step, hop, out, ws,
                               want_csc ? &ca : nullptr, stream_of(s)));
    return want_csc ? launch_block_csc(ca, stream_of(s)) : GNN_OK;
}

gnn_status gnn_gather_features(const void *table, gnn_dtype tdt, gnn_loc loc, int64_t n_rows, int64_t dim,
                               int64_t row_stride, const int64_t *ids, const int64_t *n_ids_dev, int64_t cap_ids,
                               void *out, gnn_dtype odt, gnn_stream s) {
    clear_error();
    const char *who = "gnn_gather_features";
    GNN_CHECK(loc == GNN_LOC_DEVICE || loc == GNN_LOC_HOST_PINNED, GNN_EINVAL, "%s: unknown location %d", who, loc);
    GNN_CHECK(tdt == GNN_F32 || tdt == GNN_F16 || tdt == GNN_BF16, GNN_EINVAL, "%s: unknown table dtype %d", who, tdt);
    GNN_CHECK(odt == GNN_F32 || odt == GNN_F16 || odt == GNN_BF16, GNN_EINVAL, "%s: unknown output dtype %d", who, odt);
    const bool pair_ok = (tdt == odt) || (tdt == GNN_F32 && odt == GNN_BF16) || (tdt == GNN_F16 && odt == GNN_F32) ||
                         (tdt == GNN_F16 && odt == GNN_BF16);
    GNN_CHECK(pair_ok, GNN_EUNSUPPORTED, "%s: conversion %d -> %d is not supported", who, tdt, odt);
    GNN_CHECK(dim_ok(dim), GNN_EINVAL, "%s: dim %lld out of [1, %d]", who, (long long)dim, GNN_MAX_DIM);
    GNN_CHECK(row_stride >= dim, GNN_EINVAL, "%s: row_stride %lld < dim %lld", who, (long long)row_stride,
              (long long)dim);
    GNN_CHECK(n_rows >= 0 && cap_ids >= 0, GNN_EINVAL, "%s: negative size", who);
    GNN_CHECK(table && (ids || cap_ids == 0) && (out || cap_ids == 0), GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(ids, 8) && aligned(n_ids_dev, 8), GNN_EINVAL, "%s: misaligned id arrays", who);
    GNN_CHECK(aligned(table, dtype_size(tdt)) && aligned(out, dtype_size(odt)), GNN_EINVAL, "%s: misaligned data", who);
    const void *t = nullptr;
    GNN_TRY(device_view(table, loc, &t, who));
    return launch_gather(t, tdt, dim, row_stride, ids, n_ids_dev, cap_ids, out, odt, loc == GNN_LOC_HOST_PINNED,
                         stream_of(s));
}

gnn_status gnn_aggregate_fwd(const gnn_block *b, gnn_agg kind, const void *h_src, gnn_dtype hdt, int64_t f,
                             void *out, gnn_dtype odt, gnn_stream s) {
    clear_error();
    const char *who = "gnn_aggregate_fwd";
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM, GNN_EINVAL, "%s: unknown aggregation %d", who,
              kind);
    GNN_TRY(check_block(b, false, kind == GNN_AGG_GCN_SYM, who));
    GNN_CHECK(act_dtype(hdt) && act_dtype(odt), GNN_EUNSUPPORTED, "%s: dtypes must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(f), GNN_EINVAL, "%s: f %lld out of [1, %d]", who, (long long)f, GNN_MAX_DIM);
    GNN_CHECK((h_src || b->cap_src == 0) && (out || b->cap_dst == 0), GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(h_src, dtype_size(hdt)) && aligned(out, dtype_size(odt)), GNN_EINVAL, "%s: misaligned data", who);
    return launch_aggregate_fwd(b, kind, h_src, hdt, f, out, odt, stream_of(s));
}

gnn_status gnn_aggregate_fwd_dedup(const gnn_block *b, gnn_agg kind, const void *h_src, gnn_dtype hdt, int64_t f,
                                   void *out, gnn_dtype odt, gnn_stream s) {
    clear_error();
    const char *who = "gnn_aggregate_fwd_dedup";
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM, GNN_EINVAL, "%s: unknown aggregation %d", who,
              kind);
    GNN_TRY(check_block(b, false, kind == GNN_AGG_GCN_SYM, who));
    GNN_CHECK(act_dtype(hdt) && act_dtype(odt), GNN_EUNSUPPORTED, "%s: dtypes must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(f), GNN_EINVAL, "%s: f %lld out of [1, %d]", who, (long long)f, GNN_MAX_DIM);
    GNN_CHECK((h_src || b->cap_src == 0) && (out || b->cap_dst == 0), GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(h_src, dtype_size(hdt)) && aligned(out, dtype_size(odt)), GNN_EINVAL, "%s: misaligned data", who);
    return launch_aggregate_fwd_dedup(b, kind, h_src, hdt, f, out, odt, stream_of(s));
}

gnn_status gnn_layer_fwd(const gnn_block *b, gnn_agg kind, int32_t max_row_len, const void *h_src, int64_t f,
                         const uint16_t *wt, const float *bias, int64_t n_out, void *agg_out, void *out,
                         const int64_t *labels, int64_t batch, float *g_out, float *row_loss, gnn_stream s) {
    clear_error();
    const char *who = "gnn_layer_fwd";
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM, GNN_EINVAL, "%s: unknown aggregation %d", who,
              kind);
    GNN_TRY(check_block(b, false, kind == GNN_AGG_GCN_SYM, who));
    GNN_CHECK(dim_ok(f) && dim_ok(n_out), GNN_EINVAL, "%s: f %lld or n_out %lld out of [1, %d]", who, (long long)f,
              (long long)n_out, GNN_MAX_DIM);
    GNN_CHECK(max_row_len >= 1, GNN_EINVAL, "%s: max_row_len must be >= 1", who);
    const bool last = labels != nullptr;
    GNN_CHECK(h_src && wt && agg_out && out, GNN_EINVAL, "%s: NULL pointer", who);
    if (last) {
        GNN_CHECK(g_out && row_loss, GNN_EINVAL, "%s: labels given without g_out and row_loss", who);
        GNN_CHECK(batch >= 1 && batch <= b->cap_dst, GNN_EINVAL, "%s: batch must be in [1, cap_dst]", who);
        GNN_CHECK(aligned(out, 4) && aligned(g_out, 4) && aligned(row_loss, 4) && aligned(labels, 8), GNN_EINVAL,
                  "%s: misaligned data", who);
    }
    GNN_CHECK(fused_layer_ok(kind, GNN_BF16, f, n_out, b->cap_dst, max_row_len, last, h_src, wt, agg_out),
              GNN_EUNSUPPORTED,
              "%s: shape not supported (needs f %% 4 == 0, weights of at most 2 x 8 column tiles x 8 steps or "
              "1 x 16, n_out <= 64 with labels, 8-byte aligned bf16 data)", who);
    return launch_fused_layer(b, kind, max_row_len, h_src, f, wt, bias, n_out, agg_out, out, last, labels, g_out,
                              row_loss, batch, stream_of(s));
}

gnn_status gnn_two_layer_fwd(const gnn_block *last, gnn_agg kind, int32_t fanout, const void *x_self, const void *m1,
                             int64_t f0, const uint16_t *wt1, const float *b1, int64_t f1, void *h1,
                             const uint16_t *wt2, const float *b2, int64_t n_out, void *agg_out, float *logits,
                             const int64_t *labels, int64_t batch, float *g_out, float *row_loss, float *d_a,
                             gnn_stream s) {
    clear_error();
    const char *who = "gnn_two_layer_fwd";
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM, GNN_EINVAL, "%s: unknown aggregation %d", who,
              kind);
    GNN_TRY(check_block(last, false, kind == GNN_AGG_GCN_SYM, who));
    GNN_CHECK(dim_ok(f0) && dim_ok(f1) && dim_ok(n_out), GNN_EINVAL, "%s: f0 %lld, f1 %lld or n_out %lld out of [1, %d]",
              who, (long long)f0, (long long)f1, (long long)n_out, GNN_MAX_DIM);
    GNN_CHECK(fanout >= 1, GNN_EINVAL, "%s: fanout must be >= 1", who);
    GNN_CHECK(m1 && wt1 && h1 && wt2 && agg_out && logits && labels && g_out && row_loss &&
                  (x_self || kind == GNN_AGG_GCN_SYM),
              GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(batch >= 1 && batch <= last->cap_dst, GNN_EINVAL, "%s: batch must be in [1, cap_dst]", who);
    GNN_CHECK(aligned(logits, 4) && aligned(g_out, 4) && aligned(row_loss, 4) && aligned(labels, 8) &&
                  aligned(d_a, 4),
              GNN_EINVAL, "%s: misaligned data", who);
    GNN_CHECK(two_layer_ok(kind, GNN_BF16, f0, f1, n_out, last->cap_dst, fanout,
                           kind == GNN_AGG_SAGE_MEAN ? x_self : m1, m1, wt1, wt2, h1, agg_out, nullptr),
              GNN_EUNSUPPORTED,
              "%s: shape not supported (needs f0 %% 4 == 0 with K1 <= 256, f1 %% 8 == 0 with f1 <= 256, n_out <= 64 "
              "(48 for SAGE), cap_dst <= 2048, aligned bf16 data)", who);
    return launch_two_layer(last, kind, fanout, x_self, m1, f0, wt1, b1, f1, h1, wt2, b2, n_out, agg_out, logits,
                            labels, g_out, row_loss, batch, d_a, nullptr, stream_of(s));
}

gnn_status gnn_two_layer_fwd_max(const gnn_block *last, int32_t fanout, const void *x_self, const void *m1, int64_t f0,
                                 const uint16_t *wt1, const float *b1, int64_t f1, void *h1, const uint16_t *wt2,
                                 const float *b2, int64_t n_out, void *agg_out, int32_t *argmax, float *logits,
                                 const int64_t *labels, int64_t batch, float *g_out, float *row_loss, float *d_a,
                                 gnn_stream s) {
    clear_error();
    const char *who = "gnn_two_layer_fwd_max";
    const int kind = GNN_AGG_SAGE_MAX;
    GNN_TRY(check_block(last, false, false, who));
    GNN_CHECK(dim_ok(f0) && dim_ok(f1) && dim_ok(n_out), GNN_EINVAL, "%s: f0 %lld, f1 %lld or n_out %lld out of [1, %d]",
              who, (long long)f0, (long long)f1, (long long)n_out, GNN_MAX_DIM);
    GNN_CHECK(fanout >= 1, GNN_EINVAL, "%s: fanout must be >= 1", who);
    GNN_CHECK(x_self && m1 && wt1 && h1 && wt2 && agg_out && argmax && logits && labels && g_out && row_loss,
              GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(batch >= 1 && batch <= last->cap_dst, GNN_EINVAL, "%s: batch must be in [1, cap_dst]", who);
    GNN_CHECK(aligned(logits, 4) && aligned(g_out, 4) && aligned(row_loss, 4) && aligned(labels, 8) &&
                  aligned(d_a, 4),
              GNN_EINVAL, "%s: misaligned data", who);
    GNN_CHECK(two_layer_ok(kind, GNN_BF16, f0, f1, n_out, last->cap_dst, fanout, x_self, m1, wt1, wt2, h1, agg_out,
                           argmax),
              GNN_EUNSUPPORTED,
              "%s: shape not supported (needs f0 %% 4 == 0 with 2 f0 <= 256, f1 %% 8 == 0 with f1 <= 256, n_out <= "
              "48, cap_dst <= 2048, aligned bf16 data, a 16-byte aligned argmax table)", who);
    return launch_two_layer(last, kind, fanout, x_self, m1, f0, wt1, b1, f1, h1, wt2, b2, n_out, agg_out, logits,
                            labels, g_out, row_loss, batch, d_a, argmax, stream_of(s));
}

gnn_status gnn_two_layer_bwd_workspace_size(gnn_agg kind, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_m1,
                                            int64_t cap_m2, size_t *bytes) {
    clear_error();
    const char *who = "gnn_two_layer_bwd_workspace_size";
    GNN_CHECK(bytes, GNN_EINVAL, "%s: bytes is NULL", who);
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM || kind == GNN_AGG_SAGE_MAX, GNN_EINVAL,
              "%s: unknown aggregation %d", who, kind);
    GNN_CHECK(dim_ok(f0) && dim_ok(f1) && dim_ok(n_out) && cap_m1 >= 0 && cap_m2 >= 0, GNN_EINVAL, "%s: bad size",
              who);
    *bytes = two_bwd_ws_bytes(kind, f0, f1, n_out, cap_m1, cap_m2);
    return GNN_OK;
}

gnn_status gnn_two_layer_bwd(const gnn_block *last, gnn_agg kind, const void *x_self, const void *m1, int64_t f0,
                             const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1,
                             const void *agg2, const float *d_a2, const float *g2, int64_t n_out, float *dw1,
                             float *db1, float *dw2, float *db2, void *ws, size_t ws_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_two_layer_bwd";
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM, GNN_EINVAL, "%s: unknown aggregation %d", who,
              kind);
    GNN_TRY(check_block(last, true, kind == GNN_AGG_GCN_SYM, who));
    GNN_CHECK(dim_ok(f0) && dim_ok(f1) && dim_ok(n_out), GNN_EINVAL, "%s: f0 %lld, f1 %lld or n_out %lld out of [1, %d]",
              who, (long long)f0, (long long)f1, (long long)n_out, GNN_MAX_DIM);
    GNN_CHECK(m1 && m1_rows && h1 && agg2 && d_a2 && g2 && dw1 && dw2 && ws && (x_self || kind == GNN_AGG_GCN_SYM),
              GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(cap_m1 >= 1 && cap_m1 <= last->cap_src, GNN_EINVAL, "%s: cap_m1 must be in [1, last->cap_src]", who);
    GNN_CHECK(aligned(m1_rows, 8) && aligned(g2, 4) && aligned(dw1, 4) && aligned(db1, 4) && aligned(dw2, 4) &&
                  aligned(db2, 4) && aligned(ws, 256),
              GNN_EINVAL, "%s: misaligned data", who);
    const size_t need = two_bwd_ws_bytes(kind, f0, f1, n_out, cap_m1, last->cap_dst);
    GNN_CHECK(ws_bytes >= need, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, ws_bytes, need);
    return launch_two_bwd(last, kind, kind == GNN_AGG_SAGE_MEAN ? x_self : nullptr, m1, f0, m1_rows, cap_m1, h1, f1,
                          agg2, nullptr, d_a2, g2, n_out, dw1, db1, dw2, db2, ws, stream_of(s));
}

gnn_status gnn_two_layer_bwd_max(const gnn_block *last, const void *x_self, const void *m1, int64_t f0,
                                 const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1,
                                 const void *agg2, const int32_t *argmax2, const float *d_a2, const float *g2,
                                 int64_t n_out, float *dw1, float *db1, float *dw2, float *db2, void *ws,
                                 size_t ws_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_two_layer_bwd_max";
    const int kind = GNN_AGG_SAGE_MAX;
    GNN_TRY(check_block(last, true, false, who));
    GNN_CHECK(dim_ok(f0) && dim_ok(f1) && dim_ok(n_out), GNN_EINVAL, "%s: f0 %lld, f1 %lld or n_out %lld out of [1, %d]",
              who, (long long)f0, (long long)f1, (long long)n_out, GNN_MAX_DIM);
    GNN_CHECK(x_self && m1 && m1_rows && h1 && agg2 && argmax2 && d_a2 && g2 && dw1 && dw2 && ws, GNN_EINVAL,
              "%s: NULL pointer", who);
    GNN_CHECK(cap_m1 >= 1 && cap_m1 <= last->cap_src, GNN_EINVAL, "%s: cap_m1 must be in [1, last->cap_src]", who);
    GNN_CHECK(aligned(m1_rows, 8) && aligned(g2, 4) && aligned(dw1, 4) && aligned(db1, 4) && aligned(dw2, 4) &&
                  aligned(db2, 4) && aligned(ws, 256),
              GNN_EINVAL, "%s: misaligned data", who);
    const size_t need = two_bwd_ws_bytes(kind, f0, f1, n_out, cap_m1, last->cap_dst);
    GNN_CHECK(ws_bytes >= need, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, ws_bytes, need);
    return launch_two_bwd(last, kind, x_self, m1, f0, m1_rows, cap_m1, h1, f1, agg2, argmax2, d_a2, g2, n_out, dw1,
                          db1, dw2, db2, ws, stream_of(s));
}

gnn_status gnn_aggregate_bwd(const gnn_block *b, gnn_agg kind, const float *d_a, int64_t f, const void *h_below,
                             gnn_dtype hbdt, float *d_src, gnn_stream s) {
    clear_error();
    const char *who = "gnn_aggregate_bwd";
    GNN_CHECK(kind == GNN_AGG_SAGE_MEAN || kind == GNN_AGG_GCN_SYM, GNN_EINVAL, "%s: unknown aggregation %d", who,
              kind);
    GNN_TRY(check_block(b, true, kind == GNN_AGG_GCN_SYM, who));
    GNN_CHECK(!h_below || act_dtype(hbdt), GNN_EUNSUPPORTED, "%s: h_below dtype must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(f), GNN_EINVAL, "%s: f %lld out of [1, %d]", who, (long long)f, GNN_MAX_DIM);
    GNN_CHECK((d_a || b->cap_dst == 0) && (d_src || b->cap_src == 0), GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(d_a, 4) && aligned(d_src, 4) && aligned(h_below, h_below ? dtype_size(hbdt) : 1), GNN_EINVAL,
              "%s: misaligned data", who);
    return launch_aggregate_bwd(b, kind, d_a, f, h_below, hbdt, d_src, stream_of(s));
}

gnn_status gnn_aggregate_fwd_max(const gnn_block *b, const void *h_src, gnn_dtype hdt, int64_t f, void *out,
                                 gnn_dtype odt, int32_t *argmax, gnn_stream s) {
    clear_error();
    const char *who = "gnn_aggregate_fwd_max";
    GNN_TRY(check_block(b, false, false, who));
    GNN_CHECK(act_dtype(hdt) && act_dtype(odt), GNN_EUNSUPPORTED, "%s: dtypes must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(f), GNN_EINVAL, "%s: f %lld out of [1, %d]", who, (long long)f, GNN_MAX_DIM);
    GNN_CHECK((h_src || b->cap_src == 0) && (out || b->cap_dst == 0), GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(h_src, dtype_size(hdt)) && aligned(out, dtype_size(odt)) && aligned(argmax, 4), GNN_EINVAL,
              "%s: misaligned data", who);
    return launch_aggregate_fwd_max(b, h_src, hdt, f, out, odt, argmax, stream_of(s));
}

gnn_status gnn_aggregate_bwd_max(const gnn_block *b, const int32_t *argmax, const float *d_a, int64_t f,
                                 const void *h_below, gnn_dtype hbdt, float *d_src, gnn_stream s) {
    clear_error();
    const char *who = "gnn_aggregate_bwd_max";
    GNN_TRY(check_block(b, true, false, who));
    GNN_CHECK(!h_below || act_dtype(hbdt), GNN_EUNSUPPORTED, "%s: h_below dtype must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(f), GNN_EINVAL, "%s: f %lld out of [1, %d]", who, (long long)f, GNN_MAX_DIM);
    GNN_CHECK(((d_a && argmax) || b->cap_dst == 0) && (d_src || b->cap_src == 0), GNN_EINVAL, "%s: NULL pointer",
              who);
    GNN_CHECK(aligned(d_a, 4) && aligned(d_src, 4) && aligned(argmax, 4) &&
                  aligned(h_below, h_below ? dtype_size(hbdt) : 1),
              GNN_EINVAL, "%s: misaligned data", who);
    return launch_aggregate_bwd_max(b, argmax, d_a, f, h_below, hbdt, d_src, stream_of(s));
}

gnn_status gnn_update_fwd_workspace_size(int64_t k, int64_t n_out, int64_t cap_m, gnn_dtype gemm_dt, size_t *bytes) {
    clear_error();
    GNN_CHECK(bytes, GNN_EINVAL, "gnn_update_fwd_workspace_size: bytes is NULL");
    GNN_CHECK(k >= 1 && n_out >= 1 && cap_m >= 0, GNN_EINVAL, "gnn_update_fwd_workspace_size: bad size");
    GNN_CHECK(act_dtype(gemm_dt), GNN_EUNSUPPORTED, "gnn_update_fwd_workspace_size: bad gemm dtype");
    *bytes = update_fwd_ws_bytes(k, n_out, cap_m, gemm_dt);
    return GNN_OK;
}

gnn_status gnn_update_fwd(const void *a_self, const void *a_nbr, gnn_dtype adt, int64_t k_each,
                          const int64_t *m_dev, int64_t cap_m, const float *w, const uint16_t *wt, const float *bias,
                          int64_t n_out, int32_t relu, gnn_dtype gemm_dt, void *out, gnn_dtype odt, void *ws,
                          size_t ws_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_update_fwd";
    GNN_CHECK(act_dtype(adt) && act_dtype(odt) && act_dtype(gemm_dt), GNN_EUNSUPPORTED,
              "%s: dtypes must be GNN_F32 or GNN_BF16", who);
    GNN_CHECK(dim_ok(k_each) && dim_ok(n_out), GNN_EINVAL, "%s: k_each / n_out out of [1, %d]", who, GNN_MAX_DIM);
    GNN_CHECK(cap_m >= 0 && cap_m < (1ll << 40), GNN_EINVAL, "%s: bad cap_m", who);
    GNN_CHECK(ceil_div(cap_m, 128) <= kMaxGrid, GNN_ESIZE, "%s: cap_m exceeds the grid limit", who);
    GNN_CHECK((a_self || cap_m == 0) && w && (out || cap_m == 0), GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(aligned(a_self, dtype_size(adt)) && aligned(a_nbr, dtype_size(adt)) && aligned(w, 4) &&
                  aligned(bias, 4) && aligned(out, dtype_size(odt)) && aligned(m_dev, 8),
              GNN_EINVAL, "%s: misaligned data", who);
    if (ws) {
        const int64_t K = a_nbr ? 2 * k_each : k_each;
        const size_t need = update_fwd_ws_bytes(K, n_out, cap_m, gemm_dt);
        GNN_CHECK(aligned(ws, 256), GNN_EINVAL, "%s: ws must be 256-byte aligned", who);
        GNN_CHECK(ws_bytes >= need, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, ws_bytes, need);
    }
    GNN_CHECK(aligned(wt, 8), GNN_EINVAL, "%s: wt must be 8-byte aligned", who);
    return launch_update_fwd(a_self, a_nbr, adt, k_each, m_dev, cap_m, w, gemm_dt == GNN_BF16 ? wt : nullptr, bias,
                             n_out, relu, gemm_dt, out, odt, ws, stream_of(s));
}

gnn_status gnn_update_bwd_workspace_size(int64_t k, int64_t n_out, int64_t cap_m, gnn_dtype gemm_dt, size_t *bytes) {
    clear_error();
    GNN_CHECK(bytes, GNN_EINVAL, "gnn_update_bwd_workspace_size: bytes is NULL");
    GNN_CHECK(k >= 1 && n_out >= 1 && cap_m >= 0, GNN_EINVAL, "gnn_update_bwd_workspace_size: bad size");
    GNN_CHECK(act_dtype(gemm_dt), GNN_EUNSUPPORTED, "gnn_update_bwd_workspace_size: bad gemm dtype");
    *bytes = update_bwd_ws_bytes(k, n_out, cap_m, gemm_dt);
    return GNN_OK;
}

gnn_status gnn_update_bwd(const void *a_self, const void *a_nbr, gnn_dtype adt, int64_t k_each,
                          const int64_t *m_dev, int64_t cap_m, const float *w, const float *g, int64_t n_out,
                          gnn_dtype gemm_dt, float *dw, float *db, float *d_a, void *ws, size_t ws_bytes,
                          gnn_stream s) {
    clear_error();
    const char *who = "gnn_update_bwd";
    size_t need = 0;
    GNN_TRY(check_update_bwd(a_self, a_nbr, adt, k_each, m_dev, cap_m, w, g, n_out, gemm_dt, dw, db, d_a, &need, who));
    GNN_CHECK(ws && aligned(ws, 256), GNN_EINVAL, "%s: ws must be non-NULL and 256-byte aligned", who);
    GNN_CHECK(ws_bytes >= need, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, ws_bytes, need);
    return launch_update_bwd(a_self, a_nbr, adt, k_each, m_dev, cap_m, w, g, n_out, gemm_dt, dw, db, d_a, ws,
                             nullptr, nullptr, nullptr, 0.f, stream_of(s));
}

gnn_status gnn_softmax_ce_workspace_size(int64_t b, size_t *bytes) {
    clear_error();
    GNN_CHECK(bytes && b >= 0, GNN_EINVAL, "gnn_softmax_ce_workspace_size: bad argument");
    *bytes = softmax_ce_ws_bytes(b);
    return GNN_OK;
}

gnn_status gnn_softmax_ce(const float *logits, int64_t b, int64_t c, const int64_t *labels, const int64_t *targets,
                          float *g_out, float *loss_out, void *ws, size_t ws_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_softmax_ce";
    GNN_CHECK(b >= 0 && c >= 1 && c <= GNN_MAX_DIM, GNN_EINVAL, "%s: bad shape", who);
    GNN_CHECK((logits || b == 0) && (labels || b == 0) && (g_out || b == 0) && loss_out && ws, GNN_EINVAL,
              "%s: NULL pointer", who);
    GNN_CHECK(aligned(logits, 4) && aligned(labels, 8) && aligned(targets, 8) && aligned(g_out, 4) &&
                  aligned(loss_out, 4) && aligned(ws, 4),
              GNN_EINVAL, "%s: misaligned data", who);
    GNN_CHECK(ws_bytes >= softmax_ce_ws_bytes(b), GNN_ESIZE, "%s: workspace too small", who);
    return launch_softmax_ce(logits, b, c, labels, targets, g_out, loss_out, ws, stream_of(s));
}

gnn_status gnn_sgd(float *w, const float *dw, int64_t n, float lr, gnn_stream s) {
    clear_error();
    GNN_CHECK(n >= 0, GNN_EINVAL, "gnn_sgd: negative size");
    GNN_CHECK((w && dw) || n == 0, GNN_EINVAL, "gnn_sgd: NULL pointer");
    GNN_CHECK(aligned(w, 4) && aligned(dw, 4), GNN_EINVAL, "gnn_sgd: misaligned data");
    return launch_sgd(w, dw, n, lr, stream_of(s));
}

gnn_status gnn_train_step_layout(const gnn_model *m, int64_t graph_n, int64_t batch, gnn_step_layout *out) {
    clear_error();
    GNN_TRY(check_model(m, "gnn_train_step_layout"));
    GNN_CHECK(out, GNN_EINVAL, "gnn_train_step_layout: out is NULL");
    GNN_CHECK(graph_n >= 1 && graph_n < (1ll << 31), GNN_EINVAL, "gnn_train_step_layout: bad graph size");
    GNN_CHECK(batch >= 1 && batch <= graph_n, GNN_EINVAL, "gnn_train_step_layout: batch must be in [1, n]");
    return step_layout(m, graph_n, batch, out);
}

gnn_status gnn_train_step_workspace_size(const gnn_model *m, int64_t graph_n, int64_t batch, size_t *bytes) {
    clear_error();
    GNN_CHECK(bytes, GNN_EINVAL, "gnn_train_step_workspace_size: bytes is NULL");
    gnn_step_layout o;
    GNN_TRY(gnn_train_step_layout(m, graph_n, batch, &o));
    *bytes = o.total_bytes;
    return GNN_OK;
}

gnn_status gnn_train_step_workspace_init(const gnn_model *m, int64_t graph_n, int64_t batch, void *ws,
                                         size_t ws_bytes, gnn_stream s) {
    clear_error();
    gnn_step_layout o;
    GNN_TRY(gnn_train_step_layout(m, graph_n, batch, &o));
    GNN_CHECK(ws && aligned(ws, 256), GNN_EINVAL, "gnn_train_step_workspace_init: ws must be 256-byte aligned");
    GNN_CHECK(ws_bytes >= o.total_bytes, GNN_ESIZE, "gnn_train_step_workspace_init: workspace %zu bytes, need %zu",
              ws_bytes, o.total_bytes);
    return launch_sampler_ws_init(static_cast<char *>(ws) + o.sampler_ws, graph_n, stream_of(s));
}

gnn_status gnn_model_sync_shadow(const gnn_model *m, gnn_stream s) {
    clear_error();
    const char *who = "gnn_model_sync_shadow";
    GNN_TRY(check_model(m, who));
    GNN_TRY(check_model_buffers(m, who));
    for (int l = 0; l < m->num_layers; ++l) {
        if (!m->wt[l]) continue;
        const int64_t K = (m->kind == GNN_AGG_GCN_SYM ? 1 : 2) * static_cast<int64_t>(m->dims[l]);
        GNN_TRY(launch_shadow_sync(m->w[l], K, m->dims[l + 1], m->wt[l], stream_of(s)));
    }
    return GNN_OK;
}

namespace {

// Checks shared by the one-call step and its prepare stage.
gnn_status check_prepare_args(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                              gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *targets, int64_t batch,
                              const char *who) {
    GNN_TRY(check_model(m, who));
    GNN_TRY(check_graph(g, who));
    GNN_CHECK(g->n >= 1, GNN_EINVAL, "%s: empty graph", who);
    GNN_CHECK(batch >= 1 && batch <= g->n, GNN_EINVAL, "%s: batch %lld out of [1, n]", who, (long long)batch);
    GNN_CHECK(m->kind != GNN_AGG_GCN_SYM || (gcn_norm && aligned(gcn_norm, 4)), GNN_EINVAL,
              "%s: GCN needs gcn_norm", who);
    GNN_CHECK(tdt == GNN_F32 || tdt == GNN_F16 || (tdt == GNN_BF16 && m->precision == GNN_BF16), GNN_EUNSUPPORTED,
              "%s: table dtype %d is not supported with precision %d", who, tdt, m->precision);
    GNN_CHECK(loc == GNN_LOC_DEVICE || loc == GNN_LOC_HOST_PINNED, GNN_EINVAL, "%s: unknown location", who);
    GNN_CHECK(table && targets, GNN_EINVAL, "%s: NULL pointer", who);
    GNN_CHECK(row_stride >= m->dims[0], GNN_EINVAL, "%s: row_stride below dims[0]", who);
    GNN_CHECK(aligned(targets, 8) && aligned(table, dtype_size(tdt)), GNN_EINVAL, "%s: misaligned data", who);
    return GNN_OK;
}

gnn_status check_compute_args(const gnn_model *m, const int64_t *labels, const float *loss_dev,
                              const int64_t *edges_dev, const char *who) {
    GNN_TRY(check_model_buffers(m, who));
    GNN_CHECK(labels, GNN_EINVAL, "%s: NULL labels", who);
    GNN_CHECK(aligned(labels, 8) && aligned(loss_dev, 4) && aligned(edges_dev, 8), GNN_EINVAL,
              "%s: misaligned data", who);
    return GNN_OK;
}

}  // namespace

gnn_status gnn_train_step(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                          gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *labels,
                          const int64_t *targets, int64_t batch, uint64_t seed, uint64_t step, float lr,
                          float *loss_dev, int64_t *edges_dev, void *ws, size_t ws_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_train_step";
    GNN_TRY(check_prepare_args(m, g, gcn_norm, table, tdt, loc, row_stride, targets, batch, who));
    GNN_TRY(check_compute_args(m, labels, loss_dev, edges_dev, who));
    gnn_step_layout o;
    GNN_TRY(step_layout(m, g->n, batch, &o));
    GNN_CHECK(ws && aligned(ws, 256), GNN_EINVAL, "%s: ws must be non-NULL and 256-byte aligned", who);
    GNN_CHECK(ws_bytes >= o.total_bytes, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, ws_bytes, o.total_bytes);
    const void *t = nullptr;
    GNN_TRY(device_view(table, loc, &t, who));
    return run_train_step(m, g, gcn_norm, t, tdt, loc == GNN_LOC_HOST_PINNED, row_stride, labels, targets, batch, seed, step, lr, loss_dev,
                          edges_dev, ws, stream_of(s));
}

gnn_status gnn_step_prepare_workspace_init(const gnn_model *m, int64_t graph_n, int64_t batch, void *prep_ws,
                                           size_t prep_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_step_prepare_workspace_init";
    gnn_step_layout o;
    GNN_TRY(gnn_train_step_layout(m, graph_n, batch, &o));
    GNN_CHECK(prep_ws && aligned(prep_ws, 256), GNN_EINVAL, "%s: prep_ws must be 256-byte aligned", who);
    GNN_CHECK(prep_bytes >= o.prep_bytes, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, prep_bytes,
              o.prep_bytes);
    return launch_sampler_ws_init(static_cast<char *>(prep_ws) + o.sampler_ws, graph_n, stream_of(s));
}

gnn_status gnn_step_prepare(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                            gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *targets, int64_t batch,
                            uint64_t seed, uint64_t step, void *prep_ws, size_t prep_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_step_prepare";
    GNN_TRY(check_prepare_args(m, g, gcn_norm, table, tdt, loc, row_stride, targets, batch, who));
    gnn_step_layout o;
    GNN_TRY(step_layout(m, g->n, batch, &o));
    GNN_CHECK(prep_ws && aligned(prep_ws, 256), GNN_EINVAL, "%s: prep_ws must be non-NULL and 256-byte aligned", who);
    GNN_CHECK(prep_bytes >= o.prep_bytes, GNN_ESIZE, "%s: workspace %zu bytes, need %zu", who, prep_bytes,
              o.prep_bytes);
    const void *t = nullptr;
    GNN_TRY(device_view(table, loc, &t, who));
    return run_step_prepare(m, g, gcn_norm, t, tdt, loc == GNN_LOC_HOST_PINNED, row_stride, targets, batch, seed, step, prep_ws, stream_of(s));
}

gnn_status gnn_step_compute(const gnn_model *m, int64_t graph_n, const int64_t *labels, int64_t batch, float lr,
                            float *loss_dev, int64_t *edges_dev, void *prep_ws, size_t prep_bytes, void *comp_ws,
                            size_t comp_bytes, gnn_stream s) {
    clear_error();
    const char *who = "gnn_step_compute";
    gnn_step_layout o;
    GNN_TRY(gnn_train_step_layout(m, graph_n, batch, &o));
    GNN_TRY(check_compute_args(m, labels, loss_dev, edges_dev, who));
    GNN_CHECK(prep_ws && aligned(prep_ws, 256) && comp_ws && aligned(comp_ws, 256), GNN_EINVAL,
              "%s: workspaces must be non-NULL and 256-byte aligned", who);
    GNN_CHECK(prep_bytes >= o.prep_bytes && comp_bytes >= o.compute_bytes, GNN_ESIZE,
              "%s: workspaces %zu and %zu bytes, need %zu and %zu", who, prep_bytes, comp_bytes, o.prep_bytes,
              o.compute_bytes);
    return run_step_compute(m, graph_n, labels, batch, lr, loss_dev, edges_dev, prep_ws, comp_ws, stream_of(s));
}

gnn_status gnn_train_steps(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                           gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *labels,
                           const int64_t *targets, int64_t batch, uint64_t seed, uint64_t first_step, int64_t steps,
                           float lr, float *loss_dev, int64_t *edges_dev, void *const *prep_ws, int32_t n_prep,
                           size_t prep_bytes, void *comp_ws, size_t comp_bytes, gnn_stream s, gnn_stream prep_s) {
    clear_error();
    const char *who = "gnn_train_steps";
    GNN_TRY(check_prepare_args(m, g, gcn_norm, table, tdt, loc, row_stride, targets, batch, who));
    GNN_TRY(check_compute_args(m, labels, loss_dev, edges_dev, who));
    GNN_CHECK(steps >= 0 && steps <= (int64_t{1} << 40), GNN_EINVAL, "%s: bad step count %lld", who,
              static_cast<long long>(steps));
    GNN_CHECK(n_prep >= 2 && n_prep <= GNN_MAX_PREPARE_SLOTS && prep_ws, GNN_EINVAL,
              "%s: n_prep must be in [2, %d] with a workspace array", who, GNN_MAX_PREPARE_SLOTS);
    gnn_step_layout o;
    GNN_TRY(step_layout(m, g->n, batch, &o));
    for (int i = 0; i < n_prep; ++i) {
        GNN_CHECK(prep_ws[i] && aligned(prep_ws[i], 256), GNN_EINVAL,
                  "%s: prepare workspace %d must be non-NULL and 256-byte aligned", who, i);
        for (int j = 0; j < i; ++j)
            GNN_CHECK(prep_ws[i] != prep_ws[j], GNN_EINVAL, "%s: prepare workspaces %d and %d are the same", who, j, i);
    }
    GNN_CHECK(comp_ws && aligned(comp_ws, 256), GNN_EINVAL, "%s: comp_ws must be non-NULL and 256-byte aligned", who);
    GNN_CHECK(prep_bytes >= o.prep_bytes && comp_bytes >= o.compute_bytes, GNN_ESIZE,
              "%s: workspaces %zu and %zu bytes, need %zu and %zu", who, prep_bytes, comp_bytes, o.prep_bytes,
              o.compute_bytes);
    const void *t = nullptr;
    GNN_TRY(device_view(table, loc, &t, who));
    return run_train_steps(m, g, gcn_norm, t, tdt, loc == GNN_LOC_HOST_PINNED, row_stride, labels, targets, batch,
                           seed, first_step, steps, lr, loss_dev, edges_dev, prep_ws, n_prep, comp_ws, stream_of(s),
                           stream_of(prep_s));
}

gnn_status gnn_decode_device_errors(int64_t word) {
    clear_error();
    if (word == 0) return GNN_OK;
    char text[256];
    size_t n = 0;
    auto add = [&](const char *what) {
        const int w = snprintf(text + n, sizeof(text) - n, "%s%s", n ? "; " : "", what);
        if (w > 0) n = std::min(sizeof(text) - 1, n + static_cast<size_t>(w));
    };
    if (word & GNN_DEVERR_WAIT) add("a single-pass scan gave up waiting for an earlier workgroup (GNN_DEVERR_WAIT)");
    if (word & GNN_DEVERR_RANGE) add("an index derived from device data was out of range (GNN_DEVERR_RANGE)");
    const int64_t unknown = word & ~static_cast<int64_t>(GNN_DEVERR_WAIT | GNN_DEVERR_RANGE);
    if (unknown) {
        char u[48];
        snprintf(u, sizeof(u), "unknown flags 0x%llx", static_cast<unsigned long long>(unknown));
        add(u);
    }
    return fail(GNN_EDEVICE, "device error flags 0x%llx: %s", static_cast<unsigned long long>(word), text);
}

gnn_status gnn_check_device_errors(const int64_t *word, gnn_stream s) {
    clear_error();
    GNN_CHECK(word && aligned(word, 8), GNN_EINVAL, "gnn_check_device_errors: word must be non-NULL and 8-byte aligned");
    int64_t v = 0;
    GNN_HIP(hipMemcpyAsync(&v, word, sizeof(v), hipMemcpyDeviceToHost, stream_of(s)));
    GNN_HIP(hipStreamSynchronize(stream_of(s)));
    return gnn_decode_device_errors(v);
}

gnn_status gnn_debug_sampler_fault(int64_t silent_row_tile, uint32_t spin_limit) {
    clear_error();
    GNN_CHECK(silent_row_tile >= -1, GNN_EINVAL, "gnn_debug_sampler_fault: silent_row_tile must be >= -1");
    if (silent_row_tile == -1 && spin_limit == 0) {
        set_sampler_fault(-1, samp::kSpinLimit);
        return GNN_OK;
    }
    GNN_CHECK(spin_limit >= 1, GNN_EINVAL, "gnn_debug_sampler_fault: spin_limit must be >= 1");
    set_sampler_fault(silent_row_tile, spin_limit);
    return GNN_OK;
}

}  // extern "C"
