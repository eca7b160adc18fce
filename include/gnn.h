/*
 * gnn.h -- C ABI of the MI355X (gfx950) sampled-GNN training hot path.
 *
 * One mini-batch iteration of sampled GNN training as the paper describes it
 * (HyScale-GNN, Section II-B and Figure 1): a sampler turns the input graph
 * into one bipartite block per layer, a feature loader gathers the rows of the
 * sampled input vertices (Section III-A, Feature Loader), each layer
 * aggregates neighbour features and applies the update (Section II-A,
 * equations 1-2, with the GCN and GraphSAGE operators), a loss is taken on
 * the target vertices, the same operators run backwards to produce weight
 * gradients, and the weights are updated.
 *
 * Conventions shared by every call:
 *  - Pointers marked [device] are HIP device pointers (from hipMalloc or a
 *    torch CUDA/HIP tensor); [host] pointers are ordinary host memory;
 *    [pinned] is host memory from hipHostMalloc (mapped into the device's
 *    address space).  The caller owns every buffer.  The library never
 *    allocates or frees memory and keeps no pointer after a call returns.
 *  - Every call enqueues its kernels on the given stream (a hipStream_t, or
 *    NULL for the null stream) and returns without synchronising.  Outputs
 *    are valid once the stream reaches that point; inputs must stay alive
 *    until then.
 *  - Counts produced on the device (rows of a block, sampled edges) are read
 *    from device memory by later kernels: no call ever copies them to the
 *    host.  Grids are sized by the host-side capacities and the surplus
 *    workgroups exit at once.
 *  - Matrices are dense row-major with the stated row length; activation
 *    rows of layer l have f^l elements.
 *  - bf16 values are stored as raw 16-bit patterns; narrowing from fp32
 *    rounds to nearest, ties to even.
 *  - Validation (null pointers, alignment, sizes, dtypes, capacities) runs on
 *    the host before anything is enqueued; a failed check returns an error
 *    code and enqueues nothing.  HIP launch failures return GNN_EHIP.  The
 *    text of the last error on the calling thread is in gnn_last_error().
 *    Checks that only the device can make (the sampler's bounded waits and
 *    its range checks) set flags in device memory instead, which
 *    gnn_check_device_errors reads.  Device-content errors (a vertex id >= n,
 *    a label >= C, duplicate targets) are not detected and give undefined
 *    results.
 *  - Calls on different streams may run concurrently when their buffers and
 *    workspaces do not overlap.
 */
#ifndef GNN_H
#define GNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t gnn_status;
#define GNN_OK 0
#define GNN_EINVAL (-1)        /* bad argument: null pointer, negative size, misalignment */
#define GNN_ESIZE (-2)         /* a capacity or workspace is too small */
#define GNN_EHIP (-3)          /* a HIP runtime call or kernel launch failed */
#define GNN_EUNSUPPORTED (-4)  /* valid but unsupported combination (dtype, location) */
#define GNN_EDEVICE (-5)       /* a device-side check failed (gnn_check_device_errors) */

/* Device error flags, as kept in a block's counts[3] and in a training
 * step's error word (gnn_step_layout.error).  A result computed while a flag
 * is set is undefined. */
#define GNN_DEVERR_WAIT 1      /* a single-pass scan's bounded wait for an earlier workgroup gave up */
#define GNN_DEVERR_RANGE 2     /* an index derived from device data fell outside its buffer */

/* Element types, aggregation operators and table locations.  The argument
 * types are plain 32-bit integers (not C enums), so that any value a caller
 * passes is representable and an unknown one is rejected by validation. */
typedef int32_t gnn_dtype;
typedef int32_t gnn_agg;
typedef int32_t gnn_loc;
enum { GNN_F32 = 0, GNN_BF16 = 1, GNN_F16 = 2 };
/* GNN_AGG_SAGE_MAX: GraphSAGE with the max aggregator (Section II-A); its
 * update reads [h_self || max] as the mean model reads [h_self || mean].
 * The model-level calls (gnn_train_step and its stages) take it; the
 * per-operator calls have their own entry points for it
 * (gnn_aggregate_fwd_max, gnn_aggregate_bwd_max). */
enum { GNN_AGG_SAGE_MEAN = 0, GNN_AGG_GCN_SYM = 1, GNN_AGG_SAGE_MAX = 2 };
enum { GNN_LOC_DEVICE = 0, GNN_LOC_HOST_PINNED = 1 };
typedef void *gnn_stream; /* hipStream_t */

#define GNN_MAX_LAYERS 4
#define GNN_MAX_FANOUT 1024
#define GNN_MAX_DIM 65536
#define GNN_ABI_VERSION 2

/* Text of the last error reported on the calling thread ("" if none).  Valid
 * until the next gnn_* call on this thread. */
const char *gnn_last_error(void);
int32_t gnn_abi_version(void);

/* Input graph G(V, E) (Table I): int64 CSR.  Row v lists the stored edges
 * (v, u) -- the neighbours N(v) -- in ascending u; repeated entries
 * (multi-edges) are allowed.  rowptr [device] has n+1 entries, col [device]
 * nnz entries. */
typedef struct gnn_graph {
    int64_t n;
    int64_t nnz;
    const int64_t *rowptr;
    const int64_t *col;
} gnn_graph;

/* GCN normalisation factor per vertex (GCN operator of Section II-A): the
 * degree D(v) is the input-graph degree plus the self loop, and
 * nrm[v] = fp32(1 / sqrt(D(v))) computed in double before narrowing.
 * nrm_out [device] has g->n floats. */
gnn_status gnn_gcn_norm(const gnn_graph *g, float *nrm_out, gnn_stream s);

/* ------------------------------------------------------------------------
 * Mini-batch sampler (Section III-A, Mini-batch Sampler; the GraphSAGE
 * neighbour sampler of Section VI-A).
 *
 * A block is the mini-batch topology G(V^l, E^l) of one layer: n_dst
 * destination rows and n_src sources, where the sources are the destinations
 * (same order) followed by every newly reached vertex in ascending id order.
 * Row i lists the local source index of each sampled neighbour of dst i, in
 * ascending position within i's adjacency row.  The transpose (CSC) lists,
 * for each source j, the rows i that sampled it, ascending.
 *
 * counts [device] int64[4] is written by gnn_build_block:
 *   counts[0] = n_dst, counts[1] = n_src, counts[2] = nnz (sampled edges),
 *   counts[3] = device error flags of the build (GNN_DEVERR_*; 0 when the
 *   block is valid): GNN_DEVERR_WAIT when a workgroup of the row-pointer,
 *   new-source or transpose scan gave up waiting for an earlier one (every
 *   wait is bounded, so the build always finishes), GNN_DEVERR_RANGE when a
 *   local index or transpose position fell outside the block's capacities
 *   (the access is skipped).  Read it with gnn_check_device_errors.
 * ------------------------------------------------------------------------ */
typedef struct gnn_block {
    int64_t cap_dst;   /* [host] capacity of destination rows */
    int64_t cap_src;   /* [host] capacity of src_ids / cscptr rows */
    int64_t cap_nnz;   /* [host] capacity of sampled edges */
    int64_t *counts;   /* [device] int64[4], see above */
    int64_t *src_ids;  /* [device] int64[cap_src]: global vertex id of each local source */
    int64_t *rowptr;   /* [device] int64[cap_dst + 1] */
    int32_t *col;      /* [device] int32[cap_nnz]: local source index per sampled edge */
    int64_t *cscptr;   /* [device] int64[cap_src + 1], or NULL when no transpose is wanted */
    int32_t *cscrow;   /* [device] int32[cap_nnz], or NULL together with cscptr */
    float *src_norm;   /* [device] float[cap_src]: GCN nrm of each source, or NULL */
} gnn_block;

/* Capacities that always suffice for a block of cap_dst destinations with the
 * given fanout in a graph of graph_n vertices:
 *   cap_nnz = cap_dst * fanout, cap_src = min(cap_dst + cap_nnz, graph_n). */
gnn_status gnn_block_bounds(int64_t graph_n, int64_t cap_dst, int32_t fanout, int64_t *cap_src, int64_t *cap_nnz);

/* Workspace of gnn_build_block.  It holds a per-vertex map and two
 * per-vertex bitmaps; the bitmaps must be zeroed once with
 * gnn_sampler_workspace_init and every gnn_build_block call leaves them zero
 * again.  One workspace serves any number of sequential calls on one
 * stream (calls that share it must not overlap). */
gnn_status gnn_sampler_workspace_size(int64_t graph_n, int64_t cap_dst, int32_t fanout, size_t *bytes);
gnn_status gnn_sampler_workspace_init(void *ws, size_t ws_bytes, int64_t graph_n, gnn_stream s);

/* Build one block (one hop of the sampler; hop 1 is sampled around the
 * targets and yields the block of the last layer).
 *   dst_ids   [device] destination vertex ids, distinct.
 *   n_dst_dev [device] int64 count of dst_ids, or NULL to use out->cap_dst
 *             (e.g. the targets of hop 1; for later hops pass the previous
 *             block's &counts[1]).
 *   fanout    k in [1, GNN_MAX_FANOUT].  Every dst vertex v with degree d
 *             keeps all d neighbours when d <= k, else k positions drawn
 *             without replacement by Floyd's algorithm, where draw t of
 *             vertex v is Lemire's multiply-shift of the key
 *             mix(mix(mix(mix(mix(seed)^step)^hop)^v)^t) (mix = the
 *             SplitMix64 output function) into [0, d-k+t].
 *   gcn_norm  [device] per-vertex norms (gnn_gcn_norm) to fill
 *             out->src_norm, or NULL.
 *   want_csc  nonzero to also build out->cscptr / out->cscrow.
 * Degrees must be below 2^32 and n below 2^31. */
gnn_status gnn_build_block(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids,
                           const int64_t *n_dst_dev, int32_t fanout, uint64_t seed, uint64_t step, int32_t hop,
                           int32_t want_csc, gnn_block *out, void *ws, size_t ws_bytes, gnn_stream s);

/* ------------------------------------------------------------------------
 * Feature loader (Section III-A; the Feature Loading and Data Transfer
 * stages of Section III-B): X' = X[ids].
 *   table      [device] or [pinned] (loc) n_rows x row_stride elements of tdt.
 *   ids        [device] int64 row ids; n_ids_dev [device] their count, or
 *              NULL to use cap_ids.
 *   out        [device] cap_ids x dim elements of odt.
 * Supported (tdt -> odt): F32->F32, F32->BF16, F16->F16, F16->F32,
 * F16->BF16, BF16->BF16.  Same-type copies are bit copies.  A pinned table is
 * read directly over the host link by the gather kernel (zero copy).
 * ------------------------------------------------------------------------ */
gnn_status gnn_gather_features(const void *table, gnn_dtype tdt, gnn_loc loc, int64_t n_rows, int64_t dim,
                               int64_t row_stride, const int64_t *ids, const int64_t *n_ids_dev, int64_t cap_ids,
                               void *out, gnn_dtype odt, gnn_stream s);

/* ------------------------------------------------------------------------
 * Aggregation (equation 1; GCN and GraphSAGE operators of Section II-A).
 *   h_src [device] block->cap_src x f (hdt in {F32, BF16}); row j is source j.
 *   out   [device] block->cap_dst x f (odt in {F32, BF16}).
 *   SAGE: out[i] = mean of h_src[col] over row i (zero when row i is empty).
 *   GCN:  out[i] = nrm_i^2 h_src[i] + sum over row i of nrm_i nrm_j h_src[j],
 *         each weight one fp32 product of block->src_norm entries.
 * Sums are accumulated in fp32.
 * ------------------------------------------------------------------------ */
gnn_status gnn_aggregate_fwd(const gnn_block *b, gnn_agg kind, const void *h_src, gnn_dtype hdt, int64_t f,
                             void *out, gnn_dtype odt, gnn_stream s);

/* The same aggregation with source reuse inside tiles of 16 destination
 * rows: Section IV-C's feature duplicator (each source's feature vector is
 * fetched once and handed to every destination that samples it).  A tile's
 * column indices are deduplicated in LDS, each distinct source's features
 * are read from HBM once per tile, and every row sums from LDS.  The sums
 * follow gnn_aggregate_fwd's order term for term, so the output is bitwise
 * the same; memory traffic is the tiles' distinct sources rather than their
 * edges, which pays where destinations share sources (hub-heavy blocks).
 * Arguments, layouts and errors as gnn_aggregate_fwd; tiles of more than
 * 512 edges read their sources directly. */
gnn_status gnn_aggregate_fwd_dedup(const gnn_block *b, gnn_agg kind, const void *h_src, gnn_dtype hdt, int64_t f,
                                   void *out, gnn_dtype odt, gnn_stream s);

/* Backward of the aggregation for layers above the first (the backward pass
 * repeats the forward operators in reverse, Section II-B).  Reads the block's
 * transpose; uses no atomics, so results are bitwise reproducible.
 *   d_a     [device] fp32 rows of the update input gradient: SAGE rows hold
 *           2f values (self part, then neighbour part), GCN rows f values.
 *   h_below [device] block->cap_src x f activations of the layer below
 *           (hbdt F32 or BF16) for the ReLU mask, or NULL for no mask.
 *   d_src   [device] fp32 block->cap_src x f, overwritten:
 *     SAGE: d_src[j] = [j < n_dst] d_a[j, :f] + sum_{i samples j} d_a[i, f:] / deg_i
 *     GCN:  d_src[j] = [j < n_dst] nrm_j^2 d_a[j] + sum_{i samples j} nrm_i nrm_j d_a[i]
 *     then d_src[j] *= 1[h_below[j] > 0] elementwise when h_below is given. */
gnn_status gnn_aggregate_bwd(const gnn_block *b, gnn_agg kind, const float *d_a, int64_t f, const void *h_below,
                             gnn_dtype hbdt, float *d_src, gnn_stream s);

/* GraphSAGE's max aggregator (Section II-A lists mean, max and LSTM as
 * aggregation operators; the update then reads [h_self || max] as the mean
 * path's [h_self || mean]).
 *   h_src   [device] block->cap_src x f of hdt (GNN_F32 or GNN_BF16).
 *   out     [device] block->cap_dst x f of odt (GNN_F32 or GNN_BF16):
 *           out[i, c] = max over row i's edges e of h_src[col[e], c], narrowed
 *           to odt (round to nearest even); 0 for a row without edges.
 *   argmax  [device] int32 block->cap_dst x f, or NULL when the table is
 *           not wanted (no backward follows): the local source id of the
 *           edge that holds out[i, c] (-1 for a row without edges).  The
 *           row's first edge holds the running maximum and a later edge
 *           replaces it only when strictly greater, so ties and duplicate
 *           edges go to the earliest edge, and a NaN counts only as the
 *           row's first edge.
 * The comparisons are exact, so out and argmax are bit for bit those of the
 * sequential rule.  Rows past block->counts[0] are left untouched.
 * Errors: GNN_EINVAL for a bad block, f out of range, NULL or misaligned
 * pointers; GNN_EUNSUPPORTED for other dtypes. */
gnn_status gnn_aggregate_fwd_max(const gnn_block *b, const void *h_src, gnn_dtype hdt, int64_t f, void *out,
                                 gnn_dtype odt, int32_t *argmax, gnn_stream s);

/* Backward of the max aggregator (the forward operators in reverse, Section
 * II-B): the maximum passes its gradient to the source that won it.
 *   argmax  [device] int32 block->cap_dst x f from gnn_aggregate_fwd_max.
 *   d_a     [device] fp32 rows of 2f values (self part, then max part).
 *   h_below, hbdt: the ReLU mask as in gnn_aggregate_bwd, or NULL.
 *   d_src   [device] fp32 block->cap_src x f, overwritten:
 *     d_src[j, c] = [j < n_dst] d_a[j, c] + sum over the distinct rows i that
 *                   sampled j with argmax[i, c] = j of d_a[i, f + c]
 *     then d_src[j, c] *= 1[h_below[j, c] > 0] when h_below is given.
 * Reads the block's transpose (no atomics, bitwise reproducible); each
 * column must list its rows in ascending order, as gnn_build_block makes it,
 * so that a row that sampled j several times counts once.  Sums are fp32.
 * Errors as gnn_aggregate_bwd. */
gnn_status gnn_aggregate_bwd_max(const gnn_block *b, const int32_t *argmax, const float *d_a, int64_t f,
                                 const void *h_below, gnn_dtype hbdt, float *d_src, gnn_stream s);

/* ------------------------------------------------------------------------
 * One layer's forward in one launch, bf16 (equations 1 and 2 together: the
 * aggregation of Section II-A feeding the update, as in the on-chip
 * aggregate -> update datapath of Section IV-C), with the loss of Section
 * II-B in the epilogue for the last layer.
 *   h_src   [device] bf16 block->cap_src x f (row j is source j); f % 4 == 0.
 *   wt      [device] bf16 W^T, n_out x K (K = 2f for SAGE, self rows of W
 *           first; f for GCN), as kept by gnn_model_sync_shadow.  The
 *           reduction is padded to a multiple of 32 with zero A entries
 *           that meet weights of the same row, so a non-finite weight makes
 *           its output column NaN (it is non-finite in any case).
 *   bias    [device] fp32 n_out, or NULL.
 *   agg_out [device] bf16 block->cap_dst x f: written with the aggregation
 *           (the mean for SAGE, the normalised sum for GCN), exactly what
 *           gnn_aggregate_fwd would give up to fp32 summation order.
 *   labels == NULL (hidden layer): out [device] bf16 cap_dst x n_out =
 *           ReLU([h_src[i] || agg[i]] W + b) (SAGE) or ReLU(agg W + b) (GCN),
 *           GEMM operands bf16, fp32 accumulate.
 *   labels != NULL (last layer; n_out <= 64): out [device] fp32 logits
 *           (no ReLU) for the first `batch` rows, whose targets are
 *           block->src_ids[0 .. batch); g_out [device] fp32 batch x n_out =
 *           (softmax - onehot(labels[target])) / batch; row_loss [device] fp32
 *           batch = logsumexp - logit of the label (the loss is their mean).
 *   max_row_len: the block's row-length bound (its fanout); it sizes the
 *           LDS staging of column indices; longer rows stay correct.
 * Returns GNN_EUNSUPPORTED when the weights do not fit the kernel's
 * register tiles (n_out up to 256 with K <= 256, or n_out up to 128 with
 * K <= 512) or the data are not 8-byte aligned; the caller then uses
 * gnn_aggregate_fwd and gnn_update_fwd.
 * ------------------------------------------------------------------------ */
gnn_status gnn_layer_fwd(const gnn_block *b, gnn_agg kind, int32_t max_row_len, const void *h_src, int64_t f,
                         const uint16_t *wt, const float *bias, int64_t n_out, void *agg_out, void *out,
                         const int64_t *labels, int64_t batch, float *g_out, float *row_loss, gnn_stream s);

/* ------------------------------------------------------------------------
 * Both layers of a two-layer model in one launch, bf16: layer 1's update
 * (equation 2) from its prepared aggregation, computed only for the rows
 * the last block reads; the last layer's aggregation and update (equations
 * 1 and 2) with the loss of Section II-B, as gnn_layer_fwd with labels
 * gives them; and layer 2's input gradient (the backward of equation 2).
 *   last    the last layer's block; its sources are layer 1's rows.
 *   fanout  its row-length bound (sizes the LDS staging of its indices;
 *           longer rows stay correct).
 *   x_self  [device] bf16, rows x f0: layer 1's self part of A^1 (X', the
 *           gathered features of layer 1's rows; SAGE only, may be NULL for
 *           GCN).  m1 [device] bf16, rows x f0: layer 1's aggregation.  Row j
 *           is layer-1 row j, for every source id of `last`.  f0 % 4 == 0.
 *   wt1, b1 layer 1's bf16 W^T (f1 x K1, K1 = 2 f0 for SAGE, f0 for GCN;
 *           K1 <= 256) and fp32 bias (or NULL).
 *   h1      [device] bf16, last->cap_src x f1: H^1 = ReLU(A^1 W^1 + b^1),
 *           written for every source row of `last` (each is a destination
 *           or a sampled neighbour); f1 % 8 == 0, f1 <= 256.
 *   wt2, b2 the last layer's bf16 W^T (n_out x K2, K2 = 2 f1 or f1) and
 *           fp32 bias (or NULL); n_out <= 64, and <= 48 for SAGE.
 *   agg_out [device] bf16 last->cap_dst x f1 and logits [device] fp32
 *           last->cap_dst x n_out, labels, batch, g_out and row_loss: as
 *           gnn_layer_fwd with labels.
 *   d_a     [device] fp32 last->cap_dst x K2, or NULL: dA^2 = G (W^2)^T with
 *           bf16 operands, bit for bit what gnn_update_bwd's input gradient
 *           gives for the same g_out and weights (rows from batch on are 0).
 * Bits of h1, agg_out and the logits equal those of gnn_update_fwd (A-load)
 * followed by gnn_layer_fwd.  Needs last->cap_dst <= 2048 and 16-byte
 * aligned wt1 (8 for GCN when f0 % 8 != 0), wt2, agg_out, and m1 / x_self
 * (8 bytes when f0 % 8 != 0); else GNN_EUNSUPPORTED.
 * ------------------------------------------------------------------------ */
gnn_status gnn_two_layer_fwd(const gnn_block *last, gnn_agg kind, int32_t fanout, const void *x_self, const void *m1,
                             int64_t f0, const uint16_t *wt1, const float *b1, int64_t f1, void *h1,
                             const uint16_t *wt2, const float *b2, int64_t n_out, void *agg_out, float *logits,
                             const int64_t *labels, int64_t batch, float *g_out, float *row_loss, float *d_a,
                             gnn_stream s);

/* The same launch for GraphSAGE with the max aggregator (Section II-A): layer
 * 2's aggregation is the elementwise maximum over each destination's sampled
 * H^1 rows, exactly as gnn_aggregate_fwd_max takes it (the first edge holds
 * the running maximum, a later edge replaces it only when strictly greater;
 * 0 and -1 for a row without edges).  Arguments as gnn_two_layer_fwd with
 * GraphSAGE's layout (K1 = 2 f0, K2 = 2 f1, x_self required), plus
 *   argmax  [device] int32 last->cap_dst x f1, 16-byte aligned: the local
 *           source id (row of H^1) of the edge that holds each element of
 *           agg_out, for gnn_aggregate_bwd_max.
 * Bits of h1, agg_out, argmax and the logits equal those of gnn_update_fwd
 * (A-load) followed by gnn_aggregate_fwd_max and gnn_update_fwd.  Shape and
 * alignment limits and errors as gnn_two_layer_fwd (n_out <= 48). */
gnn_status gnn_two_layer_fwd_max(const gnn_block *last, int32_t fanout, const void *x_self, const void *m1, int64_t f0,
                                 const uint16_t *wt1, const float *b1, int64_t f1, void *h1, const uint16_t *wt2,
                                 const float *b2, int64_t n_out, void *agg_out, int32_t *argmax, float *logits,
                                 const int64_t *labels, int64_t batch, float *g_out, float *row_loss, float *d_a,
                                 gnn_stream s);

/* ------------------------------------------------------------------------
 * Backward of a two-layer model below the loss (Section II-B, backward;
 * Section V: layer 1's backward is the update alone), bf16 operands, fp32
 * accumulate: the weight gradients of both layers,
 *   dW^2 = (A^2)^T G^2, db^2 = colsum(G^2)   with A^2 = [H^1 || M^2] (SAGE)
 *                                            or M^2 (GCN), the last block's rows;
 *   G^1  = ReLU'(H^1) (aggregation backward of dA^2 through `last`);
 *   dW^1 = (A^1)^T G^1, db^1 = colsum(G^1)   with A^1 = [x_self || m1] or m1.
 * G^1 is never stored: each workgroup pulls its rows through the block's
 * transpose.  No weights are updated.
 *   last    the last layer's block, with its transpose (cscptr, cscrow) and,
 *           for GCN, src_norm; its sources are layer 1's rows.
 *   x_self, m1, f0   layer 1's A^1 rows as in gnn_two_layer_fwd (bf16).
 *   m1_rows [device] int64 count of layer 1's rows (the first block's
 *           destinations), at most cap_m1 <= last->cap_src.
 *   h1      [device] bf16 H^1 (rows of `last`'s sources) x f1.
 *   agg2    [device] bf16 M^2, last->cap_dst x f1.
 *   d_a2    [device] fp32 dA^2, last->cap_dst x K2 (K2 = 2 f1 SAGE, f1 GCN),
 *           16-byte aligned: the d_a of gnn_two_layer_fwd.
 *   g2      [device] fp32 G^2, last->cap_dst x n_out (rows past the batch 0).
 *   dw1 (K1 x f1), db1 (f1, or NULL), dw2 (K2 x n_out), db2 (n_out, or NULL)
 *           [device] fp32 outputs.
 *   ws      [device] 256-byte aligned workspace of
 *           gnn_two_layer_bwd_workspace_size bytes (split partials; no state
 *           kept between calls; calls sharing it must not overlap).
 * dw1, db1, dw2 and db2 equal, bit for bit, gnn_aggregate_bwd (dA^2 -> G^1,
 * h_below = h1) followed by gnn_update_bwd on each layer with the same caps
 * (cap_m1 for layer 1, last->cap_dst for layer 2).  Needs f1 % 4 == 0 and
 * f1 > 128, K1 <= 256, f0 % 4 == 0, 8-byte aligned bf16 rows and h1;
 * else GNN_EUNSUPPORTED.
 * ------------------------------------------------------------------------ */
gnn_status gnn_two_layer_bwd_workspace_size(gnn_agg kind, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_m1,
                                            int64_t cap_m2, size_t *bytes);
gnn_status gnn_two_layer_bwd(const gnn_block *last, gnn_agg kind, const void *x_self, const void *m1, int64_t f0,
                             const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1,
                             const void *agg2, const float *d_a2, const float *g2, int64_t n_out, float *dw1,
                             float *db1, float *dw2, float *db2, void *ws, size_t ws_bytes, gnn_stream s);

/* The same for GraphSAGE with the max aggregator: layer 2's aggregation
 * backward is gnn_aggregate_bwd_max's (each maximum's gradient to the source
 * that won it, once per destination), folded into layer 1's dW as above.
 *   argmax2 [device] int32 last->cap_dst x f1, 16-byte aligned: the table
 *           gnn_two_layer_fwd_max wrote.
 * Other arguments as gnn_two_layer_bwd with GraphSAGE's layout (x_self
 * required); the workspace is gnn_two_layer_bwd_workspace_size with
 * GNN_AGG_SAGE_MAX.  dw1, db1, dw2 and db2 equal, bit for bit,
 * gnn_aggregate_bwd_max (dA^2 -> G^1, h_below = h1) followed by
 * gnn_update_bwd on each layer.  Limits and errors as gnn_two_layer_bwd. */
gnn_status gnn_two_layer_bwd_max(const gnn_block *last, const void *x_self, const void *m1, int64_t f0,
                                 const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1,
                                 const void *agg2, const int32_t *argmax2, const float *d_a2, const float *g2,
                                 int64_t n_out, float *dw1, float *db1, float *dw2, float *db2, void *ws,
                                 size_t ws_bytes, gnn_stream s);

/* ------------------------------------------------------------------------
 * Update (equation 2): Z = A W + b with A = [a_self || a_nbr] (SAGE) or
 * A = a_self (GCN, a_nbr NULL); K = 2*k_each or k_each.
 *   a_self, a_nbr [device] row-major, row length k_each, adt in {F32, BF16}.
 *   m_dev   [device] int64 row count, or NULL to use cap_m.
 *   w       [device] fp32 K x n_out row-major; bias [device] fp32 n_out or NULL.
 *   wt      [device] NULL, or the bf16 shadow W^T (n_out x K, 8-byte aligned,
 *           as kept by gnn_model_sync_shadow): with gemm_dt GNN_BF16 it is
 *           read instead of w (the same bf16 operand values).  For a bf16
 *           hidden layer (adt = odt = GNN_BF16, relu) whose W^T fits the
 *           fused layer kernel's register tiles, that kernel runs with the A
 *           rows loaded from a_self / a_nbr; a_self and a_nbr must then span
 *           cap_m rows (rows at or past the count may be read, never used),
 *           and the padding note of gnn_layer_fwd applies to wt.
 *   gemm_dt GNN_BF16: operands rounded to bf16, matrix cores, fp32 accumulate;
 *           GNN_F32: fp32 throughout.
 *   out     [device] cap_m x n_out of odt; ReLU applied when relu != 0.
 *   ws      [device] 256-byte aligned workspace of
 *           gnn_update_fwd_workspace_size bytes (the size may be 0), or NULL.
 *           With a workspace, a long reduction over few output tiles may be
 *           split across workgroups; the fp32 partial tiles are then summed
 *           in split order by a second kernel, so results stay bitwise
 *           reproducible.  No state is kept in it between calls; calls
 *           sharing one workspace must not overlap.
 * ------------------------------------------------------------------------ */
gnn_status gnn_update_fwd_workspace_size(int64_t k, int64_t n_out, int64_t cap_m, gnn_dtype gemm_dt, size_t *bytes);
gnn_status gnn_update_fwd(const void *a_self, const void *a_nbr, gnn_dtype adt, int64_t k_each,
                          const int64_t *m_dev, int64_t cap_m, const float *w, const uint16_t *wt, const float *bias,
                          int64_t n_out, int32_t relu, gnn_dtype gemm_dt, void *out, gnn_dtype odt, void *ws,
                          size_t ws_bytes, gnn_stream s);

/* Gradients of the update given g = dLoss/dZ (fp32, cap_m x n_out):
 *   dw = A^T g (K x n_out), db = column sums of g (unrounded, may be NULL),
 *   d_a = g W^T (cap_m x K, fp32) when d_a is not NULL (layers above the
 *   first; Section V, equation T_Trainer: the first layer's backward is the
 *   update alone).  The reduction over rows is split across workgroups; the
 *   fp32 partials go to ws and a second kernel sums them in split order, so
 *   results are bitwise reproducible.  Layers with K and n_out both >= 512
 *   split the rows over more workgroups, so their workspace is larger (up
 *   to 64 partial copies of dW; in bf16 also a bf16 copy of W that dA
 *   reads).  ws [device] must be 256-byte aligned
 *   and hold gnn_update_bwd_workspace_size bytes; no state is kept in it
 *   between calls; calls sharing it must not overlap. */
gnn_status gnn_update_bwd_workspace_size(int64_t k, int64_t n_out, int64_t cap_m, gnn_dtype gemm_dt, size_t *bytes);
gnn_status gnn_update_bwd(const void *a_self, const void *a_nbr, gnn_dtype adt, int64_t k_each,
                          const int64_t *m_dev, int64_t cap_m, const float *w, const float *g, int64_t n_out,
                          gnn_dtype gemm_dt, float *dw, float *db, float *d_a, void *ws, size_t ws_bytes,
                          gnn_stream s);

/* gnn_update_bwd for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, kernels and results, bit for bit, with the dW
 * partials kept in a static device array of the library instead of a
 * caller workspace.  Arguments as gnn_update_bwd without ws / ws_bytes.
 *   - The array holds 32 MiB (GNN_UPDATE_BWD_NOALLOC_MAX_SCRATCH); a shape
 *     whose gnn_update_bwd_workspace_size exceeds it returns GNN_ESIZE and
 *     enqueues nothing.  Each GPU the call runs on keeps its own copy of the
 *     array until the process ends.
 *   - The call never allocates or frees memory.  Its first call on a device
 *     looks up that device's copy (hipGetSymbolAddress, with the device
 *     current); a failed lookup returns GNN_EHIP.
 *   - Every call on one GPU shares that GPU's array: calls that overlap on
 *     one GPU (concurrent streams, or host threads) race and give undefined
 *     results; order them on one stream.  Nothing in the array needs
 *     clearing between calls. */
#define GNN_UPDATE_BWD_NOALLOC_MAX_SCRATCH (32u << 20)
gnn_status gnn_update_bwd_noalloc(const void *a_self, const void *a_nbr, gnn_dtype adt, int64_t k_each,
                                  const int64_t *m_dev, int64_t cap_m, const float *w, const float *g,
                                  int64_t n_out, gnn_dtype gemm_dt, float *dw, float *db, float *d_a,
                                  gnn_stream s);

/* Loss against the ground truth (Section II-B): mean softmax cross-entropy
 * over the b target rows of logits [device] (fp32 b x c).  The label of row
 * i is labels[targets[i]] (labels/targets [device] int64; targets NULL means
 * labels[i]).  Writes g_out [device] fp32 b x c = (softmax - onehot) / b and
 * loss_out [device] fp32 scalar.  ws must hold gnn_softmax_ce_workspace_size
 * bytes. */
gnn_status gnn_softmax_ce_workspace_size(int64_t b, size_t *bytes);
gnn_status gnn_softmax_ce(const float *logits, int64_t b, int64_t c, const int64_t *labels, const int64_t *targets,
                          float *g_out, float *loss_out, void *ws, size_t ws_bytes, gnn_stream s);

/* Plain SGD (synchronous SGD of Section II-B on one device): w -= lr * dw
 * over n fp32 values [device]. */
gnn_status gnn_sgd(float *w, const float *dw, int64_t n, float lr, gnn_stream s);

/* ------------------------------------------------------------------------
 * One whole training iteration (Section II-B, Figure 1): sample L blocks,
 * gather X', L forward layers, loss, backward in reverse order (no input
 * gradient below layer 1), SGD.
 *
 * Storage precision: with precision GNN_BF16, X', the aggregation outputs and
 * hidden activations are stored bf16 and every GEMM operand is rounded to
 * bf16 (fp32 accumulate); logits, gradients and weights stay fp32.  With
 * GNN_F32 everything is fp32.
 *
 * Feature loading: with an fp32 table in device memory and GNN_BF16, layer
 * 1's aggregation reads the table rows it sums (each element rounded to bf16
 * as the gather rounds it, so the result is bitwise that of aggregating X')
 * and X' is gathered only for the destination rows of the input layer's
 * block, which the update and the backward read; otherwise (host table,
 * other dtypes) every source row of X' is gathered.
 * ------------------------------------------------------------------------ */
typedef struct gnn_model {
    int32_t num_layers;                 /* L in [1, GNN_MAX_LAYERS] */
    int32_t kind;                       /* gnn_agg */
    int32_t precision;                  /* GNN_F32 or GNN_BF16 */
    int32_t dims[GNN_MAX_LAYERS + 1];   /* f^0 .. f^L (f^L = number of classes) */
    int32_t fanouts[GNN_MAX_LAYERS];    /* hop order: fanouts[0] is sampled around the targets */
    float *w[GNN_MAX_LAYERS];           /* [device] fp32 K_l x f^l, K_l = 2 f^{l-1} (SAGE mean or max) or
                                           f^{l-1} (GCN) */
    float *b[GNN_MAX_LAYERS];           /* [device] fp32 f^l */
    float *dw[GNN_MAX_LAYERS];          /* [device] fp32 K_l x f^l, written */
    float *db[GNN_MAX_LAYERS];          /* [device] fp32 f^l, written */
    uint16_t *wt[GNN_MAX_LAYERS];       /* [device] optional bf16 shadow f^l x K_l = bf16(W^T), 8-byte aligned,
                                           for GNN_BF16 models (NULL: the GEMMs round W as they load it) */
} gnn_model;

/* Write every non-NULL shadow m->wt[l] = bf16(m->w[l]^T) (round to nearest
 * even).  A model with shadows must be synced once before its first
 * gnn_train_step and after any change to W made outside the library;
 * gnn_train_step's SGD keeps the shadows in step with W.  The forward update
 * reads the shadow instead of W, which gives the same bf16 operand values
 * (Section II-A, equation 2, with operands rounded as in bf16 mode). */
gnn_status gnn_model_sync_shadow(const gnn_model *m, gnn_stream s);

/* Layout of a training step's internal buffers, for sizing and inspection.
 * Block h (1-based hop) is the block of layer L-h+1.
 *
 * The step has two stages: prepare (sampling of all hops, the gather of X'
 * (Section IV-B's first stage) and layer 1's aggregation, which needs no
 * weights) and compute (the rest of the forward, loss, backward and SGD).
 * Each has its own workspace.  Offsets of the prepare buffers (sampler_ws ..
 * x0, agg[1]) are bytes from the prepare workspace, those of the compute
 * buffers (agg[l >= 2] .. loss) bytes from the compute workspace.  The
 * one-call step's workspace (total_bytes) holds the prepare workspace at
 * byte 0 and the compute workspace at byte prep_bytes. */
typedef struct gnn_step_layout {
    size_t total_bytes;                 /* prep_bytes + compute_bytes */
    size_t prep_bytes, compute_bytes;   /* sizes of the two workspaces (multiples of 256) */
    size_t sampler_ws, sampler_ws_bytes;
    int64_t cap_dst[GNN_MAX_LAYERS], cap_src[GNN_MAX_LAYERS], cap_nnz[GNN_MAX_LAYERS]; /* per hop */
    size_t blk_counts[GNN_MAX_LAYERS], blk_src_ids[GNN_MAX_LAYERS], blk_rowptr[GNN_MAX_LAYERS],
        blk_col[GNN_MAX_LAYERS], blk_cscptr[GNN_MAX_LAYERS], blk_cscrow[GNN_MAX_LAYERS],
        blk_src_norm[GNN_MAX_LAYERS]; /* per hop; 0 when absent */
    size_t blk_csc_ws[GNN_MAX_LAYERS]; /* per hop with a transpose: its scratch; else 0 */
    size_t x0;                          /* gathered X' (cap_src of hop L rows; see feature loading) */
    size_t agg[GNN_MAX_LAYERS + 1];     /* per layer l: aggregation output (layer 1's is computed by the
                                           prepare stage and lives in the prepare workspace) */
    size_t h[GNN_MAX_LAYERS + 1];       /* per layer l: H^l (l < L) or logits (l = L) */
    size_t grad[GNN_MAX_LAYERS + 1];    /* per layer l: G^l = dLoss/dZ^l, fp32 */
    size_t d_a[GNN_MAX_LAYERS + 1];     /* per layer l >= 2: dLoss/dA^l, fp32 */
    size_t fwd_ws, fwd_ws_bytes;        /* update-forward workspace */
    size_t bwd_ws, bwd_ws_bytes;        /* update-backward workspace (a region per layer, layer 1 first) */
    size_t loss_ws, loss_ws_bytes;      /* loss workspace */
    size_t edges;                       /* int64 sampled edges of the step */
    size_t error;                       /* int64 device error word (GNN_DEVERR_*): the OR of counts[3] of every
                                           block of every step of the last gnn_train_step, gnn_step_compute or
                                           gnn_train_steps call on this compute workspace */
    size_t loss;                        /* fp32 loss of the step */
    size_t argmax[GNN_MAX_LAYERS + 1];  /* GNN_AGG_SAGE_MAX, per layer l >= 2: int32 argmax table of the
                                           aggregation (rows x f^{l-1}, read by the backward); else 0 */
} gnn_step_layout;

gnn_status gnn_train_step_layout(const gnn_model *m, int64_t graph_n, int64_t batch, gnn_step_layout *out);
gnn_status gnn_train_step_workspace_size(const gnn_model *m, int64_t graph_n, int64_t batch, size_t *bytes);
/* Initialise a step workspace once (sampler state); keep using it for every
 * step with the same model shape, graph size and batch. */
gnn_status gnn_train_step_workspace_init(const gnn_model *m, int64_t graph_n, int64_t batch, void *ws,
                                         size_t ws_bytes, gnn_stream s);

/* One training step.  table/tdt/loc/row_stride as in gnn_gather_features
 * (dim = m->dims[0]); labels [device] int64[graph n]; targets [device]
 * int64[batch] distinct vertex ids; gcn_norm [device] (required for GCN).
 * Writes m->dw, m->db, updates m->w, m->b in place, and writes the loss
 * (loss_dev, fp32) and the number of sampled edges sum_l |E^l| (edges_dev,
 * int64) when those pointers are not NULL. */
gnn_status gnn_train_step(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                          gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *labels,
                          const int64_t *targets, int64_t batch, uint64_t seed, uint64_t step, float lr,
                          float *loss_dev, int64_t *edges_dev, void *ws, size_t ws_bytes, gnn_stream s);

/* The two stages of gnn_train_step as separate calls, so that the prepare
 * stage of step s+1 can run on a second stream while the compute stage of
 * step s runs (two-stage feature prefetching, Section IV-B): with a pinned
 * host table, the transfer of X' over the host link is then hidden behind
 * the GPU's computation.  gnn_step_prepare(..., step=s) followed by
 * gnn_step_compute on the same prepare workspace gives the same results,
 * bit for bit, as gnn_train_step(..., step=s).
 *
 * Ownership and ordering are the caller's: a prepare workspace is written by
 * gnn_step_prepare and read by the gnn_step_compute that consumes it, so the
 * next gnn_step_prepare into it must be ordered after that compute (an event
 * on the compute stream); computes that share a model or a compute
 * workspace must be ordered among themselves.  The prepare stage reads no
 * model buffer (only its shape), so it may run while a compute updates W.
 *
 * gnn_step_prepare_workspace_init: once per prepare workspace (sampler
 *   state), as gnn_train_step_workspace_init for the one-call workspace.
 * gnn_step_prepare: arguments as gnn_train_step; writes the blocks, their
 *   transposes, X' and layer 1's aggregation into prep_ws (prep_bytes >=
 *   layout.prep_bytes).
 * gnn_step_compute: graph_n and batch as given to gnn_step_prepare; labels
 *   [device] int64[graph_n]; the targets are read back from prep_ws (the
 *   first batch sources of hop 1); writes m->dw, m->db, updates m->w, m->b
 *   (and shadows), loss_dev and edges_dev as gnn_train_step.  comp_ws
 *   (comp_bytes >= layout.compute_bytes) needs no initialisation. */
gnn_status gnn_step_prepare_workspace_init(const gnn_model *m, int64_t graph_n, int64_t batch, void *prep_ws,
                                           size_t prep_bytes, gnn_stream s);
gnn_status gnn_step_prepare(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                            gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *targets, int64_t batch,
                            uint64_t seed, uint64_t step, void *prep_ws, size_t prep_bytes, gnn_stream s);
gnn_status gnn_step_compute(const gnn_model *m, int64_t graph_n, const int64_t *labels, int64_t batch, float lr,
                            float *loss_dev, int64_t *edges_dev, void *prep_ws, size_t prep_bytes, void *comp_ws,
                            size_t comp_bytes, gnn_stream s);

/* Several training steps, pipelined: the prepare stages of later steps run
 * on prep_s while the compute stages of earlier ones run on s (the sampler /
 * feature loader / trainer pipeline of Section III-A and the two-stage
 * feature prefetching of Section IV-B, on one device).  Step i
 * (0 <= i < steps) has step number first_step + i and targets
 * targets[i * batch .. (i+1) * batch) ([device] int64, steps x batch, each
 * row distinct vertex ids).  Results are those of `steps` gnn_train_step
 * calls in order, bit for bit: the prepare stage reads no model buffer, and
 * the computes run in step order on s.
 *
 * Steps go in groups of G = max(1, n_prep / 2): the prepares of group q+1
 * overlap the computes of group q, and the two streams synchronise once per
 * group (stream events cost the host more than a launch, so a larger G
 * lowers the host cost per step; 8 slots give G = 4).
 * prep_ws: n_prep (2 .. GNN_MAX_PREPARE_SLOTS) distinct prepare workspaces of
 *   prep_bytes each, initialised with gnn_step_prepare_workspace_init.
 *   comp_ws: one compute workspace (comp_bytes).
 * loss_dev: NULL or [device] fp32[steps]; edges_dev: NULL or [device]
 *   int64[steps]: per-step loss and sampled-edge count.
 * Ordering: the first prepares wait for the work enqueued on s before the
 *   call; every compute is on s, so work enqueued on s after the call runs
 *   after all steps.  The call never waits on the host; it creates and
 *   releases its own events.  prep_s may equal s (no overlap). */
#define GNN_MAX_PREPARE_SLOTS 8
gnn_status gnn_train_steps(const gnn_model *m, const gnn_graph *g, const float *gcn_norm, const void *table,
                           gnn_dtype tdt, gnn_loc loc, int64_t row_stride, const int64_t *labels,
                           const int64_t *targets, int64_t batch, uint64_t seed, uint64_t first_step, int64_t steps,
                           float lr, float *loss_dev, int64_t *edges_dev, void *const *prep_ws, int32_t n_prep,
                           size_t prep_bytes, void *comp_ws, size_t comp_bytes, gnn_stream s, gnn_stream prep_s);

/* ------------------------------------------------------------------------
 * Device-side errors.
 *
 * gnn_decode_device_errors: host only.  Returns GNN_OK for word == 0, else
 *   GNN_EDEVICE with gnn_last_error() naming every flag set (unknown bits
 *   are reported as such).
 * gnn_check_device_errors: waits for the work enqueued on s, reads the int64
 *   word [device] (a block's &counts[3], or the step's error word at
 *   layout.error in the compute workspace, which for gnn_train_step is at
 *   byte prep_bytes + layout.error of its workspace), and decodes it as
 *   above.  This call synchronises the host with the stream.
 * ------------------------------------------------------------------------ */
gnn_status gnn_decode_device_errors(int64_t word);
gnn_status gnn_check_device_errors(const int64_t *word, gnn_stream s);

/* Test hook for the device error path, not for production use: from the
 * next sampler launch on (gnn_build_block and the training steps), row tile
 * silent_row_tile (256 destination rows each) of the row-pointer scan
 * publishes nothing, so the tile after it waits, and every row-scan wait
 * gives up after spin_limit polls and flags GNN_DEVERR_WAIT.  The block's
 * contents are then undefined.  gnn_debug_sampler_fault(-1, 0) restores
 * normal operation (the default poll limit).  Process-wide; not thread-safe
 * against concurrent sampler calls. */
gnn_status gnn_debug_sampler_fault(int64_t silent_row_tile, uint32_t spin_limit);

#ifdef __cplusplus
}
#endif

#endif /* GNN_H */
