// Internal declarations shared by the HIP sources of libgnn.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include <algorithm>

#include "gnn.h"

namespace gnn {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
gnn_status fail(gnn_status code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();
gnn_status launch_status(const char *what);  // hipGetLastError after a launch

#define GNN_CHECK(cond, code, ...)                                   \
    do {                                                             \
        if (!(cond)) return ::gnn::fail((code), __VA_ARGS__);        \
    } while (0)
#define GNN_HIP(call)                                                                  \
    do {                                                                               \
        hipError_t e_ = (call);                                                        \
        if (e_ != hipSuccess)                                                          \
            return ::gnn::fail(GNN_EHIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
    } while (0)
#define GNN_TRY(expr)                      \
    do {                                   \
        gnn_status st_ = (expr);           \
        if (st_ != GNN_OK) return st_;     \
    } while (0)
#define GNN_LAUNCHED(what) GNN_TRY(::gnn::launch_status(what))

inline hipStream_t stream_of(gnn_stream s) { return reinterpret_cast<hipStream_t>(s); }

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
__device__ __forceinline__ bool aligned_dev(const void *p, size_t a) {
    return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}
__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t round_up(size_t a, size_t b) { return (a + b - 1) / b * b; }
inline size_t dtype_size(int dt) { return dt == GNN_F32 ? 4 : 2; }

// Carves aligned sub-buffers out of a caller workspace.  With base == nullptr
// it only measures.
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base(static_cast<char *>(b)) {}
    size_t take(size_t bytes, size_t align = 256) {
        off = round_up(off, align);
        size_t at = off;
        off += round_up(bytes, 8);
        return at;
    }
    template <class T>
    T *ptr(size_t at) const { return base ? reinterpret_cast<T *>(base + at) : nullptr; }
};

// Grid limit used for capacity-sized launches (1-D grids up to 2^31-1 blocks).
constexpr int64_t kMaxGrid = (1ll << 31) - 1;

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------
// fp32 -> bf16, round to nearest even; NaNs stay NaN (quiet bit set).
// Written without branches so it vectorises inside unrolled loops.
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    const uint32_t quiet = (u >> 16) | 0x40u;
    return static_cast<uint16_t>(((u & 0x7fffffffu) > 0x7f800000u) ? quiet : rounded);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
    _Float16 v = __builtin_bit_cast(_Float16, h);
    return static_cast<float>(v);
}

// Typed element access: activations are float or raw bf16 bits (uint16_t).
template <class T> struct Elem;
template <> struct Elem<float> {
    __device__ __forceinline__ static float load(const float *p, int64_t i) { return p[i]; }
    __device__ __forceinline__ static void store(float *p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    __device__ __forceinline__ static float load(const uint16_t *p, int64_t i) { return bf16_to_f32(p[i]); }
    __device__ __forceinline__ static void store(uint16_t *p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
};

// Four consecutive elements starting at p[i] (i a multiple of 4 and the row
// 4-element aligned) as floats.
__device__ __forceinline__ float4 load4(const float *p, int64_t i) {
    return *reinterpret_cast<const float4 *>(p + i);
}
__device__ __forceinline__ float4 load4(const uint16_t *p, int64_t i) {
    uint2 v = *reinterpret_cast<const uint2 *>(p + i);
    return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                       __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
}
__device__ __forceinline__ void store4(float *p, int64_t i, float4 v) { *reinterpret_cast<float4 *>(p + i) = v; }
__device__ __forceinline__ void store4(uint16_t *p, int64_t i, float4 v) {
    uint2 o;
    o.x = static_cast<uint32_t>(f32_to_bf16(v.x)) | (static_cast<uint32_t>(f32_to_bf16(v.y)) << 16);
    o.y = static_cast<uint32_t>(f32_to_bf16(v.z)) | (static_cast<uint32_t>(f32_to_bf16(v.w)) << 16);
    *reinterpret_cast<uint2 *>(p + i) = o;
}

__device__ __forceinline__ int64_t dev_count(const int64_t *dev, int64_t fallback) {
    return dev ? *dev : fallback;
}

// ---------------------------------------------------------------------------
// validation helpers (abi.hip)
// ---------------------------------------------------------------------------
gnn_status check_block(const gnn_block *b, bool need_csc, bool need_norm, const char *who);
gnn_status check_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                            int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt,
                            const float *dw, const float *db, const float *d_a, size_t *ws_need, const char *who);

// Internal launchers reused by the training step (no host validation).
gnn_status launch_gather(const void *table, int tdt, int64_t dim, int64_t row_stride, const int64_t *ids,
                         const int64_t *n_ids_dev, int64_t cap_ids, void *out, int odt, bool host, hipStream_t s);
gnn_status launch_aggregate_fwd(const gnn_block *b, int kind, const void *h, int hdt, int64_t f, void *out, int odt,
                                hipStream_t s);
gnn_status launch_aggregate_fwd_dedup(const gnn_block *b, int kind, const void *h, int hdt, int64_t f, void *out,
                                      int odt, hipStream_t s);
gnn_status launch_aggregate_bwd(const gnn_block *b, int kind, const float *d_a, int64_t f, const void *h_below,
                                int hbdt, float *d_src, hipStream_t s);
gnn_status launch_aggregate_fwd_max(const gnn_block *b, const void *h, int hdt, int64_t f, void *out, int odt,
                                    int32_t *argmax, hipStream_t s);
gnn_status launch_aggregate_bwd_max(const gnn_block *b, const int32_t *argmax, const float *d_a, int64_t f,
                                    const void *h_below, int hbdt, float *d_src, hipStream_t s);
// Update GEMMs.  Their workspaces hold fp32 partial tiles of split
// reductions (no state survives a call).  A null forward workspace disables
// the reduction split.
size_t update_fwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt);
// wt (may be null): bf16 shadow W^T (n_out x K) read instead of w in bf16 mode.
gnn_status launch_update_fwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const uint16_t *wt, const float *bias, int64_t n_out,
                             int relu, int gemm_dt, void *out, int odt, void *ws, hipStream_t s);
size_t update_bwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m, int gemm_dt);
// w_upd / b_upd (may be null): SGD applied to them with the final gradients;
// wt_upd (may be null, needs w_upd): its bf16 shadow W^T, refreshed too.
gnn_status launch_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt, float *dw,
                             float *db, float *d_a, void *ws, float *w_upd, float *b_upd, uint16_t *wt_upd, float lr,
                             hipStream_t s);
// Forward of one layer in one launch (fused_layer.hip): aggregation into
// LDS, update on the matrix cores with W^T (bf16 shadow) in registers, and
// for the last layer (last = true) the softmax cross-entropy gradient g and
// row losses of the `batch` target rows instead of an activation.  Writes the
// aggregation output agg_out (bf16) and out (bf16 ReLU(Z), or fp32 logits).
// fused_layer_ok says whether the shapes, precision and alignment allow it.
bool fused_layer_ok(int kind, int precision, int64_t f, int64_t n_out, int64_t cap_dst, int32_t maxdeg, bool last,
                    const void *h, const uint16_t *wt, const void *agg_out);
gnn_status launch_fused_layer(const gnn_block *b, int kind, int32_t maxdeg, const void *h, int64_t f,
                              const uint16_t *wt, const float *bias, int64_t n_out, void *agg_out, void *out,
                              bool last, const int64_t *labels, float *g, float *row_loss, int64_t batch,
                              hipStream_t s);
// The same launch when the aggregation was done beforehand: the A rows are
// [a_self[i] || a_nbr[i]] (GraphSAGE) or a_nbr[i] (GCN), bf16, f wide each
// (a_self may be null for GCN); only the block's row count is read.  Check
// with fused_layer_ok(kind, GNN_BF16, f, n_out, cap_dst, 1, last, a_self or
// a_nbr, wt, a_nbr).
gnn_status launch_fused_update(const gnn_block *b, int kind, const void *a_self, const void *a_nbr, int64_t f,
                               const uint16_t *wt, const float *bias, int64_t n_out, void *out, bool last,
                               const int64_t *labels, float *g, float *row_loss, int64_t batch, hipStream_t s);
// Forward of a two-layer model in one launch (fused_two.hip): layer 1's
// update from its prepared aggregation m1 (and X' rows x_self, GraphSAGE),
// computed per tile for the rows the last block's tile reads, then the last
// layer as launch_fused_layer does with the loss.  Writes h1 (H^1, bf16),
// agg_out (M^2, bf16), the fp32 logits, g, row_loss and, when d_a is given,
// layer 2's input gradient dA^2 = G (W^2)^T (fp32, bf16 operands).  two_layer_ok says
// whether the shapes (f0 % 4 == 0 and K1 <= 256, f1 % 8 == 0 and f1 <= 256,
// n_out <= 64, or <= 48 for GraphSAGE, at most 2,048 destinations),
// precision and alignment allow it.  With the max aggregator, argmax
// (int32, 16-byte aligned, rows x f1) receives M^2's argmax table.
bool two_layer_ok(int kind, int precision, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_dst, int32_t fanout,
                  const void *x_self, const void *m1, const uint16_t *wt1, const uint16_t *wt2, const void *h1,
                  const void *agg_out, const int32_t *argmax);
gnn_status launch_two_layer(const gnn_block *last, int kind, int32_t fanout, const void *x_self, const void *m1,
                            int64_t f0, const uint16_t *wt1, const float *bias1, int64_t f1, void *h1,
                            const uint16_t *wt2, const float *bias2, int64_t n_out, void *agg_out, float *logits,
                            const int64_t *labels, float *g, float *row_loss, int64_t batch, float *d_a,
                            int32_t *argmax, hipStream_t s);
// Backward of a two-layer model below the loss (bwd_two.hip): both layers'
// dW and db, with layer 2's aggregation backward folded into layer 1's dW
// (G^1 never stored).  b2 is layer 2's block with its transpose; layer 1's A
// rows are [x_self || m1] (GraphSAGE) or m1 (GCN), bf16, f0 wide, m1_rows
// (device) of at most cap_m1; h1 is H^1 and agg2 is M^2 (bf16, f1 wide);
// d_a2 and g2 are layer 2's input and output gradients (fp32).  ws holds
// two_bwd_ws_bytes of split partials.  GNN_EUNSUPPORTED when the shapes do
// not take the folded job (bwd_pull_dev.h).
size_t two_bwd_ws_bytes(int kind, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_m1, int64_t cap_m2);
gnn_status launch_two_bwd(const gnn_block *b2, int kind, const void *x_self, const void *m1, int64_t f0,
                          const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1, const void *agg2,
                          const int32_t *arg2, const float *d_a2, const float *g2, int64_t n_out, float *dw1,
                          float *db1, float *dw2, float *db2, void *ws, hipStream_t s);
// The forward of wide layers (gemm_wide.hip): bf16 A rows and the bf16
// shadow W^T, 256 x 256 tiles for the matrix cores.  wide_fwd_ok says
// whether the shapes (K, n_out >= 512, K % 128 == 0, k_each % 64 == 0,
// n_out % 8 == 0), sizes and alignment allow it.
bool wide_fwd_ok(const void *a_self, const void *a_nbr, int adt, int64_t k_each, int64_t cap_m, int64_t n_out,
                 const uint16_t *wt, int gemm_dt, const void *out);
gnn_status launch_wide_fwd(const void *a_self, const void *a_nbr, int64_t k_each, const int64_t *m_dev,
                           int64_t cap_m, const uint16_t *wt, const float *bias, int64_t n_out, int relu, void *out,
                           int odt, void *ws, hipStream_t s);
// Workspace of the wide forward's split reduction (fp32 partial tiles).
size_t wide_fwd_ws_bytes(int64_t n_out, int64_t cap_m);
// wt = bf16(w^T) for a K x n row-major w.
gnn_status launch_shadow_sync(const float *w, int64_t K, int64_t n, uint16_t *wt, hipStream_t s);
size_t softmax_ce_ws_bytes(int64_t b);
gnn_status launch_softmax_ce(const float *logits, int64_t b, int64_t c, const int64_t *labels,
                             const int64_t *targets, float *g_out, float *loss_out, void *ws, hipStream_t s);
gnn_status launch_sgd(float *w, const float *dw, int64_t n, float lr, hipStream_t s);
size_t sampler_ws_bytes(int64_t graph_n, int64_t cap_dst, int32_t fanout);
gnn_status launch_sampler_ws_init(void *ws, int64_t graph_n, hipStream_t s);
// Builds the block's CSR part (ids, row pointer, columns, norms).  With csc
// (the block's transpose arguments, csc_dev.h) the relabel also records the
// edges' rows and counts the columns for a later launch_block_csc.
namespace csc {
struct Args;
}
gnn_status launch_build_block(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids,
                              const int64_t *n_dst_dev, int32_t fanout, uint64_t seed, uint64_t step, int32_t hop,
                              const gnn_block *out, void *ws, const csc::Args *csc, hipStream_t s);
// Error-path test hook: from the next sampler launch on, the row scan's
// tile `silent_row_tile` publishes nothing (-1: none) and its waits give up
// after `spin_limit` polls.
void set_sampler_fault(int64_t silent_row_tile, uint32_t spin_limit);
// Bound on a block's sources (gnn_block_bounds).
int64_t src_bound(int64_t graph_n, int64_t cap_dst, int32_t fanout);
// The transpose scratch inside a sampler workspace (for standalone calls).
void *sampler_csc_ws(void *ws, int64_t graph_n, int64_t cap_dst, int32_t fanout);

}  // namespace gnn
