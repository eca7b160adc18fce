// Feature loader: X' = X[ids] with an optional narrowing to bf16.
//
// The rows are cut into 4-element chunks and the flat (row, chunk) space is
// spread over the threads so that consecutive lanes read consecutive bytes of
// a row: each wavefront streams whole rows with 16-byte (fp32) or 8-byte
// (16-bit) accesses.  A pinned host table is read in place over the host
// link (zero copy).
#include "internal.h"

namespace gnn {

namespace {

constexpr int kThreads = 256;

template <class T> struct Raw4;
template <> struct Raw4<float> { using type = uint4; };
template <> struct Raw4<uint16_t> { using type = uint2; };

// Same element type on both sides: bit copy of 4-element chunks.
template <class T>
__global__ void __launch_bounds__(kThreads) gather_copy4_kernel(const T *__restrict__ table, int64_t row_stride,
                                                                 const int64_t *__restrict__ ids,
                                                                 const int64_t *n_dev, int64_t cap, int64_t dim,
                                                                 T *__restrict__ out) {
    using R = typename Raw4<T>::type;
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t chunks = dim >> 2;
    const int64_t total = n * chunks;
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; t < total;
         t += static_cast<int64_t>(gridDim.x) * kThreads) {
        const int64_t r = t / chunks;
        const int64_t c = t - r * chunks;
        const int64_t src = ids[r];
        const R v = *reinterpret_cast<const R *>(table + src * row_stride + c * 4);
        *reinterpret_cast<R *>(out + r * dim + c * 4) = v;
    }
}

// Widening / narrowing gathers on 4-element chunks.
__device__ __forceinline__ float4 load4_table(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ float4 load4_f16(const uint16_t *p) {
    const uint2 v = *reinterpret_cast<const uint2 *>(p);
    return make_float4(f16_to_f32(static_cast<uint16_t>(v.x & 0xffffu)), f16_to_f32(static_cast<uint16_t>(v.x >> 16)),
                       f16_to_f32(static_cast<uint16_t>(v.y & 0xffffu)), f16_to_f32(static_cast<uint16_t>(v.y >> 16)));
}

template <bool SRC_F16, class TOut>
__global__ void __launch_bounds__(kThreads) gather_convert4_kernel(const void *__restrict__ table,
                                                                    int64_t row_stride,
                                                                    const int64_t *__restrict__ ids,
                                                                    const int64_t *n_dev, int64_t cap, int64_t dim,
                                                                    TOut *__restrict__ out) {
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t chunks = dim >> 2;
    const int64_t total = n * chunks;
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; t < total;
         t += static_cast<int64_t>(gridDim.x) * kThreads) {
        const int64_t r = t / chunks;
        const int64_t c = t - r * chunks;
        const int64_t src = ids[r];
        const int64_t off = src * row_stride + c * 4;
        float4 v;
        if constexpr (SRC_F16)
            v = load4_f16(static_cast<const uint16_t *>(table) + off);
        else
            v = load4_table(static_cast<const float *>(table) + off);
        store4(out, r * dim + c * 4, v);
    }
}

// Element-wise fallback for rows that are not a whole number of chunks.
template <int TDT, int ODT>
__global__ void __launch_bounds__(kThreads) gather_scalar_kernel(const void *__restrict__ table, int64_t row_stride,
                                                                  const int64_t *__restrict__ ids,
                                                                  const int64_t *n_dev, int64_t cap, int64_t dim,
                                                                  void *__restrict__ out) {
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t total = n * dim;
    for (int64_t t = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; t < total;
         t += static_cast<int64_t>(gridDim.x) * kThreads) {
        const int64_t r = t / dim;
        const int64_t c = t - r * dim;
        const int64_t off = ids[r] * row_stride + c;
        if constexpr (TDT == ODT) {
            if constexpr (TDT == GNN_F32)
                static_cast<uint32_t *>(out)[t] = static_cast<const uint32_t *>(table)[off];
            else
                static_cast<uint16_t *>(out)[t] = static_cast<const uint16_t *>(table)[off];
        } else {
            float x;
            if constexpr (TDT == GNN_F32)
                x = static_cast<const float *>(table)[off];
            else
                x = f16_to_f32(static_cast<const uint16_t *>(table)[off]);
            if constexpr (ODT == GNN_F32)
                static_cast<float *>(out)[t] = x;
            else
                static_cast<uint16_t *>(out)[t] = f32_to_bf16(x);
        }
    }
}

unsigned gather_grid(int64_t work) {
    int64_t b = ceil_div(work > 0 ? work : 1, kThreads);
    if (b > (1 << 20)) b = 1 << 20;
    return static_cast<unsigned>(b);
}

}  // namespace

gnn_status launch_gather(const void *table, int tdt, int64_t dim, int64_t row_stride, const int64_t *ids,
                         const int64_t *n_ids_dev, int64_t cap_ids, void *out, int odt, hipStream_t s) {
    if (cap_ids == 0 || dim == 0) return GNN_OK;
    const size_t tsz = dtype_size(tdt), osz = dtype_size(odt);
    const bool vec = (dim % 4 == 0) && (row_stride % 4 == 0) && aligned(table, 4 * tsz) && aligned(out, 4 * osz);
    if (vec) {
        const unsigned grid = gather_grid(cap_ids * (dim / 4));
        if (tdt == odt && tdt == GNN_F32)
            gather_copy4_kernel<float><<<grid, kThreads, 0, s>>>(static_cast<const float *>(table), row_stride, ids,
                                                                 n_ids_dev, cap_ids, dim, static_cast<float *>(out));
        else if (tdt == odt)
            gather_copy4_kernel<uint16_t><<<grid, kThreads, 0, s>>>(static_cast<const uint16_t *>(table), row_stride,
                                                                    ids, n_ids_dev, cap_ids, dim,
                                                                    static_cast<uint16_t *>(out));
        else if (tdt == GNN_F32 && odt == GNN_BF16)
            gather_convert4_kernel<false, uint16_t><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                              cap_ids, dim,
                                                                              static_cast<uint16_t *>(out));
        else if (tdt == GNN_F16 && odt == GNN_BF16)
            gather_convert4_kernel<true, uint16_t><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                             cap_ids, dim,
                                                                             static_cast<uint16_t *>(out));
        else if (tdt == GNN_F16 && odt == GNN_F32)
            gather_convert4_kernel<true, float><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev, cap_ids,
                                                                          dim, static_cast<float *>(out));
        else
            return fail(GNN_EUNSUPPORTED, "gather: unsupported dtype pair %d -> %d", tdt, odt);
    } else {
        const unsigned grid = gather_grid(cap_ids * dim);
        if (tdt == GNN_F32 && odt == GNN_F32)
            gather_scalar_kernel<GNN_F32, GNN_F32><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                             cap_ids, dim, out);
        else if (tdt == GNN_F32 && odt == GNN_BF16)
            gather_scalar_kernel<GNN_F32, GNN_BF16><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                              cap_ids, dim, out);
        else if (tdt == GNN_F16 && odt == GNN_F16)
            gather_scalar_kernel<GNN_F16, GNN_F16><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                             cap_ids, dim, out);
        else if (tdt == GNN_BF16 && odt == GNN_BF16)
            gather_scalar_kernel<GNN_BF16, GNN_BF16><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                               cap_ids, dim, out);
        else if (tdt == GNN_F16 && odt == GNN_F32)
            gather_scalar_kernel<GNN_F16, GNN_F32><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                             cap_ids, dim, out);
        else if (tdt == GNN_F16 && odt == GNN_BF16)
            gather_scalar_kernel<GNN_F16, GNN_BF16><<<grid, kThreads, 0, s>>>(table, row_stride, ids, n_ids_dev,
                                                                              cap_ids, dim, out);
        else
            return fail(GNN_EUNSUPPORTED, "gather: unsupported dtype pair %d -> %d", tdt, odt);
    }
    GNN_LAUNCHED("gather");
    return GNN_OK;
}

}  // namespace gnn
