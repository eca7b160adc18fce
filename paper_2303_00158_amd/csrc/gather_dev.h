// Device side of the feature loader (see gather.hip): one job type per
// (table type, output type, vector width) variant.
//
// The rows are cut into 4-element chunks and the flat (row, chunk) space is
// spread over the threads so that consecutive lanes read consecutive bytes of
// a row: each wavefront streams whole rows with 16-byte (fp32) or 8-byte
// (16-bit) accesses.  A pinned host table is read in place over the host
// link (zero copy).
#pragma once

#include "internal.h"

namespace gnn {
namespace gath {

constexpr int kThreads = 256;

struct Args {
    const void *table;
    int64_t row_stride;
    const int64_t *ids;
    const int64_t *n_dev;  // row count on the device, or null for cap
    int64_t cap, dim;
    void *out;
};

template <class T> struct Raw4;
template <> struct Raw4<float> { using type = uint4; };
template <> struct Raw4<uint16_t> { using type = uint2; };

// Same element type on both sides: bit copy of 4-element chunks.
template <class T>
struct Copy4 {
    Args a;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const T *__restrict__ table = static_cast<const T *>(a.table);
        T *__restrict__ out = static_cast<T *>(a.out);
        const int64_t *__restrict__ ids = a.ids;
        const int64_t row_stride = a.row_stride, dim = a.dim;
        using R = typename Raw4<T>::type;
        const int64_t n = a.n_dev ? min(*a.n_dev, a.cap) : a.cap;
        const int64_t chunks = dim >> 2;
        const int64_t total = n * chunks;
        for (int64_t t = blk * kThreads + threadIdx.x; t < total; t += nblk * kThreads) {
            const int64_t r = t / chunks;
            const int64_t c = t - r * chunks;
            const int64_t src = ids[r];
            const R v = *reinterpret_cast<const R *>(table + src * row_stride + c * 4);
            *reinterpret_cast<R *>(out + r * dim + c * 4) = v;
        }
    }
};

// Widening / narrowing gathers on 4-element chunks.
__device__ __forceinline__ float4 load4_table(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ float4 load4_f16(const uint16_t *p) {
    const uint2 v = *reinterpret_cast<const uint2 *>(p);
    return make_float4(f16_to_f32(static_cast<uint16_t>(v.x & 0xffffu)), f16_to_f32(static_cast<uint16_t>(v.x >> 16)),
                       f16_to_f32(static_cast<uint16_t>(v.y & 0xffffu)), f16_to_f32(static_cast<uint16_t>(v.y >> 16)));
}

template <bool SRC_F16, class TOut>
struct Convert4 {
    Args a;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const void *__restrict__ table = a.table;
        TOut *__restrict__ out = static_cast<TOut *>(a.out);
        const int64_t *__restrict__ ids = a.ids;
        const int64_t row_stride = a.row_stride, dim = a.dim;
        const int64_t n = a.n_dev ? min(*a.n_dev, a.cap) : a.cap;
        const int64_t chunks = dim >> 2;
        const int64_t total = n * chunks;
        for (int64_t t = blk * kThreads + threadIdx.x; t < total; t += nblk * kThreads) {
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
};

// Element-wise fallback for rows that are not a whole number of chunks.
template <int TDT, int ODT>
struct Scalar {
    Args a;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const void *__restrict__ table = a.table;
        void *__restrict__ out = a.out;
        const int64_t *__restrict__ ids = a.ids;
        const int64_t row_stride = a.row_stride, dim = a.dim;
        const int64_t n = a.n_dev ? min(*a.n_dev, a.cap) : a.cap;
        const int64_t total = n * dim;
        for (int64_t t = blk * kThreads + threadIdx.x; t < total; t += nblk * kThreads) {
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
};

// Workgroups for `cap` rows of `dim` elements.
inline unsigned grid_for(int64_t cap, int64_t dim, bool vec) {
    const int64_t work = vec ? cap * (dim / 4) : cap * dim;
    int64_t b = ceil_div(work > 0 ? work : 1, kThreads);
    if (b > (1 << 20)) b = 1 << 20;
    return static_cast<unsigned>(b);
}

inline bool vec_ok(const Args &a, int tdt, int odt) {
    return (a.dim % 4 == 0) && (a.row_stride % 4 == 0) && aligned(a.table, 4 * dtype_size(tdt)) &&
           aligned(a.out, 4 * dtype_size(odt));
}

// Calls f(job) with the job of the variant serving tdt -> odt; returns false
// when the pair is not supported.
template <class F>
bool with_job(const Args &a, int tdt, int odt, F &&f) {
    if (vec_ok(a, tdt, odt)) {
        if (tdt == odt && tdt == GNN_F32) return f(Copy4<float>{a}), true;
        if (tdt == odt) return f(Copy4<uint16_t>{a}), true;
        if (tdt == GNN_F32 && odt == GNN_BF16) return f(Convert4<false, uint16_t>{a}), true;
        if (tdt == GNN_F16 && odt == GNN_BF16) return f(Convert4<true, uint16_t>{a}), true;
        if (tdt == GNN_F16 && odt == GNN_F32) return f(Convert4<true, float>{a}), true;
        return false;
    }
    if (tdt == GNN_F32 && odt == GNN_F32) return f(Scalar<GNN_F32, GNN_F32>{a}), true;
    if (tdt == GNN_F32 && odt == GNN_BF16) return f(Scalar<GNN_F32, GNN_BF16>{a}), true;
    if (tdt == GNN_F16 && odt == GNN_F16) return f(Scalar<GNN_F16, GNN_F16>{a}), true;
    if (tdt == GNN_BF16 && odt == GNN_BF16) return f(Scalar<GNN_BF16, GNN_BF16>{a}), true;
    if (tdt == GNN_F16 && odt == GNN_F32) return f(Scalar<GNN_F16, GNN_F32>{a}), true;
    if (tdt == GNN_F16 && odt == GNN_BF16) return f(Scalar<GNN_F16, GNN_BF16>{a}), true;
    return false;
}

}  // namespace gath
}  // namespace gnn
