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

// Widening / narrowing of a 4-element chunk.
__device__ __forceinline__ float4 load4_table(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ __forceinline__ float4 load4_f16(const uint16_t *p) {
    const uint2 v = *reinterpret_cast<const uint2 *>(p);
    return make_float4(f16_to_f32(static_cast<uint16_t>(v.x & 0xffffu)), f16_to_f32(static_cast<uint16_t>(v.x >> 16)),
                       f16_to_f32(static_cast<uint16_t>(v.y & 0xffffu)), f16_to_f32(static_cast<uint16_t>(v.y >> 16)));
}

// Rows of dim = 4C elements.  A wavefront is cut into S = 64 / C slots of C
// lanes (C <= 64; wider rows take ceil(C / 64) passes with S = 1), each slot
// copying one row per pass; U passes are unrolled so that U rows' id loads,
// then U rows' data loads, are in flight together.  Lanes past S * C idle.
struct RowSlots {
    int64_t C;      // chunks per row
    int S, passes;  // slots per wavefront; lane groups per row (C > 64)
    __host__ static RowSlots of(int64_t dim) {
        RowSlots r;
        r.C = dim / 4;
        r.S = r.C <= 64 ? static_cast<int>(64 / r.C) : 1;
        r.passes = r.C <= 64 ? 1 : static_cast<int>(ceil_div(r.C, 64));
        return r;
    }
};

constexpr int kUnroll = 4;

// An empty use of a loaded value: keeps the compiler from sinking the load
// into the conditional store that consumes it (which would serialise the
// unrolled rows' loads).
__device__ __forceinline__ void keep(const uint2 &v) { asm volatile("" : : "v"(v.x), "v"(v.y)); }
__device__ __forceinline__ void keep(const uint4 &v) { asm volatile("" : : "v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w)); }
__device__ __forceinline__ void keep(const float4 &v) { asm volatile("" : : "v"(v.x), "v"(v.y), "v"(v.z), "v"(v.w)); }

// The copy loop shared by the vector variants: load(off) reads the 4
// elements at table offset off, store(off, v) writes them to out.
template <class Load, class Store>
__device__ __forceinline__ void gather_rows(const Args &a, const RowSlots &rs, int64_t blk, int64_t nblk, Load &&load,
                                            Store &&store) {
    const int lane = threadIdx.x & 63;
    const int slot = lane / static_cast<int>(rs.C <= 64 ? rs.C : 64);
    const int64_t n = a.n_dev ? min(*a.n_dev, a.cap) : a.cap;
    if (n <= 0) return;  // ids[0] below is only valid when there is a row
    const int64_t waves = nblk * (kThreads / 64);
    const int64_t wave = blk * (kThreads / 64) + (threadIdx.x >> 6);
    const int64_t slots = waves * rs.S;
    for (int p = 0; p < rs.passes; ++p) {
        const int64_t c = (rs.C <= 64 ? lane % rs.C : lane) + p * 64;
        const bool lane_ok = slot < rs.S && c < rs.C;
        // kUnroll consecutive rows r0 .. r0 + kUnroll - 1 per slot and pass;
        // rows past n re-read row 0's id and store nothing
        for (int64_t r0 = (wave * rs.S + slot) * kUnroll; r0 < n; r0 += slots * kUnroll) {
            int64_t id[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int64_t r = r0 + u;
                id[u] = a.ids[r < n ? r : 0];
            }
            decltype(load(0)) v[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) v[u] = load(id[u] * a.row_stride + (lane_ok ? c : 0) * 4);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) keep(v[u]);
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int64_t r = r0 + u;
                if (lane_ok && r < n) store(r * a.dim + c * 4, v[u]);
            }
        }
    }
}

// Same element type on both sides: bit copy of 4-element chunks.
template <class T>
struct Copy4 {
    Args a;
    RowSlots rs;
    __device__ void run(int64_t blk, int64_t nblk) const {
        using R = typename Raw4<T>::type;
        const T *__restrict__ table = static_cast<const T *>(a.table);
        T *__restrict__ out = static_cast<T *>(a.out);
        gather_rows(
            a, rs, blk, nblk, [&](int64_t off) { return *reinterpret_cast<const R *>(table + off); },
            [&](int64_t off, R v) { *reinterpret_cast<R *>(out + off) = v; });
    }
};

template <bool SRC_F16, class TOut>
struct Convert4 {
    Args a;
    RowSlots rs;
    __device__ void run(int64_t blk, int64_t nblk) const {
        TOut *__restrict__ out = static_cast<TOut *>(a.out);
        if constexpr (SRC_F16) {
            const uint16_t *__restrict__ table = static_cast<const uint16_t *>(a.table);
            gather_rows(
                a, rs, blk, nblk, [&](int64_t off) { return *reinterpret_cast<const uint2 *>(table + off); },
                [&](int64_t off, uint2 v) {
                    store4(out, off,
                           make_float4(f16_to_f32(static_cast<uint16_t>(v.x & 0xffffu)),
                                       f16_to_f32(static_cast<uint16_t>(v.x >> 16)),
                                       f16_to_f32(static_cast<uint16_t>(v.y & 0xffffu)),
                                       f16_to_f32(static_cast<uint16_t>(v.y >> 16))));
                });
        } else {
            const float *__restrict__ table = static_cast<const float *>(a.table);
            gather_rows(
                a, rs, blk, nblk, [&](int64_t off) { return load4_table(table + off); },
                [&](int64_t off, float4 v) { store4(out, off, v); });
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

// Workgroups for `cap` rows of `dim` elements: the vector variants give
// each slot kUnroll rows; the scalar one a thread per element.
// A table in pinned host memory is read over the host link, which a few
// hundred wavefronts with several rows in flight each already saturate; a
// grid sized by the row count would hold every compute unit waiting on the
// link and keep concurrent work (the compute stage of the previous step) off
// the GPU.
constexpr int64_t kHostGrid = 256;

inline unsigned grid_for(int64_t cap, int64_t dim, bool vec, bool host) {
    int64_t b;
    if (vec) {
        const RowSlots rs = RowSlots::of(dim);
        b = ceil_div(cap > 0 ? cap : 1, static_cast<int64_t>(rs.S) * (kThreads / 64) * kUnroll);
    } else {
        b = ceil_div(cap * dim > 0 ? cap * dim : 1, kThreads);
    }
    // rows are strided over the grid: 2048 workgroups cover the row counts
    // of the workloads here in one or two rounds without dispatching
    // workgroups that would only read the row count and exit
    if (b > 2048) b = 2048;
    if (host && b > kHostGrid) b = kHostGrid;
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
        const RowSlots rs = RowSlots::of(a.dim);
        if (tdt == odt && tdt == GNN_F32) return f(Copy4<float>{a, rs}), true;
        if (tdt == odt) return f(Copy4<uint16_t>{a, rs}), true;
        if (tdt == GNN_F32 && odt == GNN_BF16) return f(Convert4<false, uint16_t>{a, rs}), true;
        if (tdt == GNN_F16 && odt == GNN_BF16) return f(Convert4<true, uint16_t>{a, rs}), true;
        if (tdt == GNN_F16 && odt == GNN_F32) return f(Convert4<true, float>{a, rs}), true;
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
