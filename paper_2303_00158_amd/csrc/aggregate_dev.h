// Device side of the neighbour aggregation over a sampled block, forward (pull over the block
// CSR) and backward (pull over its transpose, no atomics): the mean and GCN
// sums, and GraphSAGE's max aggregator with its argmax table.
//
// Work split: one wavefront per output row.  A row of f elements is cut into
// C = ceil(f / 4) chunks of 4; when C <= 32 the wavefront is divided into
// S = 64 / C slots that walk different edges of the row at once (f = 100:
// two slots of 25 lanes), and the slot partial sums are folded with lane
// shuffles at the end.  Up to 64 neighbour indices and weights of the row are
// held one per lane and broadcast with shuffles.  Sums are fp32.
#pragma once

#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "internal.h"

namespace gnn {
namespace agg {

template <class T> struct Tag {
    using type = T;
};

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// Elements e0 .. e0+3 of a row starting at row_off (zero past f).  Loads are
// issued unconditionally from in-bounds addresses and masked afterwards.
template <bool VEC, class T>
__device__ __forceinline__ float4 load_chunk(const T *p, int64_t row_off, int64_t e0, int64_t f) {
    if constexpr (VEC) return load4(p, row_off + e0);
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const bool ok = e0 + q < f;
        const float x = Elem<T>::load(p, row_off + (ok ? e0 + q : f - 1));
        v[q] = ok ? x : 0.f;
    }
    return make_float4(v[0], v[1], v[2], v[3]);
}

template <bool VEC, class T>
__device__ __forceinline__ void store_chunk(T *p, int64_t row_off, int64_t e0, int64_t f, float4 v) {
    if constexpr (VEC) {
        store4(p, row_off + e0, v);
        return;
    }
    const float a[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (e0 + q < f) Elem<T>::store(p, row_off + e0 + q, a[q]);
}

__device__ __forceinline__ void fma4(float4 &acc, float w, const float4 &v) {
    acc.x = fmaf(w, v.x, acc.x);
    acc.y = fmaf(w, v.y, acc.y);
    acc.z = fmaf(w, v.z, acc.z);
    acc.w = fmaf(w, v.w, acc.w);
}

__device__ __forceinline__ float4 shfl4(const float4 &v, int src) {
    return make_float4(__shfl(v.x, src, 64), __shfl(v.y, src, 64), __shfl(v.z, src, 64), __shfl(v.w, src, 64));
}

// Accumulate sum_{t in this lane's slot} w_t * x[idx_t][chunk] over one
// window of up to 64 (index, weight) pairs held one per lane.  Every lane runs
// the same number of iterations so the shuffles stay convergent.  Lanes past
// the window hold index 0 (a valid row) and the loads are issued
// unconditionally; invalid terms are masked to zero before the FMA.  The
// caller passes an in-row chunk offset for inactive lanes.  ROUND: every
// loaded value is first rounded to bf16 (round to nearest even), so that
// summing fp32 table rows gives exactly the sum over their bf16 copies.
__device__ __forceinline__ float4 round_bf16(float4 v) {
    return make_float4(bf16_to_f32(f32_to_bf16(v.x)), bf16_to_f32(f32_to_bf16(v.y)), bf16_to_f32(f32_to_bf16(v.z)),
                       bf16_to_f32(f32_to_bf16(v.w)));
}
template <bool VEC, class T, bool ROUND = false>
__device__ __forceinline__ void window_accumulate(float4 &acc, const T *x, int64_t stride, int64_t col_off,
                                                  int64_t f, int32_t my_idx, float my_w, int wn, int slot, int S,
                                                  bool active, int64_t e0) {
    for (int tb = 0; tb < wn; tb += 4 * S) {
        int32_t j[4];
        float w[4];
        bool ok[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int t = tb + q * S + slot;
            ok[q] = active && (t < wn);
            j[q] = __shfl(my_idx, t & 63, 64);
            w[q] = __shfl(my_w, t & 63, 64);
        }
        float4 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            v[q] = load_chunk<VEC>(x, static_cast<int64_t>(j[q]) * stride + col_off, e0, f);
            if constexpr (ROUND) v[q] = round_bf16(v[q]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float wq = ok[q] ? w[q] : 0.f;
            const float4 vq = ok[q] ? v[q] : make_float4(0.f, 0.f, 0.f, 0.f);
            fma4(acc, wq, vq);
        }
    }
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int KIND, class TIn, class TOut, bool VEC>
__device__ __forceinline__ void agg_fwd_row(const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                            const float *__restrict__ src_norm, const TIn *__restrict__ h, int64_t f,
                                            int C, int S, TOut *__restrict__ out, int64_t row) {
    const int lane = threadIdx.x & 63;
    const int64_t beg = rowptr[row], end = rowptr[row + 1];
    const int64_t deg = end - beg;
    const float wi = (KIND == GNN_AGG_GCN_SYM) ? src_norm[row] : 1.f;
    const int groups = (C + 63) / 64;
    const int slot = (S > 1) ? lane / C : 0;
    for (int g = 0; g < groups; ++g) {
        const int chunk = (S > 1) ? lane % C : g * 64 + lane;
        const bool active = (S > 1) ? (slot < S) : (chunk < C);
        const int64_t e0 = active ? static_cast<int64_t>(chunk) * 4 : 0;
        // the GCN self term, issued before the neighbours
        const float4 self = (KIND == GNN_AGG_GCN_SYM) ? load_chunk<VEC>(h, row * f, e0, f)
                                                        : make_float4(0.f, 0.f, 0.f, 0.f);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int64_t wb = beg; wb < end; wb += 64) {
            const int wn = static_cast<int>(min<int64_t>(64, end - wb));
            int32_t my_idx = 0;
            float my_w = 0.f;
            if (lane < wn) {
                my_idx = col[wb + lane];
                my_w = (KIND == GNN_AGG_GCN_SYM) ? wi * src_norm[my_idx] : 1.f;
            }
            window_accumulate<VEC>(acc, h, f, 0, f, my_idx, my_w, wn, slot, S, active, e0);
        }
        // fold the slots into slot 0
        for (int s2 = 1; s2 < S; ++s2) {
            const float4 o = shfl4(acc, lane + s2 * C);
            if (slot == 0) {
                acc.x += o.x;
                acc.y += o.y;
                acc.z += o.z;
                acc.w += o.w;
            }
        }
        if (slot != 0 || !active) continue;
        if (KIND == GNN_AGG_SAGE_MEAN) {
            if (deg > 0) {
                const float d = static_cast<float>(deg);
                acc.x /= d;
                acc.y /= d;
                acc.z /= d;
                acc.w /= d;
            }
        } else {
            const float ws = wi * wi;
            fma4(acc, ws, self);
        }
        store_chunk<VEC>(out, row * f, e0, f, acc);
    }
}

// ---------------------------------------------------------------------------
// backward: d_src[j] = self(j) + sum_{i in csc(j)} w_ij d_a[i, nbr part]
// ---------------------------------------------------------------------------
template <int KIND, class THB, bool VEC>
__device__ __forceinline__ void agg_bwd_row(int64_t n_dst, const int64_t *__restrict__ rowptr,
                                            const int64_t *__restrict__ cscptr, const int32_t *__restrict__ cscrow,
                                            const float *__restrict__ src_norm, const float *__restrict__ d_a,
                                            int64_t f, int C, int S, const THB *__restrict__ h_below,
                                            float *__restrict__ d_src, int64_t j) {
    const int lane = threadIdx.x & 63;
    const int64_t ka = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * f : f;
    const int64_t nbr_off = (KIND == GNN_AGG_SAGE_MEAN) ? f : 0;
    const int64_t beg = cscptr[j], end = cscptr[j + 1];
    const float wj = (KIND == GNN_AGG_GCN_SYM) ? src_norm[j] : 1.f;
    const int groups = (C + 63) / 64;
    const int slot = (S > 1) ? lane / C : 0;
    for (int g = 0; g < groups; ++g) {
        const int chunk = (S > 1) ? lane % C : g * 64 + lane;
        const bool active = (S > 1) ? (slot < S) : (chunk < C);
        const int64_t e0 = active ? static_cast<int64_t>(chunk) * 4 : 0;
        // the self term and the ReLU mask, issued before the neighbours so
        // that their latency overlaps the sum (a source past the destinations
        // reads destination row 0, unused; with no mask an in-bounds stand-in
        // address, unused; THB is float whenever h_below is null)
        const float4 self = load_chunk<VEC>(d_a, (j < n_dst ? j : 0) * ka, e0, f);
        const bool mask = h_below != nullptr;
        const float4 hb = load_chunk<VEC>(mask ? h_below : reinterpret_cast<const THB *>(d_a), mask ? j * f : 0, e0, f);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int64_t wb = beg; wb < end; wb += 64) {
            const int wn = static_cast<int>(min<int64_t>(64, end - wb));
            int32_t my_idx = 0;
            float my_w = 0.f;
            if (lane < wn) {
                my_idx = cscrow[wb + lane];
                if (KIND == GNN_AGG_GCN_SYM)
                    my_w = src_norm[my_idx] * wj;
                else
                    my_w = 1.f / static_cast<float>(rowptr[my_idx + 1] - rowptr[my_idx]);
            }
            window_accumulate<VEC>(acc, d_a, ka, nbr_off, f, my_idx, my_w, wn, slot, S, active, e0);
        }
        for (int s2 = 1; s2 < S; ++s2) {
            const float4 o = shfl4(acc, lane + s2 * C);
            if (slot == 0) {
                acc.x += o.x;
                acc.y += o.y;
                acc.z += o.z;
                acc.w += o.w;
            }
        }
        if (slot != 0 || !active) continue;
        if (j < n_dst) {
            const float ws = (KIND == GNN_AGG_GCN_SYM) ? wj * wj : 1.f;
            fma4(acc, ws, self);
        }
        if (mask) {
            if (!(hb.x > 0.f)) acc.x = 0.f;
            if (!(hb.y > 0.f)) acc.y = 0.f;
            if (!(hb.z > 0.f)) acc.z = 0.f;
            if (!(hb.w > 0.f)) acc.w = 0.f;
        }
        store_chunk<VEC>(d_src, j * f, e0, f, acc);
    }
}

// One row per wavefront, the grid's wavefronts striding over the rows (a
// grid of at most kMaxBlocks workgroups: capacity-sized grids would mostly
// hold workgroups that read the row count only to exit).
constexpr int64_t kMaxBlocks = 2048;

// The input layer's forward aggregation straight from an fp32 feature table
// (the feature loading fused into the aggregation, for tables in device
// memory): row i's p-th sampled neighbour is the global vertex gids[i k + p]
// (the sampler's staging of the block, in the block's column order), whose
// table row is read and rounded to bf16 element by element, exactly as the
// gather would have stored it in X'.  Same lanes, slots and summation order
// as agg_fwd_row over X', so the result is bitwise the same.  The GCN
// self term and weights use X' (its destination rows) and the graph's
// normalisers of the global ids (src_norm of the block holds the same
// values).
template <int KIND, bool VEC>
__device__ __forceinline__ void agg_fwd_row_table(const int64_t *__restrict__ rowptr,
                                                  const int64_t *__restrict__ gids, int32_t k,
                                                  const float *__restrict__ src_norm,
                                                  const float *__restrict__ gcn_norm, const float *__restrict__ table,
                                                  int64_t row_stride, const uint16_t *__restrict__ x_self, int64_t f,
                                                  int C, int S, uint16_t *__restrict__ out, int64_t row) {
    const int lane = threadIdx.x & 63;
    const int64_t beg = rowptr[row], end = rowptr[row + 1];
    const int64_t deg = end - beg;
    const float wi = (KIND == GNN_AGG_GCN_SYM) ? src_norm[row] : 1.f;
    const int groups = (C + 63) / 64;
    const int slot = (S > 1) ? lane / C : 0;
    for (int g = 0; g < groups; ++g) {
        const int chunk = (S > 1) ? lane % C : g * 64 + lane;
        const bool active = (S > 1) ? (slot < S) : (chunk < C);
        const int64_t e0 = active ? static_cast<int64_t>(chunk) * 4 : 0;
        const float4 self = (KIND == GNN_AGG_GCN_SYM) ? load_chunk<VEC>(x_self, row * f, e0, f)
                                                        : make_float4(0.f, 0.f, 0.f, 0.f);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int64_t wb = beg; wb < end; wb += 64) {
            const int wn = static_cast<int>(min<int64_t>(64, end - wb));
            int32_t my_idx = 0;
            float my_w = 0.f;
            if (lane < wn) {
                const int64_t gv = gids[row * k + (wb - beg) + lane];
                my_idx = static_cast<int32_t>(gv);
                my_w = (KIND == GNN_AGG_GCN_SYM) ? wi * gcn_norm[gv] : 1.f;
            }
            window_accumulate<VEC, float, true>(acc, table, row_stride, 0, f, my_idx, my_w, wn, slot, S, active, e0);
        }
        for (int s2 = 1; s2 < S; ++s2) {
            const float4 o = shfl4(acc, lane + s2 * C);
            if (slot == 0) {
                acc.x += o.x;
                acc.y += o.y;
                acc.z += o.z;
                acc.w += o.w;
            }
        }
        if (slot != 0 || !active) continue;
        if (KIND == GNN_AGG_SAGE_MEAN) {
            if (deg > 0) {
                const float d = static_cast<float>(deg);
                acc.x /= d;
                acc.y /= d;
                acc.z /= d;
                acc.w /= d;
            }
        } else {
            const float ws = wi * wi;
            fma4(acc, ws, self);
        }
        store_chunk<VEC>(out, row * f, e0, f, acc);
    }
}

template <int KIND, bool VEC>
struct FwdTableJob {
    gnn_block b;
    const int64_t *gids;
    int32_t k;
    const float *gcn_norm;
    const float *table;
    int64_t row_stride;
    const uint16_t *x_self;
    int64_t f;
    int C, S;
    uint16_t *out;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t n = b.counts[0];
        for (int64_t row = blk * kWaves + (threadIdx.x >> 6); row < n; row += nblk * kWaves)
            agg_fwd_row_table<KIND, VEC>(b.rowptr, gids, k, b.src_norm, gcn_norm, table, row_stride, x_self, f, C, S,
                                         out, row);
    }
};

template <int KIND, class TIn, class TOut, bool VEC>
struct FwdJob {
    gnn_block b;
    const TIn *h;
    int64_t f;
    int C, S;
    TOut *out;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t n = b.counts[0];
        for (int64_t row = blk * kWaves + (threadIdx.x >> 6); row < n; row += nblk * kWaves)
            agg_fwd_row<KIND, TIn, TOut, VEC>(b.rowptr, b.col, b.src_norm, h, f, C, S, out, row);
    }
};

template <int KIND, class THB, bool VEC>
struct BwdJob {
    gnn_block b;
    const float *d_a;
    int64_t f;
    int C, S;
    const THB *h_below;
    float *d_src;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t n_dst = b.counts[0], n_src = b.counts[1];
        for (int64_t j = blk * kWaves + (threadIdx.x >> 6); j < n_src; j += nblk * kWaves)
            agg_bwd_row<KIND, THB, VEC>(n_dst, b.rowptr, b.cscptr, b.cscrow, b.src_norm, d_a, f, C, S, h_below,
                                        d_src, j);
    }
};

// ---------------------------------------------------------------------------
// GraphSAGE's max aggregator, forward: out[i, c] = the maximum of h[u, c] over
// row i's edges, with argmax[i, c] the local source of the edge that holds it.
// Sequential rule: the row's first edge holds the running maximum and a later
// edge replaces it only when strictly greater (a tie, and a duplicate edge,
// go to the earliest edge).  The slots walk interleaved edges of the row,
// each applying the rule to its own edges with the row's first edge taken
// unconditionally (it belongs to slot 0); the fold keeps the greater value
// and, on equal values, the earlier edge.  That reproduces the sequential
// rule, NaN included: a NaN is only ever taken as the row's first edge, and
// then nothing replaces it.  A row without edges gives 0 and argmax -1.
// ---------------------------------------------------------------------------
struct MaxChunk {
    float v[4];
    int32_t pos[4];  // edge position in the row; INT32_MAX for none
    int32_t src[4];  // local source id; -1 for none
};

__device__ __forceinline__ void max_take(MaxChunk &m, int q, float v, int32_t pos, int32_t src) {
    m.v[q] = v;
    m.pos[q] = pos;
    m.src[q] = src;
}

template <bool VEC>
__device__ __forceinline__ void store_arg4(int32_t *p, int64_t row_off, int64_t e0, int64_t f, const int32_t *a) {
    if constexpr (VEC) {
        *reinterpret_cast<int4 *>(p + row_off + e0) = make_int4(a[0], a[1], a[2], a[3]);
        return;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (e0 + q < f) p[row_off + e0 + q] = a[q];
}

// argmax[row_off + e0 .. + 3], with `none` past f
template <bool VEC>
__device__ __forceinline__ int4 load_arg4(const int32_t *p, int64_t row_off, int64_t e0, int64_t f, int32_t none) {
    if constexpr (VEC) return *reinterpret_cast<const int4 *>(p + row_off + e0);
    int32_t a[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const bool ok = e0 + q < f;
        const int32_t x = p[row_off + (ok ? e0 + q : f - 1)];
        a[q] = ok ? x : none;
    }
    return make_int4(a[0], a[1], a[2], a[3]);
}

template <class TIn, class TOut, bool VEC>
__device__ __forceinline__ void agg_fwd_row_max(const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                                const TIn *__restrict__ h, int64_t f, int C, int S,
                                                TOut *__restrict__ out, int32_t *__restrict__ argmax, int64_t row) {
    const int lane = threadIdx.x & 63;
    const int64_t beg = rowptr[row], end = rowptr[row + 1];
    const int groups = (C + 63) / 64;
    const int slot = (S > 1) ? lane / C : 0;
    for (int g = 0; g < groups; ++g) {
        const int chunk = (S > 1) ? lane % C : g * 64 + lane;
        const bool active = (S > 1) ? (slot < S) : (chunk < C);
        const int64_t e0 = active ? static_cast<int64_t>(chunk) * 4 : 0;
        MaxChunk m;
#pragma unroll
        for (int q = 0; q < 4; ++q) max_take(m, q, -INFINITY, INT32_MAX, -1);
        for (int64_t wb = beg; wb < end; wb += 64) {
            const int wn = static_cast<int>(min<int64_t>(64, end - wb));
            const int32_t base = static_cast<int32_t>(wb - beg);
            const int32_t my_idx = (lane < wn) ? col[wb + lane] : 0;
            for (int tb = 0; tb < wn; tb += 4 * S) {
                int32_t j[4];
                bool ok[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int t = tb + u * S + slot;
                    ok[u] = active && (t < wn);
                    j[u] = __shfl(my_idx, t & 63, 64);
                }
                float4 v[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) v[u] = load_chunk<VEC>(h, static_cast<int64_t>(j[u]) * f, e0, f);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (!ok[u]) continue;
                    const int32_t pos = base + tb + u * S + slot;
                    const float x[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (pos == 0 || x[q] > m.v[q]) max_take(m, q, x[q], pos, j[u]);
                }
            }
        }
        // fold the slots into slot 0 in slot order
        for (int s2 = 1; s2 < S; ++s2) {
            const int src_lane = lane + s2 * C;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float ov = __shfl(m.v[q], src_lane, 64);
                const int32_t op = __shfl(m.pos[q], src_lane, 64);
                const int32_t os = __shfl(m.src[q], src_lane, 64);
                if (slot == 0 && (ov > m.v[q] || (ov == m.v[q] && op < m.pos[q]))) max_take(m, q, ov, op, os);
            }
        }
        if (slot != 0 || !active) continue;
        float r[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) r[q] = (m.src[q] < 0) ? 0.f : m.v[q];
        store_chunk<VEC>(out, row * f, e0, f, make_float4(r[0], r[1], r[2], r[3]));
        if (argmax) store_arg4<VEC>(argmax, row * f, e0, f, m.src);
    }
}

// Backward of the max aggregator for source j, pulled over the block's
// transpose: d_src[j, c] = [j < n_dst] d_a[j, c] + the sum of d_a[i, f + c]
// over the distinct rows i that sampled j with argmax[i, c] = j, then the
// ReLU mask.  A row that sampled j several times sits in consecutive entries
// of j's column (the columns are in ascending row order), and only the
// first of them counts: the maximum passes its gradient once.  The
// neighbour rows of d_a are read only for elements that j won.
template <class THB, bool VEC>
__device__ __forceinline__ void agg_bwd_row_max(int64_t n_dst, const int64_t *__restrict__ cscptr,
                                                const int32_t *__restrict__ cscrow, const int32_t *__restrict__ argmax,
                                                const float *__restrict__ d_a, int64_t f, int C, int S,
                                                const THB *__restrict__ h_below, float *__restrict__ d_src,
                                                int64_t j) {
    const int lane = threadIdx.x & 63;
    const int64_t ka = 2 * f;
    const int64_t beg = cscptr[j], end = cscptr[j + 1];
    const int32_t jj = static_cast<int32_t>(j);
    const int groups = (C + 63) / 64;
    const int slot = (S > 1) ? lane / C : 0;
    for (int g = 0; g < groups; ++g) {
        const int chunk = (S > 1) ? lane % C : g * 64 + lane;
        const bool active = (S > 1) ? (slot < S) : (chunk < C);
        const int64_t e0 = active ? static_cast<int64_t>(chunk) * 4 : 0;
        const float4 self = load_chunk<VEC>(d_a, (j < n_dst ? j : 0) * ka, e0, f);
        const bool mask = h_below != nullptr;
        const float4 hb = load_chunk<VEC>(mask ? h_below : reinterpret_cast<const THB *>(d_a), mask ? j * f : 0, e0, f);
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int64_t wb = beg; wb < end; wb += 64) {
            const int wn = static_cast<int>(min<int64_t>(64, end - wb));
            int32_t my_idx = 0;
            int my_first = 0;
            if (lane < wn) {
                my_idx = cscrow[wb + lane];
                my_first = (wb + lane == beg) || (cscrow[wb + lane - 1] != my_idx);
            }
            for (int tb = 0; tb < wn; tb += 4 * S) {
                int32_t i[4];
                bool ok[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    // both shuffles run in every lane: a lane left out would
                    // read as zero to the lanes that take its value
                    const int t = tb + u * S + slot;
                    i[u] = __shfl(my_idx, t & 63, 64);
                    const int first = __shfl(my_first, t & 63, 64);
                    ok[u] = active && (t < wn) && first;
                }
                int4 a[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) a[u] = load_arg4<VEC>(argmax, static_cast<int64_t>(i[u]) * f, e0, f, -1);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const bool w[4] = {ok[u] && a[u].x == jj, ok[u] && a[u].y == jj, ok[u] && a[u].z == jj,
                                       ok[u] && a[u].w == jj};
                    if (w[0] || w[1] || w[2] || w[3]) {
                        const float4 v = load_chunk<VEC>(d_a, static_cast<int64_t>(i[u]) * ka + f, e0, f);
                        acc[0] += w[0] ? v.x : 0.f;
                        acc[1] += w[1] ? v.y : 0.f;
                        acc[2] += w[2] ? v.z : 0.f;
                        acc[3] += w[3] ? v.w : 0.f;
                    }
                }
            }
        }
        for (int s2 = 1; s2 < S; ++s2) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float o = __shfl(acc[q], lane + s2 * C, 64);
                if (slot == 0) acc[q] += o;
            }
        }
        if (slot != 0 || !active) continue;
        float4 r = make_float4(acc[0], acc[1], acc[2], acc[3]);
        if (j < n_dst) {
            r.x += self.x;
            r.y += self.y;
            r.z += self.z;
            r.w += self.w;
        }
        if (mask) {
            if (!(hb.x > 0.f)) r.x = 0.f;
            if (!(hb.y > 0.f)) r.y = 0.f;
            if (!(hb.z > 0.f)) r.z = 0.f;
            if (!(hb.w > 0.f)) r.w = 0.f;
        }
        store_chunk<VEC>(d_src, j * f, e0, f, r);
    }
}

template <class TIn, class TOut, bool VEC>
struct FwdMaxJob {
    gnn_block b;
    const TIn *h;
    int64_t f;
    int C, S;
    TOut *out;
    int32_t *argmax;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t n = b.counts[0];
        for (int64_t row = blk * kWaves + (threadIdx.x >> 6); row < n; row += nblk * kWaves)
            agg_fwd_row_max<TIn, TOut, VEC>(b.rowptr, b.col, h, f, C, S, out, argmax, row);
    }
};

template <class THB, bool VEC>
struct BwdMaxJob {
    gnn_block b;
    const int32_t *argmax;
    const float *d_a;
    int64_t f;
    int C, S;
    const THB *h_below;
    float *d_src;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t n_dst = b.counts[0], n_src = b.counts[1];
        for (int64_t j = blk * kWaves + (threadIdx.x >> 6); j < n_src; j += nblk * kWaves)
            agg_bwd_row_max<THB, VEC>(n_dst, b.cscptr, b.cscrow, argmax, d_a, f, C, S, h_below, d_src, j);
    }
};

inline void split_row(int64_t f, int *C, int *S) {
    const int64_t c = ceil_div(f, 4);
    *C = static_cast<int>(c);
    *S = (c <= 32) ? static_cast<int>(64 / c) : 1;
}

inline unsigned row_grid(int64_t rows) {
    return static_cast<unsigned>(std::min<int64_t>(ceil_div(rows > 0 ? rows : 1, kWaves), kMaxBlocks));
}

// f(job) with the table-reading forward job (fp32 table -> bf16 output).
template <class F>
void with_fwd_table_job(const gnn_block *b, int kind, const int64_t *gids, int32_t k, const float *gcn_norm,
                        const float *table, int64_t row_stride, const uint16_t *x_self, int64_t f, uint16_t *out,
                        F &&fn) {
    int C, S;
    split_row(f, &C, &S);
    const bool vec = (f % 4 == 0) && (row_stride % 4 == 0) && aligned(table, 16) && aligned(x_self, 8) &&
                     aligned(out, 8);
    auto go = [&](auto kind_tag) {
        constexpr int KIND = decltype(kind_tag)::value;
        if (vec) fn(FwdTableJob<KIND, true>{*b, gids, k, gcn_norm, table, row_stride, x_self, f, C, S, out});
        else fn(FwdTableJob<KIND, false>{*b, gids, k, gcn_norm, table, row_stride, x_self, f, C, S, out});
    };
    if (kind == GNN_AGG_SAGE_MEAN) go(std::integral_constant<int, GNN_AGG_SAGE_MEAN>{});
    else go(std::integral_constant<int, GNN_AGG_GCN_SYM>{});
}

// f(job) with the forward job for (kind, hdt -> odt); false if unsupported.
template <class F>
bool with_fwd_job(const gnn_block *b, int kind, const void *h, int hdt, int64_t f, void *out, int odt, F &&fn) {
    int C, S;
    split_row(f, &C, &S);
    const bool vec = (f % 4 == 0) && aligned(h, 4 * dtype_size(hdt)) && aligned(out, 4 * dtype_size(odt));
    auto by_kind = [&](auto kind_tag, auto ti_tag, auto to_tag) {
        constexpr int KIND = decltype(kind_tag)::value;
        using TI = typename decltype(ti_tag)::type;
        using TO = typename decltype(to_tag)::type;
        const TI *hp = static_cast<const TI *>(h);
        TO *op = static_cast<TO *>(out);
        if (vec) fn(FwdJob<KIND, TI, TO, true>{*b, hp, f, C, S, op});
        else fn(FwdJob<KIND, TI, TO, false>{*b, hp, f, C, S, op});
    };
    auto by_types = [&](auto kind_tag) {
        if (hdt == GNN_F32 && odt == GNN_F32) by_kind(kind_tag, Tag<float>{}, Tag<float>{});
        else if (hdt == GNN_F32 && odt == GNN_BF16) by_kind(kind_tag, Tag<float>{}, Tag<uint16_t>{});
        else if (hdt == GNN_BF16 && odt == GNN_F32) by_kind(kind_tag, Tag<uint16_t>{}, Tag<float>{});
        else by_kind(kind_tag, Tag<uint16_t>{}, Tag<uint16_t>{});
    };
    if (!((hdt == GNN_F32 || hdt == GNN_BF16) && (odt == GNN_F32 || odt == GNN_BF16))) return false;
    if (kind == GNN_AGG_SAGE_MEAN) by_types(std::integral_constant<int, GNN_AGG_SAGE_MEAN>{});
    else by_types(std::integral_constant<int, GNN_AGG_GCN_SYM>{});
    return true;
}

// f(job) with the backward job.
template <class F>
void with_bwd_job(const gnn_block *b, int kind, const float *d_a, int64_t f, const void *h_below, int hbdt,
                  float *d_src, F &&fn) {
    int C, S;
    split_row(f, &C, &S);
    const bool vec = (f % 4 == 0) && aligned(d_a, 16) && aligned(d_src, 16) &&
                     (!h_below || aligned(h_below, 4 * dtype_size(hbdt)));
    auto by_type = [&](auto kind_tag, auto hb_tag) {
        constexpr int KIND = decltype(kind_tag)::value;
        using THB = typename decltype(hb_tag)::type;
        const THB *hb = static_cast<const THB *>(h_below);
        if (vec) fn(BwdJob<KIND, THB, true>{*b, d_a, f, C, S, hb, d_src});
        else fn(BwdJob<KIND, THB, false>{*b, d_a, f, C, S, hb, d_src});
    };
    auto by_kind = [&](auto kind_tag) {
        if (!h_below || hbdt == GNN_F32) by_type(kind_tag, Tag<float>{});
        else by_type(kind_tag, Tag<uint16_t>{});
    };
    if (kind == GNN_AGG_SAGE_MEAN) by_kind(std::integral_constant<int, GNN_AGG_SAGE_MEAN>{});
    else by_kind(std::integral_constant<int, GNN_AGG_GCN_SYM>{});
}

// f(job) with the max aggregator's forward job (argmax may be null: the
// table is not kept); false if the dtypes are unsupported.
template <class F>
bool with_fwd_max_job(const gnn_block *b, const void *h, int hdt, int64_t f, void *out, int odt, int32_t *argmax,
                      F &&fn) {
    int C, S;
    split_row(f, &C, &S);
    const bool vec = (f % 4 == 0) && aligned(h, 4 * dtype_size(hdt)) && aligned(out, 4 * dtype_size(odt)) &&
                     aligned(argmax, 16);
    auto go = [&](auto ti_tag, auto to_tag) {
        using TI = typename decltype(ti_tag)::type;
        using TO = typename decltype(to_tag)::type;
        const TI *hp = static_cast<const TI *>(h);
        TO *op = static_cast<TO *>(out);
        if (vec) fn(FwdMaxJob<TI, TO, true>{*b, hp, f, C, S, op, argmax});
        else fn(FwdMaxJob<TI, TO, false>{*b, hp, f, C, S, op, argmax});
    };
    if (!((hdt == GNN_F32 || hdt == GNN_BF16) && (odt == GNN_F32 || odt == GNN_BF16))) return false;
    if (hdt == GNN_F32 && odt == GNN_F32) go(Tag<float>{}, Tag<float>{});
    else if (hdt == GNN_F32 && odt == GNN_BF16) go(Tag<float>{}, Tag<uint16_t>{});
    else if (hdt == GNN_BF16 && odt == GNN_F32) go(Tag<uint16_t>{}, Tag<float>{});
    else go(Tag<uint16_t>{}, Tag<uint16_t>{});
    return true;
}

// f(job) with the forward job of any aggregation kind; the max aggregator
// writes its argmax table to argmax (may be null).
template <class F>
bool with_fwd_kind_job(const gnn_block *b, int kind, const void *h, int hdt, int64_t f, void *out, int odt,
                       int32_t *argmax, F &&fn) {
    if (kind == GNN_AGG_SAGE_MAX) return with_fwd_max_job(b, h, hdt, f, out, odt, argmax, fn);
    return with_fwd_job(b, kind, h, hdt, f, out, odt, fn);
}

template <class F>
void with_bwd_max_job(const gnn_block *b, const int32_t *argmax, const float *d_a, int64_t f, const void *h_below,
                      int hbdt, float *d_src, F &&fn) {
    int C, S;
    split_row(f, &C, &S);
    const bool vec = (f % 4 == 0) && aligned(d_a, 16) && aligned(d_src, 16) && aligned(argmax, 16) &&
                     (!h_below || aligned(h_below, 4 * dtype_size(hbdt)));
    auto go = [&](auto hb_tag) {
        using THB = typename decltype(hb_tag)::type;
        const THB *hb = static_cast<const THB *>(h_below);
        if (vec) fn(BwdMaxJob<THB, true>{*b, argmax, d_a, f, C, S, hb, d_src});
        else fn(BwdMaxJob<THB, false>{*b, argmax, d_a, f, C, S, hb, d_src});
    };
    if (!h_below || hbdt == GNN_F32) go(Tag<float>{});
    else go(Tag<uint16_t>{});
}

}  // namespace agg
}  // namespace gnn
