// Forward aggregation with source reuse inside a tile of destination rows:
// the idea of Section IV-C's feature duplicator (fetch each source's feature
// vector once and hand it to every destination that needs it) on gfx950.
//
// A 256-thread workgroup takes 16 destination rows at a time.  It stages
// their column indices in LDS, deduplicates them with an LDS hash table (a
// source sampled by several rows of the tile is kept once) and numbers the
// distinct sources densely.  Then, one feature slice (128 bytes of every row)
// at a time, it copies each distinct source's slice from HBM into LDS once
// and every (row, 4-feature chunk) thread sums its row from LDS.  HBM (and
// L2) traffic is the tile's distinct sources instead of its edges.
//
// The sums follow, term for term, the order of the pull kernel
// (agg_fwd_row: S slots per wavefront, each walking the edges t = s mod S of
// every 64-edge window four at a time, padded with zero terms, then folded
// slot after slot), so the output is bitwise that of gnn_aggregate_fwd.
// Tiles with more edges than the LDS staging holds read their sources from
// HBM in the same order.
#include "aggregate_dev.h"
#include "jobs.h"

namespace gnn {
namespace {

constexpr int kT = 256;          // threads
constexpr int kRows = 16;        // destination rows per tile
constexpr int kEdgeCap = 512;    // edges a tile stages and deduplicates
constexpr int kHash = 1024;      // hash slots (at most half full)
constexpr int kSliceBytes = 128; // bytes of each source row per slice
constexpr int kMaxBlocks = 2048;

template <class T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<uint16_t>(uint16_t v) { return bf16_to_f32(v); }

struct DedupArgs {
    gnn_block b;
    const void *h;
    int64_t f;
    void *out;
};

// Row `row`'s chunk e0 .. e0+3 as the pull kernel sums it.  val(j, q) is the
// value of element e0 + q of source j (zero past f); w(j) the edge weight.
template <int KIND, class Val>
__device__ __forceinline__ float4 pull_order_sum(const int32_t *cols, int64_t deg, float wi, const float *src_norm,
                                                 int C, Val &&val) {
    const int S = (C <= 32) ? 64 / C : 1;
    float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < S; ++s) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int64_t wb = 0; wb < deg; wb += 64) {
            const int wn = static_cast<int>(min<int64_t>(64, deg - wb));
            for (int tb = 0; tb < wn; tb += 4 * S) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int t = tb + q * S + s;
                    if (t < wn) {
                        const int32_t j = cols[wb + t];
                        const float w = (KIND == GNN_AGG_GCN_SYM) ? wi * src_norm[j] : 1.f;
                        agg::fma4(acc, w, val(wb + t, j));
                    } else {
                        agg::fma4(acc, 0.f, make_float4(0.f, 0.f, 0.f, 0.f));
                    }
                }
            }
        }
        if (s == 0) {
            tot = acc;
        } else {
            tot.x += acc.x;
            tot.y += acc.y;
            tot.z += acc.z;
            tot.w += acc.w;
        }
    }
    return tot;
}

template <int KIND, class TIn, class TOut>
__device__ __forceinline__ void finish(const DedupArgs &a, int64_t row, int64_t deg, float wi, int64_t e0, float4 acc) {
    const TIn *h = static_cast<const TIn *>(a.h);
    if (KIND == GNN_AGG_SAGE_MEAN) {
        if (deg > 0) {
            const float d = static_cast<float>(deg);
            acc.x /= d;
            acc.y /= d;
            acc.z /= d;
            acc.w /= d;
        }
    } else {
        agg::fma4(acc, wi * wi, agg::load_chunk<false>(h, row * a.f, e0, a.f));
    }
    agg::store_chunk<false>(static_cast<TOut *>(a.out), row * a.f, e0, a.f, acc);
}

template <int KIND, class TIn, class TOut>
__global__ void __launch_bounds__(kT) aggregate_dedup_kernel(DedupArgs a) {
    constexpr int kCps = kSliceBytes / (4 * static_cast<int>(sizeof(TIn)));  // chunks per slice
    __shared__ int64_t Rs[kRows + 1];
    __shared__ int32_t Es[kEdgeCap];
    __shared__ int16_t Ui[kEdgeCap];       // dense index of each edge's source
    __shared__ int32_t tab[kHash];          // hash table of source ids, then of dense indices
    __shared__ int32_t uniq[kEdgeCap];     // the tile's distinct sources
    __shared__ int32_t scan_tot;
    __shared__ __attribute__((aligned(16))) TIn rows[kEdgeCap * kCps * 4];  // one slice of every distinct source
    const int tid = threadIdx.x;
    const TIn *h = static_cast<const TIn *>(a.h);
    const int64_t f = a.f;
    const int C = static_cast<int>((f + 3) / 4);
    const int64_t M = a.b.counts ? min(a.b.counts[0], a.b.cap_dst) : a.b.cap_dst;
    const int64_t ntiles = (M + kRows - 1) / kRows;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t row0 = tile * kRows;
        const int rows_n = static_cast<int>(min<int64_t>(kRows, M - row0));
        for (int r = tid; r <= rows_n; r += kT) Rs[r] = a.b.rowptr[row0 + r];
        for (int i = tid; i < kHash; i += kT) tab[i] = -1;
        __syncthreads();
        const int64_t e_beg = Rs[0];
        const int64_t ne = Rs[rows_n] - e_beg;
        const bool staged = ne <= kEdgeCap;
        int U = 0;
        if (staged) {
            // stage and deduplicate the tile's sources
            for (int e = tid; e < ne; e += kT) {
                const int32_t key = a.b.col[e_beg + e];
                Es[e] = key;
                uint32_t hs = (static_cast<uint32_t>(key) * 2654435761u) >> 22;  // 10 bits
                for (;;) {
                    const int32_t prev = atomicCAS(&tab[hs], -1, key);
                    if (prev == -1 || prev == key) break;
                    hs = (hs + 1) & (kHash - 1);
                }
                Ui[e] = static_cast<int16_t>(hs);
            }
            __syncthreads();
            // dense numbering of the occupied slots: block scan, 4 slots per thread
            int occ[4], sum = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                occ[q] = tab[tid * 4 + q] >= 0 ? 1 : 0;
                sum += occ[q];
            }
            // inclusive scan of the per-thread sums over the workgroup
            __shared__ int32_t part[kT];
            part[tid] = sum;
            __syncthreads();
            for (int d = 1; d < kT; d <<= 1) {
                const int v = tid >= d ? part[tid - d] : 0;
                __syncthreads();
                part[tid] += v;
                __syncthreads();
            }
            int base = part[tid] - sum;
            if (tid == kT - 1) scan_tot = part[tid];
            int keys[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) keys[q] = tab[tid * 4 + q];
            __syncthreads();
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (occ[q]) {
                    uniq[base] = keys[q];
                    tab[tid * 4 + q] = base;  // the slot now holds the dense index
                    ++base;
                }
            }
            __syncthreads();
            U = scan_tot;
            for (int e = tid; e < ne; e += kT) Ui[e] = static_cast<int16_t>(tab[Ui[e]]);
            __syncthreads();
        }
        // slices of kCps chunks
        for (int c0 = 0; c0 < C; c0 += kCps) {
            const int cn = min(kCps, C - c0);
            if (staged) {
                // each distinct source's slice, once
                for (int i = tid; i < U * kCps; i += kT) {
                    const int u = i / kCps, c = i % kCps;
                    if (c >= cn) continue;
                    const int64_t src = static_cast<int64_t>(uniq[u]) * f;
                    const int64_t e0 = static_cast<int64_t>(c0 + c) * 4;
                    TIn *dst = rows + (u * kCps + c) * 4;
#pragma unroll
                    for (int q = 0; q < 4; ++q) dst[q] = h[src + (e0 + q < f ? e0 + q : f - 1)];
                }
                __syncthreads();
            }
            for (int it = tid; it < kRows * kCps; it += kT) {
                const int r = it / kCps, c = it % kCps;
                if (r >= rows_n || c >= cn) continue;
                const int64_t row = row0 + r;
                const int64_t rb = Rs[r] - e_beg, deg = Rs[r + 1] - Rs[r];
                const int64_t e0 = static_cast<int64_t>(c0 + c) * 4;
                const float wi = (KIND == GNN_AGG_GCN_SYM) ? a.b.src_norm[row] : 1.f;
                float4 acc;
                if (staged) {
                    acc = pull_order_sum<KIND>(Es + rb, deg, wi, a.b.src_norm, C, [&](int64_t t, int32_t) {
                        const TIn *p = rows + (Ui[rb + t] * kCps + c) * 4;
                        float v[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) v[q] = e0 + q < f ? to_f<TIn>(p[q]) : 0.f;
                        return make_float4(v[0], v[1], v[2], v[3]);
                    });
                } else {
                    acc = pull_order_sum<KIND>(a.b.col + e_beg + rb, deg, wi, a.b.src_norm, C,
                                               [&](int64_t, int32_t j) {
                        return agg::load_chunk<false>(h, static_cast<int64_t>(j) * f, e0, f);
                    });
                }
                finish<KIND, TIn, TOut>(a, row, deg, wi, e0, acc);
            }
            __syncthreads();  // the next slice overwrites the rows
        }
    }
}

template <int KIND, class TIn, class TOut>
gnn_status go(const DedupArgs &a, hipStream_t s) {
    const int64_t tiles = ceil_div(std::max<int64_t>(a.b.cap_dst, 1), kRows);
    const unsigned grid = static_cast<unsigned>(std::min<int64_t>(tiles, kMaxBlocks));
    aggregate_dedup_kernel<KIND, TIn, TOut><<<grid, kT, 0, s>>>(a);
    return launch_status("aggregate_fwd_dedup");
}

template <int KIND>
gnn_status go_types(const DedupArgs &a, int hdt, int odt, hipStream_t s) {
    if (hdt == GNN_BF16 && odt == GNN_BF16) return go<KIND, uint16_t, uint16_t>(a, s);
    if (hdt == GNN_BF16 && odt == GNN_F32) return go<KIND, uint16_t, float>(a, s);
    if (hdt == GNN_F32 && odt == GNN_BF16) return go<KIND, float, uint16_t>(a, s);
    return go<KIND, float, float>(a, s);
}

}  // namespace

gnn_status launch_aggregate_fwd_dedup(const gnn_block *b, int kind, const void *h, int hdt, int64_t f, void *out,
                                      int odt, hipStream_t s) {
    if (b->cap_dst == 0 || f == 0) return GNN_OK;
    const DedupArgs a{*b, h, f, out};
    if (kind == GNN_AGG_SAGE_MEAN) return go_types<GNN_AGG_SAGE_MEAN>(a, hdt, odt, s);
    return go_types<GNN_AGG_GCN_SYM>(a, hdt, odt, s);
}

}  // namespace gnn
