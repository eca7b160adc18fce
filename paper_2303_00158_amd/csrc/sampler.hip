// Mini-batch sampler: one block (hop) of uniform neighbour sampling without
// replacement, relabelled to local indices, with its transpose.
//
// Device workspace (sampler_ws_bytes):
//   map  int32[graph_n]  vertex -> local source index, -1 when unused
//   bits uint32[W]       one bit per vertex: "reached, not a destination"
//   ... per-call scratch
// map and bits are all -1 / 0 between calls; each call restores that state by
// resetting exactly the entries it touched.
#include "internal.h"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kBitTile = kThreads * 8;  // bitmap words per block in the scan kernels

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

__global__ void gcn_norm_kernel(const int64_t *__restrict__ rowptr, int64_t n, float *__restrict__ nrm) {
    const int64_t v = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const double D = static_cast<double>(rowptr[v + 1] - rowptr[v]) + 1.0;
    nrm[v] = static_cast<float>(1.0 / sqrt(D));
}

__global__ void fill_i32_kernel(int32_t *p, int64_t n, int32_t v) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        p[i] = v;
}

// Per destination row: sample count min(deg, k); map the destination to its
// local index; it is also source i.
__global__ void sample_count_kernel(const int64_t *__restrict__ dst, const int64_t *n_dst_dev, int64_t cap_dst,
                                    const int64_t *__restrict__ rowptr, int32_t fanout, int32_t *__restrict__ map,
                                    int64_t *__restrict__ cnt, int64_t *__restrict__ src_ids,
                                    int64_t *__restrict__ counts) {
    const int64_t n_dst = n_dst_dev ? min(*n_dst_dev, cap_dst) : cap_dst;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i == 0) counts[0] = n_dst;
    if (i >= n_dst) return;
    const int64_t v = dst[i];
    const int64_t d = rowptr[v + 1] - rowptr[v];
    cnt[i] = d < fanout ? d : fanout;
    map[v] = static_cast<int32_t>(i);
    src_ids[i] = v;
}

// One wavefront per destination row.  Rows with d <= k keep every position;
// otherwise Floyd's algorithm draws k distinct positions, held R per lane
// (slot s lives in lane s % 64, register s / 64), which are then ranked to
// write the sampled neighbours in ascending position order.
template <int R>
__global__ void __launch_bounds__(kThreads) sample_floyd_kernel(
    const int64_t *__restrict__ dst, const int64_t *__restrict__ counts, const int64_t *__restrict__ rowptr,
    const int64_t *__restrict__ col, const int64_t *__restrict__ brow, int32_t k, uint64_t seed, uint64_t step,
    uint64_t hop, int64_t *__restrict__ gcol) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x) >> 6;
    const int64_t n_dst = counts[0];
    if (row >= n_dst) return;
    const int64_t v = dst[row];
    const int64_t beg = rowptr[v];
    const int64_t d = rowptr[v + 1] - beg;
    const int64_t ob = brow[row];
    if (d <= k) {
        for (int64_t p = lane; p < d; p += 64) gcol[ob + p] = col[beg + p];
        return;
    }
    uint32_t slot[R];
#pragma unroll
    for (int r = 0; r < R; ++r) slot[r] = 0xffffffffu;
    const uint64_t pk = mix64(mix64(mix64(mix64(seed) ^ step) ^ hop) ^ static_cast<uint64_t>(v));
    for (int32_t t = 0; t < k; ++t) {
        const uint64_t j = static_cast<uint64_t>(d - k + t);
        const uint64_t key = mix64(pk ^ static_cast<uint64_t>(t));
        const uint32_t x = static_cast<uint32_t>(((key >> 32) * (j + 1)) >> 32);
        bool mine = false;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int s = r * 64 + lane;
            mine |= (s < t) && (slot[r] == x);
        }
        const bool found = __ballot(mine) != 0ull;
        const uint32_t val = found ? static_cast<uint32_t>(j) : x;
        const int treg = t >> 6;
        if (lane == (t & 63)) {
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (r == treg) slot[r] = val;
        }
    }
    // rank of each drawn position among all k (they are distinct)
    int rank[R];
#pragma unroll
    for (int r = 0; r < R; ++r) rank[r] = 0;
    for (int32_t s = 0; s < k; ++s) {
        const int sreg = s >> 6;
        uint32_t mine = 0;
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (r == sreg) mine = slot[r];
        const uint32_t other = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(mine), s & 63));
#pragma unroll
        for (int r = 0; r < R; ++r) rank[r] += (other < slot[r]) ? 1 : 0;
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int s = r * 64 + lane;
        if (s < k) gcol[ob + rank[r]] = col[beg + slot[r]];
    }
}

// Sampled ids that are not destinations: set their bit.
__global__ void mark_new_kernel(const int64_t *__restrict__ gcol, const int64_t *__restrict__ counts,
                                const int32_t *__restrict__ map, uint32_t *__restrict__ bits) {
    const int64_t nnz = counts[2];
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < nnz;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t u = gcol[e];
        if (map[u] < 0) atomicOr(&bits[u >> 5], 1u << (u & 31));
    }
}

__global__ void __launch_bounds__(kThreads) bitmap_count_kernel(const uint32_t *__restrict__ bits, int64_t words,
                                                                 int64_t *__restrict__ pc) {
    __shared__ int64_t sh[kThreads / 64];
    const int64_t w0 = static_cast<int64_t>(blockIdx.x) * kBitTile + threadIdx.x * 8;
    int64_t c = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (w0 + i < words) c += __popc(bits[w0 + i]);
    // block sum
    for (int o = 32; o > 0; o >>= 1) c += __shfl_down(c, o, 64);
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t t = 0;
        for (int w = 0; w < kThreads / 64; ++w) t += sh[w];
        pc[blockIdx.x] = t;
    }
}

// Emit the set bits in ascending vertex order as new sources n_dst + r, map
// them, and clear the bitmap.
__global__ void __launch_bounds__(kThreads) bitmap_emit_kernel(uint32_t *__restrict__ bits, int64_t words,
                                                                const int64_t *__restrict__ pcoff,
                                                                const int64_t *__restrict__ new_total,
                                                                int64_t *__restrict__ counts,
                                                                int64_t *__restrict__ src_ids,
                                                                int32_t *__restrict__ map) {
    __shared__ int64_t sh[kThreads / 64];
    const int64_t n_dst = counts[0];
    if (blockIdx.x == 0 && threadIdx.x == 0) counts[1] = n_dst + *new_total;
    const int64_t w0 = static_cast<int64_t>(blockIdx.x) * kBitTile + threadIdx.x * 8;
    uint32_t wv[8];
    int64_t c = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        wv[i] = (w0 + i < words) ? bits[w0 + i] : 0u;
        c += __popc(wv[i]);
    }
    // exclusive scan of c over the block
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t inc = c;
    for (int o = 1; o < 64; o <<= 1) {
        int64_t y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
    }
    if (lane == 63) sh[wave] = inc;
    __syncthreads();
    int64_t base = pcoff[blockIdx.x] + n_dst + inc - c;
    for (int w = 0; w < wave; ++w) base += sh[w];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        uint32_t m = wv[i];
        if (!m) continue;
        const int64_t wbase = (w0 + i) * 32;
        while (m) {
            const int b = __builtin_ctz(m);
            m &= m - 1;
            const int64_t u = wbase + b;
            src_ids[base] = u;
            map[u] = static_cast<int32_t>(base);
            ++base;
        }
        bits[w0 + i] = 0u;
    }
}

__global__ void relabel_kernel(const int64_t *__restrict__ gcol, const int64_t *__restrict__ counts,
                               const int32_t *__restrict__ map, int32_t *__restrict__ col_out) {
    const int64_t nnz = counts[2];
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < nnz;
         e += static_cast<int64_t>(gridDim.x) * blockDim.x)
        col_out[e] = map[gcol[e]];
}

__global__ void finish_kernel(const int64_t *__restrict__ src_ids, const int64_t *__restrict__ counts,
                              int32_t *__restrict__ map, const float *__restrict__ gcn_norm,
                              float *__restrict__ src_norm) {
    const int64_t n_src = counts[1];
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; j < n_src;
         j += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t u = src_ids[j];
        if (src_norm) src_norm[j] = gcn_norm[u];
        map[u] = -1;
    }
}

__global__ void edge_rows_kernel(const int64_t *__restrict__ brow, const int64_t *__restrict__ counts,
                                 int32_t *__restrict__ erow) {
    const int64_t n_dst = counts[0];
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n_dst) return;
    for (int64_t e = brow[i]; e < brow[i + 1]; ++e) erow[e] = static_cast<int32_t>(i);
}

// cscptr[j] = first position of key j in the sorted keys (lower bound).
__global__ void csc_ptr_kernel(const int32_t *__restrict__ skey, const int64_t *__restrict__ counts,
                               int64_t *__restrict__ cscptr) {
    const int64_t n_src = counts[1], nnz = counts[2];
    const int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (j > n_src) return;
    int64_t lo = 0, hi = nnz;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (skey[mid] < j) lo = mid + 1; else hi = mid;
    }
    cscptr[j] = lo;
}

struct SamplerWs {
    size_t map, bits, gcol, cnt, scan, pc, pcoff, pcscan, newtot, erow, skey, radix, total;
};

SamplerWs sampler_layout(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    const int64_t words = ceil_div(graph_n > 0 ? graph_n : 1, 32);
    const int64_t nbw = ceil_div(words, kBitTile);
    const int64_t cap_nnz = cap_dst * fanout;
    Carver c(nullptr);
    SamplerWs w;
    w.map = c.take(static_cast<size_t>(graph_n > 0 ? graph_n : 1) * 4);
    w.bits = c.take(static_cast<size_t>(words) * 4);
    w.gcol = c.take(static_cast<size_t>(cap_nnz > 0 ? cap_nnz : 1) * 8);
    w.cnt = c.take(static_cast<size_t>(cap_dst > 0 ? cap_dst : 1) * 8);
    w.scan = c.take(scan_tmp_bytes(cap_dst));
    w.pc = c.take(static_cast<size_t>(nbw) * 8);
    w.pcoff = c.take(static_cast<size_t>(nbw + 1) * 8);
    w.pcscan = c.take(scan_tmp_bytes(nbw));
    w.newtot = c.take(8);
    w.erow = c.take(static_cast<size_t>(cap_nnz > 0 ? cap_nnz : 1) * 4);
    w.skey = c.take(static_cast<size_t>(cap_nnz > 0 ? cap_nnz : 1) * 4);
    w.radix = c.take(radix_tmp_bytes(cap_nnz));
    w.total = round_up(c.off, 256);
    return w;
}

unsigned grid_for(int64_t items, int threads, int64_t max_blocks = 1 << 20) {
    int64_t b = ceil_div(items > 0 ? items : 1, threads);
    if (b > max_blocks) b = max_blocks;
    return static_cast<unsigned>(b);
}

int bits_for(int64_t v) {  // bits needed to represent values in [0, v)
    int b = 0;
    while (b < 62 && (1ll << b) < v) ++b;
    return b;
}

}  // namespace

size_t sampler_ws_bytes(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    return sampler_layout(graph_n, cap_dst, fanout).total;
}

gnn_status launch_sampler_ws_init(void *ws, int64_t graph_n, hipStream_t s) {
    SamplerWs w = sampler_layout(graph_n, 1, 1);
    char *base = static_cast<char *>(ws);
    const int64_t words = ceil_div(graph_n > 0 ? graph_n : 1, 32);
    fill_i32_kernel<<<grid_for(graph_n, kThreads, 65536), kThreads, 0, s>>>(
        reinterpret_cast<int32_t *>(base + w.map), graph_n, -1);
    GNN_LAUNCHED("sampler_ws_init(map)");
    fill_i32_kernel<<<grid_for(words, kThreads, 65536), kThreads, 0, s>>>(
        reinterpret_cast<int32_t *>(base + w.bits), words, 0);
    GNN_LAUNCHED("sampler_ws_init(bits)");
    return GNN_OK;
}

gnn_status launch_gcn_norm(const gnn_graph *g, float *nrm, hipStream_t s) {
    if (g->n == 0) return GNN_OK;
    gcn_norm_kernel<<<grid_for(g->n, kThreads, kMaxGrid), kThreads, 0, s>>>(g->rowptr, g->n, nrm);
    GNN_LAUNCHED("gcn_norm");
    return GNN_OK;
}

gnn_status launch_build_block(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids,
                              const int64_t *n_dst_dev, int32_t fanout, uint64_t seed, uint64_t step, int32_t hop,
                              bool want_csc, const gnn_block *out, void *ws, hipStream_t s) {
    const SamplerWs w = sampler_layout(g->n, out->cap_dst, fanout);
    char *base = static_cast<char *>(ws);
    int32_t *map = reinterpret_cast<int32_t *>(base + w.map);
    uint32_t *bits = reinterpret_cast<uint32_t *>(base + w.bits);
    int64_t *gcol = reinterpret_cast<int64_t *>(base + w.gcol);
    int64_t *cnt = reinterpret_cast<int64_t *>(base + w.cnt);
    int64_t *pc = reinterpret_cast<int64_t *>(base + w.pc);
    int64_t *pcoff = reinterpret_cast<int64_t *>(base + w.pcoff);
    int64_t *newtot = reinterpret_cast<int64_t *>(base + w.newtot);
    const int64_t words = ceil_div(g->n > 0 ? g->n : 1, 32);
    const int64_t nbw = ceil_div(words, kBitTile);
    const int64_t cap_dst = out->cap_dst;
    const int64_t cap_nnz = cap_dst * fanout;

    sample_count_kernel<<<grid_for(cap_dst, kThreads, kMaxGrid), kThreads, 0, s>>>(
        dst_ids, n_dst_dev, cap_dst, g->rowptr, fanout, map, cnt, out->src_ids, out->counts);
    GNN_LAUNCHED("sample_count");
    GNN_TRY(exclusive_scan(cnt, out->rowptr, out->counts, cap_dst, out->counts + 2, base + w.scan, s));

    const unsigned gw = grid_for(cap_dst * 64, kThreads, kMaxGrid);
    const uint64_t h = static_cast<uint64_t>(static_cast<int64_t>(hop));
    if (fanout <= 64)
        sample_floyd_kernel<1><<<gw, kThreads, 0, s>>>(dst_ids, out->counts, g->rowptr, g->col, out->rowptr, fanout,
                                                        seed, step, h, gcol);
    else if (fanout <= 128)
        sample_floyd_kernel<2><<<gw, kThreads, 0, s>>>(dst_ids, out->counts, g->rowptr, g->col, out->rowptr, fanout,
                                                        seed, step, h, gcol);
    else if (fanout <= 256)
        sample_floyd_kernel<4><<<gw, kThreads, 0, s>>>(dst_ids, out->counts, g->rowptr, g->col, out->rowptr, fanout,
                                                        seed, step, h, gcol);
    else if (fanout <= 512)
        sample_floyd_kernel<8><<<gw, kThreads, 0, s>>>(dst_ids, out->counts, g->rowptr, g->col, out->rowptr, fanout,
                                                        seed, step, h, gcol);
    else
        sample_floyd_kernel<16><<<gw, kThreads, 0, s>>>(dst_ids, out->counts, g->rowptr, g->col, out->rowptr,
                                                         fanout, seed, step, h, gcol);
    GNN_LAUNCHED("sample_floyd");

    const unsigned ge = grid_for(cap_nnz, kThreads, 1 << 16);
    mark_new_kernel<<<ge, kThreads, 0, s>>>(gcol, out->counts, map, bits);
    GNN_LAUNCHED("mark_new");
    bitmap_count_kernel<<<static_cast<unsigned>(nbw), kThreads, 0, s>>>(bits, words, pc);
    GNN_LAUNCHED("bitmap_count");
    GNN_TRY(exclusive_scan(pc, pcoff, nullptr, nbw, newtot, base + w.pcscan, s));
    bitmap_emit_kernel<<<static_cast<unsigned>(nbw), kThreads, 0, s>>>(bits, words, pcoff, newtot, out->counts,
                                                                       out->src_ids, map);
    GNN_LAUNCHED("bitmap_emit");
    relabel_kernel<<<ge, kThreads, 0, s>>>(gcol, out->counts, map, out->col);
    GNN_LAUNCHED("relabel");
    finish_kernel<<<grid_for(out->cap_src, kThreads, 1 << 16), kThreads, 0, s>>>(out->src_ids, out->counts, map,
                                                                                 gcn_norm, out->src_norm);
    GNN_LAUNCHED("finish");

    if (want_csc) {
        int32_t *erow = reinterpret_cast<int32_t *>(base + w.erow);
        int32_t *skey = reinterpret_cast<int32_t *>(base + w.skey);
        edge_rows_kernel<<<grid_for(cap_dst, kThreads, kMaxGrid), kThreads, 0, s>>>(out->rowptr, out->counts, erow);
        GNN_LAUNCHED("edge_rows");
        GNN_TRY(radix_sort_pairs(out->col, erow, skey, out->cscrow, out->counts + 2, cap_nnz,
                                 bits_for(out->cap_src), base + w.radix, s));
        csc_ptr_kernel<<<grid_for(out->cap_src + 1, kThreads, kMaxGrid), kThreads, 0, s>>>(skey, out->counts,
                                                                                          out->cscptr);
        GNN_LAUNCHED("csc_ptr");
    }
    return GNN_OK;
}

}  // namespace gnn
