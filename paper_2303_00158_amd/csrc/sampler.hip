// Mini-batch sampler: one block (hop) of uniform neighbour sampling without
// replacement, relabelled to local indices, with its transpose.
//
// A hop is three kernels (plus one for the transpose):
//   1. prepare   one wavefront per destination: map the destination to its
//                local index and mark it in the destination bitmap, draw its
//                sample (Floyd), write the sampled neighbour ids to a padded
//                [n_dst][k] staging array and mark them in the sample bitmap.
//   2. emit      the first workgroups scan the sample counts into the
//                block's row pointer; the rest walk the bitmaps in vertex
//                order: every vertex that was sampled and is not a
//                destination becomes the next new source (so new sources
//                come out in ascending id order); both bitmaps are cleared.
//   3. relabel   one thread per staged sample: local index via the map.
//   4. transpose one workgroup: stable radix sort of the edges by source.
// The scans in step 2 are single-pass: workgroups take tickets in the order
// they start and add the prefix of earlier tickets (decoupled look-back,
// one wavefront reading 64 predecessors at a time), so a workgroup only
// waits on workgroups that are already running.  Every wait is bounded; a
// wait that runs out flags counts[3].
//
// Device workspace (sampler_ws_bytes):
//   map   int32[graph_n]   vertex -> local source index (valid only for the
//                          vertices of the current block)
//   bits  uint32[W]        one bit per vertex: "sampled"
//   dbits uint32[W]        one bit per vertex: "destination"
//   ... per-call scratch
// Both bitmaps are all zero between calls; each call clears the words it set.
#include "sampler_dev.h"

namespace gnn {

namespace {

constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / 64;
using namespace samp;

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

template <int R>
__global__ void __launch_bounds__(kThreads) hop_prepare_kernel(HopArgs a) {
    hop_prepare_body<R>(a, blockIdx.x, gridDim.x);
}

__global__ void __launch_bounds__(kThreads) hop_emit_kernel(HopArgs a) { hop_emit_body(a); }

__global__ void __launch_bounds__(kThreads) hop_relabel_kernel(HopArgs a) {
    hop_relabel_body(a, blockIdx.x, gridDim.x);
}

// 4. stable transpose in one workgroup: LSD radix sort of (source, row) by
// source, 8 bits per pass.  Each wavefront owns a contiguous segment of the
// edge list; per pass the segments' digit histograms give every (segment,
// digit) its output offset, and the segments are scattered in order with
// ballot-based ranks, which keeps equal keys in edge order.  Then the row
// pointer of the transpose is read off the sorted keys.
__global__ void __launch_bounds__(kSortThreads) csc_build_kernel(const int32_t *__restrict__ keys_in,
                                                                  const int32_t *__restrict__ vals_in,
                                                                  const int64_t *__restrict__ counts, int key_bits,
                                                                  int32_t *ka, int32_t *va, int32_t *kb, int32_t *vb,
                                                                  int32_t *__restrict__ cscrow,
                                                                  int64_t *__restrict__ cscptr) {
    __shared__ int hist[kSortWaves][256];
    __shared__ int tot[256];
    const int64_t n = counts[2], n_src = counts[1];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t seg = ceil_div(ceil_div(n > 0 ? n : 1, kSortWaves), 64) * 64;
    const int64_t chunks = seg / 64;
    const int passes = key_bits <= 8 ? 1 : (key_bits + 7) / 8;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int32_t *ks = keys_in, *vs = vals_in;
    int32_t *kfinal = ka;
    for (int p = 0; p < passes; ++p) {
        const int shift = 8 * p;
        const bool last = p == passes - 1;
        int32_t *kd = (p % 2 == 0) ? ka : kb;
        int32_t *vd = last ? cscrow : ((p % 2 == 0) ? va : vb);
        for (int d = threadIdx.x; d < kSortWaves * 256; d += kSortThreads) (&hist[0][0])[d] = 0;
        __syncthreads();
        const int64_t s0 = wave * seg;
        const int64_t s1 = min(n, s0 + seg);
        for (int64_t q0 = s0 + lane; q0 < s1; q0 += 4 * 64) {
            int32_t kk[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) kk[b] = ks[min(q0 + b * 64, s1 - 1)];
#pragma unroll
            for (int b = 0; b < 4; ++b)
                if (q0 + b * 64 < s1) atomicAdd(&hist[wave][(kk[b] >> shift) & 255], 1);
        }
        __syncthreads();
        if (threadIdx.x < 256) {
            int s = 0;
            for (int w = 0; w < kSortWaves; ++w) s += hist[w][threadIdx.x];
            tot[threadIdx.x] = s;
        }
        __syncthreads();
        if (threadIdx.x < 256) {
            int base = 0;
            for (int d = 0; d < static_cast<int>(threadIdx.x); ++d) base += tot[d];
            for (int w = 0; w < kSortWaves; ++w) {
                const int h = hist[w][threadIdx.x];
                hist[w][threadIdx.x] = base;
                base += h;
            }
        }
        __syncthreads();
        int32_t kb[4], vb4[4];
        for (int64_t ch = 0; ch < chunks; ++ch) {
            const int64_t q = s0 + ch * 64 + lane;
            const bool valid = q < n && q < s0 + seg;
            if ((ch & 3) == 0) {
                // load the next four chunks of this segment at once
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int64_t qb = q + b * 64;
                    const int64_t qc = (qb < n) ? qb : (n > 0 ? n - 1 : 0);
                    kb[b] = ks[qc];
                    vb4[b] = vs[qc];
                }
            }
            const int32_t key = valid ? kb[ch & 3] : 0;
            const int32_t val = valid ? vb4[ch & 3] : 0;
            const int d = (key >> shift) & 255;
            uint64_t peers = __ballot(valid);
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                const bool bit = (d >> b) & 1;
                const uint64_t m = __ballot(valid && bit);
                peers &= bit ? m : ~m;
            }
            const int rank = __popcll(peers & lt);
            const int at = valid ? hist[wave][d] : 0;
            __syncthreads();
            if (valid) {
                kd[at + rank] = key;
                vd[at + rank] = val;
                if (rank == 0) hist[wave][d] = at + __popcll(peers);
            }
            __syncthreads();
        }
        __threadfence_block();
        __syncthreads();
        ks = kd;
        vs = vd;
        kfinal = kd;
    }
    // cscptr[j] = first position of key j
    if (n == 0) {
        for (int64_t j = threadIdx.x; j <= n_src; j += kSortThreads) cscptr[j] = 0;
        return;
    }
    for (int64_t pos = threadIdx.x; pos <= n; pos += kSortThreads) {
        const int64_t lo = (pos == 0) ? -1 : kfinal[pos - 1];
        const int64_t hi = (pos == n) ? n_src : kfinal[pos];
        for (int64_t j = lo + 1; j <= hi; ++j) cscptr[j] = pos;
    }
}

// Shared part: depends on graph_n only, so one serves hops of any size.
struct SharedWs {
    size_t map, bits, dbits, total;
};
SharedWs shared_layout(int64_t graph_n) {
    const int64_t words = ceil_div(graph_n > 0 ? graph_n : 1, 32);
    Carver c(nullptr);
    SharedWs w;
    w.map = c.take(static_cast<size_t>(graph_n > 0 ? graph_n : 1) * 4);
    w.bits = c.take(static_cast<size_t>(words) * 4);
    w.dbits = c.take(static_cast<size_t>(words) * 4);
    w.total = round_up(c.off, 256);
    return w;
}

// Per-hop scratch: staged samples, counts, look-back state, transpose.
struct HopWs {
    size_t gpad, cnt, status, ticket, csc, total;
};
HopWs hop_layout(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    const int64_t words = ceil_div(graph_n > 0 ? graph_n : 1, 32);
    const int64_t nb_rows = ceil_div(cap_dst > 0 ? cap_dst : 1, kThreads);
    const int64_t nb_bits = ceil_div(words, kBitTile);
    const int64_t cap_nnz = std::max<int64_t>(cap_dst * fanout, 1);
    Carver c(nullptr);
    HopWs w;
    w.gpad = c.take(static_cast<size_t>(cap_nnz) * 8);
    w.cnt = c.take(static_cast<size_t>(cap_dst > 0 ? cap_dst : 1) * 4);
    w.status = c.take(static_cast<size_t>(nb_rows + nb_bits) * 8);
    w.ticket = c.take(4);
    w.csc = c.take(block_csc_ws_bytes(cap_nnz));
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

// Transpose scratch: the row of every edge, then two key / value ping-pong
// pairs for the radix sort.
size_t block_csc_ws_bytes(int64_t cap_nnz) {
    return round_up(static_cast<size_t>(std::max<int64_t>(cap_nnz, 1)) * 4 * 5, 256);
}

size_t sampler_shared_bytes(int64_t graph_n) { return shared_layout(graph_n).total; }
size_t sampler_hop_bytes(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    return hop_layout(graph_n, cap_dst, fanout).total;
}
size_t sampler_ws_bytes(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    return sampler_shared_bytes(graph_n) + sampler_hop_bytes(graph_n, cap_dst, fanout);
}

gnn_status launch_sampler_ws_init(void *ws, int64_t graph_n, hipStream_t s) {
    const SharedWs w = shared_layout(graph_n);
    char *base = static_cast<char *>(ws);
    fill_i32_kernel<<<grid_for(graph_n, kThreads, 65536), kThreads, 0, s>>>(
        reinterpret_cast<int32_t *>(base + w.map), graph_n, -1);
    GNN_LAUNCHED("sampler_ws_init(map)");
    // bits and dbits are adjacent: clear both
    const int64_t words = static_cast<int64_t>((w.total - w.bits) / 4);
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

void *sampler_csc_ws(void *ws, int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    return static_cast<char *>(ws) + sampler_shared_bytes(graph_n) + hop_layout(graph_n, cap_dst, fanout).csc;
}

samp::HopPlan plan_hop(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids, const int64_t *n_dst_dev,
                       int32_t fanout, uint64_t seed, uint64_t step, int32_t hop, const gnn_block *out, void *shared,
                       void *scratch, void *csc_ws) {
    const SharedWs w = shared_layout(g->n);
    const HopWs hw = hop_layout(g->n, out->cap_dst, fanout);
    char *base = static_cast<char *>(shared);
    char *hbase = static_cast<char *>(scratch);
    samp::HopPlan p;
    HopArgs &a = p.a;
    a.rowptr = g->rowptr;
    a.col = g->col;
    a.gcn_norm = out->src_norm ? gcn_norm : nullptr;
    a.dst = dst_ids;
    a.n_dst_dev = n_dst_dev;
    a.cap_dst = out->cap_dst;
    a.k = fanout;
    a.seed = seed;
    a.step = step;
    a.hop = static_cast<uint64_t>(static_cast<int64_t>(hop));
    a.counts = out->counts;
    a.src_ids = out->src_ids;
    a.brow = out->rowptr;
    a.bcol = out->col;
    a.src_norm = out->src_norm;
    a.map = reinterpret_cast<int32_t *>(base + w.map);
    a.bits = reinterpret_cast<uint32_t *>(base + w.bits);
    a.dbits = reinterpret_cast<uint32_t *>(base + w.dbits);
    a.words = ceil_div(g->n > 0 ? g->n : 1, 32);
    a.gpad = reinterpret_cast<int64_t *>(hbase + hw.gpad);
    a.cnt = reinterpret_cast<int32_t *>(hbase + hw.cnt);
    a.erow = static_cast<int32_t *>(csc_ws);
    a.status = reinterpret_cast<uint64_t *>(hbase + hw.status);
    a.ticket = reinterpret_cast<int *>(hbase + hw.ticket);
    a.nb_rows = ceil_div(out->cap_dst > 0 ? out->cap_dst : 1, kThreads);
    a.nb_bits = ceil_div(a.words, kBitTile);
    p.prep_grid = grid_for(std::max<int64_t>(out->cap_dst, 1) * 64, kThreads, kMaxGrid);
    p.emit_grid = static_cast<unsigned>(a.nb_rows + a.nb_bits);
    p.relabel_grid = grid_for(std::max<int64_t>(out->cap_dst, 1) * fanout, kThreads, 1 << 16);
    p.r = fanout <= 64 ? 1 : fanout <= 128 ? 2 : fanout <= 256 ? 4 : fanout <= 512 ? 8 : 16;
    return p;
}

gnn_status launch_hop_prepare(const samp::HopPlan &p, hipStream_t s) {
    switch (p.r) {
        case 1: hop_prepare_kernel<1><<<p.prep_grid, kThreads, 0, s>>>(p.a); break;
        case 2: hop_prepare_kernel<2><<<p.prep_grid, kThreads, 0, s>>>(p.a); break;
        case 4: hop_prepare_kernel<4><<<p.prep_grid, kThreads, 0, s>>>(p.a); break;
        case 8: hop_prepare_kernel<8><<<p.prep_grid, kThreads, 0, s>>>(p.a); break;
        default: hop_prepare_kernel<16><<<p.prep_grid, kThreads, 0, s>>>(p.a); break;
    }
    GNN_LAUNCHED("hop_prepare");
    return GNN_OK;
}

gnn_status launch_hop_emit(const samp::HopPlan &p, hipStream_t s) {
    hop_emit_kernel<<<p.emit_grid, kThreads, 0, s>>>(p.a);
    GNN_LAUNCHED("hop_emit");
    return GNN_OK;
}

gnn_status launch_build_block(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids,
                              const int64_t *n_dst_dev, int32_t fanout, uint64_t seed, uint64_t step, int32_t hop,
                              const gnn_block *out, void *ws, void *csc_ws, hipStream_t s) {
    void *scratch = static_cast<char *>(ws) + sampler_shared_bytes(g->n);
    const samp::HopPlan p =
        plan_hop(g, gcn_norm, dst_ids, n_dst_dev, fanout, seed, step, hop, out, ws, scratch, csc_ws);
    GNN_TRY(launch_hop_prepare(p, s));
    GNN_TRY(launch_hop_emit(p, s));
    hop_relabel_kernel<<<p.relabel_grid, kThreads, 0, s>>>(p.a);
    GNN_LAUNCHED("hop_relabel");
    return GNN_OK;
}

gnn_status launch_block_csc(const gnn_block *out, void *csc_ws, int64_t scratch_nnz, hipStream_t s) {
    const int64_t cap_nnz = std::max<int64_t>(scratch_nnz, 1);
    int32_t *erow = static_cast<int32_t *>(csc_ws);
    int32_t *sort = erow + cap_nnz;
    csc_build_kernel<<<1, kSortThreads, 0, s>>>(out->col, erow, out->counts, bits_for(out->cap_src), sort,
                                                sort + cap_nnz, sort + 2 * cap_nnz, sort + 3 * cap_nnz, out->cscrow,
                                                out->cscptr);
    GNN_LAUNCHED("csc_build");
    return GNN_OK;
}

}  // namespace gnn
