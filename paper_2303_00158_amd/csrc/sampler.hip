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
//   3. relabel   one thread per staged sample: local index via the map
//                (and, for a block with a transpose, the count phase of the
//                transpose).
//   4. transpose scan, place and sort phases (csc_dev.h).
// The scans in step 2 are single-pass: workgroups take tickets in the order
// they start and add the prefix of earlier tickets (decoupled look-back,
// one wavefront reading 64 predecessors at a time), so a workgroup only
// waits on workgroups that are already running.  Every wait is bounded; a
// wait that runs out flags counts[3] (samp::kErrWait).
//
// Device workspace (sampler_ws_bytes):
//   map   int32[graph_n]   vertex -> local source index (valid only for the
//                          vertices of the current block)
//   bits  uint32[W]        one bit per vertex: "sampled"
//   dbits uint32[W]        one bit per vertex: "destination"
//   ... per-call scratch
// Both bitmaps are all zero between calls; each call clears the words it set.
#include <atomic>

#include "csc_dev.h"
#include "jobs.h"
#include "sampler_dev.h"

namespace gnn {

namespace {

// Error-path test hook (set_sampler_fault): the row scan's poll limit and
// the row tile that never publishes (-1: none).
std::atomic<uint32_t> g_row_spin_limit{samp::kSpinLimit};
std::atomic<int64_t> g_silent_row_tile{-1};

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
    w.csc = c.take(block_csc_ws_bytes(src_bound(graph_n, cap_dst, fanout), cap_nnz));
    w.total = round_up(c.off, 256);
    return w;
}

unsigned grid_for(int64_t items, int threads, int64_t max_blocks = 1 << 20) {
    int64_t b = ceil_div(items > 0 ? items : 1, threads);
    if (b > max_blocks) b = max_blocks;
    return static_cast<unsigned>(b);
}

// Transpose scratch: edge rows, column counters, scan look-back state.
struct CscWs {
    size_t erow, cnt, status, ticket, total;
    int64_t nb_scan;
};
CscWs csc_layout(int64_t cap_src, int64_t cap_nnz) {
    CscWs w;
    w.nb_scan = ceil_div(cap_src + 1, csc::kScanTile);
    Carver c(nullptr);
    w.erow = c.take(static_cast<size_t>(std::max<int64_t>(cap_nnz, 1)) * 4);
    w.cnt = c.take(static_cast<size_t>(std::max<int64_t>(cap_src, 1)) * 4);
    w.status = c.take(static_cast<size_t>(w.nb_scan) * 8);
    w.ticket = c.take(4);
    w.total = round_up(c.off, 256);
    return w;
}

}  // namespace

// Bound on a block's sources: destinations plus sampled edges, at most the
// graph (the capacity rule of gnn_block_bounds).
int64_t src_bound(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    return std::min<int64_t>(cap_dst + cap_dst * fanout, std::max<int64_t>(graph_n, cap_dst));
}

size_t block_csc_ws_bytes(int64_t cap_src, int64_t cap_nnz) { return csc_layout(cap_src, cap_nnz).total; }

csc::Args csc_args(const gnn_block *out, void *csc_ws, int64_t ws_src, int64_t ws_nnz) {
    const CscWs w = csc_layout(ws_src, ws_nnz);
    char *base = static_cast<char *>(csc_ws);
    csc::Args a;
    a.counts = out->counts;
    a.bcol = out->col;
    a.erow = reinterpret_cast<int32_t *>(base + w.erow);
    a.cap_src = std::min(out->cap_src, ws_src);
    a.cap_nnz = std::min(out->cap_nnz, ws_nnz);
    a.cnt = reinterpret_cast<int32_t *>(base + w.cnt);
    a.status = reinterpret_cast<uint64_t *>(base + w.status);
    a.ticket = reinterpret_cast<int *>(base + w.ticket);
    a.nb_scan = ceil_div(a.cap_src + 1, csc::kScanTile);
    a.cscptr = out->cscptr;
    a.cscrow = out->cscrow;
    return a;
}

csc::Grids csc_grids(const csc::Args &a) {
    csc::Grids g;
    g.scan = static_cast<unsigned>(a.nb_scan);
    g.place = grid_for(a.cap_nnz, csc::kThreads, 2048);
    g.sort = grid_for(ceil_div(a.cap_src, 64), csc::kThreads / 64, 2048);
    return g;
}

gnn_status launch_block_csc(const csc::Args &a, hipStream_t s) {
    const csc::Grids g = csc_grids(a);
    GNN_TRY(launch_job(csc::ScanJob{a}, g.scan, s, "csc_scan"));
    GNN_TRY(launch_job(csc::PlaceJob{a}, g.place, s, "csc_place"));
    return launch_job(csc::SortJob{a}, g.sort, s, "csc_sort");
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
                       void *scratch, const csc::Args *csc) {
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
    a.erow = csc ? csc->erow : nullptr;
    a.csc_cnt = csc ? csc->cnt : nullptr;
    a.csc_cap_src = csc ? csc->cap_src : 0;
    a.csc_status = csc ? csc->status : nullptr;
    a.csc_ticket = csc ? csc->ticket : nullptr;
    a.csc_nb = csc ? csc->nb_scan : 0;
    a.spin_limit = g_row_spin_limit.load(std::memory_order_relaxed);
    a.silent_row_tile = g_silent_row_tile.load(std::memory_order_relaxed);
    a.status = reinterpret_cast<uint64_t *>(hbase + hw.status);
    a.ticket = reinterpret_cast<int *>(hbase + hw.ticket);
    a.nb_rows = ceil_div(out->cap_dst > 0 ? out->cap_dst : 1, kThreads);
    a.nb_bits = ceil_div(a.words, kBitTile);
    // one wavefront per destination row, at most 2048 workgroups (8192
    // wavefronts) striding over the rows: capacity-sized grids would mostly
    // hold workgroups that read the row count only to exit
    p.prep_grid = grid_for(std::max<int64_t>(out->cap_dst, 1) * 64, kThreads, 2048);
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
                              const gnn_block *out, void *ws, const csc::Args *csc, hipStream_t s) {
    void *scratch = static_cast<char *>(ws) + sampler_shared_bytes(g->n);
    const samp::HopPlan p =
        plan_hop(g, gcn_norm, dst_ids, n_dst_dev, fanout, seed, step, hop, out, ws, scratch, csc);
    GNN_TRY(launch_hop_prepare(p, s));
    GNN_TRY(launch_hop_emit(p, s));
    hop_relabel_kernel<<<p.relabel_grid, kThreads, 0, s>>>(p.a);
    GNN_LAUNCHED("hop_relabel");
    return GNN_OK;
}

void set_sampler_fault(int64_t silent_row_tile, uint32_t spin_limit) {
    g_silent_row_tile.store(silent_row_tile, std::memory_order_relaxed);
    g_row_spin_limit.store(spin_limit, std::memory_order_relaxed);
}

}  // namespace gnn
