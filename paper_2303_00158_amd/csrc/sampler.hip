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
#include "internal.h"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int kBitWords = 8;                      // bitmap words per thread in the emit kernel
constexpr int kBitTile = kThreads * kBitWords;    // bitmap words per workgroup
constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / 64;
constexpr uint64_t kFlagAgg = 1ull << 62, kFlagPrefix = 2ull << 62, kValueMask = (1ull << 62) - 1;
constexpr uint32_t kSpinLimit = 1u << 22;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t load_status(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_status(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Logical workgroup index: the order in which workgroups started.
__device__ __forceinline__ int64_t take_ticket(int *ticket) {
    __shared__ int64_t t;
    if (threadIdx.x == 0) t = atomicAdd(ticket, 1);
    __syncthreads();
    return t;
}

__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Called by all 64 lanes of one wavefront: publish this workgroup's
// aggregate, add up the aggregates / prefixes of earlier tickets 64 at a
// time (lane j reads ticket blk-1-j-64w), publish the inclusive prefix, and
// return the exclusive prefix.
__device__ int64_t look_back(uint64_t *status, int64_t blk, int64_t agg, int64_t *err) {
    const int lane = threadIdx.x & 63;
    if (blk == 0) {
        if (lane == 0) store_status(&status[0], kFlagPrefix | static_cast<uint64_t>(agg));
        return 0;
    }
    if (lane == 0) store_status(&status[blk], kFlagAgg | static_cast<uint64_t>(agg));
    int64_t excl = 0;
    int64_t hi = blk - 1;
    uint32_t spins = 0;
    while (true) {
        const int64_t p = hi - lane;
        // tickets before 0 read as a zero prefix, which ends every walk
        const uint64_t s = p >= 0 ? load_status(&status[p]) : kFlagPrefix;
        const uint64_t flag = s & ~kValueMask;
        const uint64_t pre = __ballot(flag == kFlagPrefix);
        const int first = pre ? static_cast<int>(__builtin_ctzll(pre)) : 63;
        const uint64_t need = (first == 63) ? ~0ull : ((1ull << (first + 1)) - 1);
        if (__ballot(flag == 0) & need) {
            if (++spins > kSpinLimit) {
                if (lane == 0) *err = 1;  // an earlier workgroup never published: flag it and stop
                break;
            }
            continue;
        }
        excl += wave_sum64(lane <= first ? static_cast<int64_t>(s & kValueMask) : 0);
        if (pre) break;
        hi -= 64;
    }
    if (lane == 0) store_status(&status[blk], kFlagPrefix | static_cast<uint64_t>(excl + agg));
    return excl;
}

__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t *total) {
    __shared__ int64_t sh[kThreads / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
    }
    if (lane == 63) sh[wave] = inc;
    __syncthreads();
    int64_t base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
        if (w < wave) base += sh[w];
        tot += sh[w];
    }
    __syncthreads();
    *total = tot;
    return base + inc - v;
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

struct HopArgs {
    const int64_t *rowptr, *col;  // graph
    const float *gcn_norm;        // per vertex, or null
    const int64_t *dst;
    const int64_t *n_dst_dev;
    int64_t cap_dst;
    int32_t k;
    uint64_t seed, step, hop;
    // block
    int64_t *counts, *src_ids, *brow;
    int32_t *bcol;
    float *src_norm;
    // workspace
    int32_t *map;
    uint32_t *bits, *dbits;
    int64_t words;
    int64_t *gpad;      // [cap_dst][k] sampled global ids
    int32_t *cnt;       // [cap_dst] sample counts
    int32_t *erow;      // [cap_nnz] row of each edge (for the transpose) or null
    uint64_t *status;   // [nb_rows + nb_bits] look-back words
    int *ticket;
    int64_t nb_rows, nb_bits;
};

__device__ __forceinline__ void set_bit(uint32_t *bm, int64_t v) {
    atomicOr(&bm[v >> 5], 1u << (v & 31));
}

// 1. prepare: one wavefront per destination row.  R drawn positions per lane
// (slot s lives in lane s % 64, register s / 64).
template <int R>
__global__ void __launch_bounds__(kThreads) hop_prepare_kernel(HopArgs a) {
    const int64_t gtid = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const int64_t gsize = static_cast<int64_t>(gridDim.x) * kThreads;
    const int64_t n_dst = a.n_dst_dev ? min(*a.n_dst_dev, a.cap_dst) : a.cap_dst;
    // reset the look-back state of the emit kernel
    for (int64_t i = gtid; i < a.nb_rows + a.nb_bits; i += gsize) a.status[i] = 0;
    if (gtid == 0) {
        *a.ticket = 0;
        a.counts[0] = n_dst;
        a.counts[3] = 0;
    }
    const int lane = threadIdx.x & 63;
    const int64_t row = gtid >> 6;
    if (row >= n_dst) return;
    const int64_t v = a.dst[row];
    const int64_t beg = a.rowptr[v];
    const int64_t d = a.rowptr[v + 1] - beg;
    const int32_t k = a.k;
    int64_t *out = a.gpad + row * k;
    if (lane == 0) {
        a.map[v] = static_cast<int32_t>(row);
        a.src_ids[row] = v;
        if (a.src_norm) a.src_norm[row] = a.gcn_norm[v];
        a.cnt[row] = static_cast<int32_t>(d < k ? d : k);
        set_bit(a.dbits, v);
    }
    if (d <= k) {
        for (int64_t p = lane; p < d; p += 64) {
            const int64_t u = a.col[beg + p];
            out[p] = u;
            set_bit(a.bits, u);
        }
        return;
    }
    uint32_t slot[R];
#pragma unroll
    for (int r = 0; r < R; ++r) slot[r] = 0xffffffffu;
    const uint64_t pk = mix64(mix64(mix64(mix64(a.seed) ^ a.step) ^ a.hop) ^ static_cast<uint64_t>(v));
    for (int32_t t = 0; t < k; ++t) {
        const uint64_t j = static_cast<uint64_t>(d - k + t);
        const uint64_t key = mix64(pk ^ static_cast<uint64_t>(t));
        const uint32_t x = static_cast<uint32_t>(((key >> 32) * (j + 1)) >> 32);
        bool mine = false;
#pragma unroll
        for (int r = 0; r < R; ++r) mine |= (r * 64 + lane < t) && (slot[r] == x);
        const bool found = __ballot(mine) != 0ull;
        const uint32_t val = found ? static_cast<uint32_t>(j) : x;
        if (lane == (t & 63)) {
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (r == (t >> 6)) slot[r] = val;
        }
    }
    // rank of each drawn position among all k (they are distinct)
    int rank[R];
#pragma unroll
    for (int r = 0; r < R; ++r) rank[r] = 0;
    for (int32_t s = 0; s < k; ++s) {
        uint32_t mine = 0;
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (r == (s >> 6)) mine = slot[r];
        const uint32_t other = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(mine), s & 63));
#pragma unroll
        for (int r = 0; r < R; ++r) rank[r] += (other < slot[r]) ? 1 : 0;
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (r * 64 + lane < k) {
            const int64_t u = a.col[beg + slot[r]];
            out[rank[r]] = u;
            set_bit(a.bits, u);
        }
    }
}

// 2a. row pointer of the block: scan of the sample counts (logical block
// `blk` owns rows [256 blk, 256 blk + 256)).
__device__ void emit_rows(const HopArgs &a, int64_t blk, int64_t n_dst) {
    const int64_t i = blk * kThreads + threadIdx.x;
    const int64_t c = (i < n_dst) ? a.cnt[i] : 0;
    int64_t total;
    const int64_t excl_in_block = block_excl_scan(c, &total);
    __shared__ int64_t base;
    if (threadIdx.x < 64) {
        const int64_t b = look_back(a.status, blk, total, &a.counts[3]);
        if (threadIdx.x == 0) base = b;
    }
    __syncthreads();
    if (i < n_dst) a.brow[i + 1] = base + excl_in_block + c;
    if (blk == 0 && threadIdx.x == 0) a.brow[0] = 0;
    if (blk == a.nb_rows - 1 && threadIdx.x == 0) a.counts[2] = base + total;
}

// 2b. new sources in ascending vertex order (logical block `blk` owns
// kBitTile bitmap words).
__device__ void emit_sources(const HopArgs &a, int64_t blk, int64_t n_dst) {
    const int64_t w0 = blk * kBitTile + threadIdx.x * kBitWords;
    uint32_t sw[kBitWords], dw[kBitWords];
#pragma unroll
    for (int q = 0; q < kBitWords; ++q) {
        const int64_t w = (w0 + q < a.words) ? w0 + q : 0;
        sw[q] = a.bits[w];
        dw[q] = a.dbits[w];
    }
    int64_t c = 0;
#pragma unroll
    for (int q = 0; q < kBitWords; ++q) {
        if (w0 + q >= a.words) sw[q] = dw[q] = 0u;
        c += __popc(sw[q] & ~dw[q]);
    }
    int64_t total;
    const int64_t excl_in_block = block_excl_scan(c, &total);
    __shared__ int64_t base;
    if (threadIdx.x < 64) {
        const int64_t b = look_back(a.status + a.nb_rows, blk, total, &a.counts[3]);
        if (threadIdx.x == 0) base = b;
    }
    __syncthreads();
    int64_t r = n_dst + base + excl_in_block;
#pragma unroll
    for (int q = 0; q < kBitWords; ++q) {
        uint32_t m = sw[q] & ~dw[q];
        const int64_t wbase = (w0 + q) * 32;
        while (m) {
            const int b = __builtin_ctz(m);
            m &= m - 1;
            const int64_t u = wbase + b;
            a.src_ids[r] = u;
            a.map[u] = static_cast<int32_t>(r);
            if (a.src_norm) a.src_norm[r] = a.gcn_norm[u];
            ++r;
        }
        if (sw[q]) a.bits[w0 + q] = 0u;
        if (dw[q]) a.dbits[w0 + q] = 0u;
    }
    if (blk == a.nb_bits - 1 && threadIdx.x == 0) a.counts[1] = n_dst + base + total;
}

// 2. one launch, two roles: the first nb_rows tickets scan the rows, the
// rest emit the new sources.  The role is uniform per workgroup.
__global__ void __launch_bounds__(kThreads) hop_emit_kernel(HopArgs a) {
    const int64_t t = take_ticket(a.ticket);
    const int64_t n_dst = a.counts[0];
    if (t < a.nb_rows)
        emit_rows(a, t, n_dst);
    else
        emit_sources(a, t - a.nb_rows, n_dst);
}

// 3. local source index of every sampled edge.
__global__ void __launch_bounds__(kThreads) hop_relabel_kernel(HopArgs a) {
    const int64_t n_dst = a.counts[0];
    const int64_t total = n_dst * a.k;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; q < total;
         q += static_cast<int64_t>(gridDim.x) * kThreads) {
        const int64_t i = q / a.k, t = q - i * a.k;
        if (t >= a.cnt[i]) continue;
        const int64_t e = a.brow[i] + t;
        a.bcol[e] = a.map[a.gpad[q]];
        if (a.erow) a.erow[e] = static_cast<int32_t>(i);
    }
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

struct SamplerWs {
    size_t map, bits, dbits, gpad, cnt, status, ticket, csc, total;
};

// map, bits and dbits depend on graph_n only, so one workspace serves hops
// of any size.
SamplerWs sampler_layout(int64_t graph_n, int64_t cap_dst, int32_t fanout) {
    const int64_t words = ceil_div(graph_n > 0 ? graph_n : 1, 32);
    const int64_t nb_rows = ceil_div(cap_dst > 0 ? cap_dst : 1, kThreads);
    const int64_t nb_bits = ceil_div(words, kBitTile);
    const int64_t cap_nnz = std::max<int64_t>(cap_dst * fanout, 1);
    Carver c(nullptr);
    SamplerWs w;
    w.map = c.take(static_cast<size_t>(graph_n > 0 ? graph_n : 1) * 4);
    w.bits = c.take(static_cast<size_t>(words) * 4);
    w.dbits = c.take(static_cast<size_t>(words) * 4);
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
    // bits and dbits are adjacent: clear both
    fill_i32_kernel<<<grid_for(2 * words, kThreads, 65536), kThreads, 0, s>>>(
        reinterpret_cast<int32_t *>(base + w.bits), static_cast<int64_t>((w.gpad - w.bits) / 4), 0);
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
    return static_cast<char *>(ws) + sampler_layout(graph_n, cap_dst, fanout).csc;
}

gnn_status launch_build_block(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids,
                              const int64_t *n_dst_dev, int32_t fanout, uint64_t seed, uint64_t step, int32_t hop,
                              const gnn_block *out, void *ws, void *csc_ws, hipStream_t s) {
    const SamplerWs w = sampler_layout(g->n, out->cap_dst, fanout);
    char *base = static_cast<char *>(ws);
    HopArgs a;
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
    a.gpad = reinterpret_cast<int64_t *>(base + w.gpad);
    a.cnt = reinterpret_cast<int32_t *>(base + w.cnt);
    a.erow = static_cast<int32_t *>(csc_ws);
    a.status = reinterpret_cast<uint64_t *>(base + w.status);
    a.ticket = reinterpret_cast<int *>(base + w.ticket);
    a.nb_rows = ceil_div(out->cap_dst > 0 ? out->cap_dst : 1, kThreads);
    a.nb_bits = ceil_div(a.words, kBitTile);

    const unsigned gw = grid_for(std::max<int64_t>(out->cap_dst, 1) * 64, kThreads, kMaxGrid);
    if (fanout <= 64) hop_prepare_kernel<1><<<gw, kThreads, 0, s>>>(a);
    else if (fanout <= 128) hop_prepare_kernel<2><<<gw, kThreads, 0, s>>>(a);
    else if (fanout <= 256) hop_prepare_kernel<4><<<gw, kThreads, 0, s>>>(a);
    else if (fanout <= 512) hop_prepare_kernel<8><<<gw, kThreads, 0, s>>>(a);
    else hop_prepare_kernel<16><<<gw, kThreads, 0, s>>>(a);
    GNN_LAUNCHED("hop_prepare");
    hop_emit_kernel<<<static_cast<unsigned>(a.nb_rows + a.nb_bits), kThreads, 0, s>>>(a);
    GNN_LAUNCHED("hop_emit");
    hop_relabel_kernel<<<grid_for(std::max<int64_t>(out->cap_dst, 1) * fanout, kThreads, 1 << 16), kThreads, 0, s>>>(a);
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
