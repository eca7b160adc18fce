// Device side of the sampler (see sampler.hip): the hop's argument block and
// the bodies of its kernels, each taking its logical workgroup index and
// count so that a launch can run it alongside other work.
#pragma once

#include "internal.h"

namespace gnn {
namespace csc {
struct Args;
}
namespace samp {

constexpr int kThreads = 256;
constexpr int kBitWords = 8;                      // bitmap words per thread in the emit kernel
constexpr int kBitTile = kThreads * kBitWords;    // bitmap words per workgroup
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

// Device error flags of a block (its counts[3]; gnn.h names them): set
// with an atomic OR, so that concurrent checks keep every flag.
constexpr int64_t kErrWait = 1;   // a bounded wait for an earlier workgroup gave up
constexpr int64_t kErrRange = 2;  // an index derived from device data was out of range
__device__ __forceinline__ void flag_error(int64_t *err, int64_t flag) {
    atomicOr(reinterpret_cast<unsigned long long *>(err), static_cast<unsigned long long>(flag));
}

// Called by all 64 lanes of one wavefront: publish this workgroup's
// aggregate, add up the aggregates / prefixes of earlier tickets 64 at a
// time (lane j reads ticket blk-1-j-64w), publish the inclusive prefix, and
// return the exclusive prefix.  Waits for an earlier ticket give up after
// spin_limit polls and flag kErrWait.  `silent` (normally -1) names a ticket
// that publishes nothing: a host-driven test of that path.
__device__ inline int64_t look_back(uint64_t *status, int64_t blk, int64_t agg, int64_t *err,
                                    uint32_t spin_limit = kSpinLimit, int64_t silent = -1) {
    const int lane = threadIdx.x & 63;
    const bool publish = blk != silent;
    if (blk == 0) {
        if (lane == 0 && publish) store_status(&status[0], kFlagPrefix | static_cast<uint64_t>(agg));
        return 0;
    }
    if (lane == 0 && publish) store_status(&status[blk], kFlagAgg | static_cast<uint64_t>(agg));
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
            if (++spins > spin_limit) {
                if (lane == 0) flag_error(err, kErrWait);  // an earlier workgroup never published
                break;
            }
            continue;
        }
        excl += wave_sum64(lane <= first ? static_cast<int64_t>(s & kValueMask) : 0);
        if (pre) break;
        hi -= 64;
    }
    if (lane == 0 && publish) store_status(&status[blk], kFlagPrefix | static_cast<uint64_t>(excl + agg));
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
    // count phase of the transpose (when erow is set): per-column counters
    // and the transpose scan's look-back state, reset by the prepare
    int32_t *csc_cnt;
    int64_t csc_cap_src;
    uint64_t *csc_status;
    int *csc_ticket;
    int64_t csc_nb;
    // the row scan's bounded wait (kSpinLimit polls) and its silent ticket
    // (-1: none), changed only by the host's error-path test hook
    uint32_t spin_limit;
    int64_t silent_row_tile;
};

__device__ __forceinline__ void set_bit(uint32_t *bm, int64_t v) {
    atomicOr(&bm[v >> 5], 1u << (v & 31));
}

// 1. prepare: one wavefront per destination row.  R drawn positions per lane
// (slot s lives in lane s % 64, register s / 64).
template <int R>
__device__ __forceinline__ void hop_prepare_body(const HopArgs &a, int64_t blk, int64_t nblk) {
    const int64_t gtid = blk * kThreads + threadIdx.x;
    const int64_t gsize = nblk * kThreads;
    const int64_t n_dst = a.n_dst_dev ? min(*a.n_dst_dev, a.cap_dst) : a.cap_dst;
    // reset the look-back state of the emit kernel and, for a block with a
    // transpose, its column counters and scan state
    for (int64_t i = gtid; i < a.nb_rows + a.nb_bits; i += gsize) a.status[i] = 0;
    if (a.erow) {
        for (int64_t i = gtid; i < a.csc_cap_src; i += gsize) a.csc_cnt[i] = 0;
        for (int64_t i = gtid; i < a.csc_nb; i += gsize) a.csc_status[i] = 0;
        if (gtid == 0) *a.csc_ticket = 0;
    }
    if (gtid == 0) {
        *a.ticket = 0;
        a.counts[0] = n_dst;
        a.counts[3] = 0;
    }
    const int lane = threadIdx.x & 63;
    // one destination row per wavefront, the grid's wavefronts striding
    // over the rows (the row is uniform per wavefront)
    for (int64_t row = gtid >> 6; row < n_dst; row += gsize >> 6) {
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
            continue;
        }
        uint32_t slot[R];
#pragma unroll
        for (int r = 0; r < R; ++r) slot[r] = 0xffffffffu;
        const uint64_t pk = mix64(mix64(mix64(mix64(a.seed) ^ a.step) ^ a.hop) ^ static_cast<uint64_t>(v));
        // The draws' candidates x_t = floor(u_t (j_t + 1)) do not depend on
        // one another: lane t computes draw t's hash (register t / 64), and
        // only the membership test below runs draw by draw.
        uint32_t cand[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t t = r * 64 + lane;
            const uint64_t j = static_cast<uint64_t>(d - k + t);
            const uint64_t key = mix64(pk ^ static_cast<uint64_t>(t));
            cand[r] = static_cast<uint32_t>(((key >> 32) * (j + 1)) >> 32);
        }
        for (int32_t t = 0; t < k; ++t) {
            const uint64_t j = static_cast<uint64_t>(d - k + t);
            uint32_t cr = 0;
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (r == (t >> 6)) cr = cand[r];
            const uint32_t x = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(cr), t & 63));
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
}

// 2a. row pointer of the block: scan of the sample counts (logical block
// `blk` owns rows [256 blk, 256 blk + 256)).
__device__ __forceinline__ void emit_rows(const HopArgs &a, int64_t blk, int64_t n_dst) {
    const int64_t i = blk * kThreads + threadIdx.x;
    const int64_t c = (i < n_dst) ? a.cnt[i] : 0;
    int64_t total;
    const int64_t excl_in_block = block_excl_scan(c, &total);
    __shared__ int64_t base;
    if (threadIdx.x < 64) {
        const int64_t b = look_back(a.status, blk, total, &a.counts[3], a.spin_limit, a.silent_row_tile);
        if (threadIdx.x == 0) base = b;
    }
    __syncthreads();
    if (i < n_dst) a.brow[i + 1] = base + excl_in_block + c;
    if (blk == 0 && threadIdx.x == 0) a.brow[0] = 0;
    if (blk == a.nb_rows - 1 && threadIdx.x == 0) a.counts[2] = base + total;
}

// 2b. new sources in ascending vertex order (logical block `blk` owns
// kBitTile bitmap words).
__device__ __forceinline__ void emit_sources(const HopArgs &a, int64_t blk, int64_t n_dst) {
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
__device__ __forceinline__ void hop_emit_body(const HopArgs &a) {
    const int64_t t = take_ticket(a.ticket);
    const int64_t n_dst = a.counts[0];
    if (t < a.nb_rows)
        emit_rows(a, t, n_dst);
    else
        emit_sources(a, t - a.nb_rows, n_dst);
}

// 3. local source index of every sampled edge.
// With the transpose requested, also the row of every edge and the count
// phase of the transpose (per-column counts).
__device__ __forceinline__ void hop_relabel_body(const HopArgs &a, int64_t blk, int64_t nblk) {
    const int64_t n_dst = a.counts[0];
    const int64_t total = n_dst * a.k;
    const int64_t gtid = blk * kThreads + threadIdx.x, gsize = nblk * kThreads;
    for (int64_t q = gtid; q < total; q += gsize) {
        const int64_t i = q / a.k, t = q - i * a.k;
        if (t >= a.cnt[i]) continue;
        const int64_t e = a.brow[i] + t;
        const int32_t c = a.map[a.gpad[q]];
        a.bcol[e] = c;
        if (a.erow) {
            a.erow[e] = static_cast<int32_t>(i);
            if (c >= 0 && c < a.csc_cap_src)
                atomicAdd(&a.csc_cnt[c], 1);
            else
                flag_error(&a.counts[3], kErrRange);
        }
    }
}

// Jobs (see jobs.h) of the prepare and relabel steps.
template <int R> struct PrepareJob {
    HopArgs a;
    __device__ void run(int64_t blk, int64_t nblk) const { hop_prepare_body<R>(a, blk, nblk); }
};
struct RelabelJob {
    HopArgs a;
    __device__ void run(int64_t blk, int64_t nblk) const { hop_relabel_body(a, blk, nblk); }
};
// Workgroups order themselves by ticket: the logical index is not used.
struct EmitJob {
    HopArgs a;
    __device__ void run(int64_t, int64_t) const { hop_emit_body(a); }
};

// Launch parameters of one hop.
struct HopPlan {
    HopArgs a;
    unsigned prep_grid, emit_grid, relabel_grid;
    int r;  // drawn positions per lane in the prepare kernel: 1, 2, 4, 8, 16
};

// Calls f(job) with the prepare job of the plan's fanout class.
template <class F> void with_prepare_job(const HopPlan &p, F &&f) {
    switch (p.r) {
        case 1: f(PrepareJob<1>{p.a}); break;
        case 2: f(PrepareJob<2>{p.a}); break;
        case 4: f(PrepareJob<4>{p.a}); break;
        case 8: f(PrepareJob<8>{p.a}); break;
        default: f(PrepareJob<16>{p.a}); break;
    }
}

}  // namespace samp

// Host side (sampler.hip).  A hop uses the shared part of a sampler
// workspace (vertex map and bitmaps, sampler_shared_bytes) and a per-hop
// scratch (sampler_hop_bytes); hops whose steps overlap need distinct
// scratch.
size_t sampler_shared_bytes(int64_t graph_n);
size_t sampler_hop_bytes(int64_t graph_n, int64_t cap_dst, int32_t fanout);
// csc: the transpose's arguments when the hop's block gets one (the relabel
// then runs its count phase), else null.
samp::HopPlan plan_hop(const gnn_graph *g, const float *gcn_norm, const int64_t *dst_ids, const int64_t *n_dst_dev,
                       int32_t fanout, uint64_t seed, uint64_t step, int32_t hop, const gnn_block *out, void *shared,
                       void *scratch, const csc::Args *csc);
gnn_status launch_hop_prepare(const samp::HopPlan &p, hipStream_t s);
gnn_status launch_hop_emit(const samp::HopPlan &p, hipStream_t s);
}  // namespace gnn
