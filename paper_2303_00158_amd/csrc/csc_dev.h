// Transpose of a sampled block (its CSC: for every local source, the rows
// that sampled it, in ascending row order), the structure the aggregation
// backward reads so that it gathers instead of scattering.
//
// Four phases, each a job (see jobs.h) that a step can run alongside other
// work, so the transpose costs no launch of its own:
//   count  per-column edge counts (atomic increments; done by the relabel of
//          the hop, which produces the edges' columns, into counters that
//          the hop's prepare cleared)
//   scan   column pointers: exclusive scan of the counts, single pass with
//          ticket-ordered look-back; clears the counters again
//   place  every edge to a slot of its column (atomic slot counter: the
//          order inside a column is arbitrary here)
//   sort   every column in ascending row order, which makes the result
//          unique: columns of up to kShort entries by one lane with a
//          sorting network, longer ones by a wavefront that counts rows in
//          LDS and writes them out in order
// Every index a phase derives
// from device data is range-checked; a violation flags samp::kErrRange in
// counts[3] and skips the access.
#pragma once

#include "internal.h"
#include "sampler_dev.h"

namespace gnn {
namespace csc {

constexpr int kThreads = 256;
constexpr int kPer = 8;                          // columns per thread in the scan
constexpr int64_t kScanTile = kThreads * kPer;   // columns per scan workgroup
constexpr int kShort = 16;                       // longest column sorted by one lane
// rows counted per LDS pass of a long column; its 8 KB of LDS per workgroup
// is reserved by every launch the sort rides in, so it stays small
constexpr int kWindow = 1024;

struct Args {
    int64_t *counts;         // block counts: n_dst, n_src, nnz, error flag
    const int32_t *bcol;     // [nnz] column (local source) of each edge
    int32_t *erow;           // [cap_nnz] row of each edge; scratch of the sort
    int64_t cap_src, cap_nnz;
    int32_t *cnt;            // [cap_src] per-column counters
    uint64_t *status;        // [nb_scan] look-back words
    int *ticket;
    int64_t nb_scan;
    int64_t *cscptr;         // [cap_src + 1]
    int32_t *cscrow;         // [cap_nnz]
};

struct ScanJob {
    Args a;
    __device__ void run(int64_t, int64_t) const {
        const int64_t t = samp::take_ticket(a.ticket);
        const int64_t n_src = min(a.counts[1], a.cap_src);
        const int64_t j0 = t * kScanTile;
        if (j0 > n_src) return;  // every later ticket is past the end as well
        const int64_t jt = j0 + static_cast<int64_t>(threadIdx.x) * kPer;
        int32_t c[kPer];
        int64_t sum = 0;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t j = jt + q;
            c[q] = j < n_src ? a.cnt[j] : 0;
            sum += c[q];
        }
        int64_t total;
        const int64_t excl = samp::block_excl_scan(sum, &total);
        __shared__ int64_t base;
        if (threadIdx.x < 64) {
            const int64_t b = samp::look_back(a.status, t, total, &a.counts[3]);
            if (threadIdx.x == 0) base = b;
        }
        __syncthreads();
        int64_t run = base + excl;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t j = jt + q;
            if (j <= n_src) a.cscptr[j] = run;
            if (j < n_src) a.cnt[j] = 0;
            run += c[q];
        }
    }
};

struct PlaceJob {
    Args a;
    __device__ void run(int64_t blk, int64_t nblk) const {
        const int64_t nnz = min(a.counts[2], a.cap_nnz);
        const int64_t n_src = min(a.counts[1], a.cap_src);
        for (int64_t e = blk * kThreads + threadIdx.x; e < nnz; e += nblk * kThreads) {
            const int32_t c = a.bcol[e];
            if (c < 0 || c >= n_src) {
                samp::flag_error(&a.counts[3], samp::kErrRange);
                continue;
            }
            const int64_t p = a.cscptr[c] + atomicAdd(&a.cnt[c], 1);
            if (p < 0 || p >= nnz || p >= a.cscptr[c + 1]) {
                samp::flag_error(&a.counts[3], samp::kErrRange);
                continue;
            }
            a.cscrow[p] = a.erow[e];
        }
    }
};

__device__ __forceinline__ void cswap(int32_t &x, int32_t &y) {
    const int32_t lo = min(x, y), hi = max(x, y);
    x = lo;
    y = hi;
}

// One lane: sort seg[0, len) for len <= kShort (bitonic network on
// registers, padded with INT32_MAX).
__device__ __forceinline__ void sort_short(int32_t *seg, int64_t len) {
    int32_t v[kShort];
#pragma unroll
    for (int i = 0; i < kShort; ++i) v[i] = i < len ? seg[i] : INT32_MAX;
#pragma unroll
    for (int k = 2; k <= kShort; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
#pragma unroll
            for (int i = 0; i < kShort; ++i) {
                const int l = i ^ j;
                if (l > i) {
                    if ((i & k) == 0)
                        cswap(v[i], v[l]);
                    else
                        cswap(v[l], v[i]);
                }
            }
        }
    }
#pragma unroll
    for (int i = 0; i < kShort; ++i)
        if (i < len) seg[i] = v[i];
}

// Orders one wavefront's LDS (and its own global) accesses before and after
// the call; the lanes of a wavefront run together, so no workgroup barrier.
__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();
}

// One wavefront: the rows of column segment out[0, len) in ascending order.
// Rows are counted into 16-bit LDS counters (two per word), kWindow rows at
// a time, and written out in row order.  src is where the unsorted rows
// are read (out itself when one window covers all rows, else a copy).
__device__ __forceinline__ void sort_long(uint32_t *lds, const int32_t *src, int32_t *out, int64_t len,
                                          int64_t n_dst, int64_t *err) {
    const int lane = threadIdx.x & 63;
    int64_t pos = 0;
    for (int64_t w0 = 0; w0 < n_dst; w0 += kWindow) {
        for (int64_t i = lane; i < len; i += 64) {
            const int64_t r = src[i];
            if (r < 0 || r >= n_dst) {
                samp::flag_error(err, samp::kErrRange);
                continue;
            }
            if (r >= w0 && r < w0 + kWindow) {
                const int64_t o = r - w0;
                atomicAdd(&lds[o >> 1], 1u << (16 * (o & 1)));
            }
        }
        wave_sync_lds();
        const int64_t w1 = min(n_dst, w0 + kWindow);
        for (int64_t rb = w0; rb < w1; rb += 64) {
            const int64_t r = rb + lane;
            uint32_t c = 0;
            if (r < w1) {
                const int64_t o = r - w0;
                c = (lds[o >> 1] >> (16 * (o & 1))) & 0xffffu;
            }
            // exclusive scan of c over the wavefront
            uint32_t inc = c;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const uint32_t y = __shfl_up(inc, d, 64);
                if (lane >= d) inc += y;
            }
            const uint32_t tot = __shfl(inc, 63, 64);
            const int64_t at = pos + inc - c;
            for (uint32_t q = 0; q < c; ++q)
                if (at + q < len) out[at + q] = static_cast<int32_t>(r);
            pos += tot;
        }
        wave_sync_lds();
        // clear the window's counters
        for (int64_t o = lane; o < kWindow / 2; o += 64) lds[o] = 0u;
        wave_sync_lds();
    }
}

struct SortJob {
    Args a;
    __device__ void run(int64_t blk, int64_t nblk) const {
        __shared__ uint32_t lds[kThreads / 64][kWindow / 2];
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int64_t n_dst = a.counts[0];
        const int64_t n_src = min(a.counts[1], a.cap_src);
        const int64_t nnz = min(a.counts[2], a.cap_nnz);
        uint32_t *mine = lds[wave];
        for (int64_t o = lane; o < kWindow / 2; o += 64) mine[o] = 0u;
        wave_sync_lds();
        const int64_t waves = nblk * (kThreads / 64);
        for (int64_t g = blk * (kThreads / 64) + wave; g * 64 < n_src; g += waves) {
            const int64_t c = g * 64 + lane;
            int64_t p0 = 0, len = 0;
            if (c < n_src) {
                p0 = a.cscptr[c];
                const int64_t p1 = a.cscptr[c + 1];
                if (p0 < 0 || p1 < p0 || p1 > nnz) {
                    samp::flag_error(&a.counts[3], samp::kErrRange);
                    p0 = 0;
                } else {
                    len = p1 - p0;
                }
            }
            if (len >= 2 && len <= kShort) sort_short(a.cscrow + p0, len);
            uint64_t longs = __ballot(len > kShort);
            while (longs) {
                const int l = __builtin_ctzll(longs);
                longs &= longs - 1;
                const int64_t q0 = __shfl(p0, l, 64);
                const int64_t ql = __shfl(len, l, 64);
                int32_t *out = a.cscrow + q0;
                const int32_t *src = out;
                if (n_dst > kWindow) {
                    // several windows read the rows again: keep a copy in the
                    // edge-row scratch (free once the edges are placed)
                    int32_t *copy = a.erow + q0;
                    for (int64_t i = lane; i < ql; i += 64) copy[i] = out[i];
                    wave_sync_lds();
                    src = copy;
                }
                sort_long(mine, src, out, ql, n_dst, &a.counts[3]);
            }
        }
    }
};

struct Grids {
    unsigned scan, place, sort;
};

}  // namespace csc

// Host side (sampler.hip).  The transpose scratch of one block: the row of
// every edge, the per-column counters and the scan's look-back state.
size_t block_csc_ws_bytes(int64_t cap_src, int64_t cap_nnz);
// Arguments of the block's transpose in scratch sized for (ws_src, ws_nnz);
// the capacities used are the smaller of the block's and the scratch's.
csc::Args csc_args(const gnn_block *out, void *csc_ws, int64_t ws_src, int64_t ws_nnz);
csc::Grids csc_grids(const csc::Args &a);
// The scan, place and sort phases as three launches (after the relabel that
// counted).
gnn_status launch_block_csc(const csc::Args &a, hipStream_t s);

}  // namespace gnn
