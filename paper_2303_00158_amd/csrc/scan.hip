// Device-wide exclusive scan (int64) and a stable LSD radix sort of int32
// key/value pairs.  Both read their element count from device memory so no
// host synchronisation is needed; grids are sized by the host capacity.
// Neither uses global atomics, so results are deterministic.
#include "internal.h"

namespace gnn {

// ---------------------------------------------------------------------------
// block-level scan helpers (blockDim = 256, wave64)
// ---------------------------------------------------------------------------
constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

__device__ __forceinline__ int64_t wave_incl_scan(int64_t x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int64_t y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive scan of one value per thread across a 256-thread block.
__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t *sh /*[5]*/, int64_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int64_t inc = wave_incl_scan(v);
    if (lane == 63) sh[wave] = inc;
    __syncthreads();
    int64_t wbase = 0, tot = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) {
        if (w < wave) wbase += sh[w];
        tot += sh[w];
    }
    __syncthreads();
    *total = tot;
    return wbase + inc - v;
}

__global__ void __launch_bounds__(kScanThreads) scan_reduce_kernel(const int64_t *__restrict__ in,
                                                                    const int64_t *n_dev, int64_t cap,
                                                                    int64_t *__restrict__ partial) {
    __shared__ int64_t sh[8];
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * kScanItems;
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i)
        if (base + i < n) s += in[base + i];
    int64_t tot;
    block_excl_scan(s, sh, &tot);
    if (threadIdx.x == 0) partial[blockIdx.x] = tot;
}

// Single block: exclusive scan of nb partial sums in place; total to *total.
__global__ void __launch_bounds__(kScanThreads) scan_partials_kernel(int64_t *partial, int64_t nb,
                                                                      int64_t *total) {
    __shared__ int64_t sh[8];
    const int64_t per = (nb + kScanThreads - 1) / kScanThreads;
    const int64_t beg = threadIdx.x * per;
    const int64_t end = min(nb, beg + per);
    int64_t s = 0;
    for (int64_t i = beg; i < end; ++i) s += partial[i];
    int64_t tot;
    int64_t run = block_excl_scan(s, sh, &tot);
    for (int64_t i = beg; i < end; ++i) {
        int64_t v = partial[i];
        partial[i] = run;
        run += v;
    }
    if (threadIdx.x == 0) *total = tot;
}

__global__ void __launch_bounds__(kScanThreads) scan_down_kernel(const int64_t *__restrict__ in,
                                                                  const int64_t *n_dev, int64_t cap,
                                                                  const int64_t *__restrict__ partial,
                                                                  const int64_t *total, int64_t *__restrict__ out,
                                                                  int64_t *total_to) {
    __shared__ int64_t sh[8];
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kScanTile;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        out[0] = 0;
        out[n] = *total;  // also covers n == 0
        if (total_to) *total_to = *total;
    }
    if (tile0 >= n) return;
    const int64_t base = tile0 + threadIdx.x * kScanItems;
    int64_t v[kScanItems];
    int64_t s = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        v[i] = (base + i < n) ? in[base + i] : 0;
        s += v[i];
    }
    int64_t tot;
    int64_t run = partial[blockIdx.x] + block_excl_scan(s, sh, &tot);
#pragma unroll
    for (int i = 0; i < kScanItems; ++i) {
        run += v[i];
        if (base + i < n) out[base + i + 1] = run;
    }
}

size_t scan_tmp_bytes(int64_t cap) {
    int64_t nb = ceil_div(cap > 0 ? cap : 1, kScanTile);
    return static_cast<size_t>(nb + 2) * sizeof(int64_t);
}

gnn_status exclusive_scan(const int64_t *in, int64_t *out, const int64_t *n_dev, int64_t cap, int64_t *total_to,
                          void *tmp, hipStream_t s) {
    int64_t nb = ceil_div(cap > 0 ? cap : 1, kScanTile);
    GNN_CHECK(nb <= kMaxGrid, GNN_ESIZE, "scan: %lld elements exceed the grid limit", (long long)cap);
    int64_t *partial = static_cast<int64_t *>(tmp);
    int64_t *total = partial + nb;
    scan_reduce_kernel<<<dim3(static_cast<unsigned>(nb)), kScanThreads, 0, s>>>(in, n_dev, cap, partial);
    GNN_LAUNCHED("scan_reduce");
    scan_partials_kernel<<<1, kScanThreads, 0, s>>>(partial, nb, total);
    GNN_LAUNCHED("scan_partials");
    scan_down_kernel<<<dim3(static_cast<unsigned>(nb)), kScanThreads, 0, s>>>(in, n_dev, cap, partial, total, out,
                                                                             total_to);
    GNN_LAUNCHED("scan_down");
    return GNN_OK;
}

// ---------------------------------------------------------------------------
// stable LSD radix sort, 8-bit digits, one wavefront per tile of 1024 keys
// ---------------------------------------------------------------------------
constexpr int kRadixItems = 16;
constexpr int kRadixTile = 64 * kRadixItems;

__global__ void __launch_bounds__(64) radix_hist_kernel(const int32_t *__restrict__ keys, const int64_t *n_dev,
                                                         int64_t cap, int shift, int64_t nb,
                                                         int64_t *__restrict__ hist) {
    __shared__ int cnt[256];
    const int lane = threadIdx.x;
    for (int d = lane; d < 256; d += 64) cnt[d] = 0;
    __syncthreads();
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kRadixTile;
    for (int s = 0; s < kRadixItems; ++s) {
        int64_t i = tile0 + s * 64 + lane;
        if (i < n) atomicAdd(&cnt[(keys[i] >> shift) & 255], 1);
    }
    __syncthreads();
    for (int d = lane; d < 256; d += 64) hist[static_cast<int64_t>(d) * nb + blockIdx.x] = cnt[d];
}

__global__ void __launch_bounds__(64) radix_scatter_kernel(const int32_t *__restrict__ kin,
                                                            const int32_t *__restrict__ vin, const int64_t *n_dev,
                                                            int64_t cap, int shift, int64_t nb,
                                                            const int64_t *__restrict__ offs,
                                                            int32_t *__restrict__ kout, int32_t *__restrict__ vout) {
    __shared__ int run[256];
    const int lane = threadIdx.x;
    for (int d = lane; d < 256; d += 64) run[d] = 0;
    __syncthreads();
    const int64_t n = n_dev ? min(*n_dev, cap) : cap;
    const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kRadixTile;
    if (tile0 >= n) return;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int s = 0; s < kRadixItems; ++s) {
        const int64_t i = tile0 + s * 64 + lane;
        const bool valid = i < n;
        const int32_t key = valid ? kin[i] : 0;
        const int32_t val = valid ? vin[i] : 0;
        const int d = (key >> shift) & 255;
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1;
            const uint64_t m = __ballot(valid && bit);
            peers &= bit ? m : ~m;
        }
        const int rank = __popcll(peers & lt);
        if (valid) {
            const int64_t pos = offs[static_cast<int64_t>(d) * nb + blockIdx.x] + run[d] + rank;
            kout[pos] = key;
            vout[pos] = val;
        }
        __syncthreads();
        if (valid && rank == 0) run[d] += __popcll(peers);
        __syncthreads();
    }
}

size_t radix_tmp_bytes(int64_t cap) {
    int64_t nb = ceil_div(cap > 0 ? cap : 1, kRadixTile);
    size_t hist = round_up(static_cast<size_t>(256 * nb + 1) * 8, 256);
    size_t sc = round_up(scan_tmp_bytes(256 * nb), 256);
    size_t kv = round_up(static_cast<size_t>(cap > 0 ? cap : 1) * 4, 256);
    return 2 * hist + sc + 2 * kv;
}

gnn_status radix_sort_pairs(const int32_t *keys_in, const int32_t *vals_in, int32_t *keys_out, int32_t *vals_out,
                            const int64_t *n_dev, int64_t cap, int key_bits, void *tmp, hipStream_t s) {
    if (cap <= 0) return GNN_OK;
    const int64_t nb = ceil_div(cap, kRadixTile);
    GNN_CHECK(nb <= kMaxGrid, GNN_ESIZE, "radix sort: %lld keys exceed the grid limit", (long long)cap);
    Carver c(tmp);
    size_t o_hist = c.take(static_cast<size_t>(256 * nb) * 8);
    size_t o_offs = c.take(static_cast<size_t>(256 * nb + 1) * 8);
    size_t o_scan = c.take(scan_tmp_bytes(256 * nb));
    size_t o_k = c.take(static_cast<size_t>(cap) * 4);
    size_t o_v = c.take(static_cast<size_t>(cap) * 4);
    int64_t *hist = c.ptr<int64_t>(o_hist);
    int64_t *offs = c.ptr<int64_t>(o_offs);
    int32_t *tk = c.ptr<int32_t>(o_k);
    int32_t *tv = c.ptr<int32_t>(o_v);
    const int passes = key_bits <= 0 ? 1 : (key_bits + 7) / 8;
    const int32_t *ksrc = keys_in;
    const int32_t *vsrc = vals_in;
    for (int p = 0; p < passes; ++p) {
        // the last pass must land in keys_out / vals_out
        const bool to_out = ((passes - 1 - p) % 2) == 0;
        int32_t *kdst = to_out ? keys_out : tk;
        int32_t *vdst = to_out ? vals_out : tv;
        radix_hist_kernel<<<dim3(static_cast<unsigned>(nb)), 64, 0, s>>>(ksrc, n_dev, cap, 8 * p, nb, hist);
        GNN_LAUNCHED("radix_hist");
        GNN_TRY(exclusive_scan(hist, offs, nullptr, 256 * nb, nullptr, c.ptr<void>(o_scan), s));
        radix_scatter_kernel<<<dim3(static_cast<unsigned>(nb)), 64, 0, s>>>(ksrc, vsrc, n_dev, cap, 8 * p, nb,
                                                                            offs, kdst, vdst);
        GNN_LAUNCHED("radix_scatter");
        ksrc = kdst;
        vsrc = vdst;
    }
    return GNN_OK;
}

}  // namespace gnn
