// Forward update (equation 2) for wide layers, where the product is bound by
// the matrix cores rather than by memory: Z = [A_self || A_nbr] W + b with
// bf16 operands (A rows and the bf16 shadow W^T), fp32 accumulation, bias,
// optional ReLU and a bf16 or fp32 store.  The host-table model's first
// layer (K = 1,536, n_out = 1,024) is the case it is written for.
//
// Tiling for gfx950 (CDNA4):
//  * one 512-thread workgroup per CU computes a 256 x 256 output tile with
//    v_mfma_f32_16x16x32_bf16; its eight wavefronts (2 x 4) own 128 x 64
//    blocks, 128 accumulator registers per lane, so the two wavefronts on
//    each SIMD keep accumulators and fragments in registers.  (Measured
//    against four wavefronts of 128 x 128 with v_mfma_f32_32x32x16_bf16,
//    which read half the LDS bytes per flop but leave one wavefront per
//    SIMD to cover every wait: 0.66 against 0.83 PFLOP/s at 26,624 x 1,536
//    x 1,024; and against reading the next chunk's fragments during the
//    current chunk's MFMAs: no gain);
//  * the reduction runs in 32-deep chunks.  Both operand tiles of a chunk
//    (2 x 16 KB) are copied from memory straight into LDS by buffer loads
//    with the LDS bit (no register staging, so the register file holds the
//    accumulators and fragments only), in a ring of four LDS stages
//    (128 KB): the copies of a chunk are issued three chunks ahead of its
//    use, so every load has three chunks of matrix-core work (3 x 64 MFMAs
//    per SIMD) to land; each wavefront waits for its own copies of the
//    chunk it is about to use, and a barrier publishes them;
//  * LDS rows are 64 bytes (32 bf16); their four 16-byte granules are
//    XOR-swizzled by bits 1..2 of the row, so that the fragment reads (16
//    rows of one granule) are free of bank conflicts;
//  * tiles are dealt to the eight XCDs in contiguous ranges of the
//    row-major tile order, so the workgroups on one XCD share A rows (and
//    all of W^T) in that XCD's L2;
//  * tiles are 224 rows high instead of 256 (wavefronts of 112 x 64) where
//    that fills the CUs' last round better: the kernel's time goes by
//    rounds of 256 workgroups, so 476 tiles of 224 rows beat 416 of 256;
//  * the epilogue stages each wavefront's quadrant through LDS 16 rows at a
//    time and writes row-contiguous 16-byte (bf16) or 32-byte (fp32)
//    chunks, with bias and ReLU applied on the way.
#include "gemm_wide_dev.h"

namespace gnn {

namespace {

using namespace wide;

// Workgroup layout: NW wavefronts as 2 x (NW / 2), each owning a 128 x WN
// block of the tile; each wavefront copies CPW 16-row blocks of each
// operand per chunk.
template <int NW> struct Layout {
    static constexpr int kThreads = NW * 64;
    static constexpr int WC = NW / 2;
    static constexpr int WN = kTile / WC;      // columns per wavefront
    static constexpr int WJ = WN / 16;         // MFMA column tiles per wavefront
    static constexpr int CPW = 16 / NW;        // 16-row blocks per operand per wavefront per chunk
    // vmcnt(2 chunks of copies) | expcnt(7, no wait) | lgkmcnt(0)
    static constexpr int kWaitTwo = ((4 * CPW) & 15) | (((4 * CPW) >> 4) << 14) | 0x70;
};

struct WideArgs {
    const uint16_t *a0, *a1;  // A = [a0 || a1] (a1 null: A = a0), rows of k_each bf16 values each
    int64_t k_each, K;
    const int64_t *m_dev;
    int64_t cap_m;
    const uint16_t *wt;       // W^T, n_out x K bf16
    int64_t n_out;
    const float *bias;        // n_out, or null
    int relu;
    void *out;                // cap_m x n_out, bf16 or fp32
    int64_t tiles_m, tiles_n, per_xcd;
    float *part;              // split partial tiles, or null (no split)
    int64_t grid;             // the launch's workgroups
};

constexpr int64_t kCus = 256;

// Reduction splits when only T tiles hold rows (the row count is on the
// device): none unless the tiles fill at most a quarter of the CUs (the
// fp32 partials cost more than a split saves above that: at 6,000 rows of
// K = 1,536 two splits took 98 us against 86), else the largest divisor S
// of the q four-chunk groups with S T workgroups in one round of the CUs
// (and in the grid).
__host__ __device__ inline int wide_split(int64_t T, int64_t q, int64_t grid) {
    if (T > kCus / 4) return 1;
    const int64_t lim = (grid < kCus ? grid : kCus) / (T > 0 ? T : 1);
    int best = 1;
    for (int64_t sp = 2; sp <= lim && sp <= q; ++sp)
        if (q % sp == 0) best = static_cast<int>(sp);
    return best;
}

// Buffer descriptors over the operands: a load past the buffer's bytes
// returns zeros, so rows beyond the capacities need no clamping (they only
// feed outputs that are not stored).  Offsets are 32-bit: each operand must
// stay below 2 GB (checked by the host).
struct Descs {
    __amdgpu_buffer_rsrc_t a0, a1, wt;
};
template <int NW> struct Operands {
    Descs d;
    int a_off[Layout<NW>::CPW], b_off[Layout<NW>::CPW];  // this lane's byte offsets, chunk 0
};

// A wavefront's copy instruction fills 1 KB of LDS: lane l writes the 16
// bytes at l * 16, i.e. row l / 4 of a 16-row block at granule position
// l % 4, which holds the row's logical granule (l % 4) ^ ((l / 8) % 4)
// under the swizzle.  Wavefront w copies row blocks w + NW i of each tile.
template <int NW>
__device__ __forceinline__ Operands<NW> make_operands(const WideArgs &p, int64_t row0, int64_t col0) {
    Operands<NW> o;
    const int64_t ald = p.a1 ? p.k_each : p.K;
    const int64_t rows_a = p.cap_m - row0, rows_b = p.n_out - col0;
    const uint16_t *a0 = p.a0 + row0 * ald;
    const uint16_t *a1 = (p.a1 ? p.a1 : p.a0) + row0 * ald;
    const uint16_t *wt = p.wt + col0 * p.K;
    o.d.a0 = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(a0), 0, static_cast<int>(rows_a * ald * 2),
                                             0x00020000);
    o.d.a1 = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(a1), 0, static_cast<int>(rows_a * ald * 2),
                                             0x00020000);
    o.d.wt = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(wt), 0, static_cast<int>(rows_b * p.K * 2),
                                             0x00020000);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = (lane & 3) ^ ((lane >> 3) & 3);
#pragma unroll
    for (int i = 0; i < Layout<NW>::CPW; ++i) {
        const int r = (wave + NW * i) * 16 + (lane >> 2);
        o.a_off[i] = static_cast<int>((r * ald + g * 8) * 2);
        o.b_off[i] = static_cast<int>((r * p.K + g * 8) * 2);
    }
    return o;
}

// Issue this wavefront's copies of chunk k0 into the tiles As / Bs.
template <int NW>
__device__ __forceinline__ void copy_chunk(const WideArgs &p, const Operands<NW> &o, int64_t k0, uint16_t *As,
                                           uint16_t *Bs) {
    // which half of [a0 || a1] the chunk lies in (k_each is a multiple of 32)
    const bool hi = p.a1 != nullptr && k0 >= p.k_each;
    const __amdgpu_buffer_rsrc_t ra = hi ? o.d.a1 : o.d.a0;
    const int ak = static_cast<int>((hi ? k0 - p.k_each : k0) * 2), bk = static_cast<int>(k0 * 2);
    const int wave = threadIdx.x >> 6;
#if defined(__HIP_DEVICE_COMPILE__)  // the LDS-bit buffer load exists for the device pass only
#pragma unroll
    for (int i = 0; i < Layout<NW>::CPW; ++i) {
        const int blk = (wave + NW * i) * 512;  // elements: 16 rows x 32
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(As + blk), 16, o.a_off[i] + ak, 0, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(o.d.wt, (lds_void *)(Bs + blk), 16, o.b_off[i] + bk, 0, 0, 0);
    }
#endif
}

// MFMAs of one wavefront on one staged chunk: the FI A fragments are read
// first; the B fragments follow one at a time, each read while the FI MFMAs
// of the previous one run.
template <int NW, int FI>
__device__ __forceinline__ void mma_chunk(f32x4 (&acc)[FI][Layout<NW>::WJ], const uint16_t *As, const uint16_t *Bs) {
    constexpr int WJ = Layout<NW>::WJ;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ra = (wave / Layout<NW>::WC) * 16 * FI + (lane & 15);
    const int rb = (wave % Layout<NW>::WC) * Layout<NW>::WN + (lane & 15);
    const int kq = (lane >> 4) * 8;
    bf16x8 a[FI];
#pragma unroll
    for (int i = 0; i < FI; ++i) a[i] = *reinterpret_cast<const bf16x8 *>(As + sw_idx(ra + 16 * i, kq));
    bf16x8 b = *reinterpret_cast<const bf16x8 *>(Bs + sw_idx(rb, kq));
#pragma unroll
    for (int j = 0; j < WJ; ++j) {
        bf16x8 bn = b;
        if (j < WJ - 1) bn = *reinterpret_cast<const bf16x8 *>(Bs + sw_idx(rb + 16 * (j + 1), kq));
#pragma unroll
        for (int i = 0; i < FI; ++i) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b, acc[i][j], 0, 0, 0);
        b = bn;
    }
    // scheduling: FI + 1 LDS reads (A fragments and the first B), then per B
    // fragment one LDS read among its FI MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, FI + 1, 0);
#pragma unroll
    for (int j = 0; j < WJ - 1; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, FI - 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, FI, 0);
}

// FI A fragments per wavefront: tiles of 32 FI rows (256 or 224) by 256
// columns.  The copies always fill 256 LDS rows; with 224-row tiles the last
// 32 are the next tile's rows (or zeros past the capacity) and go unused.
template <int NW, int FI, class TO>
__global__ void __launch_bounds__(NW * 64, 1) wide_fwd_kernel(WideArgs p) {
    constexpr int TM = 32 * FI;
    using LY = Layout<NW>;
    constexpr int WJ = LY::WJ;
    __shared__ __attribute__((aligned(16))) uint16_t lds0[2][kTileElems];
    __shared__ __attribute__((aligned(16))) uint16_t lds1[2][kTileElems];
    __shared__ __attribute__((aligned(16))) uint16_t lds2[2][kTileElems];
    __shared__ __attribute__((aligned(16))) uint16_t lds3[2][kTileElems];
    // tile of this workgroup: XCD x = blockIdx % 8 takes tiles
    // [x * per_xcd, (x + 1) * per_xcd) of the row-major tile order.  With a
    // split (few tiles hold rows), work item w = s T + t is split s of tile
    // t, dealt to the XCDs the same way.
    const int64_t b = blockIdx.x;
    const int64_t M = p.m_dev ? min(*p.m_dev, p.cap_m) : p.cap_m;
    const int64_t T = ceil_div(M, int64_t(TM)) * p.tiles_n;
    const int64_t nch_all = p.K / kBK;
    const int S = p.part ? wide_split(T, nch_all / 4, p.grid) : 1;
    int64_t t, c_beg = 0, nch = nch_all;
    int split = 0;
    if (S == 1) {
        t = (b % kXcds) * p.per_xcd + b / kXcds;
        if (t >= p.tiles_m * p.tiles_n) return;
    } else {
        const int64_t w = (b % kXcds) * ceil_div(T * S, int64_t(kXcds)) + b / kXcds;
        if (w >= T * S) return;
        split = static_cast<int>(w / T);
        t = w % T;
        nch = nch_all / S;
        c_beg = split * nch;
    }
    const int64_t tm = t / p.tiles_n, tn = t % p.tiles_n;
    const int64_t row0 = tm * TM, col0 = tn * kTile;
    if (row0 >= M) return;

    f32x4 acc[FI][WJ];
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < WJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const Operands<NW> ops = make_operands<NW>(p, row0, col0);
    // Chunk c goes to stage c % 4.  The chunk count is a multiple of 4
    // (K % 128 == 0), so the loop body takes four chunks with no exit
    // between them; copies past the last chunk re-read it into a stage
    // nobody reads any more, so the copies need no branch.
    const int64_t last = (c_beg + nch - 1) * kBK;
    auto at = [&](int64_t c) { return min((c_beg + c) * kBK, last); };
    copy_chunk<NW>(p, ops, at(0), lds0[0], lds0[1]);
    copy_chunk<NW>(p, ops, at(1), lds1[0], lds1[1]);
    copy_chunk<NW>(p, ops, at(2), lds2[0], lds2[1]);
    for (int64_t c = 0; c < nch; c += 4) {
        chunk_barrier<LY::kWaitTwo>();
        copy_chunk<NW>(p, ops, at(c + 3), lds3[0], lds3[1]);
        mma_chunk<NW, FI>(acc, lds0[0], lds0[1]);
        chunk_barrier<LY::kWaitTwo>();
        copy_chunk<NW>(p, ops, at(c + 4), lds0[0], lds0[1]);
        mma_chunk<NW, FI>(acc, lds1[0], lds1[1]);
        chunk_barrier<LY::kWaitTwo>();
        copy_chunk<NW>(p, ops, at(c + 5), lds1[0], lds1[1]);
        mma_chunk<NW, FI>(acc, lds2[0], lds2[1]);
        chunk_barrier<LY::kWaitTwo>();
        copy_chunk<NW>(p, ops, at(c + 6), lds2[0], lds2[1]);
        mma_chunk<NW, FI>(acc, lds3[0], lds3[1]);
    }
    chunk_barrier<0x0070>();  // vmcnt(0) lgkmcnt(0): the ring is drained

    // epilogue: per wavefront, 8 slabs of 16 rows x WN columns through LDS
    // (the first half of the wavefronts in stage 0, the rest in stage 1)
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int WN = LY::WN, LD = WN + 4, CGN = WN / 8, RPP = 64 / CGN;
    float *slab = (wave < NW / 2 ? reinterpret_cast<float *>(&lds0[0][0])
                                 : reinterpret_cast<float *>(&lds1[0][0])) + (wave % (NW / 2)) * 16 * LD;
    const int64_t wrow0 = row0 + (wave / LY::WC) * 16 * FI, wcol0 = col0 + (wave % LY::WC) * WN;
    const int cg = lane % CGN;               // this lane's 8-column group
    const int64_t gc = wcol0 + cg * 8;
    float bv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) bv[e] = (p.bias && gc + e < p.n_out) ? p.bias[gc + e] : 0.f;
#pragma unroll
    for (int i = 0; i < FI; ++i) {
#pragma unroll
        for (int j = 0; j < WJ; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) slab[((lane >> 4) * 4 + q) * LD + j * 16 + (lane & 15)] = acc[i][j][q];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int s2 = 0; s2 < 16 / RPP; ++s2) {
            const int r = lane / CGN + RPP * s2;  // 0..15
            const float4 v0 = *reinterpret_cast<const float4 *>(slab + r * LD + cg * 8);
            const float4 v1 = *reinterpret_cast<const float4 *>(slab + r * LD + cg * 8 + 4);
            float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
            const int64_t gr = wrow0 + i * 16 + r;
            if (S > 1) {
                // the split's fp32 partial tile (TM x 256, row-major); bias
                // and activation come with the sum of the splits
                if (gr < M && gc < p.n_out) {
                    float *o = p.part + ((split * T + t) * TM + (gr - row0)) * kTile + (gc - col0);
                    *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
                    *reinterpret_cast<float4 *>(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
                }
                continue;
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                v[e] += bv[e];
                if (p.relu) v[e] = fmaxf(v[e], 0.f);
            }
            if (gr < M && gc < p.n_out) {
                if constexpr (sizeof(TO) == 2) {
                    uint4 o;
                    o.x = pack_bf16(v[0], v[1]);
                    o.y = pack_bf16(v[2], v[3]);
                    o.z = pack_bf16(v[4], v[5]);
                    o.w = pack_bf16(v[6], v[7]);
                    *reinterpret_cast<uint4 *>(static_cast<uint16_t *>(p.out) + gr * p.n_out + gc) = o;
                } else {
                    float *o = static_cast<float *>(p.out) + gr * p.n_out + gc;
                    *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
                    *reinterpret_cast<float4 *>(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// out = act(sum over the splits, in order, of the partial tiles + bias) for
// the rows held on the device, when the forward kernel split (it decides the
// same way from the same row count); else nothing.
template <class TO>
__global__ void __launch_bounds__(256) wide_fwd_reduce_kernel(WideArgs p, int64_t tm_rows) {
    const int64_t M = p.m_dev ? min(*p.m_dev, p.cap_m) : p.cap_m;
    const int64_t T = ceil_div(M, tm_rows) * p.tiles_n;
    const int S = wide_split(T, p.K / kBK / 4, p.grid);
    if (S == 1) return;
    const int64_t groups = p.n_out / 8;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < M * groups;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t r = i / groups, c = (i - r * groups) * 8;
        const int64_t t = (r / tm_rows) * p.tiles_n + c / kTile;
        const float *src = p.part + (t * tm_rows + r % tm_rows) * kTile + c % kTile;
        const int64_t stride = T * tm_rows * kTile;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
        for (int sp = 0; sp < S; ++sp) {
            const float4 x = *reinterpret_cast<const float4 *>(src + sp * stride);
            const float4 y = *reinterpret_cast<const float4 *>(src + sp * stride + 4);
            v[0] += x.x; v[1] += x.y; v[2] += x.z; v[3] += x.w;
            v[4] += y.x; v[5] += y.y; v[6] += y.z; v[7] += y.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            v[e] += p.bias ? p.bias[c + e] : 0.f;
            if (p.relu) v[e] = fmaxf(v[e], 0.f);
        }
        if constexpr (sizeof(TO) == 2) {
            uint4 o;
            o.x = pack_bf16(v[0], v[1]);
            o.y = pack_bf16(v[2], v[3]);
            o.z = pack_bf16(v[4], v[5]);
            o.w = pack_bf16(v[6], v[7]);
            *reinterpret_cast<uint4 *>(static_cast<uint16_t *>(p.out) + r * p.n_out + c) = o;
        } else {
            float *o = static_cast<float *>(p.out) + r * p.n_out + c;
            *reinterpret_cast<float4 *>(o) = make_float4(v[0], v[1], v[2], v[3]);
            *reinterpret_cast<float4 *>(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
        }
    }
}

constexpr int kWideWaves = 8;

}  // namespace

bool wide_fwd_ok(const void *a_self, const void *a_nbr, int adt, int64_t k_each, int64_t cap_m, int64_t n_out,
                 const uint16_t *wt, int gemm_dt, const void *out) {
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    // 32-bit buffer offsets: each operand below 2 GB
    const bool fits = cap_m * k_each * 2 < (int64_t(1) << 31) && n_out * K * 2 < (int64_t(1) << 31);
    return gemm_dt == GNN_BF16 && adt == GNN_BF16 && wt != nullptr && K >= 512 && n_out >= 512 &&
           k_each % kBK == 0 && K % (kStages * kBK) == 0 && n_out % 8 == 0 && fits && aligned(a_self, 16) &&
           aligned(a_nbr, 16) && aligned(wt, 16) && aligned(out, 16);
}

namespace {

// Tile height and grid: 256 or 224 rows, whichever takes the fewest rows x
// rounds of the CUs (at 26,624 rows and four column tiles: 416 tiles fill
// 1.6 rounds of 256 CUs, 476 fill 1.9; the shorter tiles finish sooner).
struct WideGrid {
    int fi;
    int64_t tiles_m, tiles_n, per_xcd, blocks;
};
WideGrid wide_grid(int64_t cap_m, int64_t n_out) {
    WideGrid g{};
    g.tiles_n = ceil_div(n_out, kTile);
    auto cost = [&](int64_t tm) { return ceil_div(ceil_div(cap_m, tm) * g.tiles_n, kCus) * tm; };
    g.fi = cost(224) < cost(256) ? 7 : 8;
    g.tiles_m = ceil_div(cap_m, int64_t(32 * g.fi));
    g.per_xcd = ceil_div(g.tiles_m * g.tiles_n, kXcds);
    g.blocks = g.per_xcd * kXcds;
    return g;
}

}  // namespace

size_t wide_fwd_ws_bytes(int64_t n_out, int64_t cap_m) {
    // at most one round of the CUs (or the grid) of partial tiles
    const WideGrid g = wide_grid(cap_m, n_out);
    return round_up(static_cast<size_t>(std::min<int64_t>(kCus, g.blocks)) * 32 * g.fi * kTile * 4, size_t(256));
}

gnn_status launch_wide_fwd(const void *a_self, const void *a_nbr, int64_t k_each, const int64_t *m_dev,
                           int64_t cap_m, const uint16_t *wt, const float *bias, int64_t n_out, int relu, void *out,
                           int odt, void *ws, hipStream_t s) {
    WideArgs p{};
    p.a0 = static_cast<const uint16_t *>(a_self);
    p.a1 = static_cast<const uint16_t *>(a_nbr);
    p.k_each = k_each;
    p.K = a_nbr ? 2 * k_each : k_each;
    p.m_dev = m_dev;
    p.cap_m = cap_m;
    p.wt = wt;
    p.n_out = n_out;
    p.bias = bias;
    p.relu = relu;
    p.out = out;
    const WideGrid g = wide_grid(cap_m, n_out);
    p.tiles_m = g.tiles_m;
    p.tiles_n = g.tiles_n;
    p.per_xcd = g.per_xcd;
    p.grid = g.blocks;
    GNN_CHECK(g.blocks <= kMaxGrid, GNN_ESIZE, "update_fwd: cap_m exceeds the grid limit");
    // With a workspace and the row count on the device, the reduction is
    // split when few tiles hold rows: the kernel decides from the row count,
    // and a second kernel sums the splits (or does nothing when there were
    // none).  A row count known here (cap_m) never leaves room for a split:
    // the grid has no more workgroups than tiles.
    const int64_t tm_rows = 32 * g.fi;
    const bool split = ws && m_dev;
    p.part = split ? static_cast<float *>(ws) : nullptr;
    constexpr int NT = Layout<kWideWaves>::kThreads;
    const unsigned gb = static_cast<unsigned>(g.blocks);
    if (odt == GNN_BF16) {
        if (g.fi == 8) wide_fwd_kernel<kWideWaves, 8, uint16_t><<<gb, NT, 0, s>>>(p);
        else wide_fwd_kernel<kWideWaves, 7, uint16_t><<<gb, NT, 0, s>>>(p);
    } else {
        if (g.fi == 8) wide_fwd_kernel<kWideWaves, 8, float><<<gb, NT, 0, s>>>(p);
        else wide_fwd_kernel<kWideWaves, 7, float><<<gb, NT, 0, s>>>(p);
    }
    GNN_LAUNCHED("update_fwd_wide");
    if (split) {
        const unsigned rg = static_cast<unsigned>(std::min<int64_t>(ceil_div(cap_m * (n_out / 8), int64_t(256)), 512));
        if (odt == GNN_BF16) wide_fwd_reduce_kernel<uint16_t><<<rg, 256, 0, s>>>(p, tm_rows);
        else wide_fwd_reduce_kernel<float><<<rg, 256, 0, s>>>(p, tm_rows);
        GNN_LAUNCHED("update_fwd_wide_reduce");
    }
    return GNN_OK;
}

}  // namespace gnn
