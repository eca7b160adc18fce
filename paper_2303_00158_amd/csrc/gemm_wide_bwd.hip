// Update gradients (the backward of equation 2) for wide layers, where the
// products are bound by the matrix cores rather than by memory:
//   dW = A^T G, db = colsum(G)   (K x n_out; reduction over the M rows,
//                                 split across workgroups)
//   dA = G W^T                   (M x K; reduction over n_out)
// with bf16 operands, fp32 accumulation and fp32 results, on the 256 x 256
// tiles of gemm_wide_dev.h.  The host-table model's first layer (K = 1,536,
// n_out = 1,024) is the case they are written for.
//
// Operands: A's tiles (dW, T layout) and those of a bf16 copy of W (dA, N
// layout, made by a small kernel first) are copied from memory straight into
// LDS by buffer loads with the LDS bit, three chunks ahead of their use.  G
// (fp32) is loaded into registers one (dW) or two (dA) chunks ahead,
// converted to bf16 (v_cvt_pk_bf16_f32) and written to LDS behind the MFMAs
// of the chunk before: T layout for dW, N layout for dA.  The workgroups of
// dW's first K tile also take db from those fp32 registers.
//
// dW and dA share one launch, dW's workgroups first: dW has one workgroup
// per CU at most (its splits fill one wave) and dA's tiles are short, so the
// CUs dW leaves idle, and those it frees, take dA's tiles instead of dA
// rounding up to whole waves on its own.
// Buffer descriptors bound every load: rows past a split's end (dW) or past
// the capacity read as zeros.
//
// dW's splits write fp32 partial tiles (and, from the first K tile, their
// db row) in the layout the engine's reduction job sums in split order
// (gemm_bwd_dev.h), so SGD and the bf16 shadow refresh are shared.
#include "gemm_bwd_dev.h"
#include "gemm_wide_dev.h"
#include "jobs.h"

namespace gnn {

namespace {

using namespace wide;
using gemm::part_ld;
using gemm::split_range;

constexpr int kWgThreads = 512;  // 8 wavefronts as 2 x 4, each a 128 x 64 block
constexpr int kCus = 256;

// ---------------------------------------------------------------------------
// problems
// ---------------------------------------------------------------------------

struct DinArgs {
    const float *g;            // M x n_out
    const uint16_t *wb;        // bf16 W, K x n_pad (zero past n_out)
    const int64_t *m_dev;
    int64_t cap_m, K, n_out, n_pad;
    float *d_a;                // M x K
    int64_t tiles_m, tiles_n, per_xcd;
};

struct DwArgs {
    const uint16_t *a0, *a1;   // A = [a0 || a1] (a1 null: A = a0), k_each bf16 per row each
    int64_t k_each, K;
    const float *g;            // M x n_out
    const int64_t *m_dev;
    int64_t cap_m, n_out;
    int want_db;
    float *part;               // nsplit x (K + 1) x part_ld(n_out)
    int64_t k_tiles, tiles, nsplit, per_xcd;
};

// The fp32 operand's registers for one chunk: 16 floats per thread.
struct GRegs {
    float4 v[4];
};

__device__ __forceinline__ float4 load_b128(__amdgpu_buffer_rsrc_t r, int off) {
    return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ uint4 cvt8(const float4 &x, const float4 &y) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    auto p = [](float a, float b) {
        bf16x2 v;
        v[0] = static_cast<__bf16>(a);
        v[1] = static_cast<__bf16>(b);
        return __builtin_bit_cast(uint32_t, v);
    };
    return make_uint4(p(x.x, x.y), p(x.z, x.w), p(y.x, y.y), p(y.z, y.w));
}

// dA = G W^T: the A operand is G (staged, N layout), the B operand is the
// bf16 W (copied, N layout); the reduction runs over n_out.
struct DinProb {
    static constexpr bool kTA = false, kTB = false, kStagedA = true;
    using Args = DinArgs;
    struct Work {
        __amdgpu_buffer_rsrc_t rg, rw;
        int w_off[2];          // this lane's byte offsets into W's tile, chunk 0
        int g_off;             // this thread's byte offset into G's tile (first of its rows), chunk 0
        int g_col;             // first G column this thread loads, chunk 0
        int g_ld;              // bytes between this thread's rows (8 rows of G)
        int64_t row0, col0, M, nch;
    };
    __device__ static bool setup(const Args &p, int64_t blk, Work &w) {
        const int64_t t = (blk % wide::kXcds) * p.per_xcd + blk / wide::kXcds;
        if (t >= p.tiles_m * p.tiles_n) return false;
        const int64_t tm = t / p.tiles_n, tn = t % p.tiles_n;
        w.M = p.m_dev ? min(*p.m_dev, p.cap_m) : p.cap_m;
        w.row0 = tm * kTile;
        w.col0 = tn * kTile;
        if (w.row0 >= w.M) return false;
        w.nch = ceil_div(p.n_out, int64_t(kBK));
        w.rg = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p.g + w.row0 * p.n_out), 0,
                                                 static_cast<int>((p.cap_m - w.row0) * p.n_out * 4), 0x00020000);
        w.rw = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.wb + w.col0 * p.n_pad), 0,
                                                 static_cast<int>((p.K - w.col0) * p.n_pad * 2), 0x00020000);
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int gr = (lane & 3) ^ ((lane >> 3) & 3);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int r = (wave + 8 * i) * 16 + (lane >> 2);
            w.w_off[i] = static_cast<int>((r * p.n_pad + gr * 8) * 2);
        }
        // thread -> rows 32 wave + lane / 8 + 8 e (e < 4), columns 4 (lane % 8)
        // .. + 3: each load instruction reads 8 whole 128-byte row segments
        w.g_col = (lane & 7) * 4;
        w.g_off = static_cast<int>(((wave * 32 + (lane >> 3)) * p.n_out + w.g_col) * 4);
        w.g_ld = static_cast<int>(8 * p.n_out * 4);
        return true;
    }
    __device__ static void dma(const Args &, const Work &w, int64_t c, uint16_t *, uint16_t *Bs) {
#if defined(__HIP_DEVICE_COMPILE__)
        const int wave = threadIdx.x >> 6;
        const int ck = static_cast<int>(c * kBK * 2);
#pragma unroll
        for (int i = 0; i < 2; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(w.rw, (lds_void *)(Bs + (wave + 8 * i) * 512), 16,
                                                     w.w_off[i] + ck, 0, 0, 0);
#endif
    }
    __device__ static void gload(const Args &, const Work &w, int64_t c, GRegs &r) {
        const int ck = static_cast<int>(c * kBK * 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) r.v[e] = load_b128(w.rg, w.g_off + ck + w.g_ld * e);
    }
    struct Sums {};
    // Chunk c's registers to LDS.  Columns past n_out belong to the next row:
    // they are zeroed here (not at the load, which would wait for it), so
    // that they cannot meet W's zero padding as NaN.
    __device__ static void gwrite(const Args &p, const Work &w, const GRegs &r, uint16_t *As, Sums &, int64_t c,
                                  bool) {
        const int lane = threadIdx.x & 63, row = (threadIdx.x >> 6) * 32 + (lane >> 3);
        const bool in = c * kBK + w.g_col < p.n_out;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint4 v = cvt8(in ? r.v[e] : make_float4(0.f, 0.f, 0.f, 0.f), r.v[e]);
            *reinterpret_cast<uint2 *>(As + sw_idx(row + 8 * e, w.g_col)) = make_uint2(v.x, v.y);
        }
    }
};

// dW = A^T G: the A operand is A^T (copied, T layout), the B operand is G^T
// (staged, T layout); the reduction runs over this split's rows.
struct DwProb {
    static constexpr bool kTA = true, kTB = true, kStagedA = false;
    using Args = DwArgs;
    struct Work {
        __amdgpu_buffer_rsrc_t ra, rg;
        int a_off[2];          // this lane's byte offsets into A's chunk, chunk 0
        int g_off;             // this thread's byte offset into G's chunk, chunk 0
        int64_t ald;           // A's row stride (elements)
        int64_t row0, col0;    // tile origin: K row, n_out column
        int64_t nch;
        int split;
        bool do_db;            // the first K tile's workgroups write db
    };
    __device__ static bool setup(const Args &p, int64_t blk, Work &w) {
        const int64_t t = (blk % wide::kXcds) * p.per_xcd + blk / wide::kXcds;
        if (t >= p.tiles * p.nsplit) return false;
        w.split = static_cast<int>(t / p.tiles);
        const int64_t tile = t % p.tiles;
        const int64_t tk = tile % p.k_tiles, tn = tile / p.k_tiles;
        const int64_t M = p.m_dev ? min(*p.m_dev, p.cap_m) : p.cap_m;
        int64_t r_beg, r_end;
        split_range<kBK>(M, static_cast<int>(p.nsplit), w.split, &r_beg, &r_end);
        w.nch = ceil_div(r_end - r_beg, int64_t(kBK));
        w.row0 = tk * kTile;
        w.col0 = tn * kTile;
        w.do_db = p.want_db && tk == 0;
        // the K tile lies in one half of [a0 || a1] (k_each % 256 == 0 when a1 is given)
        const bool hi = p.a1 != nullptr && w.row0 >= p.k_each;
        w.ald = p.a1 ? p.k_each : p.K;
        const uint16_t *abase = (hi ? p.a1 : p.a0) + r_beg * w.ald + (hi ? w.row0 - p.k_each : w.row0);
        // Rows past the split read as zeros (the bound ends where the next
        // row of the split range would start).  Columns past K (GCN layers
        // with K % 256 != 0) run into the following row; their products only
        // reach rows of dW past K, which are not stored.  The same holds for
        // G's columns past n_out.
        const int64_t a_col = hi ? w.row0 - p.k_each : w.row0, rows = r_end - r_beg;
        w.ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(abase), 0,
                                                 static_cast<int>(rows > 0 ? (rows * w.ald - a_col) * 2 : 0), 0x00020000);
        w.rg = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p.g + r_beg * p.n_out + w.col0), 0,
                                                 static_cast<int>(rows > 0 ? (rows * p.n_out - w.col0) * 4 : 0),
                                                 0x00020000);
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            // copy instruction wave + 8 i fills reduction rows 2 (wave + 8 i) and + 1
            const int k = 2 * (wave + 8 * i) + (lane >> 5);
            const int u = t_unit(k, lane & 31);
            w.a_off[i] = static_cast<int>((k * w.ald + u * 8) * 2);
        }
        // thread -> reduction rows 4 (tid / 64) .. + 3, columns 4 (tid % 64) .. + 3
        w.g_off = static_cast<int>((((threadIdx.x >> 6) * 4) * p.n_out + (threadIdx.x & 63) * 4) * 4);
        return true;
    }
    __device__ static void dma(const Args &, const Work &w, int64_t c, uint16_t *As, uint16_t *) {
#if defined(__HIP_DEVICE_COMPILE__)
        const int wave = threadIdx.x >> 6;
        const int ck = static_cast<int>(c * kBK * w.ald * 2);
#pragma unroll
        for (int i = 0; i < 2; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(w.ra, (lds_void *)(As + (wave + 8 * i) * 512), 16,
                                                     w.a_off[i] + ck, 0, 0, 0);
#endif
    }
    __device__ static void gload(const Args &p, const Work &w, int64_t c, GRegs &r) {
        const int ck = static_cast<int>(c * kBK * p.n_out * 4), ld = static_cast<int>(p.n_out * 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) r.v[e] = load_b128(w.rg, w.g_off + ck + ld * e);
    }
    struct Sums {
        float4 s;
    };
    // Row 4 (tid / 64) + e of the chunk, columns 4 (tid % 64) .. + 3: one
    // wavefront writes whole 512-byte rows, free of bank conflicts.
    __device__ static void gwrite(const Args &, const Work &w, const GRegs &r, uint16_t *Bs, Sums &cs, int64_t,
                                  bool count) {
        const int k0 = (threadIdx.x >> 6) * 4, c = (threadIdx.x & 63) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint4 v = cvt8(r.v[e], r.v[e]);
            *reinterpret_cast<uint2 *>(Bs + t_idx(k0 + e, c)) = make_uint2(v.x, v.y);
        }
        if (w.do_db && count) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                cs.s.x += r.v[e].x;
                cs.s.y += r.v[e].y;
                cs.s.z += r.v[e].z;
                cs.s.w += r.v[e].w;
            }
        }
    }
};

// ---------------------------------------------------------------------------
// the pipelined matrix-core loop
// ---------------------------------------------------------------------------

// MFMAs of one wavefront on one staged chunk (a 128 x 64 block).  With both
// operands in the N layout the eight A fragments are read first and the B
// fragments follow one at a time, each read while the eight MFMAs of the
// previous one run.  With both in the T layout (two reads per fragment, and
// an address per read) the four B fragments are read first and the A
// fragments stream, which holds 16 fewer registers.
template <bool TA, bool TB>
__device__ __forceinline__ void mma_chunk(f32x4 (&acc)[8][4], const uint16_t *As, const uint16_t *Bs) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ra = (wave >> 2) * 128, rb = (wave & 3) * 64;
    if constexpr (TA && TB) {
        bf16x8 b[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = frag_t(Bs, rb + 16 * j, lane);
        bf16x8 a = frag_t(As, ra, lane);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            bf16x8 an = a;
            if (i < 7) an = frag_t(As, ra + 16 * (i + 1), lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b[j], acc[i][j], 0, 0, 0);
            a = an;
        }
        // 10 LDS reads (B fragments and the first A), then per A fragment
        // its two reads among its 4 MFMAs
        __builtin_amdgcn_sched_group_barrier(0x100, 10, 0);
#pragma unroll
        for (int i = 0; i < 7; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        return;
    }
    bf16x8 a[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = frag<TA>(As, ra + 16 * i, lane);
    bf16x8 b = frag<TB>(Bs, rb, lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        bf16x8 bn = b;
        if (j < 3) bn = frag<TB>(Bs, rb + 16 * (j + 1), lane);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b, acc[i][j], 0, 0, 0);
        b = bn;
    }
    constexpr int RA = TA ? 2 : 1, RB = TB ? 2 : 1;  // LDS reads per fragment
    __builtin_amdgcn_sched_group_barrier(0x100, 8 * RA + RB, 0);
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, RB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 7, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
}

// Store a wavefront's 128 x 64 block of fp32 results (rows < nrows, columns
// < ncols, row stride ld) through LDS as row-contiguous 32-byte chunks.
__device__ __forceinline__ void store_block(const f32x4 (&acc)[8][4], float *slab, int64_t grow0, int64_t gcol0,
                                            int64_t nrows, int64_t ncols, float *out, int64_t ld) {
    constexpr int WN = 64, LD = WN + 4, CGN = WN / 8, RPP = 64 / CGN;
    const int lane = threadIdx.x & 63;
    const int cg = lane % CGN;
    const int64_t gc = gcol0 + cg * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) slab[((lane >> 4) * 4 + q) * LD + j * 16 + (lane & 15)] = acc[i][j][q];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int s2 = 0; s2 < 16 / RPP; ++s2) {
            const int r = lane / CGN + RPP * s2;
            const int64_t gr = grow0 + i * 16 + r;
            if (gr < nrows && gc < ncols) {
                float *o = out + gr * ld + gc;
                *reinterpret_cast<float4 *>(o) = *reinterpret_cast<const float4 *>(slab + r * LD + cg * 8);
                *reinterpret_cast<float4 *>(o + 4) = *reinterpret_cast<const float4 *>(slab + r * LD + cg * 8 + 4);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// One 256 x 256 tile: chunk c's copied operand goes to stage c % 4 three
// chunks ahead; its staged operand is loaded into registers R chunks ahead
// of the step that writes it, which is the step before its use, after that
// step's MFMAs.  Per wavefront and
// chunk the copies are 2 instructions and the staged loads 4, so (issue
// order: copies of c + 3, then loads of c + 1 + R, per step c):
//  * at step c, the copies of chunk c are complete once at most
//    4 + 2 (2 + 4) = 16 later operations are outstanding;
//  * the loads of chunk c + 1 are complete once at most 2 (R = 1) or
//    2 + 4 + 2 (R = 2) later operations are outstanding.
//
// The four stages are separate LDS arrays, so that the compiler sees that a
// stage's LDS writes and reads do not touch the stages whose copies are in
// flight (with one array it waits for every copy before each LDS write).
struct Ring {
    uint16_t *st[kStages][2];
};

template <class P, int R>
__device__ __forceinline__ void run_tile(const typename P::Args &p, const typename P::Work &w, f32x4 (&acc)[8][4],
                                         const Ring &ring, typename P::Sums &cs) {
    auto st = ring.st;
    constexpr int kWaitCopy = waitcnt(16, 0);
    constexpr int kWaitLoad = waitcnt(R == 1 ? 2 : 8, 15);
    const int64_t nch = w.nch;
    const int64_t last = nch - 1;
    auto at = [&](int64_t c) { return min(c, last); };
    auto staged = [&](int s) { return P::kStagedA ? st[s][0] : st[s][1]; };
    GRegs g[R];
    P::dma(p, w, at(0), st[0][0], st[0][1]);
    P::dma(p, w, at(1), st[1][0], st[1][1]);
    P::gload(p, w, at(0), g[0]);
    __builtin_amdgcn_s_waitcnt(waitcnt(0, 15));
    P::gwrite(p, w, g[0], staged(0), cs, at(0), true);
    if constexpr (R == 1) {
        P::dma(p, w, at(2), st[2][0], st[2][1]);
        P::gload(p, w, at(1), g[0]);
    } else {
        P::gload(p, w, at(1), g[1]);
        P::dma(p, w, at(2), st[2][0], st[2][1]);
        P::gload(p, w, at(2), g[0]);
    }
    for (int64_t c4 = 0; c4 < nch; c4 += 4) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int64_t c = c4 + s;
            chunk_barrier<kWaitCopy>();
            P::dma(p, w, at(c + 3), st[(s + 3) & 3][0], st[(s + 3) & 3][1]);
            if (c < nch) mma_chunk<P::kTA, P::kTB>(acc, st[s][0], st[s][1]);
            // behind the MFMAs (which run on while these issue): chunk c + 1's
            // registers to LDS, then the loads of chunk c + 1 + R
            __builtin_amdgcn_s_waitcnt(kWaitLoad);
            GRegs &gr = g[(s + 1) % R];
            P::gwrite(p, w, gr, staged((s + 1) & 3), cs, at(c + 1), c + 1 < nch);
            P::gload(p, w, at(c + 1 + R), gr);
        }
    }
    chunk_barrier<waitcnt(0, 0)>();  // the ring is drained
}

// The LDS of a workgroup: the ring's four stages as separate arrays.
#define WIDE_RING                                                                                           \
    __shared__ __attribute__((aligned(16))) uint16_t st0[2][kTileElems];                                    \
    __shared__ __attribute__((aligned(16))) uint16_t st1[2][kTileElems];                                    \
    __shared__ __attribute__((aligned(16))) uint16_t st2[2][kTileElems];                                    \
    __shared__ __attribute__((aligned(16))) uint16_t st3[2][kTileElems];                                    \
    Ring ring{{{st0[0], st0[1]}, {st1[0], st1[1]}, {st2[0], st2[1]}, {st3[0], st3[1]}}}

// The epilogue's per-wavefront slabs (16 x 68 floats each): wavefronts 0-3
// in stage 0, 4-7 in stage 1.
__device__ __forceinline__ float *slab_of(const Ring &ring) {
    const int wave = threadIdx.x >> 6;
    return reinterpret_cast<float *>(wave < 4 ? ring.st[0][0] : ring.st[1][0]) + (wave & 3) * 16 * 68;
}

// One dA tile (blk counts dA's tiles).
template <int R> __device__ __forceinline__ void dinput_tile(const DinArgs &p, int64_t blk, const Ring &ring) {
    DinProb::Work w;
    if (!DinProb::setup(p, blk, w)) return;
    f32x4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    DinProb::Sums cs;
    run_tile<DinProb, R>(p, w, acc, ring, cs);
    const int wave = threadIdx.x >> 6;
    store_block(acc, slab_of(ring), w.row0 + (wave >> 2) * 128, w.col0 + (wave & 3) * 64, w.M, p.K, p.d_a, p.K);
}

// One dW partial tile (blk counts dW's workgroups).
template <int R> __device__ __forceinline__ void dweight_tile(const DwArgs &p, int64_t blk, const Ring &ring) {
    DwProb::Work w;
    if (!DwProb::setup(p, blk, w)) return;
    f32x4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    DwProb::Sums cs;
    cs.s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (w.nch > 0) run_tile<DwProb, R>(p, w, acc, ring, cs);
    const int64_t ldp = part_ld(p.n_out);
    float *pp = p.part + static_cast<int64_t>(w.split) * (p.K + 1) * ldp;
    const int wave = threadIdx.x >> 6;
    store_block(acc, slab_of(ring), w.row0 + (wave >> 2) * 128, w.col0 + (wave & 3) * 64, p.K, p.n_out, pp, ldp);
    if (w.do_db) {
        // the 8 threads of a column group hold sums over rows 4 (tid / 64)
        // .. + 3 (+ 32 per chunk); fold them in row-group order
        float *cbuf = reinterpret_cast<float *>(ring.st[2][0]);  // 8 x 256 floats, clear of the slabs
        *reinterpret_cast<float4 *>(cbuf + (threadIdx.x >> 6) * kTile + (threadIdx.x & 63) * 4) = cs.s;
        __syncthreads();
        if (threadIdx.x < kTile && w.col0 + threadIdx.x < p.n_out) {
            float sum = 0.f;
            for (int r = 0; r < 8; ++r) sum += cbuf[r * kTile + threadIdx.x];
            pp[p.K * ldp + w.col0 + threadIdx.x] = sum;
        }
    }
}

template <int R> __global__ void __launch_bounds__(kWgThreads, 1) wide_dweight_kernel(DwArgs p) {
    WIDE_RING;
    dweight_tile<R>(p, blockIdx.x, ring);
}

// dW's workgroups (n_dw of them, a multiple of 8) and then dA's tiles in one
// grid: the dispatcher hands the long dW workgroups out first and fills the
// CUs they leave, and those they free, with dA's tiles.  Block indices keep
// their XCD (block % 8) in both ranges.
template <int RW, int RA>
__global__ void __launch_bounds__(kWgThreads, 1) wide_dw_din_kernel(DwArgs pw, DinArgs pa, int64_t n_dw) {
    WIDE_RING;
    const int64_t b = blockIdx.x;
    if (b < n_dw) dweight_tile<RW>(pw, b, ring);
    else dinput_tile<RA>(pa, b - n_dw, ring);
}

// wb[k][n] = bf16(w[k][n]) for n < n_out, 0 for n_out <= n < n_pad; eight
// elements per thread (n_out and n_pad are multiples of 8).
__global__ void __launch_bounds__(256) wide_w_bf16_kernel(const float *__restrict__ w, int64_t K, int64_t n_out,
                                                          int64_t n_pad, uint16_t *__restrict__ wb) {
    const int64_t groups = n_pad / 8;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (t >= K * groups) return;
    const int64_t k = t / groups, n = (t - k * groups) * 8;
    uint4 o = make_uint4(0, 0, 0, 0);
    if (n < n_out) {
        const float4 x = *reinterpret_cast<const float4 *>(w + k * n_out + n);
        const float4 y = *reinterpret_cast<const float4 *>(w + k * n_out + n + 4);
        o = make_uint4(pack_bf16(x.x, x.y), pack_bf16(x.z, x.w), pack_bf16(y.x, y.y), pack_bf16(y.z, y.w));
    }
    *reinterpret_cast<uint4 *>(wb + k * n_pad + n) = o;
}

// chunks of the staged operand in registers ahead of their LDS write: two
// for dA (one measured 1-3% slower), one for dW (whose transposing reads
// hold an address per read)
constexpr int kLeadDin = 2, kLeadDw = 1;

int64_t wb_bytes(int64_t K, int64_t n_out) { return round_up(K * round_up(n_out, int64_t(kBK)) * 2, int64_t(256)); }

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

namespace gbwd {

WideBwdPlan plan_wide_bwd(int64_t K, int64_t n_out, int64_t cap_m) {
    WideBwdPlan p{};
    p.k_tiles = ceil_div(K, int64_t(kTile));
    p.tiles = p.k_tiles * ceil_div(n_out, int64_t(kTile));
    const int64_t nch = std::max<int64_t>(ceil_div(cap_m, int64_t(kBK)), 1);
    const int64_t max_split = std::max<int64_t>(1, std::min<int64_t>({kCus / p.tiles, 64, nch}));
    // dW alone: one workgroup per CU, as many splits as fill the chip in one wave
    p.nsplit = max_split;
    // dW with dA in the same launch: dW's workgroups take tiles x S CUs for
    // ceil(nch / S) chunks while the other CUs run dA tiles (n_out / 32
    // chunks, each about 1.25 of a dW chunk, plus ~2.6 chunks of epilogue);
    // the dA tiles left when dW ends take whole rounds of all CUs.  S
    // minimises that estimate (fewer splits than max_split leave more CUs to
    // dA from the start and fewer partials to reduce).
    const double ta = 1.25 * static_cast<double>(ceil_div(n_out, int64_t(kBK))) + 2.6;
    const double da_tiles = static_cast<double>(ceil_div(cap_m, int64_t(kTile)) * p.k_tiles);
    double best = 0;
    for (int64_t sp = 1; sp <= max_split; ++sp) {
        const double tw = static_cast<double>(ceil_div(nch, sp));
        const double free_cus = static_cast<double>(kCus - p.tiles * sp);
        const double left = std::max(0.0, da_tiles - free_cus * tw / ta);
        const double t = tw + std::ceil(left / kCus) * ta;
        if (sp == 1 || t < best) {
            best = t;
            p.nsplit_da = sp;
        }
    }
    p.part_bytes = round_up(p.nsplit * (K + 1) * part_ld(n_out) * 4, int64_t(256));  // nsplit >= nsplit_da
    p.ws_bytes = p.part_bytes + wb_bytes(K, n_out);
    return p;
}

bool wide_bwd_shape(int64_t K, int64_t n_out, int gemm_dt) {
    return gemm_dt == GNN_BF16 && K >= 512 && n_out >= 512 && n_out % 8 == 0 && K % 8 == 0;
}

bool wide_bwd_ok(const Args &a) {
    const int64_t K = a.K();
    if (!wide_bwd_shape(K, a.n_out, a.gemm_dt) || a.adt != GNN_BF16 || a.cap_m <= 0) return false;
    if (a.a_nbr && a.k_each % kTile != 0) return false;  // a K tile must lie in one half of [a_self || a_nbr]
    // 32-bit buffer offsets
    const int64_t lim = int64_t(1) << 31;
    if (a.cap_m * a.n_out * 4 >= lim || a.cap_m * a.k_each * 2 >= lim || wb_bytes(K, a.n_out) >= lim) return false;
    return aligned(a.a_self, 16) && aligned(a.a_nbr, 16) && aligned(a.g, 16) && aligned(a.w, 16) && aligned(a.d_a, 16) &&
           aligned(a.part, 256);
}

gnn_status launch_wide_bwd_gemms(const Args &a, hipStream_t s) {
    const int64_t K = a.K();
    const WideBwdPlan pl = plan_wide_bwd(K, a.n_out, a.cap_m);
    const int64_t n_pad = round_up(a.n_out, int64_t(kBK));
    DwArgs w{};
    w.a0 = static_cast<const uint16_t *>(a.a_self);
    w.a1 = static_cast<const uint16_t *>(a.a_nbr);
    w.k_each = a.k_each;
    w.K = K;
    w.g = a.g;
    w.m_dev = a.m_dev;
    w.cap_m = a.cap_m;
    w.n_out = a.n_out;
    w.want_db = a.db != nullptr;
    w.part = a.part;
    w.k_tiles = pl.k_tiles;
    w.tiles = pl.tiles;
    w.nsplit = a.d_a ? pl.nsplit_da : pl.nsplit;
    w.per_xcd = ceil_div(pl.tiles * w.nsplit, int64_t(wide::kXcds));
    const int64_t n_dw = w.per_xcd * wide::kXcds;
    if (!a.d_a) {
        wide_dweight_kernel<kLeadDw><<<static_cast<unsigned>(n_dw), kWgThreads, 0, s>>>(w);
        GNN_LAUNCHED("update_dweight_wide");
        return GNN_OK;
    }
    uint16_t *wb = reinterpret_cast<uint16_t *>(reinterpret_cast<char *>(a.part) + pl.part_bytes);
    wide_w_bf16_kernel<<<static_cast<unsigned>(ceil_div(K * (n_pad / 8), int64_t(256))), 256, 0, s>>>(a.w, K, a.n_out,
                                                                                                  n_pad, wb);
    GNN_LAUNCHED("update_bwd_wide_w");
    DinArgs d{};
    d.g = a.g;
    d.wb = wb;
    d.m_dev = a.m_dev;
    d.cap_m = a.cap_m;
    d.K = K;
    d.n_out = a.n_out;
    d.n_pad = n_pad;
    d.d_a = a.d_a;
    d.tiles_m = ceil_div(a.cap_m, int64_t(kTile));
    d.tiles_n = ceil_div(K, int64_t(kTile));
    d.per_xcd = ceil_div(d.tiles_m * d.tiles_n, int64_t(wide::kXcds));
    const int64_t blocks = n_dw + d.per_xcd * wide::kXcds;
    GNN_CHECK(blocks <= kMaxGrid, GNN_ESIZE, "update_bwd: cap_m exceeds the grid limit");
    wide_dw_din_kernel<kLeadDw, kLeadDin><<<static_cast<unsigned>(blocks), kWgThreads, 0, s>>>(w, d, n_dw);
    GNN_LAUNCHED("update_dweight_dinput_wide");
    return GNN_OK;
}

}  // namespace gbwd

}  // namespace gnn
