// Matrix-core GEMM engine shared by the update kernels (gemm_fwd.hip,
// gemm_bwd.hip).
//
// The update's dense products (equation 2 and its gradients) on the CDNA4
// matrix cores.
//
//   forward   Z  = [A_self || A_nbr] W + b  (ReLU, narrowing epilogue)
//   input     dA = G W^T                    (layers above the first)
//   weights   dW = A^T G, db = colsum(G)    (optionally followed by SGD)
//
// One engine serves all three: a 256-thread workgroup (4 wavefronts as 2 x 2)
// computes a BM x BN tile (64 x 64 or 128 x 128) of C = P Q^T, walking the
// reduction in chunks of BK (64 for bf16, 32 for fp32).  Both operand tiles
// are staged in LDS with the reduction index contiguous (Ps[row][r],
// Qs[col][r]); each operand source knows its memory layout.
//   bf16: v_mfma_f32_16x16x32_bf16, operands rounded to bf16 on staging;
//   fp32: v_mfma_f32_16x16x4_f32.
// Accumulation is fp32.
//
// The shapes of a sampled mini-batch are small, so every kernel here is
// bound by memory latency rather than bandwidth or matrix-core rate.  The
// engine is written around that:
//  * a ring of two register stages keeps two chunks of loads in flight while
//    the matrix cores work on an earlier one (deeper rings measured slower:
//    more code and registers for the same latency);
//  * every global load is issued from a clamped, in-bounds address with no
//    per-element branch, so a chunk's loads issue back to back;
//  * epilogue operands (bias, the weights an SGD step updates) are loaded
//    once, before the stores, never inside a load-use chain;
//  * reductions that are split across workgroups never synchronise inside
//    the kernel: each split writes a row-major partial tile and a separate
//    reduction kernel sums the partials in split order.  (A device-scope
//    fence per workgroup costs an L2 writeback on this part, far more than
//    one extra launch.)  The fixed order keeps results bitwise reproducible.
#pragma once

#include "internal.h"

namespace gnn {
namespace gemm {

constexpr int kThreads = 256;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Staged tiles in LDS: row r (a tile row), reduction index k.  bf16 rows
// are unpadded and their 16-byte granules (8 elements) are XOR-swizzled by
// bits 2..3 of the row.  That spreads over all banks both the MFMA operand
// reads (16 rows x one granule) and the transposing commits of SrcCols
// (4 consecutive rows x half a granule per thread).  fp32 rows are padded.
template <bool BF16> struct Cfg;
template <> struct Cfg<true> {
    using T = uint16_t;
    static constexpr int BK = 64, LDK = BK;
    __device__ __forceinline__ static int idx(int r, int k) {
        return r * LDK + ((((k >> 3) ^ (((r >> 2) & 3) << 1)) << 3) | (k & 7));
    }
};
template <> struct Cfg<false> {
    using T = float;
    static constexpr int BK = 32, LDK = BK + 4;
    __device__ __forceinline__ static int idx(int r, int k) { return r * LDK + k; }
};

// A chunk of four source elements kept in its storage form until commit:
// raw bits for 16-bit sources (no ALU work touches in-flight loads), floats
// for fp32 sources.
template <class TX> struct Raw;
template <> struct Raw<uint16_t> {
    using type = uint2;
    __device__ __forceinline__ static type load(const uint16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
    __device__ __forceinline__ static type load_each(const uint16_t *p0, const uint16_t *p1, const uint16_t *p2,
                                                     const uint16_t *p3) {
        return make_uint2(static_cast<uint32_t>(*p0) | (static_cast<uint32_t>(*p1) << 16),
                          static_cast<uint32_t>(*p2) | (static_cast<uint32_t>(*p3) << 16));
    }
    __device__ __forceinline__ static float4 to_f32(type v) {
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                           __uint_as_float(v.y & 0xffff0000u));
    }
    __device__ __forceinline__ static uint2 to_bf16(type v) { return v; }
    __device__ __forceinline__ static float elem(type v, int e) {
        const uint32_t w = e < 2 ? v.x : v.y;
        return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    }
    // element e as bf16 bits
    __device__ __forceinline__ static uint32_t bits(type v, int e) {
        const uint32_t w = e < 2 ? v.x : v.y;
        return (e & 1) ? (w >> 16) : (w & 0xffffu);
    }
};
template <> struct Raw<float> {
    using type = float4;
    __device__ __forceinline__ static type load(const float *p) { return *reinterpret_cast<const float4 *>(p); }
    __device__ __forceinline__ static type load_each(const float *p0, const float *p1, const float *p2, const float *p3) {
        return make_float4(*p0, *p1, *p2, *p3);
    }
    __device__ __forceinline__ static float4 to_f32(type v) { return v; }
    __device__ __forceinline__ static uint2 to_bf16(type v) {
        return make_uint2(static_cast<uint32_t>(f32_to_bf16(v.x)) | (static_cast<uint32_t>(f32_to_bf16(v.y)) << 16),
                          static_cast<uint32_t>(f32_to_bf16(v.z)) | (static_cast<uint32_t>(f32_to_bf16(v.w)) << 16));
    }
    __device__ __forceinline__ static float elem(type v, int e) {
        return e == 0 ? v.x : (e == 1 ? v.y : (e == 2 ? v.z : v.w));
    }
    __device__ __forceinline__ static uint32_t bits(type v, int e) { return f32_to_bf16(elem(v, e)); }
};

// ---------------------------------------------------------------------------
// operand sources: fetch(s, r0) loads this thread's chunks of the tile for
// reduction offset r0 into register stage s; commit(s, lds) writes stage s
// to LDS.  Stage indices must be compile-time constants after unrolling.
// ---------------------------------------------------------------------------

// Rows of a row-major matrix, 4 consecutive reduction elements per chunk
// ("R-contiguous").  The matrix may be the concatenation [x0 || x1] of two
// matrices of row length `split` (x1 == nullptr: one matrix of row length
// ld).  Element (tile row t, red r) = X[row0 + t][r].  Requires rows >= 1,
// cols >= 1; with VEC, cols and split are multiples of 4 and the rows are
// 4-element aligned.
template <bool BF16, int ROWS, class TX, bool VEC, int D>
struct SrcRows {
    static constexpr int BK = Cfg<BF16>::BK;
    static constexpr int CPR = BK / 4;                       // chunks per tile row
    static constexpr int NCH = ROWS * BK / 4 / kThreads;     // chunks per thread
    const TX *x0, *x1;
    int64_t ld, split, rows, cols, row0;
    typename Raw<TX>::type reg[D][NCH];
    // branch-free choice between the two halves of the concatenation
    __device__ __forceinline__ const TX *addr(int64_t t, int64_t r) const {
        const bool hi = x1 != nullptr && r >= split;
        const TX *base = hi ? x1 : x0;
        return base + (hi ? t * split + (r - split) : t * ld + r);
    }
    // Out-of-range indices are clamped to valid ones: tile rows past `rows`
    // only feed output rows that are never stored, and reduction indices past
    // the range are zeroed in LDS by zero_tail().
    __device__ __forceinline__ void fetch(int s, int64_t r0) {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int64_t t = row0 + q / CPR, r = r0 + (q % CPR) * 4;
            const int64_t tc = t < rows ? t : rows - 1;
            if constexpr (VEC) {
                reg[s][i] = Raw<TX>::load(addr(tc, r < cols ? r : 0));
            } else {
                reg[s][i] = Raw<TX>::load_each(addr(tc, r < cols ? r : 0), addr(tc, r + 1 < cols ? r + 1 : 0),
                                               addr(tc, r + 2 < cols ? r + 2 : 0), addr(tc, r + 3 < cols ? r + 3 : 0));
            }
        }
    }
    __device__ __forceinline__ void commit(int s, typename Cfg<BF16>::T *lds) const {
        using CV = Cfg<BF16>;
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int q = threadIdx.x + i * kThreads;
            typename CV::T *p = lds + CV::idx(q / CPR, (q % CPR) * 4);
            if constexpr (BF16)
                *reinterpret_cast<uint2 *>(p) = Raw<TX>::to_bf16(reg[s][i]);
            else
                *reinterpret_cast<float4 *>(p) = Raw<TX>::to_f32(reg[s][i]);
        }
    }
};

// Columns of a row-major matrix Y, read as element (tile row t, red r) =
// Y[r][col0 + t]: each thread loads 4 consecutive tile rows ("T-contiguous")
// for NCH consecutive reduction indices, and transposes the 4 x 4 blocks in
// registers so that LDS receives 4 consecutive reduction elements per write.
// Y may be the concatenation [y0 || y1] along its columns (each of width
// `split`).  Requires ncols >= 1; with VEC, ncols and split are multiples of 4.
template <bool BF16, int ROWS, class TY, bool VEC, int D>
struct SrcCols {
    static constexpr int BK = Cfg<BF16>::BK;
    static constexpr int TPR = ROWS / 4;                     // threads per reduction index
    static constexpr int RPP = kThreads / TPR;               // reduction indices per pass
    static constexpr int NCH = BK / RPP;                     // consecutive reduction indices per thread
    const TY *y0, *y1;
    int64_t ld, split, ncols, r_end, col0;
    typename Raw<TY>::type reg[D][NCH];
    __device__ __forceinline__ int my_t() const { return (threadIdx.x % TPR) * 4; }
    __device__ __forceinline__ int my_r(int i) const { return (threadIdx.x / TPR) * NCH + i; }
    __device__ __forceinline__ const TY *addr(int64_t r, int64_t t) const {
        const bool hi = y1 != nullptr && t >= split;
        const TY *base = hi ? y1 : y0;
        return base + (hi ? r * split + (t - split) : r * ld + t);
    }
    // Clamped like SrcRows: columns past ncols only feed outputs that are not
    // stored; reduction rows past r_end are zeroed in LDS.
    __device__ __forceinline__ void fetch(int s, int64_t r0) {
        const int64_t t = col0 + my_t();
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int64_t r = r0 + my_r(i);
            const int64_t rc = r < r_end ? r : r_end - 1;
            if constexpr (VEC) {
                reg[s][i] = Raw<TY>::load(addr(rc, t < ncols ? t : 0));
            } else {
                reg[s][i] = Raw<TY>::load_each(addr(rc, t < ncols ? t : 0), addr(rc, t + 1 < ncols ? t + 1 : 0),
                                               addr(rc, t + 2 < ncols ? t + 2 : 0), addr(rc, t + 3 < ncols ? t + 3 : 0));
            }
        }
    }
    __device__ __forceinline__ void commit(int s, typename Cfg<BF16>::T *lds) const {
        using CV = Cfg<BF16>;
        const int tt = my_t();
        if constexpr (NCH % 4 == 0) {
#pragma unroll
            for (int g = 0; g < NCH / 4; ++g) {
                const int kk = my_r(4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    typename CV::T *p = lds + CV::idx(tt + e, kk);
                    if constexpr (BF16) {
                        const uint2 v = make_uint2(
                            Raw<TY>::bits(reg[s][4 * g + 0], e) | (Raw<TY>::bits(reg[s][4 * g + 1], e) << 16),
                            Raw<TY>::bits(reg[s][4 * g + 2], e) | (Raw<TY>::bits(reg[s][4 * g + 3], e) << 16));
                        *reinterpret_cast<uint2 *>(p) = v;
                    } else {
                        const float4 v = make_float4(Raw<TY>::elem(reg[s][4 * g + 0], e),
                                                     Raw<TY>::elem(reg[s][4 * g + 1], e),
                                                     Raw<TY>::elem(reg[s][4 * g + 2], e),
                                                     Raw<TY>::elem(reg[s][4 * g + 3], e));
                        *reinterpret_cast<float4 *>(p) = v;
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int kk = my_r(i);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if constexpr (BF16)
                        lds[CV::idx(tt + e, kk)] = static_cast<uint16_t>(Raw<TY>::bits(reg[s][i], e));
                    else
                        lds[CV::idx(tt + e, kk)] = Raw<TY>::elem(reg[s][i], e);
                }
            }
        }
    }
    // fp32 sums of stage s over this thread's reduction rows below r_end
    // (when `tail` is false every fetched row is in range).
    __device__ __forceinline__ void add_colsum(int s, float4 &sum, int64_t r0, bool tail) const {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            if (tail && r0 + my_r(i) >= r_end) continue;
            const float4 v = Raw<TY>::to_f32(reg[s][i]);
            sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
        }
    }
};

// ---------------------------------------------------------------------------
// the tile engine
// ---------------------------------------------------------------------------
template <int BM, int BN>
struct Acc {
    static constexpr int WI = BM / 32, WJ = BN / 32;  // 16 x 16 MFMA tiles per wavefront
    f32x4 c[WI][WJ];
};

template <int BM, int BN>
__device__ __forceinline__ int acc_row(int i, int q) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return (wave >> 1) * (BM / 2) + i * 16 + (lane >> 4) * 4 + q;
}
template <int BM, int BN>
__device__ __forceinline__ int acc_col(int j) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    return (wave & 1) * (BN / 2) + j * 16 + (lane & 15);
}

template <bool BF16, int BM, int BN>
__device__ __forceinline__ void mma_chunk(Acc<BM, BN> &acc, const typename Cfg<BF16>::T *Ps,
                                          const typename Cfg<BF16>::T *Qs) {
    using CV = Cfg<BF16>;
    constexpr int WI = Acc<BM, BN>::WI, WJ = Acc<BM, BN>::WJ;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const int ra = (wave >> 1) * (BM / 2) + lr, rb = (wave & 1) * (BN / 2) + lr;
    if constexpr (BF16) {
#pragma unroll
        for (int kk = 0; kk < CV::BK; kk += 32) {
            bf16x8 a[WI], b[WJ];
#pragma unroll
            for (int i = 0; i < WI; ++i)
                a[i] = *reinterpret_cast<const bf16x8 *>(Ps + CV::idx(ra + i * 16, kk + lg * 8));
#pragma unroll
            for (int j = 0; j < WJ; ++j)
                b[j] = *reinterpret_cast<const bf16x8 *>(Qs + CV::idx(rb + j * 16, kk + lg * 8));
#pragma unroll
            for (int i = 0; i < WI; ++i)
#pragma unroll
                for (int j = 0; j < WJ; ++j)
                    acc.c[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc.c[i][j], 0, 0, 0);
        }
    } else {
#pragma unroll
        for (int kk = 0; kk < CV::BK; kk += 4) {
            float a[WI], b[WJ];
#pragma unroll
            for (int i = 0; i < WI; ++i) a[i] = Ps[CV::idx(ra + i * 16, kk + lg)];
#pragma unroll
            for (int j = 0; j < WJ; ++j) b[j] = Qs[CV::idx(rb + j * 16, kk + lg)];
#pragma unroll
            for (int i = 0; i < WI; ++i)
#pragma unroll
                for (int j = 0; j < WJ; ++j)
                    acc.c[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc.c[i][j], 0, 0, 0);
        }
    }
}

// LDS for the operand tiles, reused as the epilogue staging area.
template <int BM, int BN>
constexpr int lds_bytes() {
    constexpr int ops = (BM + BN) * 36 * 4;  // fp32 [*][36]; bf16 [*][64] takes less
    constexpr int stage = (BM / 2) * (BN + 4) * 4;
    return ops > stage ? ops : stage;
}

// Zero reduction columns [valid, BK) of both LDS tiles (last chunk only).
template <bool BF16, int BM, int BN>
__device__ __forceinline__ void zero_tail(typename Cfg<BF16>::T *Ps, typename Cfg<BF16>::T *Qs, int valid) {
    using CV = Cfg<BF16>;
    const int w = CV::BK - valid;
    for (int q = threadIdx.x; q < (BM + BN) * w; q += kThreads) {
        const int row = q / w, col = valid + q % w;
        if (row < BM)
            Ps[CV::idx(row, col)] = typename CV::T(0);
        else
            Qs[CV::idx(row - BM, col)] = typename CV::T(0);
    }
}

// acc = sum over r in [r_beg, r_end) of P[.., r] Q[.., r], with a ring of D
// register stages.  colsum(sq, stage, r0, tail) is called once per chunk
// with the right operand's staged registers.
//
// Every stage is fetched unconditionally, also for chunks past the end
// (their clamped addresses re-read cached lines and the data is never
// committed): the number of loads in flight behind each stage is then the
// same on every path, so the wait before a commit covers that stage alone.
//
// run_tile is tile_prefetch (the first D chunks' loads) followed by tile_rest,
// so a caller can issue a tile's first loads early and finish it later.
template <bool BF16, int D, class SP, class SQ>
__device__ __forceinline__ void tile_prefetch(SP &sp, SQ &sq, int64_t r_beg) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
        sp.fetch(s, r_beg + s * Cfg<BF16>::BK);
        sq.fetch(s, r_beg + s * Cfg<BF16>::BK);
    }
}

template <int BM, int BN>
__device__ __forceinline__ void zero_acc(Acc<BM, BN> &acc) {
#pragma unroll
    for (int i = 0; i < Acc<BM, BN>::WI; ++i)
#pragma unroll
        for (int j = 0; j < Acc<BM, BN>::WJ; ++j) acc.c[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// The rest of run_tile after tile_prefetch (r_beg < r_end, acc zeroed).
template <bool BF16, int D, int BM, int BN, class SP, class SQ, class ColSum>
__device__ __forceinline__ void tile_rest(Acc<BM, BN> &acc, SP &sp, SQ &sq, int64_t r_beg, int64_t r_end, char *lds,
                                          ColSum &&colsum) {
    using CV = Cfg<BF16>;
    using T = typename CV::T;
    T *Ps = reinterpret_cast<T *>(lds);
    T *Qs = Ps + BM * CV::LDK;
    const int64_t nch = ceil_div(r_end - r_beg, CV::BK);
    // one chunk through stage s: commit, refill the stage D chunks ahead,
    // multiply
    auto step = [&](int s, int64_t c) {
        const int64_t r0 = r_beg + c * CV::BK;
        const bool tail = r0 + CV::BK > r_end;
        colsum(sq, s, r0, tail);
        sp.commit(s, Ps);
        sq.commit(s, Qs);
        if (tail) {
            __syncthreads();
            zero_tail<BF16, BM, BN>(Ps, Qs, static_cast<int>(r_end - r0));
        }
        __syncthreads();
        sp.fetch(s, r0 + D * CV::BK);
        sq.fetch(s, r0 + D * CV::BK);
        mma_chunk<BF16, BM, BN>(acc, Ps, Qs);
        __syncthreads();
    };
    // Whole groups of D chunks, then the remainder outside the loop, so that
    // the loop's back edge sees the same loads in flight on every path.
    int64_t c0 = 0;
    for (; c0 + D <= nch; c0 += D) {
#pragma unroll
        for (int s = 0; s < D; ++s) step(s, c0 + s);
    }
#pragma unroll
    for (int s = 0; s < D - 1; ++s)
        if (c0 + s < nch) step(s, c0 + s);
}

template <bool BF16, int D, int BM, int BN, class SP, class SQ, class ColSum>
__device__ __forceinline__ void run_tile(Acc<BM, BN> &acc, SP &sp, SQ &sq, int64_t r_beg, int64_t r_end, char *lds,
                                         ColSum &&colsum) {
    zero_acc(acc);
    if (r_beg >= r_end) return;
    tile_prefetch<BF16, D>(sp, sq, r_beg);
    tile_rest<BF16, D>(acc, sp, sq, r_beg, r_end, lds, colsum);
}

// ---------------------------------------------------------------------------
// epilogue: the tile is staged through LDS so that every thread ends up with
// row-contiguous 4-column chunks.  The chunk set of a thread is known before
// the staging (TileOut), so callers load epilogue operands up front.
// ---------------------------------------------------------------------------
template <int BM, int BN>
struct TileOut {
    static constexpr int CPR = BN / 4;              // 4-column chunks per row
    static constexpr int RPI = kThreads / CPR;      // rows per pass
    static constexpr int PER_HALF = (BM / 2) / RPI; // passes per half tile
    static constexpr int NIT = 2 * PER_HALF;
    __device__ __forceinline__ static int col() { return (threadIdx.x % CPR) * 4; }
    __device__ __forceinline__ static int row(int it) {
        return (it / PER_HALF) * (BM / 2) + (it % PER_HALF) * RPI + threadIdx.x / CPR;
    }
};

// emit(it, tile_row, tile_col, float4) for each of this thread's NIT chunks.
template <int BM, int BN, class Emit>
__device__ __forceinline__ void emit_tile(const Acc<BM, BN> &acc, char *lds, Emit &&emit) {
    using TO = TileOut<BM, BN>;
    float *st = reinterpret_cast<float *>(lds);
    constexpr int LD = BN + 4, HR = BM / 2;
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        __syncthreads();
        if ((wave >> 1) == half) {
#pragma unroll
            for (int i = 0; i < Acc<BM, BN>::WI; ++i)
#pragma unroll
                for (int j = 0; j < Acc<BM, BN>::WJ; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        st[(acc_row<BM, BN>(i, q) - half * HR) * LD + acc_col<BM, BN>(j)] = acc.c[i][j][q];
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < TO::PER_HALF; ++k) {
            const int it = half * TO::PER_HALF + k;
            const int r = TO::row(it), c = TO::col();
            emit(it, r, c, *reinterpret_cast<const float4 *>(st + (r - half * HR) * LD + c));
        }
    }
}

// Four consecutive elements p[i..i+3] of a row whose valid length ends at
// `lim` (exclusive), as floats.  With VEC the row is 4-aligned and i < lim
// implies i + 3 < lim; past-the-end elements read a clamped index.
template <bool VEC>
__device__ __forceinline__ float4 load4_clamped(const float *p, int64_t row_base, int64_t i, int64_t lim) {
    if constexpr (VEC) {
        return *reinterpret_cast<const float4 *>(p + row_base + (i < lim ? i : 0));
    } else {
        const int64_t last = lim - 1;
        return make_float4(p[row_base + min(i, last)], p[row_base + min(i + 1, last)], p[row_base + min(i + 2, last)],
                           p[row_base + min(i + 3, last)]);
    }
}

// Store elements i..i+3 (those below lim) of a row; VEC as in load4_clamped.
template <bool VEC, class TO>
__device__ __forceinline__ void store4_masked(TO *p, int64_t row_base, int64_t i, int64_t lim, float4 v) {
    if (i >= lim) return;
    if constexpr (VEC) {
        store4(p, row_base + i, v);
    } else {
        const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (i + e < lim) Elem<TO>::store(p, row_base + i + e, vv[e]);
    }
}

// ---------------------------------------------------------------------------
// launch plans
// ---------------------------------------------------------------------------
inline int bk_of(bool bf16) { return bf16 ? Cfg<true>::BK : Cfg<false>::BK; }

// 128 x 128 tiles only when even they give two workgroups per CU.
inline int pick_tile(int64_t rows, int64_t cols) {
    const int64_t t128 = ceil_div(std::max<int64_t>(rows, 1), 128) * ceil_div(std::max<int64_t>(cols, 1), 128);
    return t128 >= 512 ? 128 : 64;
}

// Register stages in flight per tile size.
template <int TILE> constexpr int depth() { return TILE == 64 ? 2 : 1; }

// Workgroup -> output tile mapping.  Workgroups are dealt round-robin to
// the 8 XCDs (each with its own L2).  With at least 8 row tiles,
// consecutive workgroups of one XCD take the column tiles of one row block,
// so the row block's operand rows are fetched into that XCD's L2 once
// (row tiles past mt in the last group have nothing to do).  With fewer
// row tiles the tiles are dealt row-major so that every XCD gets work.
constexpr int kXcds = 8;
struct TileMap {
    int64_t mt, nt;  // row and column tiles
    __host__ __device__ bool grouped() const { return mt >= kXcds; }
    __host__ __device__ int64_t blocks() const { return grouped() ? ceil_div(mt, kXcds) * kXcds * nt : mt * nt; }
    __device__ void tile_of(int64_t b, int64_t *x, int64_t *y) const {
        if (!grouped()) {
            *x = b % mt;
            *y = b / mt;
            return;
        }
        const int64_t per_group = kXcds * nt;
        const int64_t g = b / per_group, j = b % per_group;
        *x = g * kXcds + j % kXcds;
        *y = j / kXcds;
    }
};

// Workgroup -> (split, tile) for reductions split over rows (dW): all tiles
// of one split run on one XCD, where they share the split's operand rows,
// and consecutive splits go to consecutive XCDs.  nsplit is padded to a
// multiple of 8; workgroups of padding splits have nothing to do.
struct SplitMap {
    int64_t tiles;  // output tiles
    int nsplit;
    __host__ __device__ int64_t blocks() const { return ceil_div(nsplit, kXcds) * kXcds * tiles; }
    __device__ void of(int64_t b, int *split, int64_t *tile) const {
        *split = static_cast<int>((b / (kXcds * tiles)) * kXcds + b % kXcds);
        *tile = (b / kXcds) % tiles;
    }
};

// Reduction range of split `split` out of `nsplit` over [0, total), in
// whole chunks.
template <int BK>
__device__ __forceinline__ void split_range(int64_t total, int nsplit, int split, int64_t *beg, int64_t *end) {
    const int64_t per = ceil_div(ceil_div(total, nsplit), BK) * BK;
    *beg = min(total, split * per);
    *end = min(total, *beg + per);
}

// Leading dimension of the fp32 partial tiles of a split reduction.
__host__ __device__ inline int64_t part_ld(int64_t cols) { return (cols + 3) / 4 * 4; }

// Sum over splits s = 0..nsplit-1, in that order, of the float4 at
// p + s * stride.  Loads are issued sixteen splits at a time (one round trip
// for the usual split counts).
__device__ __forceinline__ float4 sum_splits(const float *p, int64_t stride, int nsplit) {
    constexpr int kAtOnce = 16;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < nsplit; s0 += kAtOnce) {
        float4 v[kAtOnce];
#pragma unroll
        for (int g = 0; g < kAtOnce; ++g)
            v[g] = *reinterpret_cast<const float4 *>(p + static_cast<int64_t>(min(s0 + g, nsplit - 1)) * stride);
#pragma unroll
        for (int g = 0; g < kAtOnce; ++g) {
            if (s0 + g < nsplit) {
                acc.x += v[g].x;
                acc.y += v[g].y;
                acc.z += v[g].z;
                acc.w += v[g].w;
            }
        }
    }
    return acc;
}

// Bias add and ReLU (non-positive and NaN inputs give 0) of the forward
// epilogue.
__device__ __forceinline__ float4 bias_act(float4 v, float4 b, int relu) {
    float4 z = make_float4(v.x + b.x, v.y + b.y, v.z + b.z, v.w + b.w);
    if (relu) {
        z.x = z.x > 0.f ? z.x : 0.f;
        z.y = z.y > 0.f ? z.y : 0.f;
        z.z = z.z > 0.f ? z.z : 0.f;
        z.w = z.w > 0.f ? z.w : 0.f;
    }
    return z;
}

}  // namespace gemm
}  // namespace gnn
