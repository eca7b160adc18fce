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
// computes a BM x BN tile (128 x 128 or 64 x 64) of C = P Q^T, walking the
// reduction in chunks of BK (64 for bf16, 32 for fp32).  Both operand tiles
// are staged in LDS with the reduction index contiguous (Ps[row][r],
// Qs[col][r]); each operand source knows its memory layout.  The next chunk
// is fetched into registers while the matrix cores work on the current one.
// Every global load is issued unconditionally from a clamped, in-bounds
// address and masked afterwards, so a chunk's loads are all in flight at once.
//   bf16: v_mfma_f32_16x16x32_bf16, operands rounded to bf16 on staging;
//   fp32: v_mfma_f32_16x16x4_f32.
// Accumulation is fp32.
//
// The shapes of a sampled mini-batch are small and latency-bound, so the
// reduction can be split over blockIdx.z.  Each split writes its partial
// tile to the workspace in register order, and the last workgroup to finish
// a tile (an integer ticket per tile) sums all partials in split order and
// runs the epilogue.  The order of the sum is fixed, so results are bitwise
// reproducible, and no extra kernel launch is needed.
#pragma once

#include "internal.h"

namespace gnn {
namespace gemm {

constexpr int kThreads = 256;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <bool BF16> struct Cfg;
template <> struct Cfg<true> {
    using T = uint16_t;
    static constexpr int BK = 64, LDK = BK + 8;
    __device__ __forceinline__ static T cvt(float x) { return f32_to_bf16(x); }
};
template <> struct Cfg<false> {
    using T = float;
    static constexpr int BK = 32, LDK = BK + 4;
    __device__ __forceinline__ static T cvt(float x) { return x; }
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
};

// ---------------------------------------------------------------------------
// operand sources: fetch() loads this thread's chunks of the tile for
// reduction offset r0 into registers; commit() writes them to LDS.
// ---------------------------------------------------------------------------

// Rows of a row-major matrix, 4 consecutive reduction elements per chunk
// ("R-contiguous").  The matrix may be the concatenation [x0 || x1] of two
// matrices of row length `split` (x1 == nullptr: one matrix of row length
// ld).  Element (tile row t, red r) = X[row0 + t][r].  Requires rows >= 1,
// cols >= 1; with VEC, cols and split are multiples of 4 and the rows are
// 4-element aligned.
template <bool BF16, int ROWS, class TX, bool VEC>
struct SrcRows {
    static constexpr int BK = Cfg<BF16>::BK;
    static constexpr int CPR = BK / 4;                       // chunks per tile row
    static constexpr int NCH = ROWS * BK / 4 / kThreads;     // chunks per thread
    const TX *x0, *x1;
    int64_t ld, split, rows, cols, row0;
    typename Raw<TX>::type reg[NCH];
    __device__ __forceinline__ const TX *addr(int64_t t, int64_t r) const {
        return (x1 != nullptr && r >= split) ? x1 + t * split + (r - split) : x0 + t * ld + r;
    }
    // Out-of-range indices are clamped to valid ones: tile rows past `rows`
    // only feed output rows that are never stored, and reduction indices past
    // the range are zeroed in LDS by zero_tail().
    __device__ void fetch(int64_t r0) {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int64_t t = row0 + q / CPR, r = r0 + (q % CPR) * 4;
            const int64_t tc = t < rows ? t : rows - 1;
            if constexpr (VEC) {
                reg[i] = Raw<TX>::load(addr(tc, r < cols ? r : 0));
            } else {
                reg[i] = Raw<TX>::load_each(addr(tc, r < cols ? r : 0), addr(tc, r + 1 < cols ? r + 1 : 0),
                                            addr(tc, r + 2 < cols ? r + 2 : 0), addr(tc, r + 3 < cols ? r + 3 : 0));
            }
        }
    }
    __device__ void commit(typename Cfg<BF16>::T *lds) const {
        using CV = Cfg<BF16>;
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int q = threadIdx.x + i * kThreads;
            typename CV::T *p = lds + (q / CPR) * CV::LDK + (q % CPR) * 4;
            if constexpr (BF16)
                *reinterpret_cast<uint2 *>(p) = Raw<TX>::to_bf16(reg[i]);
            else
                *reinterpret_cast<float4 *>(p) = Raw<TX>::to_f32(reg[i]);
        }
    }
};

// Columns of a row-major matrix Y, read as element (tile row t, red r) =
// Y[r][col0 + t], 4 consecutive tile rows per chunk ("T-contiguous").  Y may
// be the concatenation [y0 || y1] along its columns (each of width `split`).
// Requires ncols >= 1; with VEC, ncols and split are multiples of 4.
template <bool BF16, int ROWS, class TY, bool VEC>
struct SrcCols {
    static constexpr int BK = Cfg<BF16>::BK;
    static constexpr int TPR = ROWS / 4;                     // threads per reduction index
    static constexpr int RPP = kThreads / TPR;               // reduction indices per pass
    static constexpr int NCH = BK / RPP;
    const TY *y0, *y1;
    int64_t ld, split, ncols, r_end, col0;
    typename Raw<TY>::type reg[NCH];
    __device__ __forceinline__ int my_t() const { return (threadIdx.x % TPR) * 4; }
    __device__ __forceinline__ int my_r(int i) const { return threadIdx.x / TPR + i * RPP; }
    __device__ __forceinline__ const TY *addr(int64_t r, int64_t t) const {
        return (y1 != nullptr && t >= split) ? y1 + r * split + (t - split) : y0 + r * ld + t;
    }
    // Clamped like SrcRows: columns past ncols only feed outputs that are not
    // stored; reduction rows past r_end are zeroed in LDS.
    __device__ void fetch(int64_t r0) {
        const int64_t t = col0 + my_t();
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int64_t r = r0 + my_r(i);
            const int64_t rc = r < r_end ? r : r_end - 1;
            if constexpr (VEC) {
                reg[i] = Raw<TY>::load(addr(rc, t < ncols ? t : 0));
            } else {
                reg[i] = Raw<TY>::load_each(addr(rc, t < ncols ? t : 0), addr(rc, t + 1 < ncols ? t + 1 : 0),
                                            addr(rc, t + 2 < ncols ? t + 2 : 0), addr(rc, t + 3 < ncols ? t + 3 : 0));
            }
        }
    }
    __device__ void commit(typename Cfg<BF16>::T *lds) const {
        using CV = Cfg<BF16>;
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int kk = my_r(i), tt = my_t();
            if constexpr (BF16) {
                const uint2 b = Raw<TY>::to_bf16(reg[i]);
                lds[(tt + 0) * CV::LDK + kk] = static_cast<uint16_t>(b.x & 0xffffu);
                lds[(tt + 1) * CV::LDK + kk] = static_cast<uint16_t>(b.x >> 16);
                lds[(tt + 2) * CV::LDK + kk] = static_cast<uint16_t>(b.y & 0xffffu);
                lds[(tt + 3) * CV::LDK + kk] = static_cast<uint16_t>(b.y >> 16);
            } else {
                const float4 v = Raw<TY>::to_f32(reg[i]);
                lds[(tt + 0) * CV::LDK + kk] = v.x;
                lds[(tt + 1) * CV::LDK + kk] = v.y;
                lds[(tt + 2) * CV::LDK + kk] = v.z;
                lds[(tt + 3) * CV::LDK + kk] = v.w;
            }
        }
    }
    // fp32 sums of the fetched values over this thread's reduction rows
    // below r_end (when `tail` is false every fetched row is in range).
    __device__ void add_colsum(float4 &s, int64_t r0, bool tail) const {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            if (tail && r0 + my_r(i) >= r_end) continue;
            const float4 v = Raw<TY>::to_f32(reg[i]);
            s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
    }
};

// ---------------------------------------------------------------------------
// the tile engine
// ---------------------------------------------------------------------------
template <int BM, int BN>
struct Acc {
    static constexpr int WI = BM / 32, WJ = BN / 32;  // 16 x 16 MFMA tiles per wavefront
    static constexpr int N = WI * WJ * 4;             // floats per thread
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
    const typename CV::T *pa = Ps + ((wave >> 1) * (BM / 2) + lr) * CV::LDK;
    const typename CV::T *pb = Qs + ((wave & 1) * (BN / 2) + lr) * CV::LDK;
    if constexpr (BF16) {
#pragma unroll
        for (int kk = 0; kk < CV::BK; kk += 32) {
            bf16x8 a[WI], b[WJ];
#pragma unroll
            for (int i = 0; i < WI; ++i) a[i] = *reinterpret_cast<const bf16x8 *>(pa + i * 16 * CV::LDK + kk + lg * 8);
#pragma unroll
            for (int j = 0; j < WJ; ++j) b[j] = *reinterpret_cast<const bf16x8 *>(pb + j * 16 * CV::LDK + kk + lg * 8);
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
            for (int i = 0; i < WI; ++i) a[i] = pa[i * 16 * CV::LDK + kk + lg];
#pragma unroll
            for (int j = 0; j < WJ; ++j) b[j] = pb[j * 16 * CV::LDK + kk + lg];
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
    constexpr int ops = (BM + BN) * 72 * 2;  // bf16 [*][72] and fp32 [*][36] take the same bytes
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
        (row < BM ? Ps + row * CV::LDK : Qs + (row - BM) * CV::LDK)[col] = typename CV::T(0);
    }
}

// acc = sum over r in [r_beg, r_end) of P[.., r] Q[.., r].  colsum(src, r0,
// tail) is called once per chunk with the right operand's staged registers.
template <bool BF16, int BM, int BN, class SP, class SQ, class ColSum>
__device__ __forceinline__ void run_tile(Acc<BM, BN> &acc, SP &sp, SQ &sq, int64_t r_beg, int64_t r_end, char *lds,
                                         ColSum &&colsum) {
    using CV = Cfg<BF16>;
    using T = typename CV::T;
    T *Ps = reinterpret_cast<T *>(lds);
    T *Qs = Ps + BM * CV::LDK;
#pragma unroll
    for (int i = 0; i < Acc<BM, BN>::WI; ++i)
#pragma unroll
        for (int j = 0; j < Acc<BM, BN>::WJ; ++j) acc.c[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (r_beg >= r_end) return;
    sp.fetch(r_beg);
    sq.fetch(r_beg);
    for (int64_t r0 = r_beg; r0 < r_end; r0 += CV::BK) {
        const bool tail = r0 + CV::BK > r_end;
        colsum(sq, r0, tail);  // reads the staged registers, which the commit waits for anyway
        sp.commit(Ps);
        sq.commit(Qs);
        if (tail) {
            __syncthreads();
            zero_tail<BF16, BM, BN>(Ps, Qs, static_cast<int>(r_end - r0));
        }
        __syncthreads();
        if (r0 + CV::BK < r_end) {
            sp.fetch(r0 + CV::BK);
            sq.fetch(r0 + CV::BK);
        }
        mma_chunk<BF16, BM, BN>(acc, Ps, Qs);
        __syncthreads();
    }
}

// Split reduction.  Returns false when this workgroup is not the last of its
// tile (it has written its partial and must exit); otherwise acc holds the
// sum over all splits in split order.
template <int BM, int BN>
__device__ __forceinline__ bool reduce_splits(Acc<BM, BN> &acc, float *part, int *tickets, int tile, int ntiles,
                                              int nsplit, int split) {
    if (nsplit == 1) return true;
    constexpr int WI = Acc<BM, BN>::WI, WJ = Acc<BM, BN>::WJ, NA = Acc<BM, BN>::N;
    __shared__ int is_last;
    float4 *mine = reinterpret_cast<float4 *>(part + (static_cast<int64_t>(split) * ntiles + tile) * kThreads * NA) +
                   threadIdx.x * (NA / 4);
#pragma unroll
    for (int i = 0; i < WI; ++i)
#pragma unroll
        for (int j = 0; j < WJ; ++j)
            mine[i * WJ + j] = make_float4(acc.c[i][j][0], acc.c[i][j][1], acc.c[i][j][2], acc.c[i][j][3]);
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) is_last = (atomicAdd(&tickets[tile], 1) == nsplit - 1);
    __syncthreads();
    if (!is_last) return false;
    __threadfence();
#pragma unroll
    for (int i = 0; i < WI; ++i)
#pragma unroll
        for (int j = 0; j < WJ; ++j) acc.c[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < nsplit; ++s) {
        const float4 *src = reinterpret_cast<const float4 *>(part + (static_cast<int64_t>(s) * ntiles + tile) *
                                                                        kThreads * NA) + threadIdx.x * (NA / 4);
        float4 v[WI * WJ];
#pragma unroll
        for (int x = 0; x < WI * WJ; ++x) v[x] = src[x];
#pragma unroll
        for (int i = 0; i < WI; ++i)
#pragma unroll
            for (int j = 0; j < WJ; ++j) {
                acc.c[i][j][0] += v[i * WJ + j].x;
                acc.c[i][j][1] += v[i * WJ + j].y;
                acc.c[i][j][2] += v[i * WJ + j].z;
                acc.c[i][j][3] += v[i * WJ + j].w;
            }
    }
    if (threadIdx.x == 0) tickets[tile] = 0;  // ready for the next launch
    return true;
}

// Write the tile through LDS so global stores are row-contiguous:
// out[(row0 + r) * ld + col0 + c] = f(col, value) for rows < rows_valid,
// columns < cols_valid.  Two passes of BM/2 rows.
template <int BM, int BN, class TO, class F>
__device__ __forceinline__ void store_tile(const Acc<BM, BN> &acc, char *lds, TO *out, int64_t ld, int64_t row0,
                                           int64_t col0, int64_t rows_valid, int64_t cols_valid, F &&f) {
    float *st = reinterpret_cast<float *>(lds);
    constexpr int LD = BN + 4, HR = BM / 2;
    const int wave = threadIdx.x >> 6;
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
        for (int q = threadIdx.x; q < HR * (BN / 4); q += kThreads) {
            const int r = q / (BN / 4), c = (q % (BN / 4)) * 4;
            const int64_t gr = row0 + half * HR + r;
            if (gr >= rows_valid) continue;
            const int64_t gc = col0 + c;
            const float4 v = *reinterpret_cast<const float4 *>(st + r * LD + c);
            const float vv[4] = {v.x, v.y, v.z, v.w};
            if (gc + 3 < cols_valid && aligned_dev(out + gr * ld + gc, sizeof(TO) * 4)) {
                float o[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = f(gc + e, vv[e]);
                store4(out, gr * ld + gc, make_float4(o[0], o[1], o[2], o[3]));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (gc + e < cols_valid) Elem<TO>::store(out, gr * ld + gc + e, f(gc + e, vv[e]));
            }
        }
    }
}

// Reduction range of split `split` out of `nsplit` over [0, total), in
// whole chunks.
template <int BK>
__device__ __forceinline__ void split_range(int64_t total, int nsplit, int split, int64_t *beg, int64_t *end) {
    const int64_t per = ceil_div(ceil_div(total, nsplit), BK) * BK;
    *beg = min(total, split * per);
    *end = min(total, *beg + per);
}

// ---------------------------------------------------------------------------
// launch plans
// ---------------------------------------------------------------------------
struct Plan {
    int tile;  // 128 or 64 (square tiles)
    dim3 grid;
    int ntiles, nsplit;
};

// Every GEMM workspace starts with a fixed ticket area (independent of the
// shape, so a workspace can be reused by calls of different shapes without
// partial tiles ever landing on tickets).  Launches with more tiles than
// tickets run unsplit.
constexpr size_t kTicketBytes = 32768;
constexpr int kMaxTickets = static_cast<int>(kTicketBytes / 4);

inline int bk_of(bool bf16) { return bf16 ? Cfg<true>::BK : Cfg<false>::BK; }

inline Plan make_plan(int tile, int64_t rows, int64_t cols, int64_t red, bool bf16, int max_split, int target) {
    Plan p;
    p.tile = tile;
    const int64_t mt = ceil_div(std::max<int64_t>(rows, 1), tile), nt = ceil_div(std::max<int64_t>(cols, 1), tile);
    p.ntiles = static_cast<int>(mt * nt);
    int64_t s = 1;
    if (p.ntiles <= kMaxTickets) {
        s = ceil_div(target, p.ntiles);
        s = std::min<int64_t>(s, ceil_div(std::max<int64_t>(red, 1), bk_of(bf16)));
        s = std::min<int64_t>(s, max_split);
        s = std::max<int64_t>(s, 1);
    }
    p.nsplit = static_cast<int>(s);
    p.grid = dim3(static_cast<unsigned>(mt), static_cast<unsigned>(nt), static_cast<unsigned>(p.nsplit));
    return p;
}

// Output tiles of rows x cols with a reduction of `red`: big outputs use
// 128 x 128 tiles unsplit; small ones 64 x 64 tiles with the reduction split
// to reach about one workgroup per CU.
inline Plan plan_fwd(int64_t rows, int64_t cols, int64_t red, bool bf16) {
    const int64_t t128 = ceil_div(std::max<int64_t>(rows, 1), 128) * ceil_div(std::max<int64_t>(cols, 1), 128);
    if (t128 >= 192) return make_plan(128, rows, cols, red, bf16, 1, 256);
    return make_plan(64, rows, cols, red, bf16, 8, 256);
}

inline Plan plan_dw(int64_t K, int64_t n_out, int64_t cap_m, bool bf16) {
    const int64_t t64 = ceil_div(K, 64) * ceil_div(n_out, 64);
    if (t64 >= 512) return make_plan(128, K, n_out, cap_m, bf16, 16, 512);
    return make_plan(64, K, n_out, cap_m, bf16, 16, 256);
}

inline size_t part_bytes(const Plan &p) {
    const size_t per_thread = static_cast<size_t>(p.tile / 32) * (p.tile / 32) * 4;
    return p.nsplit > 1 ? static_cast<size_t>(p.nsplit) * p.ntiles * kThreads * per_thread * 4 : 0;
}

inline size_t dbpart_bytes(const Plan &p, int64_t n_out) {
    return static_cast<size_t>(p.nsplit) * ceil_div(n_out, p.tile) * p.tile * 4;
}

}  // namespace gemm
}  // namespace gnn
