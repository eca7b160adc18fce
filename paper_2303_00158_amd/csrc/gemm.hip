// The update's dense products (equation 2 and its gradients) on the CDNA4
// matrix cores.
//
//   forward   Z  = [A_self || A_nbr] W + b  (ReLU, narrowing epilogue)
//   input     dA = G W^T                    (layers above the first)
//   weights   dW = A^T G, db = colsum(G)    (split over rows, fixed-order reduce)
//
// One engine serves all three: a 256-thread workgroup (4 wavefronts as 2 x 2)
// computes a 128 x 128 tile of C = P Q, stepping through the reduction in
// chunks of 32.  Both operand tiles are staged in LDS with the reduction index
// contiguous (Ps[row][r], Qs[col][r]); each operand source knows its own
// memory layout and writes the tile in that form.  The next chunk is fetched
// into registers while the matrix cores work on the current one.
//   bf16 mode: v_mfma_f32_16x16x16_bf16, operands rounded to bf16 on staging;
//   fp32 mode: v_mfma_f32_16x16x4_f32.
// Accumulation is fp32 in both.
#include "internal.h"

namespace gnn {

namespace {

constexpr int kThreads = 256;
constexpr int BM = 128, BN = 128, BK = 32;
constexpr int PAD = 8;
constexpr int LDK = BK + PAD;            // LDS row length in elements
constexpr int kChunks = (BM * BK) / (4 * kThreads);  // 4-element chunks per thread per operand tile (= 4)

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Element type staged in LDS: raw bf16 bits or fp32.
template <bool BF16> struct Stage;
template <> struct Stage<true> {
    using T = uint16_t;
    __device__ __forceinline__ static T cvt(float x) { return f32_to_bf16(x); }
};
template <> struct Stage<false> {
    using T = float;
    __device__ __forceinline__ static T cvt(float x) { return x; }
};

// ---------------------------------------------------------------------------
// operand sources.  Each fetches kChunks 4-element chunks into registers for
// reduction offset r0 and then writes them into an LDS tile [128][LDK].
//   "R-contiguous": the 4 elements run along the reduction index;
//   "T-contiguous": the 4 elements run along the tile's row index.
// ---------------------------------------------------------------------------

// Activation rows: element (row m, red k) of [a_self || a_nbr], row length
// k_each each (R-contiguous).  Used as the left operand of the forward GEMM.
template <class TA>
struct SrcActRows {
    const TA *self, *nbr;
    int64_t k_each, K, rows;  // rows = valid row count
    int64_t row0;
    bool vec;
    float4 reg[kChunks];
    __device__ void fetch(int64_t r0) {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int tr = q >> 3, tk = (q & 7) * 4;
            const int64_t m = row0 + tr, k = r0 + tk;
            float v[4] = {0.f, 0.f, 0.f, 0.f};
            if (m < rows) {
                if (vec && k + 3 < K) {
                    const bool s = k < k_each;
                    const float4 x = s ? load4(self, m * k_each + k) : load4(nbr, m * k_each + (k - k_each));
                    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int64_t kk = k + e;
                        if (kk < K)
                            v[e] = kk < k_each ? Elem<TA>::load(self, m * k_each + kk)
                                               : Elem<TA>::load(nbr, m * k_each + (kk - k_each));
                    }
                }
            }
            reg[i] = make_float4(v[0], v[1], v[2], v[3]);
        }
    }
    template <class T, class CV>
    __device__ void commit(T *lds) const {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int tr = q >> 3, tk = (q & 7) * 4;
            T *p = lds + tr * LDK + tk;
            p[0] = CV::cvt(reg[i].x); p[1] = CV::cvt(reg[i].y); p[2] = CV::cvt(reg[i].z); p[3] = CV::cvt(reg[i].w);
        }
    }
};

// fp32 row-major matrix X (rows x cols, row length ld) read as element
// (tile row t, red r) = X[t][r]  (R-contiguous).  Used for G as the left
// operand of dA = G W^T, and for W as the right operand of dA (col k, red n).
struct SrcRowsR {
    const float *x;
    int64_t ld, rows, cols;  // valid extent: t < rows, r < cols
    int64_t row0;
    bool vec;
    float4 reg[kChunks];
    __device__ void fetch(int64_t r0) {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int tr = q >> 3, tk = (q & 7) * 4;
            const int64_t t = row0 + tr, r = r0 + tk;
            float v[4] = {0.f, 0.f, 0.f, 0.f};
            if (t < rows) {
                if (vec && r + 3 < cols) {
                    const float4 a = load4(x, t * ld + r);
                    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (r + e < cols) v[e] = x[t * ld + r + e];
                }
            }
            reg[i] = make_float4(v[0], v[1], v[2], v[3]);
        }
    }
    template <class T, class CV>
    __device__ void commit(T *lds) const {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int tr = q >> 3, tk = (q & 7) * 4;
            T *p = lds + tr * LDK + tk;
            p[0] = CV::cvt(reg[i].x); p[1] = CV::cvt(reg[i].y); p[2] = CV::cvt(reg[i].z); p[3] = CV::cvt(reg[i].w);
        }
    }
};

// Matrix Y read as element (tile row t, red r) = Y[r][t] with Y row-major of
// row length ld (T-contiguous).  Y elements are TY (fp32 or bf16); optionally
// Y is the two-pointer activation [self || nbr] indexed Y[r][t] with t the
// column.  Used for W as the right operand of the forward GEMM (col n, red k)
// and for A and G in the weight-gradient GEMM (red m).
template <class TY>
struct SrcColsT {
    const TY *y;       // Y, or A_self when nbr != nullptr
    const TY *nbr;     // second half of the columns (t >= split), or nullptr
    int64_t ld;        // row length of y (and nbr)
    int64_t split;     // columns t < split come from y, the rest from nbr
    int64_t ncols;     // valid t < ncols
    int64_t r_end;     // valid r < r_end
    int64_t row0;      // first tile row (t)
    bool vec;
    float4 reg[kChunks];
    __device__ void fetch(int64_t r0) {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int tk = q >> 5, tt = (q & 31) * 4;
            const int64_t r = r0 + tk, t = row0 + tt;
            float v[4] = {0.f, 0.f, 0.f, 0.f};
            if (r < r_end) {
                const bool whole = vec && t + 3 < ncols && (nbr == nullptr || t + 3 < split || t >= split);
                if (whole) {
                    const float4 a = (nbr == nullptr || t < split) ? load4(y, r * ld + t) : load4(nbr, r * ld + (t - split));
                    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int64_t tt2 = t + e;
                        if (tt2 < ncols)
                            v[e] = (nbr == nullptr || tt2 < split) ? Elem<TY>::load(y, r * ld + tt2)
                                                                   : Elem<TY>::load(nbr, r * ld + (tt2 - split));
                    }
                }
            }
            reg[i] = make_float4(v[0], v[1], v[2], v[3]);
        }
    }
    template <class T, class CV>
    __device__ void commit(T *lds) const {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int q = threadIdx.x + i * kThreads;
            const int tk = q >> 5, tt = (q & 31) * 4;
            lds[(tt + 0) * LDK + tk] = CV::cvt(reg[i].x);
            lds[(tt + 1) * LDK + tk] = CV::cvt(reg[i].y);
            lds[(tt + 2) * LDK + tk] = CV::cvt(reg[i].z);
            lds[(tt + 3) * LDK + tk] = CV::cvt(reg[i].w);
        }
    }
};

// ---------------------------------------------------------------------------
// the tile engine
// ---------------------------------------------------------------------------
template <bool BF16>
struct Acc {
    f32x4 c[4][4];
};

template <bool BF16>
__device__ __forceinline__ void mma_tile(Acc<BF16> &acc, const typename Stage<BF16>::T *Ps,
                                         const typename Stage<BF16>::T *Qs, int wm, int wn, int lane) {
    const int lr = lane & 15, lg = lane >> 4;
    if constexpr (BF16) {
#pragma unroll
        for (int kk = 0; kk < BK; kk += 16) {
            s16x4 a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[i] = *reinterpret_cast<const s16x4 *>(Ps + (wm * 64 + i * 16 + lr) * LDK + kk + lg * 4);
                b[i] = *reinterpret_cast<const s16x4 *>(Qs + (wn * 64 + i * 16 + lr) * LDK + kk + lg * 4);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc.c[i][j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a[i], b[j], acc.c[i][j], 0, 0, 0);
        }
    } else {
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[i] = Ps[(wm * 64 + i * 16 + lr) * LDK + kk + lg];
                b[i] = Qs[(wn * 64 + i * 16 + lr) * LDK + kk + lg];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc.c[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc.c[i][j], 0, 0, 0);
        }
    }
}

// C tile += P[row0.., r_beg..r_end) Q[.., col0..]; returns in acc.
template <bool BF16, class SP, class SQ>
__device__ __forceinline__ void run_tile(Acc<BF16> &acc, SP &sp, SQ &sq, int64_t r_beg, int64_t r_end) {
    using T = typename Stage<BF16>::T;
    __shared__ __attribute__((aligned(16))) T Ps[BM * LDK];
    __shared__ __attribute__((aligned(16))) T Qs[BN * LDK];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc.c[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (r_beg >= r_end) return;
    sp.fetch(r_beg);
    sq.fetch(r_beg);
    for (int64_t r0 = r_beg; r0 < r_end; r0 += BK) {
        sp.template commit<T, Stage<BF16>>(Ps);
        sq.template commit<T, Stage<BF16>>(Qs);
        __syncthreads();
        if (r0 + BK < r_end) {
            sp.fetch(r0 + BK);
            sq.fetch(r0 + BK);
        }
        mma_tile<BF16>(acc, Ps, Qs, wm, wn, lane);
        __syncthreads();
    }
}

// Visit every accumulator element: f(row_in_tile, col_in_tile, value).
template <bool BF16, class F>
__device__ __forceinline__ void for_each_acc(const Acc<BF16> &acc, F &&f) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) f(wm * 64 + i * 16 + lg * 4 + q, wn * 64 + j * 16 + lr, acc.c[i][j][q]);
}

// ---------------------------------------------------------------------------
// forward: out = act([self || nbr] W + b)
// ---------------------------------------------------------------------------
template <bool BF16, class TA, class TO>
__global__ void __launch_bounds__(kThreads) update_fwd_kernel(const TA *__restrict__ a_self,
                                                               const TA *__restrict__ a_nbr, int64_t k_each,
                                                               const int64_t *m_dev, int64_t cap_m,
                                                               const float *__restrict__ w,
                                                               const float *__restrict__ bias, int64_t n_out,
                                                               int relu, bool vec_a, bool vec_w,
                                                               TO *__restrict__ out) {
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * BM;
    const int64_t col0 = static_cast<int64_t>(blockIdx.y) * BN;
    if (row0 >= M) return;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    SrcActRows<TA> sp{a_self, a_nbr, k_each, K, M, row0, vec_a, {}};
    SrcColsT<float> sq{w, nullptr, n_out, n_out, n_out, K, col0, vec_w, {}};
    Acc<BF16> acc;
    run_tile<BF16>(acc, sp, sq, 0, K);
    for_each_acc<BF16>(acc, [&](int r, int c, float v) {
        const int64_t m = row0 + r, n = col0 + c;
        if (m < M && n < n_out) {
            float z = v + (bias ? bias[n] : 0.f);
            if (relu && !(z > 0.f)) z = 0.f;
            Elem<TO>::store(out, m * n_out + n, z);
        }
    });
}

// ---------------------------------------------------------------------------
// input gradient: d_a = g W^T   (M x K; reduction over n_out)
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ void __launch_bounds__(kThreads) update_dinput_kernel(const float *__restrict__ g,
                                                                  const float *__restrict__ w, const int64_t *m_dev,
                                                                  int64_t cap_m, int64_t K, int64_t n_out, bool vec,
                                                                  float *__restrict__ d_a) {
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * BM;
    const int64_t col0 = static_cast<int64_t>(blockIdx.y) * BN;
    if (row0 >= M) return;
    SrcRowsR sp{g, n_out, M, n_out, row0, vec, {}};
    SrcRowsR sq{w, n_out, K, n_out, col0, vec, {}};
    Acc<BF16> acc;
    run_tile<BF16>(acc, sp, sq, 0, n_out);
    for_each_acc<BF16>(acc, [&](int r, int c, float v) {
        const int64_t m = row0 + r, k = col0 + c;
        if (m < M && k < K) d_a[m * K + k] = v;
    });
}

// ---------------------------------------------------------------------------
// weight gradient partials: part[p] = A[rows of p]^T g[rows of p]   (K x N)
// ---------------------------------------------------------------------------
template <bool BF16, class TA>
__global__ void __launch_bounds__(kThreads) update_dweight_kernel(const TA *__restrict__ a_self,
                                                                   const TA *__restrict__ a_nbr, int64_t k_each,
                                                                   const float *__restrict__ g, const int64_t *m_dev,
                                                                   int64_t cap_m, int64_t n_out, int parts,
                                                                   bool vec_a, bool vec_g,
                                                                   float *__restrict__ part) {
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * BM;  // over K
    const int64_t col0 = static_cast<int64_t>(blockIdx.y) * BN;  // over n_out
    const int p = blockIdx.z;
    const int64_t per = ceil_div(ceil_div(M, parts), BK) * BK;
    const int64_t r_beg = min(M, p * per), r_end = min(M, r_beg + per);
    SrcColsT<TA> sp{a_self, a_nbr, k_each, k_each, K, r_end, row0, vec_a, {}};
    SrcColsT<float> sq{g, nullptr, n_out, n_out, n_out, r_end, col0, vec_g, {}};
    Acc<BF16> acc;
    run_tile<BF16>(acc, sp, sq, r_beg, r_end);
    float *dst = part + static_cast<int64_t>(p) * K * n_out;
    for_each_acc<BF16>(acc, [&](int r, int c, float v) {
        const int64_t k = row0 + r, n = col0 + c;
        if (k < K && n < n_out) dst[k * n_out + n] = v;
    });
}

// Column sums of g over the rows of part p: dbpart[p][n].
__global__ void __launch_bounds__(kThreads) colsum_part_kernel(const float *__restrict__ g, const int64_t *m_dev,
                                                                int64_t cap_m, int64_t n_out, int parts,
                                                                float *__restrict__ dbpart) {
    __shared__ float sh[4][64];
    const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
    const int p = blockIdx.y;
    const int64_t per = ceil_div(ceil_div(M, parts), BK) * BK;
    const int64_t r_beg = min(M, p * per), r_end = min(M, r_beg + per);
    const int64_t n = static_cast<int64_t>(blockIdx.x) * 64 + (threadIdx.x & 63);
    const int grp = threadIdx.x >> 6;
    float s = 0.f;
    if (n < n_out)
        for (int64_t m = r_beg + grp; m < r_end; m += 4) s += g[m * n_out + n];
    sh[grp][threadIdx.x & 63] = s;
    __syncthreads();
    if (grp == 0 && n < n_out)
        dbpart[static_cast<int64_t>(p) * n_out + n] = ((sh[0][threadIdx.x] + sh[1][threadIdx.x]) + sh[2][threadIdx.x]) +
                                                      sh[3][threadIdx.x];
}

// Fixed-order sum over the parts.
__global__ void reduce_parts_kernel(const float *__restrict__ part, int parts, int64_t len, float *__restrict__ out) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < len;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        float s = 0.f;
        for (int p = 0; p < parts; ++p) s += part[static_cast<int64_t>(p) * len + i];
        out[i] = s;
    }
}

int num_parts(int64_t cap_m) {
    int64_t p = ceil_div(cap_m > 0 ? cap_m : 1, 512);
    if (p > 64) p = 64;
    return static_cast<int>(p);
}

}  // namespace

gnn_status launch_update_fwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *bias, int64_t n_out, int relu, int gemm_dt,
                             void *out, int odt, hipStream_t s) {
    if (cap_m == 0 || n_out == 0) return GNN_OK;
    const dim3 grid(static_cast<unsigned>(ceil_div(cap_m, BM)), static_cast<unsigned>(ceil_div(n_out, BN)));
    const size_t asz = dtype_size(adt);
    const bool vec_a = (k_each % 4 == 0) && aligned(a_self, 4 * asz) && (!a_nbr || aligned(a_nbr, 4 * asz));
    const bool vec_w = (n_out % 4 == 0) && aligned(w, 16);
    const bool bf = gemm_dt == GNN_BF16;
#define FWD(BFV, TA, TO)                                                                                     \
    update_fwd_kernel<BFV, TA, TO><<<grid, kThreads, 0, s>>>(static_cast<const TA *>(a_self),               \
                                                              static_cast<const TA *>(a_nbr), k_each, m_dev, \
                                                              cap_m, w, bias, n_out, relu, vec_a, vec_w,     \
                                                              static_cast<TO *>(out))
    if (bf) {
        if (adt == GNN_BF16 && odt == GNN_BF16) FWD(true, uint16_t, uint16_t);
        else if (adt == GNN_BF16 && odt == GNN_F32) FWD(true, uint16_t, float);
        else if (adt == GNN_F32 && odt == GNN_BF16) FWD(true, float, uint16_t);
        else FWD(true, float, float);
    } else {
        if (adt == GNN_BF16 && odt == GNN_BF16) FWD(false, uint16_t, uint16_t);
        else if (adt == GNN_BF16 && odt == GNN_F32) FWD(false, uint16_t, float);
        else if (adt == GNN_F32 && odt == GNN_BF16) FWD(false, float, uint16_t);
        else FWD(false, float, float);
    }
#undef FWD
    GNN_LAUNCHED("update_fwd");
    return GNN_OK;
}

size_t update_bwd_ws_bytes(int64_t k, int64_t n_out, int64_t cap_m) {
    const int parts = num_parts(cap_m);
    return round_up(static_cast<size_t>(parts) * k * n_out * 4, 256) + round_up(static_cast<size_t>(parts) * n_out * 4, 256);
}

gnn_status launch_update_bwd(const void *a_self, const void *a_nbr, int adt, int64_t k_each, const int64_t *m_dev,
                             int64_t cap_m, const float *w, const float *g, int64_t n_out, int gemm_dt, float *dw,
                             float *db, float *d_a, void *ws, hipStream_t s) {
    if (n_out == 0) return GNN_OK;
    const int64_t K = a_nbr ? 2 * k_each : k_each;
    const int parts = num_parts(cap_m);
    float *part = static_cast<float *>(ws);
    float *dbpart = reinterpret_cast<float *>(static_cast<char *>(ws) +
                                              round_up(static_cast<size_t>(parts) * K * n_out * 4, 256));
    const size_t asz = dtype_size(adt);
    const bool vec_a = (k_each % 4 == 0) && aligned(a_self, 4 * asz) && (!a_nbr || aligned(a_nbr, 4 * asz));
    const bool vec_g = (n_out % 4 == 0) && aligned(g, 16) && aligned(w, 16);
    const bool bf = gemm_dt == GNN_BF16;
    // weight gradient
    {
        const dim3 grid(static_cast<unsigned>(ceil_div(K, BM)), static_cast<unsigned>(ceil_div(n_out, BN)),
                        static_cast<unsigned>(parts));
#define DW(BFV, TA)                                                                                                \
    update_dweight_kernel<BFV, TA><<<grid, kThreads, 0, s>>>(static_cast<const TA *>(a_self),                     \
                                                              static_cast<const TA *>(a_nbr), k_each, g, m_dev,    \
                                                              cap_m, n_out, parts, vec_a, vec_g, part)
        if (bf) {
            if (adt == GNN_BF16) DW(true, uint16_t); else DW(true, float);
        } else {
            if (adt == GNN_BF16) DW(false, uint16_t); else DW(false, float);
        }
#undef DW
        GNN_LAUNCHED("update_dweight");
        reduce_parts_kernel<<<static_cast<unsigned>(ceil_div(K * n_out, 256)), 256, 0, s>>>(part, parts, K * n_out, dw);
        GNN_LAUNCHED("reduce_dweight");
    }
    if (db) {
        const dim3 grid(static_cast<unsigned>(ceil_div(n_out, 64)), static_cast<unsigned>(parts));
        colsum_part_kernel<<<grid, kThreads, 0, s>>>(g, m_dev, cap_m, n_out, parts, dbpart);
        GNN_LAUNCHED("colsum_part");
        reduce_parts_kernel<<<static_cast<unsigned>(ceil_div(n_out, 256)), 256, 0, s>>>(dbpart, parts, n_out, db);
        GNN_LAUNCHED("reduce_dbias");
    }
    if (d_a && cap_m > 0) {
        const dim3 grid(static_cast<unsigned>(ceil_div(cap_m, BM)), static_cast<unsigned>(ceil_div(K, BN)));
        if (bf)
            update_dinput_kernel<true><<<grid, kThreads, 0, s>>>(g, w, m_dev, cap_m, K, n_out, vec_g, d_a);
        else
            update_dinput_kernel<false><<<grid, kThreads, 0, s>>>(g, w, m_dev, cap_m, K, n_out, vec_g, d_a);
        GNN_LAUNCHED("update_dinput");
    }
    return GNN_OK;
}

}  // namespace gnn
