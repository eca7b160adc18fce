// Forward of one layer in one launch: the aggregation of a row tile
// (equation 1; the GraphSAGE-mean and GCN definitions of Section II-A) goes
// straight into LDS and feeds the update (equation 2) on the matrix cores,
// the on-chip aggregate -> update datapath of Section IV-C.  For the last
// layer the epilogue also computes the softmax cross-entropy gradient and
// row losses (Section II-B's loss), so the logits never make a round trip
// before the backward pass.
//
// Layout of the work, for a 512-thread workgroup (8 wavefronts):
//  * weights stay in registers: wavefront w owns output column tiles
//    w, w + 8, ... (16 columns each) and holds their bf16 W^T fragments for
//    every 32-wide reduction step, loaded once per workgroup (before the row
//    count is even known, so their latency hides behind the first tile);
//  * the workgroup walks row tiles of BM (16 or 32) destination rows; per
//    tile the row pointers and then the column indices are staged in LDS,
//    every thread aggregates (row, 4- or 8-feature chunk) items with up to 8
//    neighbour loads in flight, and the bf16 A tile ([self || mean] for
//    GraphSAGE, the normalised sum for GCN) lands in LDS;
//  * v_mfma_f32_16x16x32_bf16 over the A tile and the register-resident
//    W^T, then bias, ReLU (hidden layers) and bf16 stores, or the loss.
// The aggregation output is also written to HBM: the backward pass needs it
// for the weight gradient.  Sums are fp32 over the edges in block order; the
// stored A values are rounded to bf16 (round to nearest even) exactly as the
// separate aggregation kernel stores them.
#include "internal.h"

namespace gnn {

namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kLogitLd = 65;  // row stride of the staged logits (fp32)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct FusedArgs {
    const int64_t *counts;  // counts[0] = destination rows M (null: M = cap_dst)
    const int64_t *rowptr;  // block CSR [M + 1]
    const int32_t *col;     // local source ids
    const float *src_norm;  // GCN normalisers per local source (destinations first), else null
    int64_t cap_dst;
    int32_t es_cap;         // column indices a tile can stage in LDS (BM x the expected row-length bound)
    const uint16_t *h;      // H^{l-1}, bf16, row-major [sources x f]
    int64_t f;
    const uint16_t *wt;     // bf16 W^T [n_out x K]
    const float *bias;      // [n_out] or null
    int64_t n_out;
    uint16_t *agg_out;      // bf16 [M x f]: the mean (GraphSAGE) or the normalised sum (GCN)
    void *out;              // hidden: bf16 H^l = ReLU(Z) [M x n_out]; last layer: fp32 logits
    // last layer only
    const int64_t *labels;  // [graph n]
    const int64_t *targets; // vertex ids of the destination rows (the block's first sources)
    float *g;               // (softmax - onehot) / b, [b x n_out]
    float *row_loss;        // [b]
    int64_t b;
    int kpad, ldk;          // K rounded up to 32; LDS row stride of the A tile (kpad + 8)
    // A-load mode (a_nbr != null): the aggregation was done beforehand; the
    // A rows are [a_self[i] || a_nbr[i]] (GraphSAGE) or a_nbr[i] (GCN), bf16
    const uint16_t *a_self, *a_nbr;
};

// A 16-byte MFMA operand fragment of bf16 W^T row n: elements k0 .. k0+7,
// zero outside [0, n_out) x [0, K).  K is a multiple of 4, so each 4-element
// half lies wholly inside or outside the row.
__device__ __forceinline__ bf16x8 load_wfrag(const uint16_t *wt, int64_t K, int64_t n_out, int64_t n, int64_t k0) {
    uint2 lo = make_uint2(0u, 0u), hi = make_uint2(0u, 0u);
    const bool nok = n < n_out;
    const uint16_t *row = wt + (nok ? n : 0) * K;
    if (nok && k0 < K) lo = *reinterpret_cast<const uint2 *>(row + k0);
    if (nok && k0 + 4 < K) hi = *reinterpret_cast<const uint2 *>(row + k0 + 4);
    const uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
    return __builtin_bit_cast(bf16x8, u);
}

// Features e0 .. e0 + CW - 1 (CW = 4 or 8 bf16, one 8- or 16-byte access) of
// a row, as floats.
template <int CW> struct Chunk;
template <> struct Chunk<4> {
    using raw = uint2;
    float v[4];
    __device__ __forceinline__ static raw load(const uint16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
    __device__ __forceinline__ void set(raw u) {
        v[0] = __uint_as_float(u.x << 16);
        v[1] = __uint_as_float(u.x & 0xffff0000u);
        v[2] = __uint_as_float(u.y << 16);
        v[3] = __uint_as_float(u.y & 0xffff0000u);
    }
    __device__ __forceinline__ raw bf16() const {
        return make_uint2(static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16),
                          static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16));
    }
    __device__ __forceinline__ static void store(uint16_t *p, raw u) { *reinterpret_cast<uint2 *>(p) = u; }
    __device__ __forceinline__ static raw zero() { return make_uint2(0u, 0u); }
};
template <> struct Chunk<8> {
    using raw = uint4;
    float v[8];
    __device__ __forceinline__ static raw load(const uint16_t *p) { return *reinterpret_cast<const uint4 *>(p); }
    __device__ __forceinline__ void set(raw u) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    __device__ __forceinline__ raw bf16() const {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = static_cast<uint32_t>(f32_to_bf16(v[2 * i])) | (static_cast<uint32_t>(f32_to_bf16(v[2 * i + 1])) << 16);
        return make_uint4(w[0], w[1], w[2], w[3]);
    }
    __device__ __forceinline__ static void store(uint16_t *p, raw u) { *reinterpret_cast<uint4 *>(p) = u; }
    __device__ __forceinline__ static raw zero() { return make_uint4(0u, 0u, 0u, 0u); }
};

// One (row, chunk) item of the aggregation: the chunk of the A row (self and
// mean for GraphSAGE, the normalised sum for GCN) into LDS and the
// aggregation output.  The edges [rb, re) of the row are read from Es, eight
// neighbour loads in flight.
template <int KIND, int CW>
__device__ __forceinline__ void aggregate_item(const FusedArgs &a, const int32_t *Es, int rb, int re, int64_t row,
                                               int64_t e0, uint16_t *arow) {
    using Ch = Chunk<CW>;
    const uint16_t *__restrict__ h = a.h;
    const int64_t f = a.f;
    const float wi = (KIND == GNN_AGG_GCN_SYM) ? a.src_norm[row] : 1.f;
    const typename Ch::raw self_raw = Ch::load(h + row * f + e0);
    Ch acc;
#pragma unroll
    for (int i = 0; i < CW; ++i) acc.v[i] = 0.f;
    for (int e = rb; e < re; e += 8) {
        typename Ch::raw v[8];
        float w[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int j = Es[e + q < re ? e + q : rb];
            v[q] = Ch::load(h + static_cast<int64_t>(j) * f + e0);
            w[q] = (KIND == GNN_AGG_GCN_SYM) ? wi * a.src_norm[j] : 1.f;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (e + q < re) {
                Ch x;
                x.set(v[q]);
#pragma unroll
                for (int i = 0; i < CW; ++i)
                    acc.v[i] = (KIND == GNN_AGG_GCN_SYM) ? fmaf(w[q], x.v[i], acc.v[i]) : acc.v[i] + x.v[i];
            }
        }
    }
    if (KIND == GNN_AGG_SAGE_MEAN) {
        if (re > rb) {
            const float d = static_cast<float>(re - rb);
#pragma unroll
            for (int i = 0; i < CW; ++i) acc.v[i] /= d;
        }
        const typename Ch::raw m = acc.bf16();
        Ch::store(arow + e0, self_raw);
        Ch::store(arow + f + e0, m);
        Ch::store(a.agg_out + row * f + e0, m);
    } else {
        const float ws = wi * wi;
        Ch x;
        x.set(self_raw);
#pragma unroll
        for (int i = 0; i < CW; ++i) acc.v[i] = fmaf(ws, x.v[i], acc.v[i]);
        const typename Ch::raw m = acc.bf16();
        Ch::store(arow + e0, m);
        Ch::store(a.agg_out + row * f + e0, m);
    }
}

template <int KIND, int CW>
__device__ __forceinline__ void zero_item(int64_t f, int64_t e0, uint16_t *arow) {
    Chunk<CW>::store(arow + e0, Chunk<CW>::zero());
    if (KIND == GNN_AGG_SAGE_MEAN) Chunk<CW>::store(arow + f + e0, Chunk<CW>::zero());
}

// A-load mode: the A tile's rows straight from HBM.  Chunk c of a row is
// features c * CW .. of the self part (c < C, GraphSAGE) or of the
// aggregation part.  Up to four chunks per thread are loaded before any is
// stored, so their loads are in flight together.
template <int KIND, int CW>
__device__ __forceinline__ void load_a_tile(const FusedArgs &a, int64_t row0, int rows, int C, uint16_t *As) {
    using Ch = Chunk<CW>;
    const int KC = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * C : C;  // chunks per A row
    const int total = rows * KC;
    constexpr int kU = 4;
    for (int base = threadIdx.x; base < total; base += kU * kThreads) {
        typename Ch::raw v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int it = base + u * kThreads;
            const int q = it < total ? it : 0;
            const int r = q / KC, c = q % KC;
            const bool self = KIND == GNN_AGG_SAGE_MEAN && c < C;
            const uint16_t *src = self ? a.a_self : a.a_nbr;
            const int64_t e0 = static_cast<int64_t>(c - ((KIND == GNN_AGG_SAGE_MEAN && !self) ? C : 0)) * CW;
            v[u] = Ch::load(src + (row0 + r) * a.f + e0);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int it = base + u * kThreads;
            if (it < total) Ch::store(As + (it / KC) * a.ldk + (it % KC) * CW, v[u]);
        }
    }
}

// LOGITS: the last layer (fp32 logits, softmax cross-entropy in the
// epilogue; n_out <= 64 so wavefronts 0..3 hold every column); otherwise a
// hidden layer (bias, ReLU, bf16 output).  TPW column tiles per wavefront,
// KSM reduction steps held in registers (kpad / 32 <= KSM).
template <int KIND, int BM, int TPW, int KSM, bool LOGITS>
__global__ void __launch_bounds__(kThreads) fused_layer_kernel(FusedArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    uint16_t *As = reinterpret_cast<uint16_t *>(smem);  // BM x ldk bf16; reused for the logits
    const size_t as_bytes = static_cast<size_t>(
        max(BM * a.ldk * 2, LOGITS ? BM * kLogitLd * 4 : 0));
    int64_t *Rs = reinterpret_cast<int64_t *>(smem + ((as_bytes + 15) & ~size_t(15)));  // BM + 1 row pointers
    int32_t *Es = reinterpret_cast<int32_t *>(Rs + BM + 1);                              // es_cap columns
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t f = a.f;
    const int64_t K = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * f : f;
    const int KS = a.kpad / 32;
    const int CT = static_cast<int>((a.n_out + 15) / 16);

    // this wavefront's weight fragments and bias values
    bf16x8 wf[TPW][KSM];
    float bv[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int64_t n = static_cast<int64_t>(wave + kWaves * t) * 16 + (lane & 15);
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks)
            wf[t][ks] = ks < KS ? load_wfrag(a.wt, K, a.n_out, n, ks * 32 + 8 * (lane >> 4)) : bf16x8{};
        bv[t] = (a.bias && n < a.n_out) ? a.bias[n] : 0.f;
    }

    const int64_t M = a.counts ? min(a.counts[0], a.cap_dst) : a.cap_dst;
    const int64_t ntiles = (M + BM - 1) / BM;
    // 8-feature chunks (16-byte accesses) when rows allow it
    const bool load_a = a.a_nbr != nullptr;
    const bool w8 = (f % 8) == 0 && (load_a ? aligned_dev(a.a_self, 16) && aligned_dev(a.a_nbr, 16)
                                            : aligned_dev(a.h, 16) && aligned_dev(a.agg_out, 16));
    const int cw = w8 ? 8 : 4;
    const int C = static_cast<int>(f / cw);  // chunks per row
    const int kq = static_cast<int>((a.kpad - K) / 4);  // zero 4-element groups of the reduction tail

    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t row0 = tile * BM;
        const int rows = static_cast<int>(min<int64_t>(BM, M - row0));
        if (load_a) {
            if (w8) load_a_tile<KIND, 8>(a, row0, rows, C, As);
            else load_a_tile<KIND, 4>(a, row0, rows, C, As);
            const int KC = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * C : C;
            for (int q = tid; q < (BM - rows) * KC; q += kThreads) {
                uint16_t *dst = As + (rows + q / KC) * a.ldk + (q % KC) * cw;
                *reinterpret_cast<uint2 *>(dst) = make_uint2(0u, 0u);
                if (w8) *reinterpret_cast<uint2 *>(dst + 4) = make_uint2(0u, 0u);
            }
        } else {
        for (int r = tid; r <= rows; r += kThreads) Rs[r] = a.rowptr[row0 + r];
        __syncthreads();
        const int64_t e_beg = Rs[0];
        const int64_t ne = Rs[rows] - e_beg;
        // a tile with more edges than the staging area reads its indices in
        // place (rows longer than the bound the launch was sized for)
        const bool staged = ne <= a.es_cap;
        if (staged)
            for (int e = tid; e < ne; e += kThreads) Es[e] = a.col[e_beg + e];
        const int32_t *E = staged ? Es : a.col + e_beg;
        __syncthreads();

        // aggregation into the A tile (and the aggregation output)
        for (int it = tid; it < BM * C; it += kThreads) {
            const int r = it / C, c = it % C;
            const int64_t e0 = static_cast<int64_t>(c) * cw;
            uint16_t *arow = As + r * a.ldk;
            if (r >= rows) {
                if (w8) zero_item<KIND, 8>(f, e0, arow);
                else zero_item<KIND, 4>(f, e0, arow);
                continue;
            }
            const int rb = static_cast<int>(Rs[r] - e_beg), re = static_cast<int>(Rs[r + 1] - e_beg);
            if (w8) aggregate_item<KIND, 8>(a, E, rb, re, row0 + r, e0, arow);
            else aggregate_item<KIND, 4>(a, E, rb, re, row0 + r, e0, arow);
        }
        }  // aggregation mode
        for (int q = tid; q < BM * kq; q += kThreads) {
            const int r = q / kq, k = static_cast<int>(K) + (q % kq) * 4;
            *reinterpret_cast<uint2 *>(As + r * a.ldk + k) = make_uint2(0u, 0u);
        }
        __syncthreads();

        // the update on the matrix cores
        f32x4 acc[BM / 16][TPW];
#pragma unroll
        for (int rt = 0; rt < BM / 16; ++rt)
#pragma unroll
            for (int t = 0; t < TPW; ++t) acc[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
        bool any = false;
#pragma unroll
        for (int t = 0; t < TPW; ++t) any |= (wave + kWaves * t) < CT;
        if (any) {
#pragma unroll
            for (int ks = 0; ks < KSM; ++ks) {
                if (ks < KS) {
#pragma unroll
                    for (int rt = 0; rt < BM / 16; ++rt) {
                        const bf16x8 af = *reinterpret_cast<const bf16x8 *>(
                            As + (rt * 16 + (lane & 15)) * a.ldk + ks * 32 + 8 * (lane >> 4));
#pragma unroll
                        for (int t = 0; t < TPW; ++t)
                            acc[rt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[t][ks], acc[rt][t], 0, 0, 0);
                    }
                }
            }
        }

        if constexpr (!LOGITS) {
            uint16_t *out = static_cast<uint16_t *>(a.out);
#pragma unroll
            for (int t = 0; t < TPW; ++t) {
                const int64_t n = static_cast<int64_t>(wave + kWaves * t) * 16 + (lane & 15);
                if (n >= a.n_out) continue;
#pragma unroll
                for (int rt = 0; rt < BM / 16; ++rt)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r = rt * 16 + 4 * (lane >> 4) + q;
                        if (r < rows) {
                            const float z = acc[rt][t][q] + bv[t];
                            out[(row0 + r) * a.n_out + n] = f32_to_bf16(z > 0.f ? z : 0.f);
                        }
                    }
            }
            __syncthreads();  // the next tile overwrites Rs, Es and As
        } else {
            // logits through LDS, then one group of TPR threads per row
            float *Ls = reinterpret_cast<float *>(smem);
            __syncthreads();  // every wavefront is done reading As
            if (wave < CT) {
                const int n = wave * 16 + (lane & 15);
#pragma unroll
                for (int rt = 0; rt < BM / 16; ++rt)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        Ls[(rt * 16 + 4 * (lane >> 4) + q) * kLogitLd + n] = acc[rt][0][q] + bv[0];
            }
            __syncthreads();
            constexpr int TPR = kThreads / BM;  // 32 or 16 threads per row, within one wavefront
            const int r = tid / TPR, j = tid % TPR;
            const int64_t row = row0 + r;
            const bool live = r < rows && row < a.b;
            const float *zr = Ls + r * kLogitLd;
            float mx = -INFINITY;
            for (int n = j; n < a.n_out; n += TPR) mx = fmaxf(mx, zr[n]);
#pragma unroll
            for (int o = TPR / 2; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
            float s = 0.f;
            for (int n = j; n < a.n_out; n += TPR) s += expf(zr[n] - mx);
#pragma unroll
            for (int o = TPR / 2; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
            if (live) {
                const float lse = mx + logf(s);
                const int64_t y = a.labels[a.targets[row]];
                const float inv_b = 1.f / static_cast<float>(a.b);
                float *lg = static_cast<float *>(a.out) + row * a.n_out;
                for (int n = j; n < a.n_out; n += TPR) {
                    const float p = expf(zr[n] - lse);
                    a.g[row * a.n_out + n] = (p - (n == y ? 1.f : 0.f)) * inv_b;
                    lg[n] = zr[n];
                }
                if (j == 0) a.row_loss[row] = lse - zr[y];
            }
            __syncthreads();
        }
    }
}

struct Shape {
    int bm, tpw, ksm;
    bool ok;
};

Shape fused_shape(int kind, int64_t f, int64_t n_out, int64_t cap_dst, int32_t maxdeg, bool logits) {
    Shape sh{0, 0, 0, false};
    if (f <= 0 || f % 4 != 0 || n_out <= 0) return sh;
    const int64_t K = kind == GNN_AGG_SAGE_MEAN ? 2 * f : f;
    const int64_t ks = ceil_div(K, 32), ct = ceil_div(n_out, 16);
    const int64_t tpw = ceil_div(ct, kWaves);
    if (logits && n_out > 64) return sh;
    if (tpw == 1 && ks <= 16) sh = Shape{0, 1, 16, true};
    else if (tpw == 2 && ks <= 8) sh = Shape{0, 2, 8, true};
    else return sh;
    sh.bm = cap_dst >= 4096 ? 32 : 16;
    return sh;
}

// Column indices staged per tile: BM rows of the expected length, at most
// 2048 (longer tiles read theirs in place).
int32_t es_cap_of(const Shape &sh, int32_t maxdeg) {
    return static_cast<int32_t>(std::min<int64_t>(static_cast<int64_t>(sh.bm) * std::max(maxdeg, 1), 2048));
}

size_t fused_lds(const Shape &sh, int ldk, bool logits, int32_t maxdeg) {
    const size_t as = std::max<size_t>(static_cast<size_t>(sh.bm) * ldk * 2,
                                       logits ? static_cast<size_t>(sh.bm) * kLogitLd * 4 : 0);
    return round_up(as, 16) + static_cast<size_t>(sh.bm + 1) * 8 + static_cast<size_t>(es_cap_of(sh, maxdeg)) * 4;
}

template <int KIND, int BM, int TPW, int KSM, bool LOGITS>
gnn_status go(const FusedArgs &a, unsigned grid, size_t lds, hipStream_t s) {
    fused_layer_kernel<KIND, BM, TPW, KSM, LOGITS><<<grid, kThreads, lds, s>>>(a);
    return launch_status("fused_layer");
}

template <int KIND, bool LOGITS>
gnn_status go_shape(const Shape &sh, const FusedArgs &a, unsigned grid, size_t lds, hipStream_t s) {
    if (sh.bm == 32) {
        if (sh.tpw == 1) return go<KIND, 32, 1, 16, LOGITS>(a, grid, lds, s);
        return go<KIND, 32, 2, 8, LOGITS>(a, grid, lds, s);
    }
    if (sh.tpw == 1) return go<KIND, 16, 1, 16, LOGITS>(a, grid, lds, s);
    return go<KIND, 16, 2, 8, LOGITS>(a, grid, lds, s);
}

}  // namespace

bool fused_layer_ok(int kind, int precision, int64_t f, int64_t n_out, int64_t cap_dst, int32_t maxdeg, bool last,
                    const void *h, const uint16_t *wt, const void *agg_out) {
    // (in A-load mode h is the self part and agg_out the aggregation)
    if (precision != GNN_BF16 || wt == nullptr) return false;
    if (!aligned(h, 8) || !aligned(wt, 8) || !aligned(agg_out, 8)) return false;
    const Shape sh = fused_shape(kind, f, n_out, cap_dst, maxdeg, last);
    if (!sh.ok) return false;
    const int64_t K = kind == GNN_AGG_SAGE_MEAN ? 2 * f : f;
    const int kpad = static_cast<int>(ceil_div(K, 32) * 32);
    return fused_lds(sh, kpad + 8, last, maxdeg) <= 64 * 1024;
}

namespace {

gnn_status launch_fused(const gnn_block *b, int kind, int32_t maxdeg, const void *h, int64_t f, const uint16_t *wt,
                        const float *bias, int64_t n_out, void *agg_out, const void *a_self, const void *a_nbr,
                        void *out, bool last, const int64_t *labels, float *g, float *row_loss, int64_t batch,
                        hipStream_t s) {
    const Shape sh = fused_shape(kind, f, n_out, b->cap_dst, maxdeg, last);
    GNN_CHECK(sh.ok, GNN_EUNSUPPORTED, "fused_layer: shape not supported");
    const int64_t K = kind == GNN_AGG_SAGE_MEAN ? 2 * f : f;
    FusedArgs a{};
    a.counts = b->counts;
    a.rowptr = b->rowptr;
    a.col = b->col;
    a.src_norm = b->src_norm;
    a.cap_dst = b->cap_dst;
    a.es_cap = es_cap_of(sh, maxdeg);
    a.h = static_cast<const uint16_t *>(h);
    a.f = f;
    a.wt = wt;
    a.bias = bias;
    a.n_out = n_out;
    a.agg_out = static_cast<uint16_t *>(agg_out);
    a.out = out;
    a.labels = labels;
    a.targets = b->src_ids;
    a.g = g;
    a.row_loss = row_loss;
    a.b = batch;
    a.kpad = static_cast<int>(ceil_div(K, 32) * 32);
    a.ldk = a.kpad + 8;
    a.a_self = static_cast<const uint16_t *>(a_self);
    a.a_nbr = static_cast<const uint16_t *>(a_nbr);
    const size_t lds = fused_lds(sh, a.ldk, last, maxdeg);
    const unsigned grid = static_cast<unsigned>(std::min<int64_t>(ceil_div(std::max<int64_t>(b->cap_dst, 1), sh.bm),
                                                                  256));
    if (kind == GNN_AGG_SAGE_MEAN)
        return last ? go_shape<GNN_AGG_SAGE_MEAN, true>(sh, a, grid, lds, s)
                    : go_shape<GNN_AGG_SAGE_MEAN, false>(sh, a, grid, lds, s);
    return last ? go_shape<GNN_AGG_GCN_SYM, true>(sh, a, grid, lds, s)
                : go_shape<GNN_AGG_GCN_SYM, false>(sh, a, grid, lds, s);
}

}  // namespace

gnn_status launch_fused_layer(const gnn_block *b, int kind, int32_t maxdeg, const void *h, int64_t f,
                              const uint16_t *wt, const float *bias, int64_t n_out, void *agg_out, void *out,
                              bool last, const int64_t *labels, float *g, float *row_loss, int64_t batch,
                              hipStream_t s) {
    return launch_fused(b, kind, maxdeg, h, f, wt, bias, n_out, agg_out, nullptr, nullptr, out, last, labels, g,
                        row_loss, batch, s);
}

gnn_status launch_fused_update(const gnn_block *b, int kind, const void *a_self, const void *a_nbr, int64_t f,
                               const uint16_t *wt, const float *bias, int64_t n_out, void *out, bool last,
                               const int64_t *labels, float *g, float *row_loss, int64_t batch, hipStream_t s) {
    GNN_CHECK(a_nbr && (kind != GNN_AGG_SAGE_MEAN || a_self), GNN_EINVAL, "fused_update: NULL A operand");
    return launch_fused(b, kind, 1, a_self ? a_self : a_nbr, f, wt, bias, n_out, nullptr, a_self, a_nbr, out, last,
                        labels, g, row_loss, batch, s);
}

}  // namespace gnn
