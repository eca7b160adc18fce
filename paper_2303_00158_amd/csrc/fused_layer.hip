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
//  * the workgroup walks row tiles of BM (4, 8, 16 or 32) destination rows; per
//    tile the row pointers and then the column indices are staged in LDS,
//    every thread aggregates (row, 4- or 8-feature chunk) items with up to
//    kNbr neighbour loads in flight, and the bf16 A tile ([self || mean] for
//    GraphSAGE, the normalised sum for GCN) lands in LDS;
//  * v_mfma_f32_16x16x32_bf16 over the A tile and the register-resident
//    W^T, then bias, ReLU (hidden layers) and bf16 stores, or the loss.
// The aggregation output is also written to HBM: the backward pass needs it
// for the weight gradient.  Sums are fp32 over the edges in block order; the
// stored A values are rounded to bf16 (round to nearest even) exactly as the
// separate aggregation kernel stores them.
#include "fused_dev.h"

namespace gnn {

namespace {

using namespace fl;

struct FusedArgs {
    const int64_t *counts;  // M = min((counts[0] & cnt_keep) | cnt_add, cap_dst) (never null)
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
    int kpad, ldk;          // KSM x 32 (the reduction length the kernel runs); A tile row stride (kpad + 8)
    // A-load mode (a_nbr != null): the aggregation was done beforehand; the
    // A rows are [a_self[i] || a_nbr[i]] (GraphSAGE) or a_nbr[i] (GCN), bf16
    const uint16_t *a_self, *a_nbr;
    int64_t cnt_keep, cnt_add;  // -1, 0 with a device row count; 0, cap_dst without one
};

// Every kernel argument in one batch of scalar loads at entry (in_sgpr).
__device__ __forceinline__ void args_up_front(const FusedArgs &a) {
    in_sgpr(a.counts), in_sgpr(a.rowptr), in_sgpr(a.col), in_sgpr(a.src_norm), in_sgpr(a.cap_dst);
    in_sgpr(a.es_cap), in_sgpr(a.h), in_sgpr(a.f), in_sgpr(a.wt), in_sgpr(a.bias), in_sgpr(a.n_out);
    in_sgpr(a.agg_out), in_sgpr(a.out), in_sgpr(a.labels), in_sgpr(a.targets), in_sgpr(a.g), in_sgpr(a.row_loss);
    in_sgpr(a.b), in_sgpr(a.kpad), in_sgpr(a.ldk), in_sgpr(a.a_self), in_sgpr(a.a_nbr), in_sgpr(a.cnt_keep);
    in_sgpr(a.cnt_add);
}

// One (row, chunk) item of the aggregation: the chunk of the A row (self and
// mean for GraphSAGE, the normalised sum for GCN) into LDS and the
// aggregation output.  The edges [rb, re) of the row are read from Es, kNbr
// neighbour loads in flight (a row of the usual fanouts takes one or two
// rounds of load latency).
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
    for (int e = rb; e < re; e += kNbr) {
        typename Ch::raw v[kNbr];
        float w[kNbr];
#pragma unroll
        for (int q = 0; q < kNbr; ++q) {
            const int j = Es[e + q < re ? e + q : rb];
            v[q] = Ch::load(h + static_cast<int64_t>(j) * f + e0);
            w[q] = (KIND == GNN_AGG_GCN_SYM) ? wi * a.src_norm[j] : 1.f;
        }
#pragma unroll
        for (int q = 0; q < kNbr; ++q) {
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

// A-load mode: the A tile's rows straight from HBM.  Item q of a tile is
// chunk q % KC of row q / KC (KC chunks per A row); chunk c holds features
// c * CW .. of the self part (c < C, GraphSAGE) or of the aggregation part.
// A round is kU items per thread, all loaded before any is stored so that
// their loads are in flight together.  The loads read any row inside the
// capacity (rows at or past the row count are stored as zeros), so a tile's
// first round can be issued before the row count has arrived.
constexpr int kU = 4;
template <int KIND, int CW>
__device__ __forceinline__ void load_a_round(const FusedArgs &a, int64_t row0, int C, int items, int base,
                                             uint4 (&v)[kU]) {
    const int KC = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * C : C;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int it = base + u * kThreads;
        const int q = it < items ? it : 0;
        const int r = q / KC, c = q % KC;
        const bool self = KIND == GNN_AGG_SAGE_MEAN && c < C;
        const uint16_t *src = self ? a.a_self : a.a_nbr;
        const int64_t e0 = static_cast<int64_t>(c - ((KIND == GNN_AGG_SAGE_MEAN && !self) ? C : 0)) * CW;
        const int64_t row = min<int64_t>(row0 + r, a.cap_dst - 1);
        if constexpr (CW == 8) {
            v[u] = Chunk<8>::load(src + row * a.f + e0);
        } else {
            const uint2 w = Chunk<4>::load(src + row * a.f + e0);
            v[u] = make_uint4(w.x, w.y, 0u, 0u);
        }
    }
}
template <int KIND, int CW>
__device__ __forceinline__ void store_a_round(const FusedArgs &a, int rows, int C, int items, int base,
                                              const uint4 (&v)[kU], uint16_t *As) {
    const int KC = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * C : C;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
        const int it = base + u * kThreads;
        if (it >= items) continue;
        const int r = it / KC;
        uint16_t *dst = As + r * a.ldk + (it % KC) * CW;
        const uint4 x = r < rows ? v[u] : make_uint4(0u, 0u, 0u, 0u);
        if constexpr (CW == 8) Chunk<8>::store(dst, x);
        else Chunk<4>::store(dst, make_uint2(x.x, x.y));
    }
}

// LOGITS: the last layer (fp32 logits, softmax cross-entropy in the
// epilogue; n_out <= 64 so wavefronts 0..3 hold every column); otherwise a
// hidden layer (bias, ReLU, bf16 output).  TPW column tiles per wavefront,
// KSM reduction steps held in registers (kpad = 32 KSM >= K; the A tile's
// columns K .. kpad are zero, so every step runs unconditionally).  W16: 16-byte
// weight loads (see load_wfrag).  LOADA: A-load
// mode (a_nbr set), else aggregation mode.
template <int KIND, int BM, int TPW, int KSM, bool LOGITS, bool LOADA, bool W16>
__global__ void __launch_bounds__(kThreads) fused_layer_kernel(FusedArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    args_up_front(a);
    // the A tile has AR >= BM rows (whole 16-row matrix-core tiles; rows
    // BM .. AR stay zero)
    constexpr int RT = (BM + 15) / 16, AR = 16 * RT;
    uint16_t *As = reinterpret_cast<uint16_t *>(smem);  // AR x ldk bf16; reused for the logits
    const size_t as_bytes = static_cast<size_t>(
        max(AR * a.ldk * 2, LOGITS ? AR * kLogitLd * 4 : 0));
    int64_t *Rs = reinterpret_cast<int64_t *>(smem + ((as_bytes + 15) & ~size_t(15)));  // BM + 1 row pointers
    int32_t *Es = reinterpret_cast<int32_t *>(Rs + BM + 1);                              // es_cap columns
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t f = a.f;
    const int64_t K = (KIND == GNN_AGG_SAGE_MEAN) ? 2 * f : f;
    const int CT = static_cast<int>((a.n_out + 15) / 16);
    // epilogue: TPR threads per row (64, 32 or 16, within one wavefront);
    // with BM = 4 only the first 4 x 64 threads have a row
    constexpr int TPR = kThreads / BM > 64 ? 64 : kThreads / BM;
    // 8-feature chunks (16-byte accesses) when rows allow it
    constexpr bool load_a = LOADA;
    const bool w8 = (f % 8) == 0 && (load_a ? aligned_dev(a.a_self, 16) && aligned_dev(a.a_nbr, 16)
                                            : aligned_dev(a.h, 16) && aligned_dev(a.agg_out, 16));
    const int cw = w8 ? 8 : 4;
    const int C = static_cast<int>(f / cw);  // chunks per row
    const int a_items = AR * ((KIND == GNN_AGG_SAGE_MEAN) ? 2 * C : C);
    const int kq = static_cast<int>((a.kpad - K) / 4);  // zero 4-element groups of the reduction tail

    // A tile's first loads do not wait for the row count: its row pointers
    // (aggregation) or first A round (A-load), and in the last layer its
    // target ids, are read inside the block's capacity and issued before the
    // weights, since the vector-memory counter completes loads in issue
    // order.  Only rows below the count use what they read.
    int64_t rp = 0, tg = 0;
    uint4 va[kU];
    auto prefetch = [&](int64_t row0) {
        if (load_a) {
            if (w8) load_a_round<KIND, 8>(a, row0, C, a_items, tid, va);
            else load_a_round<KIND, 4>(a, row0, C, a_items, tid, va);
        } else if (tid <= BM) {
            rp = a.rowptr[min<int64_t>(row0 + tid, a.cap_dst)];
        }
        if (LOGITS) tg = a.targets[min<int64_t>(row0 + tid / TPR, a.cap_dst - 1)];
    };
    prefetch(static_cast<int64_t>(blockIdx.x) * BM);

    // The row count: a scalar load (it waits on its own counter, not behind
    // the vector loads) whose use is branch-free arithmetic, so that nothing
    // waits for it before the weights have been issued.
    typedef const __attribute__((address_space(4))) int64_t *const_i64;
    const int64_t M = min((*(const_i64)a.counts & a.cnt_keep) | a.cnt_add, a.cap_dst);

    // this wavefront's weight fragments and bias values
    bf16x8 wf[TPW][KSM];
    float bv[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int64_t n = static_cast<int64_t>(wave + kWaves * t) * 16 + (lane & 15);
        if (wave + kWaves * t < CT) {  // (uniform per wavefront)
            // columns n >= n_out read row 0: they only feed outputs that are never stored
            const uint32_t row = static_cast<uint32_t>((n < a.n_out ? n : 0) * K);
#pragma unroll
            for (int ks = 0; ks < KSM; ++ks)
                wf[t][ks] = load_wfrag<W16>(a.wt, row, static_cast<uint32_t>(K), ks * 32 + 8 * (lane >> 4));
        } else {
#pragma unroll
            for (int ks = 0; ks < KSM; ++ks) wf[t][ks] = bf16x8{};
        }
        // (a null bias reads W^T instead; the epilogue discards it)
        bv[t] = (a.bias ? a.bias : reinterpret_cast<const float *>(a.wt))[n < a.n_out ? n : 0];
    }
    for (int64_t tile = blockIdx.x; tile * BM < a.cap_dst; tile += gridDim.x) {
        const int64_t row0 = tile * BM;
        const int rows = static_cast<int>(min<int64_t>(BM, M - row0));
        if (rows <= 0) break;
        if (tile != blockIdx.x) prefetch(row0);  // later tiles (few workgroups have any)
        const int er = tid / TPR;  // this thread's row in the last layer's epilogue
        const bool live = LOGITS && er < rows && row0 + er < a.b;
        if (load_a) {
            for (int base = tid; base < a_items; base += kU * kThreads) {
                if (base != tid) {
                    if (w8) load_a_round<KIND, 8>(a, row0, C, a_items, base, va);
                    else load_a_round<KIND, 4>(a, row0, C, a_items, base, va);
                }
                if (w8) store_a_round<KIND, 8>(a, rows, C, a_items, base, va, As);
                else store_a_round<KIND, 4>(a, rows, C, a_items, base, va, As);
            }
        } else {
        if (tid <= rows) Rs[tid] = rp;
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
        for (int it = tid; it < AR * C; it += kThreads) {
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
        for (int q = tid; q < AR * kq; q += kThreads) {
            const int r = q / kq, k = static_cast<int>(K) + (q % kq) * 4;
            *reinterpret_cast<uint2 *>(As + r * a.ldk + k) = make_uint2(0u, 0u);
        }
        // last layer: the row's label, in flight during the matrix-core work
        // (the target id's load was issued with the weights, which the matrix
        // cores need by now anyway)
        const int64_t y = live ? a.labels[tg] : 0;
        __syncthreads();

        // The bias as the epilogue uses it.  The empty asm keeps the choice
        // inside the loop: hoisted before it, the choice would wait for the
        // bias load, and with it for every load issued before it.
        float bias_t[TPW];
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            bias_t[t] = bv[t];
            asm volatile("" : "+v"(bias_t[t]));
            if (!a.bias) bias_t[t] = 0.f;
        }

        // the update on the matrix cores
        f32x4 acc[RT][TPW];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int t = 0; t < TPW; ++t) acc[rt][t] = f32x4{0.f, 0.f, 0.f, 0.f};
        bool any = false;
#pragma unroll
        for (int t = 0; t < TPW; ++t) any |= (wave + kWaves * t) < CT;
        if (any) {
#pragma unroll
            for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const bf16x8 af = *reinterpret_cast<const bf16x8 *>(
                        As + (rt * 16 + (lane & 15)) * a.ldk + ks * 32 + 8 * (lane >> 4));
#pragma unroll
                    for (int t = 0; t < TPW; ++t)
                        acc[rt][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf[t][ks], acc[rt][t], 0, 0, 0);
                }
        }

        if constexpr (!LOGITS) {
            uint16_t *out = static_cast<uint16_t *>(a.out);
#pragma unroll
            for (int t = 0; t < TPW; ++t) {
                const int64_t n = static_cast<int64_t>(wave + kWaves * t) * 16 + (lane & 15);
                if (n >= a.n_out) continue;
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r = rt * 16 + 4 * (lane >> 4) + q;
                        if (r < rows) {
                            const float z = acc[rt][t][q] + bias_t[t];
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
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        Ls[(rt * 16 + 4 * (lane >> 4) + q) * kLogitLd + n] = acc[rt][0][q] + bias_t[0];
            }
            __syncthreads();
            softmax_ce_row<TPR>(Ls + er * kLogitLd, tid % TPR, live, row0 + er, y, a.n_out, a.b,
                                static_cast<float *>(a.out), a.g, a.row_loss);
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
    // the reduction runs KSM steps over a zero-padded A tile: half the steps
    // when K fits them (GCN's K = f; small layers)
    if (tpw == 1 && ks <= 8) sh = Shape{0, 1, 8, true};
    else if (tpw == 1 && ks <= 16) sh = Shape{0, 1, 16, true};
    else if (tpw == 2 && ks <= 4) sh = Shape{0, 2, 4, true};
    else if (tpw == 2 && ks <= 8) sh = Shape{0, 2, 8, true};
    else return sh;
    // rows per tile: enough workgroups to spread the gather over the CUs
    // (each CU keeps a bounded number of misses in flight)
    sh.bm = cap_dst >= 8192 ? 32 : cap_dst >= 4096 ? 16 : cap_dst >= 2048 ? 8 : 4;
    return sh;
}

// Column indices staged per tile: BM rows of the expected length, at most
// 2048 (longer tiles read theirs in place).
int32_t es_cap_of(const Shape &sh, int32_t maxdeg) {
    return static_cast<int32_t>(std::min<int64_t>(static_cast<int64_t>(sh.bm) * std::max(maxdeg, 1), 2048));
}

size_t fused_lds(const Shape &sh, int ldk, bool logits, int32_t maxdeg) {
    const size_t ar = round_up(static_cast<size_t>(sh.bm), 16);  // A tile rows
    const size_t as = std::max<size_t>(ar * ldk * 2, logits ? ar * kLogitLd * 4 : 0);
    return round_up(as, 16) + static_cast<size_t>(sh.bm + 1) * 8 + static_cast<size_t>(es_cap_of(sh, maxdeg)) * 4;
}

template <int KIND, int BM, int TPW, int KSM, bool LOGITS>
gnn_status go(const FusedArgs &a, unsigned grid, size_t lds, hipStream_t s) {
    const int64_t K = KIND == GNN_AGG_SAGE_MEAN ? 2 * a.f : a.f;
    const bool w16 = K % 8 == 0 && aligned(a.wt, 16);
    if (a.a_nbr) {
        if (w16) fused_layer_kernel<KIND, BM, TPW, KSM, LOGITS, true, true><<<grid, kThreads, lds, s>>>(a);
        else fused_layer_kernel<KIND, BM, TPW, KSM, LOGITS, true, false><<<grid, kThreads, lds, s>>>(a);
    } else {
        if (w16) fused_layer_kernel<KIND, BM, TPW, KSM, LOGITS, false, true><<<grid, kThreads, lds, s>>>(a);
        else fused_layer_kernel<KIND, BM, TPW, KSM, LOGITS, false, false><<<grid, kThreads, lds, s>>>(a);
    }
    return launch_status("fused_layer");
}

template <int KIND, int BM, bool LOGITS>
gnn_status go_steps(const Shape &sh, const FusedArgs &a, unsigned grid, size_t lds, hipStream_t s) {
    if (sh.tpw == 1) return sh.ksm == 8 ? go<KIND, BM, 1, 8, LOGITS>(a, grid, lds, s)
                                        : go<KIND, BM, 1, 16, LOGITS>(a, grid, lds, s);
    return sh.ksm == 4 ? go<KIND, BM, 2, 4, LOGITS>(a, grid, lds, s) : go<KIND, BM, 2, 8, LOGITS>(a, grid, lds, s);
}

template <int KIND, bool LOGITS>
gnn_status go_shape(const Shape &sh, const FusedArgs &a, unsigned grid, size_t lds, hipStream_t s) {
    if (sh.bm == 4) return go_steps<KIND, 4, LOGITS>(sh, a, grid, lds, s);
    if (sh.bm == 8) return go_steps<KIND, 8, LOGITS>(sh, a, grid, lds, s);
    if (sh.bm == 32) return go_steps<KIND, 32, LOGITS>(sh, a, grid, lds, s);
    return go_steps<KIND, 16, LOGITS>(sh, a, grid, lds, s);
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
    (void)K;
    return fused_lds(sh, sh.ksm * 32 + 8, last, maxdeg) <= 64 * 1024;
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
    // without a device row count, M = cap_dst and the count load reads W^T
    a.counts = b->counts ? b->counts : reinterpret_cast<const int64_t *>(wt);
    a.cnt_keep = b->counts ? -1 : 0;
    a.cnt_add = b->counts ? 0 : b->cap_dst;
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
    a.kpad = sh.ksm * 32;
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
