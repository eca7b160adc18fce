// Forward of a two-layer model in one launch: layer 1's update, layer 2's
// aggregation and update, and the loss.
//
// Layer 1's aggregation M^1 is made by the prepare stage (it needs no
// weights), so a row of H^1 = ReLU([X'[j] || M^1[j]] W^1 + b^1) (equation 2;
// for GCN the A^1 row is M^1[j] alone) costs one A^1 row and the layer's
// weights.  A tile of the last block's destinations needs H^1 only on its own
// rows (GraphSAGE's self term, GCN's self loop) and on the rows its sampled
// edges name.  The workgroup gathers exactly those A^1 rows, in edge order,
// computes their H^1 rows on the matrix cores with W^1 in registers, keeps
// them in LDS for the aggregation of equation 1 and writes them out for the
// backward pass; the A^2 tile then goes through the update with W^2 in
// registers and the softmax cross-entropy epilogue (Section II-B's loss).
// This is the on-chip aggregate -> update datapath of Section IV-C carried
// across the layer boundary.
//
// A row that several tiles sample is computed by each of them.  The copies
// are identical (an output element is one fp32 sum over K in a fixed order,
// whatever other rows share its matrix-core tile), so their stores race
// harmlessly.  At small mini-batches the last block has about as many edges
// as sources, so little is computed twice, and the launch that had to
// produce all of H^1 before any aggregation could start is gone.
//
// The arithmetic is that of the two launches it replaces (layer 1's update
// in A-load mode, then the fused last layer): H^1 bits, the aggregation's
// fp32 sums in edge order, the A^2 bits and the logits are the same.
#include "fused_dev.h"

namespace gnn {

namespace {

using namespace fl;

constexpr int kBm = 4;      // destinations per tile
constexpr int kSrows = 112;  // H^1 rows per pass: seven 16-row matrix-core tiles (kBm x 27 edges)
constexpr int kTpw1 = 2;    // layer-1 output column tiles per wavefront (f1 <= 256)
constexpr int kU = 8;       // A^1 chunks per thread in flight
constexpr int kLdh = 256 + 8;  // H^1 tile row stride (elements; f1 <= 256)
constexpr int kEsMax = kThreads;  // column indices a tile stages (one per thread)

constexpr int cmax(int x, int y) { return x > y ? x : y; }

struct TwoArgs {
    const int64_t *counts;   // M = min((counts[0] & cnt_keep) | cnt_add, cap_dst) (never null)
    int64_t cnt_keep, cnt_add;
    const int64_t *rowptr;   // last block CSR [M + 1]
    const int32_t *col;      // its local source ids = rows of H^1
    const float *src_norm;   // GCN normalisers of its sources, else null
    int64_t cap_dst;
    int32_t es_cap;          // column indices a tile stages in LDS
    const uint16_t *x_self;  // X' rows, GraphSAGE's self part of A^1, bf16 [rows x f0]
    const uint16_t *m1;      // M^1 rows, bf16 [rows x f0]
    int64_t f0;
    const uint16_t *wt1;     // bf16 (W^1)^T [f1 x K1]
    const float *bias1;      // [f1] or null
    int64_t f1;
    uint16_t *h1;            // H^1, bf16 [layer-1 rows x f1]
    const uint16_t *wt2;     // bf16 (W^2)^T [n_out x K2]
    const float *bias2;      // [n_out] or null
    int64_t n_out;
    uint16_t *agg_out;       // M^2, bf16 [cap_dst x f1]
    int32_t *argmax;         // max aggregator: int32 argmax table of M^2 [rows x f1], else null
    float *logits;           // [cap_dst x n_out]
    const int64_t *labels;   // [graph n]
    const int64_t *targets;  // vertex ids of the destinations
    float *g;                // (softmax - onehot) / b, [b x n_out]
    float *row_loss;         // [b]
    int64_t b;
    float *d_a;              // dA^2 = G (W^2)^T, fp32 [cap_dst x K2], or null
};

__device__ __forceinline__ void args_up_front(const TwoArgs &a) {
    in_sgpr(a.counts), in_sgpr(a.cnt_keep), in_sgpr(a.cnt_add), in_sgpr(a.rowptr), in_sgpr(a.col);
    in_sgpr(a.src_norm), in_sgpr(a.cap_dst), in_sgpr(a.es_cap), in_sgpr(a.x_self), in_sgpr(a.m1), in_sgpr(a.f0);
    in_sgpr(a.wt1), in_sgpr(a.bias1), in_sgpr(a.f1), in_sgpr(a.h1), in_sgpr(a.wt2), in_sgpr(a.bias2);
    in_sgpr(a.n_out), in_sgpr(a.agg_out), in_sgpr(a.logits), in_sgpr(a.labels), in_sgpr(a.targets), in_sgpr(a.g);
    in_sgpr(a.row_loss), in_sgpr(a.b), in_sgpr(a.d_a);
}

// Row of H^1 behind tile row s: the destinations first (a destination is
// its own source), then the source of each edge of the tile.
__device__ __forceinline__ int64_t s_row(int s, int rows, int64_t row0, const int32_t *E) {
    return s < rows ? row0 + s : static_cast<int64_t>(E[s - rows]);
}

// The A^1 rows of tile rows s0 .. s0 + ns into A1s, and zeros in rows
// ns .. rz (the rest of the last 16-row tile in use).  Item q is chunk
// q % KC of tile row q / KC; for GraphSAGE chunks below C0 come from X', the
// rest from M^1.  kU items per thread are loaded before any is stored, so
// their loads are in flight together.
template <bool SAGE, int CW0, int LDK1>
__device__ __forceinline__ void gather_a1(const TwoArgs &a, const int32_t *E, int64_t row0, int rows, int s0, int ns,
                                          int rz, int C0, uint16_t *A1s) {
    using Ch = Chunk<CW0>;
    const int KC = SAGE ? 2 * C0 : C0;
    const int items = ns * KC;
    for (int base = threadIdx.x; base < items; base += kU * kThreads) {
        typename Ch::raw v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int it = base + u * kThreads;
            const int q = it < items ? it : 0;
            const int r = q / KC, c = q % KC;
            const int64_t j = s_row(s0 + r, rows, row0, E);
            const bool self = SAGE && c < C0;
            const int64_t e0 = static_cast<int64_t>(self || !SAGE ? c : c - C0) * CW0;
            v[u] = Ch::load((self ? a.x_self : a.m1) + j * a.f0 + e0);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int it = base + u * kThreads;
            if (it < items) Ch::store(A1s + (it / KC) * LDK1 + (it % KC) * CW0, v[u]);
        }
    }
    for (int q = items + threadIdx.x; q < rz * KC; q += kThreads)
        Ch::store(A1s + (q / KC) * LDK1 + (q % KC) * CW0, Ch::zero());
}

// A 16-byte MFMA fragment of bf16 W^T (elements k .. k+7 of the row
// starting at element `row`) through a buffer descriptor: a wavefront that
// owns no columns holds a descriptor with no records, so its loads return
// zeros without a memory access.  Every wavefront thus issues the same
// branch-free sequence of loads, which keeps the compiler's count of loads
// in flight exact (a branch around them makes it wait for all of them at the
// join, and with them for everything issued before).  Clamping as load_wfrag.
template <bool W16>
__device__ __forceinline__ bf16x8 wfrag_buf(__amdgpu_buffer_rsrc_t r, uint32_t row, uint32_t K, uint32_t k) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    if constexpr (W16) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(2u * (row + min(k, K - 8))), 0, 0);
        return __builtin_bit_cast(bf16x8, v);
    } else {
        const uint32_t last = K - 4;
        const u32x2 lo = __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(2u * (row + min(k, last))), 0, 0);
        const u32x2 hi = __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(2u * (row + min(k + 4u, last))), 0, 0);
        return __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
    }
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const uint16_t *p, bool own, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p), 0, own ? static_cast<int>(bytes) : 0,
                                             0x00020000);
}

// One workgroup per tile of kBm destinations.  KSM1: reduction steps of
// layer 1 (32 KSM1 >= K1); CW0: features per A^1 chunk (8 when f0 % 8 == 0,
// else 4).  Layer 2 runs 32 KSM2 >= K2 = 2 f1 (GraphSAGE) or f1 (GCN) with
// f1 <= 256.  W^1 rows are read 16 bytes at a time when K1 % 8 == 0 (always
// for GraphSAGE, and for GCN when CW0 == 8), W^2 rows always (K2 % 8 == 0).
//
// Load order, which the vector-memory counter completes in: row pointers and
// target ids; the tile's column indices; W^1 (in flight while the indices
// are staged and the A^1 rows gathered); the A^1 rows; W^2 after layer 1
// (needed last).  A load's wait then covers only what was issued before it.
template <int KIND, int KSM1, int CW0>
__global__ void __launch_bounds__(kThreads) two_layer_kernel(TwoArgs a) {
    constexpr bool SAGE = KIND != GNN_AGG_GCN_SYM;  // A = [h_self || aggregation]
    constexpr bool MAXA = KIND == GNN_AGG_SAGE_MAX;
    constexpr bool W16A = SAGE || CW0 == 8;
    constexpr int KSM2 = SAGE ? 16 : 8;
    constexpr int TPR = kThreads / kBm > 64 ? 64 : kThreads / kBm;  // epilogue threads per destination
    constexpr int LDK1 = 32 * KSM1 + 8, LDK2 = 32 * KSM2 + 8;  // LDS row strides (elements)
    constexpr int LDW2 = 32 * KSM2 + 8;                          // staged W^2 rows
    constexpr int A_ELEMS = cmax(cmax(kSrows * LDK1, 16 * LDK2), 16 * kLogitLd * 2);
    __shared__ __attribute__((aligned(16))) uint16_t A1s[A_ELEMS];  // A^1 tile; then the A^2 tile, then the logits
    __shared__ __attribute__((aligned(16))) uint16_t Hs[kSrows * kLdh];
    __shared__ int64_t Rs[kBm + 1];  // row pointers
    __shared__ int32_t Es[kEsMax];   // column indices
    __shared__ float Ns[kEsMax];     // GCN: their normalisers
    __shared__ float Gs[kWaves * 64];  // bf16-rounded gradient rows (dA^2's left operand)
    args_up_front(a);
    uint16_t *A2s = A1s;
    float *Ls = reinterpret_cast<float *>(A1s);
    // (the wavefront index as a scalar, so that per-wavefront buffer
    // descriptors live in scalar registers)
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t f0 = a.f0, f1 = a.f1;
    const int64_t K1 = SAGE ? 2 * f0 : f0, K2 = SAGE ? 2 * f1 : f1;
    const int C0 = static_cast<int>(f0 / CW0);
    const int C1 = static_cast<int>(f1 / 8);  // 8-feature chunks of an H^1 row
    const int CT1 = static_cast<int>((f1 + 15) / 16), CT2 = static_cast<int>((a.n_out + 15) / 16);
    const int kq1 = static_cast<int>((32 * KSM1 - K1) / 4), kq2 = static_cast<int>((32 * KSM2 - K2) / 4);

    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kBm;
    int64_t rp = 0;
    if (tid <= kBm) rp = a.rowptr[min<int64_t>(row0 + tid, a.cap_dst)];
    const int64_t tg = a.targets[min<int64_t>(row0 + tid / TPR, a.cap_dst - 1)];
    // the row count: a scalar load, used through branch-free arithmetic
    typedef const __attribute__((address_space(4))) int64_t *const_i64;
    const int64_t M = min((*(const_i64)a.counts & a.cnt_keep) | a.cnt_add, a.cap_dst);
    const int rows = static_cast<int>(min<int64_t>(kBm, M - row0));
    if (rows <= 0) return;  // (uniform)
    const int er = tid / TPR;  // this thread's destination in the loss epilogue
    const bool live = er < rows && row0 + er < a.b;
    if (tid <= rows) Rs[tid] = rp;
    __syncthreads();
    const int64_t e_beg = Rs[0];
    const int ne = static_cast<int>(Rs[rows] - e_beg);
    // a tile with more edges than the staging area reads its indices in
    // place (rows longer than the fanout the launch was sized for)
    const bool staged = ne <= a.es_cap;
    int32_t cj = 0;
    if (staged && tid < ne) cj = a.col[e_beg + tid];  // (es_cap <= kThreads)
    __builtin_amdgcn_sched_barrier(0);

    // layer 1's weights: wavefront w owns output column tiles w and w + 8
    bf16x8 wf1[kTpw1][KSM1];
    float bv1[kTpw1];
#pragma unroll
    for (int t = 0; t < kTpw1; ++t) {
        const int ct = wave + kWaves * t;
        const int64_t n = static_cast<int64_t>(ct) * 16 + (lane & 15);
        const __amdgpu_buffer_rsrc_t r = rows_rsrc(a.wt1, ct < CT1, f1 * K1 * 2);
        const uint32_t row = static_cast<uint32_t>((n < f1 ? n : 0) * K1);
#pragma unroll
        for (int ks = 0; ks < KSM1; ++ks)
            wf1[t][ks] = wfrag_buf<W16A>(r, row, static_cast<uint32_t>(K1), ks * 32 + 8 * (lane >> 4));
        // (a null bias reads W^T instead; the epilogue discards it)
        bv1[t] = (a.bias1 ? a.bias1 : reinterpret_cast<const float *>(a.wt1))[n < f1 ? n : 0];
    }
    __builtin_amdgcn_sched_barrier(0);
    if (staged && tid < ne) Es[tid] = cj;
    const int64_t y = live ? a.labels[tg] : 0;
    // the A^1 tile's reduction padding (columns K1 .. 32 KSM1) is zero
    for (int q = tid; q < kSrows * kq1; q += kThreads) {
        const int r = q / kq1, k = static_cast<int>(K1) + (q % kq1) * 4;
        *reinterpret_cast<uint2 *>(A1s + r * LDK1 + k) = make_uint2(0u, 0u);
    }
    __syncthreads();
    if (!SAGE && staged && tid < ne) Ns[tid] = a.src_norm[cj];
    // The rest of the tile, instantiated for indices staged in LDS and for
    // indices read in place, so that each copy reads them through one
    // address space (a pointer that may be either makes every index read
    // a flat access, which waits for all vector loads in flight).
    auto rest = [&](auto staged_tag) {
    constexpr bool STAGED = decltype(staged_tag)::value;
    const int32_t *E;
    if constexpr (STAGED) E = Es;
    else E = a.col + e_beg;

    // this thread's aggregation item: destination ar, features 8 ac ..
    // 8 ac + 7; its edges are [rb, re) of the tile
    const int ar = tid / C1, ac = tid % C1;
    const bool item = tid < kBm * C1 && ar < rows;
    int rb = 0, re = 0;
    float wi = 1.f;
    if (item) {
        rb = static_cast<int>(Rs[ar] - e_beg);
        re = static_cast<int>(Rs[ar + 1] - e_beg);
        if (!SAGE) wi = a.src_norm[row0 + ar];
    }
    Chunk<8> acc;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc.v[i] = 0.f;
    // max aggregator: acc holds the running maximum, am the local source of
    // the edge that holds it (-1 before the row's first edge)
    int32_t am[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) am[i] = -1;
    uint4 self_raw = make_uint4(0u, 0u, 0u, 0u);

    // layer 2's weights (wavefronts 0 .. CT2 - 1, one column tile each,
    // n_out <= 64), loaded in the last pass once its stores are issued
    bf16x8 wf2[KSM2];
    float bias2_t = 0.f;

    // tile rows: the destinations, then the source of each edge; all of
    // them in one pass unless the tile has more than kSrows - kBm edges
    const int NS = rows + ne;
    for (int s0 = 0; s0 < NS; s0 += kSrows) {
        const int ns = min(kSrows, NS - s0);
        const int nrt = (ns + 15) / 16;  // 16-row matrix-core tiles in use
        gather_a1<SAGE, CW0, LDK1>(a, E, row0, rows, s0, ns, nrt * 16, C0, A1s);
        __syncthreads();
        // the bias as the epilogue uses it, chosen here: hoisted above the
        // gather, the choice would wait for the bias load and with it for all
        // of W^1 (the empty asm keeps it here)
        float bias_t[kTpw1];
#pragma unroll
        for (int t = 0; t < kTpw1; ++t) {
            bias_t[t] = bv1[t];
            asm volatile("" : "+v"(bias_t[t]));
            if (!a.bias1) bias_t[t] = 0.f;
        }
        // layer 2's weights in the last pass: they stream in while the
        // matrix cores work on layer 1 (no other memory traffic then)
        if (s0 + kSrows >= NS && wave < CT2) {  // (uniform per wavefront)
            const int64_t n = static_cast<int64_t>(wave) * 16 + (lane & 15);
            const uint32_t row = static_cast<uint32_t>((n < a.n_out ? n : 0) * K2);
#pragma unroll
            for (int ks = 0; ks < KSM2; ++ks)
                wf2[ks] = load_wfrag<true>(a.wt2, row, static_cast<uint32_t>(K2), ks * 32 + 8 * (lane >> 4));
            bias2_t = (a.bias2 ? a.bias2 : reinterpret_cast<const float *>(a.wt2))[n < a.n_out ? n : 0];
        }
        // layer 1's update of these rows, one 16-row tile at a time, then
        // bias and ReLU to bf16 into the H^1 tile
        if (wave < CT1) {
            for (int rt = 0; rt < nrt; ++rt) {
                f32x4 acc1[kTpw1];
#pragma unroll
                for (int t = 0; t < kTpw1; ++t) acc1[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSM1; ++ks) {
                    const bf16x8 af = *reinterpret_cast<const bf16x8 *>(
                        A1s + (rt * 16 + (lane & 15)) * LDK1 + ks * 32 + 8 * (lane >> 4));
#pragma unroll
                    for (int t = 0; t < kTpw1; ++t)
                        acc1[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf1[t][ks], acc1[t], 0, 0, 0);
                }
#pragma unroll
                for (int t = 0; t < kTpw1; ++t) {
                    const int n = (wave + kWaves * t) * 16 + (lane & 15);
                    if (wave + kWaves * t >= CT1 || n >= f1) continue;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float z = acc1[t][q] + bias_t[t];
                        Hs[(rt * 16 + 4 * (lane >> 4) + q) * kLdh + n] = f32_to_bf16(z > 0.f ? z : 0.f);
                    }
                }
            }
        }
        __syncthreads();
        // the pass's H^1 rows out to HBM, 16 bytes per thread and item
        for (int q = tid; q < ns * C1; q += kThreads) {
            const int sr = q / C1, c = q % C1;
            Chunk<8>::store(a.h1 + s_row(s0 + sr, rows, row0, E) * f1 + c * 8,
                            *reinterpret_cast<const uint4 *>(Hs + sr * kLdh + c * 8));
        }
        // equation 1 over this pass's edges of the item's destination, in
        // edge order
        if (item) {
            if (s0 == 0) self_raw = *reinterpret_cast<const uint4 *>(Hs + ar * kLdh + ac * 8);
            const int lo = max(rb, s0 - rows), hi = min(re, s0 + ns - rows);
            // (four rows read ahead of their sums; rows past hi read the
            // tile's first row and are not summed)
            for (int e0 = lo; e0 < hi; e0 += 4) {
                uint4 raw[4];
                float w[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int e = e0 + u < hi ? e0 + u : lo;
                    raw[u] = *reinterpret_cast<const uint4 *>(Hs + (rows + e - s0) * kLdh + ac * 8);
                    w[u] = SAGE ? 1.f : wi * (STAGED ? Ns[e] : a.src_norm[E[e]]);
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (e0 + u >= hi) break;
                    Chunk<8> x;
                    x.set(raw[u]);
                    if constexpr (MAXA) {
                        // the row's first edge is taken, a later one only
                        // when strictly greater (ties go to the earliest)
                        const int32_t src = E[e0 + u];
#pragma unroll
                        for (int i = 0; i < 8; ++i)
                            if (am[i] < 0 || x.v[i] > acc.v[i]) {
                                acc.v[i] = x.v[i];
                                am[i] = src;
                            }
                    } else if (SAGE) {
#pragma unroll
                        for (int i = 0; i < 8; ++i) acc.v[i] = acc.v[i] + x.v[i];
                    } else {
#pragma unroll
                        for (int i = 0; i < 8; ++i) acc.v[i] = fmaf(w[u], x.v[i], acc.v[i]);
                    }
                }
            }
        }
        __syncthreads();  // the next pass overwrites both tiles
    }

    // the A^2 tile (16 rows; zero past the destinations and past K2) and M^2
    if (item) {
        uint16_t *arow = A2s + ar * LDK2;
        if constexpr (MAXA) {
            // the maximum of bf16 values is one of them: exact in bf16; a
            // row without edges gives 0 and argmax -1
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (am[i] < 0) acc.v[i] = 0.f;
            const uint4 m = acc.bf16();
            Chunk<8>::store(arow + ac * 8, self_raw);
            Chunk<8>::store(arow + f1 + ac * 8, m);
            Chunk<8>::store(a.agg_out + (row0 + ar) * f1 + ac * 8, m);
            int4 *ap = reinterpret_cast<int4 *>(a.argmax + (row0 + ar) * f1 + ac * 8);
            ap[0] = make_int4(am[0], am[1], am[2], am[3]);
            ap[1] = make_int4(am[4], am[5], am[6], am[7]);
        } else if (SAGE) {
            if (re > rb) {
                const float d = static_cast<float>(re - rb);
#pragma unroll
                for (int i = 0; i < 8; ++i) acc.v[i] /= d;
            }
            const uint4 m = acc.bf16();
            Chunk<8>::store(arow + ac * 8, self_raw);
            Chunk<8>::store(arow + f1 + ac * 8, m);
            Chunk<8>::store(a.agg_out + (row0 + ar) * f1 + ac * 8, m);
        } else {
            const float ws = wi * wi;
            Chunk<8> x;
            x.set(self_raw);
#pragma unroll
            for (int i = 0; i < 8; ++i) acc.v[i] = fmaf(ws, x.v[i], acc.v[i]);
            const uint4 m = acc.bf16();
            Chunk<8>::store(arow + ac * 8, m);
            Chunk<8>::store(a.agg_out + (row0 + ar) * f1 + ac * 8, m);
        }
    }
    {
        const int kp2 = 32 * KSM2, zr = (16 - rows) * (kp2 / 4), zc = rows * kq2, kd = kq2 > 0 ? kq2 : 1;
        for (int q = tid; q < zr + zc; q += kThreads) {
            const int r = q < zr ? rows + q / (kp2 / 4) : (q - zr) / kd;
            const int k = q < zr ? (q % (kp2 / 4)) * 4 : static_cast<int>(K2) + ((q - zr) % kd) * 4;
            *reinterpret_cast<uint2 *>(A2s + r * LDK2 + k) = make_uint2(0u, 0u);
        }
    }
    __syncthreads();
    // layer 2's update (wavefronts 0 .. CT2 - 1)
    f32x4 acc2 = f32x4{0.f, 0.f, 0.f, 0.f};
    if (wave < CT2) {
#pragma unroll
        for (int ks = 0; ks < KSM2; ++ks) {
            const bf16x8 af =
                *reinterpret_cast<const bf16x8 *>(A2s + (lane & 15) * LDK2 + ks * 32 + 8 * (lane >> 4));
            acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, wf2[ks], acc2, 0, 0, 0);
        }
        // W^2 into the H^1 tile's space (free since the aggregation) for
        // the input gradient below: [16 CT2][LDW2] (two_shape keeps it
        // inside the tile; the padded row stride spreads a fragment's 16
        // rows over all LDS banks)
        if (a.d_a) {
#pragma unroll
            for (int ks = 0; ks < KSM2; ++ks)
                *reinterpret_cast<bf16x8 *>(Hs + (wave * 16 + (lane & 15)) * LDW2 + ks * 32 + 8 * (lane >> 4)) = wf2[ks];
        }
    }
    asm volatile("" : "+v"(bias2_t));
    if (!a.bias2) bias2_t = 0.f;
    __syncthreads();  // every wavefront is done reading the A^2 tile
    if (wave < CT2) {
        const int n = wave * 16 + (lane & 15);
#pragma unroll
        for (int q = 0; q < 4; ++q) Ls[(4 * (lane >> 4) + q) * kLogitLd + n] = acc2[q] + bias2_t;
    }
    __syncthreads();
    // the staged W^2 values dA^2 needs, read now (the barrier above made
    // them visible), during the softmax
    constexpr int KP2 = 32 * KSM2, KTW = KP2 / 16 / kWaves;
    uint32_t w[KTW][2][8];
#pragma unroll
    for (int i = 0; i < KTW; ++i) {
        if (!a.d_a) break;  // (uniform)
        const int k = (wave + kWaves * i) * 16 + (lane & 15);  // < KP2
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int n = st * 32 + 8 * (lane >> 4) + t;
                const bool in = n < a.n_out;
                const uint32_t v = Hs[(in ? n : 0) * LDW2 + k];
                w[i][st][t] = in ? v : 0u;
            }
    }
    softmax_ce_row<TPR>(Ls + er * kLogitLd, tid % TPR, live, row0 + er, y, a.n_out, a.b, a.logits, a.g, a.row_loss,
                        Gs + er * 64, 64);
    if (a.d_a) {
        // dA^2 = G (W^2)^T on the matrix cores with the operands and steps of
        // the update's input-gradient GEMM: bf16(G) rows against the bf16
        // W^2 rows (the shadow holds exactly those values), classes in two
        // zero-padded steps of 32 in order, so the result is bit for bit that
        // GEMM's.  G comes from LDS (the rows of this tile; matrix rows 4 ..
        // 15 are zero), W^2 from the copy staged above.  Wavefront w computes
        // output column tiles w, w + 8, ...  Every operand read is
        // unconditional, from an in-bounds address, and masked afterwards (a
        // read under a condition becomes a branch with its own wait), and all
        // of a wavefront's reads are issued before its first product.
        __syncthreads();  // the gradient rows are staged
        bf16x8 ga[2];
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            const int r = lane & 15, n0 = st * 32 + 8 * (lane >> 4);
            const float4 lo = *reinterpret_cast<const float4 *>(Gs + (r & 7) * 64 + n0);
            const float4 hi = *reinterpret_cast<const float4 *>(Gs + (r & 7) * 64 + n0 + 4);
            const uint32_t keep = r < kBm ? 0xffffffffu : 0u;
            // (the values are bf16 already: the high halves are exact)
            const uint32_t p0 = (__float_as_uint(lo.x) >> 16) | (__float_as_uint(lo.y) & 0xffff0000u);
            const uint32_t p1 = (__float_as_uint(lo.z) >> 16) | (__float_as_uint(lo.w) & 0xffff0000u);
            const uint32_t p2 = (__float_as_uint(hi.x) >> 16) | (__float_as_uint(hi.y) & 0xffff0000u);
            const uint32_t p3 = (__float_as_uint(hi.z) >> 16) | (__float_as_uint(hi.w) & 0xffff0000u);
            ga[st] = __builtin_bit_cast(bf16x8, make_uint4(p0 & keep, p1 & keep, p2 & keep, p3 & keep));
        }
#pragma unroll
        for (int i = 0; i < KTW; ++i) {
            const int kt = wave + kWaves * i, k = kt * 16 + (lane & 15);
            f32x4 d = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                const uint32_t *v = w[i][st];
                const uint4 p = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16),
                                           v[6] | (v[7] << 16));
                d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ga[st], __builtin_bit_cast(bf16x8, p), d, 0, 0, 0);
            }
            // lanes 0 .. 15 hold rows 0 .. 3 of column k
            if (kt * 16 < K2 && (lane >> 4) == 0) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (q < rows) a.d_a[(row0 + q) * K2 + k] = d[q];
            }
        }
    }
    };
    if (staged) rest(std::true_type{});
    else rest(std::false_type{});
}

struct TwoShape {
    int ksm1, cw0;
    int32_t es_cap;
    bool ok;
};

TwoShape two_shape(int kind, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_dst, int32_t fanout) {
    TwoShape sh{};
    const bool sage = kind != GNN_AGG_GCN_SYM;
    const int64_t K1 = sage ? 2 * f0 : f0;
    if (f0 <= 0 || f0 % 4 != 0 || K1 > 256) return sh;
    if (f1 <= 0 || f1 % 8 != 0 || f1 > 16 * kWaves * kTpw1) return sh;
    if (n_out <= 0 || n_out > 64 || cap_dst <= 0 || cap_dst > 2048) return sh;
    // W^2 staged in the H^1 tile's LDS for the input gradient
    if (ceil_div(n_out, 16) * 16 * ((sage ? 512 : 256) + 8) > static_cast<int64_t>(kSrows) * kLdh) return sh;
    sh.ksm1 = K1 <= 128 ? 4 : K1 <= 224 ? 7 : 8;  // (zero-padded steps add exact zeros)
    sh.cw0 = f0 % 8 == 0 ? 8 : 4;
    sh.es_cap = static_cast<int32_t>(std::min<int64_t>(static_cast<int64_t>(kBm) * std::max(fanout, 1), kEsMax));
    sh.ok = true;
    return sh;
}

// One workgroup per tile (at most 512).
template <int KIND>
gnn_status two_go(const TwoShape &sh, const TwoArgs &a, unsigned grid, hipStream_t s) {
    auto go = [&](auto ksm) {
        constexpr int KSM1 = decltype(ksm)::value;
        if (sh.cw0 == 8) two_layer_kernel<KIND, KSM1, 8><<<grid, kThreads, 0, s>>>(a);
        else two_layer_kernel<KIND, KSM1, 4><<<grid, kThreads, 0, s>>>(a);
    };
    if (sh.ksm1 == 4) go(std::integral_constant<int, 4>{});
    else if (sh.ksm1 == 7) go(std::integral_constant<int, 7>{});
    else go(std::integral_constant<int, 8>{});
    return launch_status("two_layer_fwd");
}

}  // namespace

bool two_layer_ok(int kind, int precision, int64_t f0, int64_t f1, int64_t n_out, int64_t cap_dst, int32_t fanout,
                  const void *x_self, const void *m1, const uint16_t *wt1, const uint16_t *wt2, const void *h1,
                  const void *agg_out, const int32_t *argmax) {
    if (precision != GNN_BF16 || !wt1 || !wt2 || !m1 || !h1 || !agg_out) return false;
    if (kind == GNN_AGG_SAGE_MAX && (!argmax || !aligned(argmax, 16))) return false;
    const TwoShape sh = two_shape(kind, f0, f1, n_out, cap_dst, fanout);
    if (!sh.ok) return false;
    const size_t ra = sh.cw0 == 8 ? 16 : 8;
    const bool sage = kind != GNN_AGG_GCN_SYM;
    if (!aligned(m1, ra) || (sage && (!x_self || !aligned(x_self, ra)))) return false;
    if ((sage || sh.cw0 == 8) ? !aligned(wt1, 16) : !aligned(wt1, 8)) return false;
    return aligned(wt2, 16) && aligned(h1, 2) && aligned(agg_out, 16);
}

gnn_status launch_two_layer(const gnn_block *last, int kind, int32_t fanout, const void *x_self, const void *m1,
                            int64_t f0, const uint16_t *wt1, const float *bias1, int64_t f1, void *h1,
                            const uint16_t *wt2, const float *bias2, int64_t n_out, void *agg_out, float *logits,
                            const int64_t *labels, float *g, float *row_loss, int64_t batch, float *d_a,
                            int32_t *argmax, hipStream_t s) {
    const TwoShape sh = two_shape(kind, f0, f1, n_out, last->cap_dst, fanout);
    GNN_CHECK(sh.ok, GNN_EUNSUPPORTED, "two_layer_fwd: shape not supported");
    TwoArgs a{};
    a.counts = last->counts ? last->counts : reinterpret_cast<const int64_t *>(wt1);
    a.cnt_keep = last->counts ? -1 : 0;
    a.cnt_add = last->counts ? 0 : last->cap_dst;
    a.rowptr = last->rowptr;
    a.col = last->col;
    a.src_norm = last->src_norm;
    a.cap_dst = last->cap_dst;
    a.es_cap = sh.es_cap;
    a.x_self = static_cast<const uint16_t *>(kind != GNN_AGG_GCN_SYM ? x_self : m1);
    a.m1 = static_cast<const uint16_t *>(m1);
    a.f0 = f0;
    a.wt1 = wt1;
    a.bias1 = bias1;
    a.f1 = f1;
    a.h1 = static_cast<uint16_t *>(h1);
    a.wt2 = wt2;
    a.bias2 = bias2;
    a.n_out = n_out;
    a.agg_out = static_cast<uint16_t *>(agg_out);
    a.argmax = argmax;
    a.logits = logits;
    a.labels = labels;
    a.targets = last->src_ids;
    a.g = g;
    a.row_loss = row_loss;
    a.b = batch;
    a.d_a = d_a;
    const unsigned grid = static_cast<unsigned>(ceil_div(last->cap_dst, kBm));
    if (kind == GNN_AGG_SAGE_MAX) return two_go<GNN_AGG_SAGE_MAX>(sh, a, grid, s);
    return kind == GNN_AGG_SAGE_MEAN ? two_go<GNN_AGG_SAGE_MEAN>(sh, a, grid, s)
                                     : two_go<GNN_AGG_GCN_SYM>(sh, a, grid, s);
}

}  // namespace gnn
