// The backward pass of a two-layer model below the loss in one launch: layer
// 2's weight-gradient partials and layer 1's, with layer 2's aggregation
// backward folded into the latter.
//
// Below layer 2 the backward pass needs G^1 only for layer 1's update
// gradients: G^1 = ReLU'(H^1) (P^T dA^2_nbr + self), dW^1 = (A^1)^T G^1 and
// db^1 = colsum(G^1) (Section II-B, backward; Section V: layer 1's backward
// is the update alone).  The unfused path writes G^1 (fp32) with the
// aggregation backward and reads it back in the dW GEMM, one launch later.
// Here each workgroup pulls the rows of G^1 it multiplies straight through
// the block transpose.
//
// The work is bound by memory: by chains of dependent round trips (about a
// microsecond each here) and by the bytes each compute unit has in flight.
// So a workgroup owns a small piece (one row split of at most 128 rows, as
// the dW GEMM's split plan gives it, one 64-column tile of G^1 and all of K,
// up to 256: one 64-row slice of dW per wavefront), each G^1 value is made
// once, and the loads take three round trips:
//   1. everything that does not depend on the transpose, at once: the
//      split's transpose row pointers, its A^1 chunks (registers), its H^1
//      mask and dA^2 self rows, and layer 2's dW tile (below);
//   2. the split's edges' destination rows (cscrow), 256 edges per pass;
//   3. their dA^2 neighbour rows (the tile's 64 columns), loaded straight
//      into LDS (16 bytes per lane), and their weights.
// Then each thread sums its rows' edges from LDS in edge order, applies the
// self term and the mask, and the finished G^1 values go to LDS as bf16 for
// the matrix cores (with their fp32 column sums for db).
//
// Workgroup b also computes tile b of layer 2's dW partials (a DweightJob
// tile): its loads go out with step 1 and its matrix-core work runs while
// layer 1's partial stores drain, so layer 2 costs no launch and no round
// trip of its own.
//
// Every arithmetic step is the unfused path's, in its order: the edge sum of
// the aggregation backward (one wavefront row walk, edges in transpose
// order, fma), the self term and the ReLU mask, then the dW GEMM's bf16
// staging, its column sums, its MFMA sequence and its split partials.  The
// partials are therefore bitwise those of aggregate backward + dW GEMM
// whenever the aggregation backward walks a row's edges in one sequence
// (G^1 wider than 128 columns); narrower layers take the unfused path.
#pragma once

#include "aggregate_dev.h"
#include "gemm_bwd_dev.h"

namespace gnn {
namespace gbwd {

constexpr int kPullChunks = 2;                // 64-row chunks per group
constexpr int kPullRows = 64 * kPullChunks;  // rows of G^1 per group
constexpr int kPullEdges = 256;               // edges staged in LDS per pass
constexpr int kPullMaxK = 256;                // K rows of dW per workgroup (4 wavefronts x 64)

template <int KIND, bool VA, class L2>
struct DweightPullJob {
    const uint16_t *a_self, *a_nbr;  // A^1 = [a_self || a_nbr] (bf16), k_each wide each
    int64_t k_each;
    const int64_t *m_dev;            // rows of A^1 (= sources of block b)
    int64_t cap_m;
    gnn_block b;                     // layer 2's block with its transpose
    const float *d_a;                // dA^2 (fp32): b's destination rows, (SAGE ? 2 : 1) * f wide
    const uint16_t *h;               // H^1 (bf16, f wide): the ReLU mask
    int64_t f;                       // width of G^1 (layer 1's output)
    int want_db;
    float *part;                     // split partials, laid out as the dW GEMM's
    SplitMap map;                    // tiles: the 64-column tiles of G^1
    L2 l2;                           // layer 2's dW tiles
    int64_t l2_blocks;
    const int32_t *argmax;           // max aggregator: layer 2's argmax table (b's destinations x f), else null

    __device__ void run(int64_t blk, int64_t) const {
        using CV = Cfg<true>;
        constexpr int BK = CV::BK, NC = kPullChunks;
        constexpr bool SAGE = KIND != GNN_AGG_GCN_SYM;  // dA^2 rows [self || aggregation part]
        // the max aggregator stages each edge's argmax row beside its dA^2
        // row, in an array of its own (the job runs one workgroup per CU at
        // its register use, so the LDS costs no occupancy)
        constexpr bool MAXA = KIND == GNN_AGG_SAGE_MAX;
        constexpr int PE = kPullEdges;
        using SA = SrcCols<true, kPullMaxK, uint16_t, VA, NC>;
        // vst: the staged edge rows, then the matrix-core operands, the
        // epilogue staging and layer 2's tile
        __shared__ __attribute__((aligned(16))) float vst[kPullEdges * 64];
        __shared__ float wst[kPullEdges];
        __shared__ int32_t dstl[kPullEdges];
        __shared__ int32_t cpl[kPullRows + 1];
        __shared__ float cs[16][64];
        __shared__ __attribute__((aligned(16))) int32_t ast[MAXA ? kPullEdges * 64 : 4];
        static_assert(L2::kLdsBytes + sizeof(typename L2::ColSums) <= sizeof(vst), "layer 2's tile needs more LDS");
        static_assert(sizeof(float) * 4 * 64 * 64 <= sizeof(vst), "epilogue staging needs more LDS");
        static_assert((kPullMaxK + 64) * BK * 2 <= sizeof(vst), "operand tiles need more LDS");
        uint16_t *Ps = reinterpret_cast<uint16_t *>(vst), *Qs = Ps + kPullMaxK * BK;
        auto finish2 = [&](typename L2::Tile &t2) {
            l2.finish(t2, reinterpret_cast<char *>(vst),
                      *reinterpret_cast<typename L2::ColSums *>(vst + L2::kLdsBytes / 4));
        };

        const int tid = threadIdx.x, lane = tid & 63;
        const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int lr = lane & 15, lg = lane >> 4;
        // layer 2's tile: its loads now, the rest at the end
        typename L2::Tile t2;
        bool has2 = blk < l2_blocks && l2.begin(blk, t2);

        int split;
        int64_t tile;
        map.of(blk, &split, &tile);
        const bool live = split < map.nsplit;
        const int64_t K = a_nbr ? 2 * k_each : k_each;
        const int64_t col0 = tile * 64;
        const int64_t M = m_dev ? min(*m_dev, cap_m) : cap_m;
        int64_t r_beg = 0, r_end = 0;
        if (live) split_range<BK>(M, map.nsplit, split, &r_beg, &r_end);
        const int64_t ka = SAGE ? 2 * f : f, nbr_off = SAGE ? f : 0;
        // this thread's G^1 elements in the GEMM's staging layout: rows
        // rr*4 .. rr*4+3 of every 64-row chunk, columns tt .. tt+3
        const int rr = tid / 16, tt = (tid % 16) * 4;
        const bool col_ok = col0 + tt < f;
        const int64_t ccol = col_ok ? col0 + tt : 0;
        const bool wave_k = static_cast<int64_t>(wave) * 64 < K;

        SA sp{a_self, a_nbr, k_each, k_each, K, r_end, 0, {}};
        f32x4 acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        float4 colsum = make_float4(0.f, 0.f, 0.f, 0.f);
        const int64_t n_dst = b.counts[0];

        for (int64_t g0 = r_beg; g0 < r_end; g0 += kPullRows) {
            const int64_t g1 = min(r_end, g0 + kPullRows);
            const int nr = static_cast<int>(g1 - g0);
            // step 1: the transpose's row pointers first, then everything
            // else of the group (edge offsets are clamped to the block's
            // capacity, so a damaged transpose cannot send reads out of it)
            const int64_t eb_raw = b.cscptr[g1], ea_raw = b.cscptr[g0];
            const int64_t cp_raw = b.cscptr[g0 + min(tid, nr)];
#pragma unroll
            for (int c = 0; c < NC; ++c) sp.fetch(c, g0 + c * BK);
            uint2 hb[NC][4];
            float4 sf[NC][4];
            float wj[NC][4];
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int x = c * 64 + rr * 4 + i;
                    const int64_t r = g0 + (x < nr ? x : 0);
                    hb[c][i] = *reinterpret_cast<const uint2 *>(h + r * f + ccol);
                    sf[c][i] = load4(d_a, (r < n_dst ? r : 0) * ka + ccol);
                    if constexpr (!SAGE) wj[c][i] = b.src_norm[r];
                }
            const int64_t Eb = min(max(eb_raw, int64_t(0)), b.cap_nnz);
            const int64_t Ea = min(max(ea_raw, int64_t(0)), Eb);
            if (tid <= nr) cpl[tid] = static_cast<int32_t>(min(max(cp_raw, Ea), Eb) - Ea);
            float4 gv[NC][4];
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) gv[c][i] = make_float4(0.f, 0.f, 0.f, 0.f);
            for (int64_t pb = Ea;; pb += PE) {
                const int64_t pe = min(Eb, pb + PE);
                const int n = static_cast<int>(pe - pb);
                // step 2: the edges' destination rows (and, for the max
                // aggregator, whether the previous edge names the same row)
                int32_t dst = tid < n ? b.cscrow[pb + tid] : 0;
                int32_t prev = -1;
                if (MAXA && tid < n && pb + tid > Ea) prev = b.cscrow[pb + tid - 1];
                dst = min(max(dst, 0), static_cast<int32_t>(b.cap_dst - 1));
                dstl[tid] = dst;
                __syncthreads();
                // step 3: the neighbour rows into LDS, 4 edges (16 lanes x 16
                // bytes each) per wavefront instruction, and the weights
                {
                    const int w0 = wave * (PE / 4);
                    const int nw = min(max(n - w0, 0), PE / 4);
                    const int64_t cq = col0 + (lane & 15) * 4;
                    const int64_t cl = cq < f ? cq : 0;
                    for (int i = 0; i < nw; i += 4) {
                        const int slot = w0 + i + (lane >> 4);
                        if (slot < n) {
                            const float *src = d_a + static_cast<int64_t>(dstl[slot]) * ka + nbr_off + cl;
                            __builtin_amdgcn_global_load_lds(src, vst + (w0 + i) * 64, 16, 0, 0);
                            if constexpr (MAXA) {
                                const int32_t *asrc = argmax + static_cast<int64_t>(dstl[slot]) * f + cl;
                                __builtin_amdgcn_global_load_lds(asrc, ast + (w0 + i) * 64, 16, 0, 0);
                            }
                        }
                    }
                }
                if (tid < n) {
                    float w;
                    if constexpr (MAXA) {
                        // 1: the first of a run of entries naming one row
                        // (a destination that sampled this source several
                        // times passes its gradient once); the column's
                        // first entry counts whatever precedes it
                        w = prev == b.cscrow[pb + tid] ? 0.f : 1.f;
                    } else if constexpr (SAGE) {
                        const int64_t d0 = b.rowptr[dst], d1 = b.rowptr[dst + 1];
                        w = 1.f / static_cast<float>(d1 - d0);
                    } else {
                        w = b.src_norm[dst];
                    }
                    wst[tid] = w;
                }
                __builtin_amdgcn_s_waitcnt(0);
                __syncthreads();
                const bool last = pe >= Eb;
                const int32_t lo_p = static_cast<int32_t>(pb - Ea), hi_p = static_cast<int32_t>(pe - Ea);
#pragma unroll
                for (int c = 0; c < NC; ++c)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int x = c * 64 + rr * 4 + i;
                        if (x >= nr) continue;
                        const int32_t lo = max(cpl[x], lo_p), hi = min(cpl[x + 1], hi_p);
                        if constexpr (MAXA) {
                            // the maximum passes its gradient to the source
                            // that won it: add where argmax names this row
                            const int32_t jj = static_cast<int32_t>(g0 + x);
                            for (int32_t e = lo; e < hi; ++e) {
                                if (e != cpl[x] && wst[e - lo_p] == 0.f) continue;
                                const int4 am = *reinterpret_cast<const int4 *>(ast + (e - lo_p) * 64 + tt);
                                const float4 v = *reinterpret_cast<const float4 *>(vst + (e - lo_p) * 64 + tt);
                                gv[c][i].x += am.x == jj ? v.x : 0.f;
                                gv[c][i].y += am.y == jj ? v.y : 0.f;
                                gv[c][i].z += am.z == jj ? v.z : 0.f;
                                gv[c][i].w += am.w == jj ? v.w : 0.f;
                            }
                            continue;
                        }
                        for (int32_t e = lo; e < hi; ++e) {
                            float we = wst[e - lo_p];
                            if constexpr (!SAGE) we = we * wj[c][i];
                            agg::fma4(gv[c][i], we, *reinterpret_cast<const float4 *>(vst + (e - lo_p) * 64 + tt));
                        }
                    }
                __syncthreads();
                if (last) break;
            }
            // self term, ReLU mask; rows past the split and columns past f
            // are zero (as the GEMM's tail zeroing leaves them)
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int x = c * 64 + rr * 4 + i;
                    float4 g = gv[c][i];
                    if (g0 + x < n_dst) {
                        float ws = 1.f;
                        if constexpr (!SAGE) ws = wj[c][i] * wj[c][i];
                        agg::fma4(g, ws, sf[c][i]);
                    }
                    const uint2 m = hb[c][i];
                    if (!(__uint_as_float(m.x << 16) > 0.f)) g.x = 0.f;
                    if (!(__uint_as_float(m.x & 0xffff0000u) > 0.f)) g.y = 0.f;
                    if (!(__uint_as_float(m.y << 16) > 0.f)) g.z = 0.f;
                    if (!(__uint_as_float(m.y & 0xffff0000u) > 0.f)) g.w = 0.f;
                    if (x >= nr || !col_ok) g = make_float4(0.f, 0.f, 0.f, 0.f);
                    gv[c][i] = g;
                    if (want_db && x < nr) {
                        colsum.x += g.x;
                        colsum.y += g.y;
                        colsum.z += g.z;
                        colsum.w += g.w;
                    }
                }
            // the group's chunks through the matrix cores
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int64_t r0 = g0 + c * BK;
                if (r0 >= g1) break;
                // the tail chunk: A's reduction rows past the split are zero
                // (the clamped loads repeat the last row)
#pragma unroll
                for (int i = 0; i < SA::NCH; ++i)
                    if (r0 + sp.my_r(i) >= r_end) sp.reg[c][i] = make_uint2(0u, 0u);
                sp.commit(c, Ps);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t b0 = Raw<float>::bits(gv[c][0], e), b1 = Raw<float>::bits(gv[c][1], e);
                    const uint32_t b2 = Raw<float>::bits(gv[c][2], e), b3 = Raw<float>::bits(gv[c][3], e);
                    *reinterpret_cast<uint2 *>(Qs + CV::idx(tt + e, rr * 4)) = make_uint2(b0 | (b1 << 16), b2 | (b3 << 16));
                }
                __syncthreads();
                if (wave_k) {
#pragma unroll
                    for (int kk = 0; kk < BK; kk += 32) {
                        bf16x8 a[4], bq[4];
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            a[i] = *reinterpret_cast<const bf16x8 *>(Ps + CV::idx(wave * 64 + i * 16 + lr, kk + lg * 8));
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            bq[j] = *reinterpret_cast<const bf16x8 *>(Qs + CV::idx(j * 16 + lr, kk + lg * 8));
#pragma unroll
                        for (int i = 0; i < 4; ++i)
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], bq[j], acc[i][j], 0, 0, 0);
                    }
                }
                __syncthreads();
            }
        }
        if (!live) {  // an idle split: layer 2's tile only
            if (has2) finish2(t2);
            return;
        }
        // partials: dW rows of this wavefront's K slice, then db
        const int64_t ldp = part_ld(f);
        float *pp = part + static_cast<int64_t>(split) * (K + 1) * ldp;
        if (want_db) {
            cs[rr][tt + 0] = colsum.x;
            cs[rr][tt + 1] = colsum.y;
            cs[rr][tt + 2] = colsum.z;
            cs[rr][tt + 3] = colsum.w;
        }
        float *st = vst + wave * 64 * 64;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) st[(i * 16 + lg * 4 + q) * 64 + j * 16 + lr] = acc[i][j][q];
        __syncthreads();
        if (want_db && tid < 64 && col0 + tid < ldp) {
            float sum = 0.f;
            for (int k = 0; k < 16; ++k) sum += cs[k][tid];
            pp[K * ldp + col0 + tid] = sum;
        }
        const int c4 = (lane & 15) * 4;
#pragma unroll
        for (int it = 0; it < 16; ++it) {
            const int row = it * 4 + (lane >> 4);
            const int64_t k = static_cast<int64_t>(wave) * 64 + row;
            if (k < K && col0 + c4 < ldp)
                *reinterpret_cast<float4 *>(pp + k * ldp + col0 + c4) = *reinterpret_cast<const float4 *>(st + row * 64 + c4);
        }
        if (has2) {
            __syncthreads();  // the staging area is reused
            finish2(t2);
        }
    }
};

}  // namespace gbwd
}  // namespace gnn

namespace gnn {

// Host side (bwd_two.hip): the backward of a two-layer model below the loss
// as dW partials for both layers (layer 2's aggregation backward folded into
// layer 1's) and their split reductions.
struct TwoBwdPlan {
    gbwd::Args a1, a2;  // the two layers' update backward (no dA)
    gbwd::Plan p1, p2;
    gnn_block b2;       // layer 2's block
    const float *d_a2;
    const uint16_t *h1;
    gbwd::SplitMap pm;  // the folded job's (split, column tile) map
    const int32_t *arg2;  // max aggregator: layer 2's argmax table, else null
    unsigned grid;      // its workgroups
    bool gemm_ok;       // both dW GEMMs take the bf16 64 x 64 variants with vector A loads
    bool pull;          // and the folded job applies
};

// kind: the aggregator; b2: layer 2's block (with its transpose); layer 1's A
// rows [x_self || m1] (GraphSAGE) or m1 (GCN), bf16, f0 wide, with their row
// count m1_rows (device) and capacity cap_m1; H^1 (bf16, f1 wide); M^2 =
// agg2 (bf16, f1 wide) and, for the max aggregator, its argmax table arg2
// (int32, 16-byte aligned); dA^2 and G^2 (fp32); per layer the weight
// gradient outputs, the partial region (sized by gbwd::dw_part_bytes of the
// plan) and the SGD targets (null: no update).
TwoBwdPlan plan_two_bwd(int kind, const gnn_block &b2, const void *x_self, const void *m1, int64_t f0,
                        const int64_t *m1_rows, int64_t cap_m1, const uint16_t *h1, int64_t f1, const void *agg2,
                        const int32_t *arg2,
                        const float *d_a2, const float *g2, int64_t n_out, const float *w1, float *dw1, float *db1,
                        float *part1, float *w1_upd, float *b1_upd, uint16_t *wt1_upd, const float *w2, float *dw2,
                        float *db2, float *part2, float *w2_upd, float *b2_upd, uint16_t *wt2_upd, float lr);
// The partials of both layers in one launch (requires t.pull).
gnn_status launch_two_bwd_partials(const TwoBwdPlan &t, int kind, hipStream_t s);

}  // namespace gnn
