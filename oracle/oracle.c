/*
 * CPU oracle for sampled mini-batch GNN training (GCN and GraphSAGE with the
 * mean aggregator; the max aggregator's forward and backward too).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The GPU product path never
 * links, imports or calls it, and this file shares no code, header, table or
 * constant with that path.
 *
 * Every routine is the plain definition of one step of the training
 * iteration described in the paper (Section II-A, equations 1-2 and the GCN
 * and GraphSAGE layer definitions; Section II-B for the mini-batch workflow;
 * Section V, equation T_Trainer, for which backward steps exist).  Floating
 * point values are widened to double, combined with sequential sums in
 * double precision, and narrowed only where the storage precision of the
 * training step says a value is stored.  OpenMP (when compiled in) splits
 * loops over independent output rows only, so results do not depend on the
 * thread count.
 *
 * Storage dtype codes: 0 = fp32, 1 = bf16 (raw uint16 bits), 2 = fp16 (raw
 * uint16 bits), 3 = fp64 (oracle-only, used for finite-difference checks).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F16 = 2, ORC_F64 = 3 };
enum { ORC_SAGE_MEAN = 0, ORC_GCN_SYM = 1 };

/* ------------------------------------------------------------------------ */
/* Scalar conversions written from the IEEE 754 binary16 / bfloat16 formats. */
/* ------------------------------------------------------------------------ */

static uint32_t f32_bits(float x) { uint32_t u; memcpy(&u, &x, 4); return u; }
static float bits_f32(uint32_t u) { float x; memcpy(&x, &u, 4); return x; }

/* bfloat16 is the upper half of a binary32; narrowing rounds to nearest,
 * ties to even.  NaNs stay NaN (quiet bit forced). */
uint16_t orc_f32_to_bf16(float x)
{
    uint32_t u = f32_bits(x);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

float orc_bf16_to_f32(uint16_t h) { return bits_f32((uint32_t)h << 16); }

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
float orc_f16_to_f32(uint16_t h)
{
    uint32_t sign = (uint32_t)(h >> 15) & 1u;
    int32_t exp = (h >> 10) & 0x1f;
    uint32_t frac = h & 0x3ffu;
    double mag;
    if (exp == 0x1f) {
        uint32_t u = (sign << 31) | 0x7f800000u | (frac << 13);
        return bits_f32(u);
    }
    if (exp == 0)
        mag = ldexp((double)frac, -24);           /* subnormal: frac * 2^-24 */
    else
        mag = ldexp((double)(1024 + frac), exp - 25); /* (1 + frac/1024) * 2^(exp-15) */
    return (float)(sign ? -mag : mag);
}

static double load_elem(const void *p, int dt, int64_t i)
{
    switch (dt) {
    case ORC_F32: return (double)((const float *)p)[i];
    case ORC_BF16: return (double)orc_bf16_to_f32(((const uint16_t *)p)[i]);
    case ORC_F16: return (double)orc_f16_to_f32(((const uint16_t *)p)[i]);
    default: return ((const double *)p)[i];
    }
}

/* Narrow a double to the storage type: to fp32 by round-to-nearest, then to
 * bf16 by round-to-nearest-even (the point where the GPU rounds its fp32
 * accumulator). */
static void store_elem(void *p, int dt, int64_t i, double v)
{
    switch (dt) {
    case ORC_F32: ((float *)p)[i] = (float)v; break;
    case ORC_BF16: ((uint16_t *)p)[i] = orc_f32_to_bf16((float)v); break;
    case ORC_F64: ((double *)p)[i] = v; break;
    default: break;
    }
}

/* Value a GEMM operand takes: with bf16 GEMM arithmetic every operand is
 * rounded to bf16 on input; otherwise the stored value is used. */
static double gemm_operand(double stored, int gemm_dt)
{
    if (gemm_dt == ORC_BF16)
        return (double)orc_bf16_to_f32(orc_f32_to_bf16((float)stored));
    return stored;
}

void orc_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Neighbour sampler (Section II-B; GraphSAGE neighbour sampler of VI-A).     */
/* ------------------------------------------------------------------------ */

/* SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014). */
uint64_t orc_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* Random key of draw t for vertex v at hop `hop` of training step `step`. */
uint64_t orc_sample_key(uint64_t seed, uint64_t step, uint64_t hop, uint64_t v, uint64_t t)
{
    uint64_t k = orc_mix64(seed);
    k = orc_mix64(k ^ step);
    k = orc_mix64(k ^ hop);
    k = orc_mix64(k ^ v);
    return orc_mix64(k ^ t);
}

/* Uniform integer in [0, bound) from the upper 32 bits of a key (Lemire's
 * multiply-shift, without the rejection step).  bound <= 2^32. */
uint64_t orc_bounded(uint64_t key, uint64_t bound)
{
    return ((key >> 32) * bound) >> 32;
}

static int cmp_i64(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

/* Positions (0-based offsets into v's adjacency row) sampled without
 * replacement: all d of them when d <= k, otherwise k drawn by Floyd's
 * algorithm (Bentley and Floyd, CACM 1987), then sorted ascending. */
int64_t orc_sample_positions(int64_t d, int32_t k, uint64_t seed, uint64_t step, int32_t hop,
                             int64_t v, int64_t *pos)
{
    if (d <= (int64_t)k) {
        for (int64_t p = 0; p < d; ++p) pos[p] = p;
        return d;
    }
    int64_t cnt = 0;
    for (int32_t t = 0; t < k; ++t) {
        int64_t j = d - k + t;
        int64_t x = (int64_t)orc_bounded(orc_sample_key(seed, step, (uint64_t)hop, (uint64_t)v, (uint64_t)t),
                                         (uint64_t)(j + 1));
        int found = 0;
        for (int64_t s = 0; s < cnt; ++s)
            if (pos[s] == x) { found = 1; break; }
        pos[cnt++] = found ? j : x;
    }
    qsort(pos, (size_t)cnt, sizeof(int64_t), cmp_i64);
    return cnt;
}

/* GCN symmetric normalisation factor per vertex: D(v) is the input-graph
 * degree plus the self loop, nrm(v) = fp32(1 / sqrt(D(v))). */
void orc_gcn_norm(int64_t n, const int64_t *rowptr, float *nrm)
{
    for (int64_t v = 0; v < n; ++v) {
        double D = (double)(rowptr[v + 1] - rowptr[v]) + 1.0;
        nrm[v] = (float)(1.0 / sqrt(D));
    }
}

typedef struct { int64_t id; int64_t pos; } id_pos;

static int cmp_id_pos(const void *a, const void *b)
{
    int64_t x = ((const id_pos *)a)->id, y = ((const id_pos *)b)->id;
    return (x > y) - (x < y);
}

static int64_t find_id(const id_pos *arr, int64_t n, int64_t id)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (arr[mid].id < id) lo = mid + 1; else hi = mid;
    }
    return (lo < n && arr[lo].id == id) ? arr[lo].pos : -1;
}

/* One hop of the mini-batch sampler: the bipartite block whose destination
 * rows are `dst` and whose sources are dst followed by every newly reached
 * vertex in ascending id order.  Returns 0, or -2 if a capacity is too
 * small, or -1 for a vertex id out of range.
 * Outputs: src_ids[n_src]; block CSR brow[n_dst+1] / bcol[nnz] with local
 * source indices in sampled order; its stable transpose cscptr[n_src+1] /
 * cscrow[nnz] (rows ascending within each source). */
int orc_build_block(int64_t n, const int64_t *rowptr, const int64_t *col,
                    const int64_t *dst, int64_t n_dst, int32_t fanout,
                    uint64_t seed, uint64_t step, int32_t hop,
                    int64_t cap_src, int64_t cap_nnz,
                    int64_t *src_ids, int64_t *n_src_out, int64_t *brow, int32_t *bcol,
                    int64_t *nnz_out, int64_t *cscptr, int32_t *cscrow)
{
    int64_t total = 0;
    for (int64_t i = 0; i < n_dst; ++i) {
        if (dst[i] < 0 || dst[i] >= n) return -1;
        int64_t d = rowptr[dst[i] + 1] - rowptr[dst[i]];
        total += d < fanout ? d : fanout;
    }
    if (total > cap_nnz) return -2;

    int64_t *gid = (int64_t *)malloc(sizeof(int64_t) * (size_t)(total > 0 ? total : 1));
    int64_t *pos = (int64_t *)malloc(sizeof(int64_t) * (size_t)(fanout > 0 ? fanout : 1));
    id_pos *dsorted = (id_pos *)malloc(sizeof(id_pos) * (size_t)(n_dst > 0 ? n_dst : 1));
    if (!gid || !pos || !dsorted) { free(gid); free(pos); free(dsorted); return -3; }

    /* sampled neighbour lists, in row order */
    brow[0] = 0;
    int64_t e = 0;
    for (int64_t i = 0; i < n_dst; ++i) {
        int64_t v = dst[i];
        int64_t d = rowptr[v + 1] - rowptr[v];
        int64_t cnt = orc_sample_positions(d, fanout, seed, step, hop, v, pos);
        for (int64_t t = 0; t < cnt; ++t) gid[e++] = col[rowptr[v] + pos[t]];
        brow[i + 1] = e;
    }

    /* dst membership */
    for (int64_t i = 0; i < n_dst; ++i) { dsorted[i].id = dst[i]; dsorted[i].pos = i; }
    qsort(dsorted, (size_t)n_dst, sizeof(id_pos), cmp_id_pos);

    /* new sources: sorted unique of sampled ids that are not destinations */
    int64_t *cand = (int64_t *)malloc(sizeof(int64_t) * (size_t)(total > 0 ? total : 1));
    int64_t nc = 0;
    for (int64_t t = 0; t < total; ++t)
        if (find_id(dsorted, n_dst, gid[t]) < 0) cand[nc++] = gid[t];
    qsort(cand, (size_t)nc, sizeof(int64_t), cmp_i64);
    int64_t nu = 0;
    for (int64_t t = 0; t < nc; ++t)
        if (nu == 0 || cand[nu - 1] != cand[t]) cand[nu++] = cand[t];

    int64_t n_src = n_dst + nu;
    if (n_src > cap_src) { free(gid); free(pos); free(dsorted); free(cand); return -2; }
    for (int64_t i = 0; i < n_dst; ++i) src_ids[i] = dst[i];
    for (int64_t t = 0; t < nu; ++t) src_ids[n_dst + t] = cand[t];

    /* local source index of each sampled edge */
    for (int64_t t = 0; t < total; ++t) {
        int64_t p = find_id(dsorted, n_dst, gid[t]);
        if (p < 0) {
            int64_t lo = 0, hi = nu;
            while (lo < hi) {
                int64_t mid = lo + (hi - lo) / 2;
                if (cand[mid] < gid[t]) lo = mid + 1; else hi = mid;
            }
            p = n_dst + lo;
        }
        bcol[t] = (int32_t)p;
    }

    /* stable transpose: walking rows in order places each source's rows in
     * ascending order */
    if (cscptr) {
        for (int64_t j = 0; j <= n_src; ++j) cscptr[j] = 0;
        for (int64_t t = 0; t < total; ++t) cscptr[bcol[t] + 1]++;
        for (int64_t j = 0; j < n_src; ++j) cscptr[j + 1] += cscptr[j];
        int64_t *fill = (int64_t *)calloc((size_t)(n_src > 0 ? n_src : 1), sizeof(int64_t));
        for (int64_t i = 0; i < n_dst; ++i)
            for (int64_t t = brow[i]; t < brow[i + 1]; ++t) {
                int32_t j = bcol[t];
                cscrow[cscptr[j] + fill[j]++] = (int32_t)i;
            }
        free(fill);
    }
    *n_src_out = n_src;
    *nnz_out = total;
    free(gid); free(pos); free(dsorted); free(cand);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Feature loader: X' = X[ids] (Section III-A, Feature Loader).               */
/* ------------------------------------------------------------------------ */

void orc_gather(const void *table, int tdt, int64_t dim, int64_t row_stride, const int64_t *ids,
                int64_t n_ids, void *out, int odt)
{
    for (int64_t r = 0; r < n_ids; ++r) {
        int64_t base = ids[r] * row_stride;
        for (int64_t c = 0; c < dim; ++c) {
            int64_t o = r * dim + c;
            if (tdt == odt && (tdt == ORC_F32 || tdt == ORC_BF16 || tdt == ORC_F16)) {
                /* same type: a bit copy (NaN payloads preserved) */
                if (tdt == ORC_F32) ((uint32_t *)out)[o] = ((const uint32_t *)table)[base + c];
                else ((uint16_t *)out)[o] = ((const uint16_t *)table)[base + c];
            } else if (odt == ORC_BF16) {
                float x = (tdt == ORC_F32) ? ((const float *)table)[base + c]
                                           : (float)load_elem(table, tdt, base + c);
                ((uint16_t *)out)[o] = orc_f32_to_bf16(x);
            } else {
                store_elem(out, odt, o, load_elem(table, tdt, base + c));
            }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Aggregation (equation 1 with the GCN and GraphSAGE operators).             */
/* ------------------------------------------------------------------------ */

/* Edge weight of the GCN operator: nrm(v) * nrm(u) as one fp32 product. */
static double gcn_weight(const float *src_norm, int64_t i, int64_t j)
{
    float w = src_norm[i] * src_norm[j];
    return (double)w;
}

/* Forward aggregation for the dst rows of one block.
 *   SAGE: out[i] = mean of h[col] over the sampled neighbours (0 if none).
 *   GCN:  out[i] = nrm_i^2 h[i] + sum_e nrm_i nrm_col h[col]
 * h has n_src rows; row i of h is dst i itself (destinations come first). */
void orc_aggregate_fwd(int kind, int64_t n_dst, const int64_t *brow, const int32_t *bcol,
                       const float *src_norm, const void *h, int hdt, int64_t f, void *out, int odt)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_dst; ++i) {
        double *acc = (double *)calloc((size_t)f, sizeof(double));
        int64_t deg = brow[i + 1] - brow[i];
        if (kind == ORC_GCN_SYM) {
            double ws = gcn_weight(src_norm, i, i);
            for (int64_t c = 0; c < f; ++c) acc[c] = ws * load_elem(h, hdt, i * f + c);
        }
        for (int64_t e = brow[i]; e < brow[i + 1]; ++e) {
            int64_t j = bcol[e];
            double w = (kind == ORC_GCN_SYM) ? gcn_weight(src_norm, i, j) : 1.0;
            for (int64_t c = 0; c < f; ++c) acc[c] += w * load_elem(h, hdt, j * f + c);
        }
        for (int64_t c = 0; c < f; ++c) {
            double v = acc[c];
            if (kind == ORC_SAGE_MEAN) v = deg > 0 ? v / (double)deg : 0.0;
            store_elem(out, odt, i * f + c, v);
        }
        free(acc);
    }
}

/* Backward of the aggregation for layers above the first: the transpose of
 * the forward operator applied to dA, followed by the ReLU mask of the
 * layer below (when h_below is given):
 *   SAGE (dA has 2f columns: self part then neighbour part):
 *     dH[j] = [j < n_dst] dA[j, 0:f] + sum_{(i,e): col_e = j} dA[i, f:2f] / deg_i
 *   GCN (dA has f columns):
 *     dH[j] = [j < n_dst] nrm_j^2 dA[j] + sum_{(i,e): col_e = j} nrm_i nrm_j dA[i]
 *   G[j]  = dH[j] * 1[h_below[j] > 0]
 * The sum walks the forward block's edges (a scatter over rows), which is the
 * definition of the transpose; it does not use the CSC. */
void orc_aggregate_bwd(int kind, int64_t n_dst, int64_t n_src, const int64_t *brow, const int32_t *bcol,
                       const float *src_norm, const void *d_a, int adt, int64_t f,
                       const void *h_below, int hbdt, void *d_src, int odt)
{
    int64_t ka = (kind == ORC_SAGE_MEAN) ? 2 * f : f;
    double *acc = (double *)calloc((size_t)(n_src * f > 0 ? n_src * f : 1), sizeof(double));
    for (int64_t j = 0; j < n_dst; ++j)
        for (int64_t c = 0; c < f; ++c) {
            double g = load_elem(d_a, adt, j * ka + c);
            acc[j * f + c] = (kind == ORC_GCN_SYM) ? gcn_weight(src_norm, j, j) * g : g;
        }
    for (int64_t i = 0; i < n_dst; ++i) {
        int64_t deg = brow[i + 1] - brow[i];
        for (int64_t e = brow[i]; e < brow[i + 1]; ++e) {
            int64_t j = bcol[e];
            for (int64_t c = 0; c < f; ++c) {
                if (kind == ORC_SAGE_MEAN)
                    acc[j * f + c] += load_elem(d_a, adt, i * ka + f + c) / (double)deg;
                else
                    acc[j * f + c] += gcn_weight(src_norm, i, j) * load_elem(d_a, adt, i * ka + c);
            }
        }
    }
    for (int64_t j = 0; j < n_src; ++j)
        for (int64_t c = 0; c < f; ++c) {
            double v = acc[j * f + c];
            if (h_below && !(load_elem(h_below, hbdt, j * f + c) > 0.0)) v = 0.0;
            store_elem(d_src, odt, j * f + c, v);
        }
    free(acc);
}

/* GraphSAGE with the max aggregator (Section II-A names mean, max and LSTM
 * as aggregation operators):
 *   out[i, c] = max over row i's sampled neighbours u of h[u, c]
 * (zero, and argmax -1, for a row with no neighbours).  The row's first edge
 * holds the running maximum and a later edge replaces it only when strictly
 * greater, so a tie, and a duplicate edge, goes to the earliest edge;
 * argmax[i, c] is that edge's source (its local id).  The comparison is on
 * the stored values (no rounding); the maximum is narrowed to out's dtype. */
void orc_aggregate_fwd_max(int64_t n_dst, const int64_t *brow, const int32_t *bcol, const void *h, int hdt,
                           int64_t f, void *out, int odt, int32_t *argmax)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_dst; ++i)
        for (int64_t c = 0; c < f; ++c) {
            double best = 0.0;
            int32_t arg = -1;
            for (int64_t e = brow[i]; e < brow[i + 1]; ++e) {
                double v = load_elem(h, hdt, (int64_t)bcol[e] * f + c);
                if (arg < 0 || v > best) {
                    best = v;
                    arg = bcol[e];
                }
            }
            store_elem(out, odt, i * f + c, best);
            argmax[i * f + c] = arg;
        }
}

/* Backward of the max aggregator (Section II-B: the backward pass applies the
 * forward operators in reverse).  The maximum passes its gradient to the
 * source that won it; the concatenation's self part passes to the
 * destination itself (dA has 2f columns: self part, then max part):
 *   dH[j, c] = [j < n_dst] dA[j, c] + sum_{i: argmax[i, c] = j} dA[i, f + c]
 *   G[j, c]  = dH[j, c] * 1[h_below[j, c] > 0]   (when h_below is given)
 * The sum scatters over the argmax table; it does not use the block. */
void orc_aggregate_bwd_max(int64_t n_dst, int64_t n_src, const int32_t *argmax, const void *d_a, int adt, int64_t f,
                           const void *h_below, int hbdt, void *d_src, int odt)
{
    double *acc = (double *)calloc((size_t)(n_src * f > 0 ? n_src * f : 1), sizeof(double));
    for (int64_t j = 0; j < n_dst; ++j)
        for (int64_t c = 0; c < f; ++c) acc[j * f + c] = load_elem(d_a, adt, j * 2 * f + c);
    for (int64_t i = 0; i < n_dst; ++i)
        for (int64_t c = 0; c < f; ++c) {
            int32_t j = argmax[i * f + c];
            if (j >= 0) acc[(int64_t)j * f + c] += load_elem(d_a, adt, i * 2 * f + f + c);
        }
    for (int64_t j = 0; j < n_src; ++j)
        for (int64_t c = 0; c < f; ++c) {
            double v = acc[j * f + c];
            if (h_below && !(load_elem(h_below, hbdt, j * f + c) > 0.0)) v = 0.0;
            store_elem(d_src, odt, j * f + c, v);
        }
    free(acc);
}

/* ------------------------------------------------------------------------ */
/* Update (equation 2): Z = A W + b, with A = [a_self || a_nbr] for SAGE.      */
/* ------------------------------------------------------------------------ */

/* A as an m x K double matrix of GEMM operand values. */
static double *operand_A(int64_t m, const void *a_self, const void *a_nbr, int adt, int64_t k_each, int gemm_dt,
                         int64_t *K_out)
{
    int64_t K = a_nbr ? 2 * k_each : k_each;
    double *A = (double *)malloc(sizeof(double) * (size_t)(m * K > 0 ? m * K : 1));
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < m; ++r)
        for (int64_t k = 0; k < K; ++k) {
            double s = (k < k_each) ? load_elem(a_self, adt, r * k_each + k)
                                    : load_elem(a_nbr, adt, r * k_each + (k - k_each));
            A[r * K + k] = gemm_operand(s, gemm_dt);
        }
    *K_out = K;
    return A;
}

/* Z[r][c] = b[c] + sum_k A[r][k] W[k][c]; H = ReLU(Z) when relu != 0. */
void orc_update_fwd(int64_t m, const void *a_self, const void *a_nbr, int adt, int64_t k_each,
                    const void *w, int wdt, const void *bias, int bdt, int64_t nout, int relu, int gemm_dt,
                    void *out, int odt)
{
    int64_t K;
    double *A = operand_A(m, a_self, a_nbr, adt, k_each, gemm_dt, &K);
    double *Wt = (double *)malloc(sizeof(double) * (size_t)(K * nout > 0 ? K * nout : 1));
    for (int64_t k = 0; k < K; ++k)
        for (int64_t c = 0; c < nout; ++c)
            Wt[c * K + k] = gemm_operand(load_elem(w, wdt, k * nout + c), gemm_dt);
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < m; ++r)
        for (int64_t c = 0; c < nout; ++c) {
            double s = 0.0;
            for (int64_t k = 0; k < K; ++k) s += A[r * K + k] * Wt[c * K + k];
            s += bias ? load_elem(bias, bdt, c) : 0.0;
            if (relu && !(s > 0.0)) s = 0.0;
            store_elem(out, odt, r * nout + c, s);
        }
    free(A);
    free(Wt);
}

/* Gradients of Z = A W + b given G = dLoss/dZ:
 *   dW = A^T G, db = column sums of G (unrounded), dA = G W^T (optional). */
void orc_update_bwd(int64_t m, const void *a_self, const void *a_nbr, int adt, int64_t k_each,
                    const void *w, int wdt, const void *g, int gdt, int64_t nout, int gemm_dt,
                    void *dw, void *db, void *d_a, int dt_out)
{
    int64_t K;
    double *A = operand_A(m, a_self, a_nbr, adt, k_each, gemm_dt, &K);
    double *Gq = (double *)malloc(sizeof(double) * (size_t)(m * nout > 0 ? m * nout : 1));
    for (int64_t i = 0; i < m * nout; ++i) Gq[i] = gemm_operand(load_elem(g, gdt, i), gemm_dt);
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < K; ++k)
        for (int64_t c = 0; c < nout; ++c) {
            double s = 0.0;
            for (int64_t r = 0; r < m; ++r) s += A[r * K + k] * Gq[r * nout + c];
            store_elem(dw, dt_out, k * nout + c, s);
        }
    if (db)
        for (int64_t c = 0; c < nout; ++c) {
            double s = 0.0;
            for (int64_t r = 0; r < m; ++r) s += load_elem(g, gdt, r * nout + c);
            store_elem(db, dt_out, c, s);
        }
    if (d_a) {
        double *Wq = (double *)malloc(sizeof(double) * (size_t)(K * nout > 0 ? K * nout : 1));
        for (int64_t i = 0; i < K * nout; ++i) Wq[i] = gemm_operand(load_elem(w, wdt, i), gemm_dt);
#pragma omp parallel for schedule(static)
        for (int64_t r = 0; r < m; ++r)
            for (int64_t k = 0; k < K; ++k) {
                double s = 0.0;
                for (int64_t c = 0; c < nout; ++c) s += Gq[r * nout + c] * Wq[k * nout + c];
                store_elem(d_a, dt_out, r * K + k, s);
            }
        free(Wq);
    }
    free(A);
    free(Gq);
}

/* ------------------------------------------------------------------------ */
/* Loss against the ground truth (Section II-B): mean softmax cross-entropy.  */
/* ------------------------------------------------------------------------ */

/* Returns the mean loss; writes G = (softmax(Z) - onehot(y)) / B. */
double orc_softmax_ce(int64_t b, int64_t c, const void *logits, int ldt, const int64_t *y,
                      void *g, int gdt)
{
    double total = 0.0;
    for (int64_t i = 0; i < b; ++i) {
        double mx = -INFINITY;
        for (int64_t k = 0; k < c; ++k) {
            double z = load_elem(logits, ldt, i * c + k);
            if (z > mx) mx = z;
        }
        double s = 0.0;
        for (int64_t k = 0; k < c; ++k) s += exp(load_elem(logits, ldt, i * c + k) - mx);
        double lse = mx + log(s);
        total += lse - load_elem(logits, ldt, i * c + y[i]);
        for (int64_t k = 0; k < c; ++k) {
            double p = exp(load_elem(logits, ldt, i * c + k) - lse);
            store_elem(g, gdt, i * c + k, (p - (k == y[i] ? 1.0 : 0.0)) / (double)b);
        }
    }
    return b > 0 ? total / (double)b : 0.0;
}

/* Plain SGD step: w <- w - lr * dw. */
void orc_sgd(int64_t n, void *w, int wdt, const void *dw, int dwdt, double lr)
{
    for (int64_t i = 0; i < n; ++i)
        store_elem(w, wdt, i, load_elem(w, wdt, i) - lr * load_elem(dw, dwdt, i));
}
