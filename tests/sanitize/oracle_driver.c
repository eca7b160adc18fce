/* Runs every function of the CPU oracle on small, edge-case-heavy inputs so
 * that an AddressSanitizer / UndefinedBehaviorSanitizer build of oracle.c
 * can report any out-of-bounds access, leak or undefined operation.  It
 * checks no values (the Python pins do that); it exits 0 when every call
 * returned its documented status. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

enum { F32 = 0, BF16 = 1, F16 = 2 };
enum { SAGE = 0, GCN = 1 };

uint16_t orc_f32_to_bf16(float x);
float orc_bf16_to_f32(uint16_t h);
float orc_f16_to_f32(uint16_t h);
void orc_set_threads(int n);
uint64_t orc_mix64(uint64_t z);
uint64_t orc_sample_key(uint64_t seed, uint64_t step, uint64_t hop, uint64_t v, uint64_t t);
uint64_t orc_bounded(uint64_t key, uint64_t bound);
int64_t orc_sample_positions(int64_t d, int32_t k, uint64_t seed, uint64_t step, int32_t hop, int64_t v,
                             int64_t *pos);
void orc_gcn_norm(int64_t n, const int64_t *rowptr, float *nrm);
int orc_build_block(int64_t n, const int64_t *rowptr, const int64_t *col, const int64_t *dst, int64_t n_dst,
                    int32_t fanout, uint64_t seed, uint64_t step, int32_t hop, int64_t cap_src, int64_t cap_nnz,
                    int64_t *src_ids, int64_t *n_src_out, int64_t *brow, int32_t *bcol, int64_t *nnz_out,
                    int64_t *cscptr, int32_t *cscrow);
void orc_gather(const void *table, int tdt, int64_t dim, int64_t row_stride, const int64_t *ids, int64_t n_ids,
                void *out, int odt);
void orc_aggregate_fwd(int kind, int64_t n_dst, const int64_t *brow, const int32_t *bcol, const float *src_norm,
                       const void *h, int hdt, int64_t f, void *out, int odt);
void orc_aggregate_bwd(int kind, int64_t n_dst, int64_t n_src, const int64_t *brow, const int32_t *bcol,
                       const float *src_norm, const void *d_a, int adt, int64_t f, const void *h_below, int hbdt,
                       void *d_src, int odt);
void orc_update_fwd(int64_t m, const void *a_self, const void *a_nbr, int adt, int64_t k_each, const void *w,
                    int wdt, const void *bias, int bdt, int64_t nout, int relu, int gemm_dt, void *out, int odt);
void orc_update_bwd(int64_t m, const void *a_self, const void *a_nbr, int adt, int64_t k_each, const void *w,
                    int wdt, const void *g, int gdt, int64_t nout, int gemm_dt, void *dw, void *db, void *d_a,
                    int dt_out);
double orc_softmax_ce(int64_t b, int64_t c, const void *logits, int ldt, const int64_t *y, void *g, int gdt);
void orc_sgd(int64_t n, void *w, int wdt, const void *dw, int dwdt, double lr);

static uint64_t rng = 88172645463325252ull;
static uint64_t next(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return rng;
}
static float unif(void) { return (float)((next() >> 11) * (1.0 / 9007199254740992.0)) * 2.f - 1.f; }

#define CHECK(c)                                                    \
    do {                                                            \
        if (!(c)) {                                                 \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            return 1;                                               \
        }                                                           \
    } while (0)

/* A multigraph of n vertices: vertex 0 a hub linked to every other vertex,
 * vertices 1..3 isolated, the rest with a few random neighbours (repeats
 * kept), rows sorted ascending. */
static void make_graph(int64_t n, int64_t **rowptr_o, int64_t **col_o) {
    int64_t *deg = calloc((size_t)n, sizeof(int64_t));
    int64_t *rowptr = malloc(sizeof(int64_t) * (size_t)(n + 1));
    deg[0] = n - 4;
    for (int64_t v = 4; v < n; ++v) deg[v] = 1 + (int64_t)(next() % 9);
    rowptr[0] = 0;
    for (int64_t v = 0; v < n; ++v) rowptr[v + 1] = rowptr[v] + deg[v];
    int64_t *col = malloc(sizeof(int64_t) * (size_t)(rowptr[n] > 0 ? rowptr[n] : 1));
    for (int64_t v = 0; v < n; ++v) {
        int64_t *r = col + rowptr[v];
        if (v == 0) {
            for (int64_t u = 4; u < n; ++u) r[u - 4] = u;
        } else {
            r[0] = 0;  /* everyone's first neighbour is the hub */
            for (int64_t p = 1; p < deg[v]; ++p) r[p] = 4 + (int64_t)(next() % (uint64_t)(n - 4));
            for (int64_t a = 1; a < deg[v]; ++a)  /* insertion sort */
                for (int64_t b = a; b > 0 && r[b - 1] > r[b]; --b) {
                    int64_t t = r[b]; r[b] = r[b - 1]; r[b - 1] = t;
                }
        }
    }
    free(deg);
    *rowptr_o = rowptr;
    *col_o = col;
}

int main(void) {
    orc_set_threads(2);
    /* conversions, including NaN, infinities and ties */
    const float specials[] = {0.f, -0.f, 1.f, 1.00390625f, 3.0e38f, -3.0e38f, 1.0e-40f, 0.f / 0.f, 1.f / 0.f};
    for (size_t i = 0; i < sizeof(specials) / sizeof(specials[0]); ++i)
        (void)orc_bf16_to_f32(orc_f32_to_bf16(specials[i]));
    for (uint32_t h = 0; h < 65536; h += 7) (void)orc_f16_to_f32((uint16_t)h);
    /* sampling */
    int64_t pos[300];
    CHECK(orc_sample_positions(5, 10, 1, 2, 1, 7, pos) == 5);
    CHECK(orc_sample_positions(300, 300, 1, 2, 1, 7, pos) == 300);
    CHECK(orc_sample_positions(1000, 1, 1, 2, 1, 7, pos) == 1);
    CHECK(orc_sample_positions(1000, 300, 1, 2, 2, 9, pos) == 300);
    CHECK(orc_sample_positions(0, 3, 1, 2, 2, 9, pos) == 0);
    (void)orc_bounded(orc_mix64(0), 0);
    (void)orc_bounded(~0ull, ~0ull);

    const int64_t n = 200;
    int64_t *rowptr, *col;
    make_graph(n, &rowptr, &col);
    float *nrm = malloc(sizeof(float) * (size_t)n);
    orc_gcn_norm(n, rowptr, nrm);

    /* blocks: hop 1 around targets that include the hub and isolated
     * vertices, hop 2 around hop 1's sources; an empty batch; a capacity
     * that is too small; an out-of-range id */
    int64_t dst[] = {0, 1, 2, 57, 150, 199, 33, 4};
    const int64_t n_dst = 8;
    const int32_t k1 = 3, k2 = 5;
    int64_t cap_nnz1 = n_dst * k1, cap_src1 = n_dst + cap_nnz1;
    int64_t *src1 = malloc(sizeof(int64_t) * (size_t)cap_src1), *brow1 = malloc(sizeof(int64_t) * (size_t)(n_dst + 1));
    int32_t *bcol1 = malloc(sizeof(int32_t) * (size_t)cap_nnz1), *cscrow1 = malloc(sizeof(int32_t) * (size_t)cap_nnz1);
    int64_t *cscptr1 = malloc(sizeof(int64_t) * (size_t)(cap_src1 + 1));
    int64_t n_src1 = 0, nnz1 = 0;
    CHECK(orc_build_block(n, rowptr, col, dst, n_dst, k1, 3, 4, 1, cap_src1, cap_nnz1, src1, &n_src1, brow1, bcol1,
                          &nnz1, cscptr1, cscrow1) == 0);
    int64_t cap_nnz2 = n_src1 * k2, cap_src2 = n_src1 + cap_nnz2;
    int64_t *src2 = malloc(sizeof(int64_t) * (size_t)cap_src2), *brow2 = malloc(sizeof(int64_t) * (size_t)(n_src1 + 1));
    int32_t *bcol2 = malloc(sizeof(int32_t) * (size_t)cap_nnz2), *cscrow2 = malloc(sizeof(int32_t) * (size_t)cap_nnz2);
    int64_t *cscptr2 = malloc(sizeof(int64_t) * (size_t)(cap_src2 + 1));
    int64_t n_src2 = 0, nnz2 = 0;
    CHECK(orc_build_block(n, rowptr, col, src1, n_src1, k2, 3, 4, 2, cap_src2, cap_nnz2, src2, &n_src2, brow2, bcol2,
                          &nnz2, cscptr2, cscrow2) == 0);
    int64_t e_src = 0, e_nnz = 0, e_brow[1];
    CHECK(orc_build_block(n, rowptr, col, dst, 0, k1, 3, 4, 1, 1, 1, src1, &e_src, e_brow, bcol1, &e_nnz, cscptr1,
                          cscrow1) == 0);
    CHECK(orc_build_block(n, rowptr, col, dst, n_dst, k1, 3, 4, 1, cap_src1, 2, src1, &n_src1, brow1, bcol1, &nnz1,
                          cscptr1, cscrow1) == -2);
    int64_t bad[] = {0, n};
    CHECK(orc_build_block(n, rowptr, col, bad, 2, k1, 3, 4, 1, cap_src1, cap_nnz1, src1, &n_src1, brow1, bcol1,
                          &nnz1, cscptr1, cscrow1) == -1);
    CHECK(orc_build_block(n, rowptr, col, dst, n_dst, k1, 3, 4, 1, cap_src1, cap_nnz1, src1, &n_src1, brow1, bcol1,
                          &nnz1, cscptr1, cscrow1) == 0);

    /* gather in every supported type pair, with a row stride */
    const int64_t f0 = 12, stride = 16;
    float *table = malloc(sizeof(float) * (size_t)(n * stride));
    uint16_t *table16 = malloc(sizeof(uint16_t) * (size_t)(n * stride));
    for (int64_t i = 0; i < n * stride; ++i) {
        table[i] = unif();
        table16[i] = (uint16_t)(next() & 0x7bff);
    }
    float *x32 = malloc(sizeof(float) * (size_t)(n_src2 * f0));
    uint16_t *x16 = malloc(sizeof(uint16_t) * (size_t)(n_src2 * f0));
    orc_gather(table, F32, f0, stride, src2, n_src2, x32, F32);
    orc_gather(table, F32, f0, stride, src2, n_src2, x16, BF16);
    orc_gather(table16, F16, f0, stride, src2, n_src2, x16, F16);
    orc_gather(table16, F16, f0, stride, src2, n_src2, x32, F32);
    orc_gather(table16, F16, f0, stride, src2, n_src2, x16, BF16);
    orc_gather(table, F32, f0, stride, src2, 0, x32, F32);

    float *nrm2 = malloc(sizeof(float) * (size_t)n_src2);
    for (int64_t j = 0; j < n_src2; ++j) nrm2[j] = nrm[src2[j]];
    for (int kind = SAGE; kind <= GCN; ++kind)
        for (int dt = F32; dt <= BF16; ++dt) {
            const void *h = dt == F32 ? (const void *)x32 : (const void *)x16;
            const int64_t K = kind == SAGE ? 2 * f0 : f0, nout = 7;
            void *agg = malloc(4 * (size_t)(n_src1 * f0));
            orc_aggregate_fwd(kind, n_src1, brow2, bcol2, nrm2, h, dt, f0, agg, dt);
            float *w = malloc(sizeof(float) * (size_t)(K * nout)), *b = malloc(sizeof(float) * (size_t)nout);
            for (int64_t i = 0; i < K * nout; ++i) w[i] = unif();
            for (int64_t i = 0; i < nout; ++i) b[i] = unif();
            float *z = malloc(sizeof(float) * (size_t)(n_src1 * nout));
            const void *as = kind == SAGE ? h : agg, *an = kind == SAGE ? agg : NULL;
            orc_update_fwd(n_src1, as, an, dt, f0, w, F32, b, F32, nout, 1, dt, z, F32);
            orc_update_fwd(0, as, an, dt, f0, w, F32, NULL, F32, nout, 0, dt, z, F32);
            float *g = malloc(sizeof(float) * (size_t)(n_src1 * nout)), *dw = malloc(sizeof(float) * (size_t)(K * nout));
            float *db = malloc(sizeof(float) * (size_t)nout), *da = malloc(sizeof(float) * (size_t)(n_src1 * K));
            for (int64_t i = 0; i < n_src1 * nout; ++i) g[i] = unif();
            orc_update_bwd(n_src1, as, an, dt, f0, w, F32, g, F32, nout, dt, dw, db, da, F32);
            orc_update_bwd(n_src1, as, an, dt, f0, w, F32, g, F32, nout, dt, dw, NULL, NULL, F32);
            /* the backward aggregation of the hop-1 block: d_a rows of
             * its destinations, gradients for its sources */
            const int64_t ka = kind == SAGE ? 2 * f0 : f0;
            float *dA = malloc(sizeof(float) * (size_t)(n_dst * ka)), *dsrc = malloc(sizeof(float) * (size_t)(n_src1 * f0));
            for (int64_t i = 0; i < n_dst * ka; ++i) dA[i] = unif();
            float *nrm1 = malloc(sizeof(float) * (size_t)n_src1);
            for (int64_t j = 0; j < n_src1; ++j) nrm1[j] = nrm[src1[j]];
            orc_aggregate_bwd(kind, n_dst, n_src1, brow1, bcol1, nrm1, dA, F32, f0, h, dt, dsrc, F32);
            orc_aggregate_bwd(kind, n_dst, n_src1, brow1, bcol1, nrm1, dA, F32, f0, NULL, F32, dsrc, F32);
            free(agg); free(w); free(b); free(z); free(g); free(dw); free(db); free(da); free(dA); free(dsrc);
            free(nrm1);
        }
    /* loss and SGD */
    const int64_t B = 9, C = 5;
    float logits[45], gl[45];
    int64_t y[9];
    for (int i = 0; i < 45; ++i) logits[i] = 30.f * unif();
    for (int i = 0; i < 9; ++i) y[i] = (int64_t)(next() % C);
    (void)orc_softmax_ce(B, C, logits, F32, y, gl, F32);
    (void)orc_softmax_ce(0, C, logits, F32, y, gl, F32);
    orc_sgd(45, logits, F32, gl, F32, 0.1);
    orc_sgd(0, logits, F32, gl, F32, 0.1);

    free(rowptr); free(col); free(nrm); free(src1); free(brow1); free(bcol1); free(cscrow1); free(cscptr1);
    free(src2); free(brow2); free(bcol2); free(cscrow2); free(cscptr2); free(table); free(table16); free(x32);
    free(x16); free(nrm2);
    printf("oracle driver: ok\n");
    return 0;
}
