/* Drives the host-side validation of every C-ABI entry point with bad and
 * good arguments, for an AddressSanitizer / UndefinedBehaviorSanitizer
 * build of the library's host code.  Nothing here reaches the GPU: every
 * call is rejected (or answered) before any HIP call, so the driver runs on
 * a machine without one.  Exits 0 when every status is the documented one. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "gnn.h"

#define EXPECT(call, want)                                                                  \
    do {                                                                                    \
        gnn_status st_ = (call);                                                            \
        if (st_ != (want)) {                                                                \
            fprintf(stderr, "line %d: %s returned %d, expected %d (%s)\n", __LINE__, #call, \
                    (int)st_, (int)(want), gnn_last_error());                               \
            return 1;                                                                       \
        }                                                                                   \
    } while (0)

static gnn_model model(int kind, int precision, const int *dims, const int *fan, int L) {
    gnn_model m;
    memset(&m, 0, sizeof(m));
    m.num_layers = L;
    m.kind = kind;
    m.precision = precision;
    for (int i = 0; i <= L; ++i) m.dims[i] = dims[i];
    for (int i = 0; i < L; ++i) m.fanouts[i] = fan[i];
    return m;
}

int main(void) {
    if (gnn_abi_version() != GNN_ABI_VERSION) return 1;
    int64_t cs = 0, cn = 0;
    EXPECT(gnn_block_bounds(100, 10, 0, &cs, &cn), GNN_EINVAL);
    if (strstr(gnn_last_error(), "fanout") == NULL) return 1;
    EXPECT(gnn_block_bounds(100, 10, 25, &cs, &cn), GNN_OK);
    EXPECT(gnn_block_bounds(1000000000, 1024, 25, &cs, &cn), GNN_OK);
    EXPECT(gnn_block_bounds(100, -1, 25, &cs, &cn), GNN_EINVAL);
    EXPECT(gnn_block_bounds(100, 10, 25, NULL, &cn), GNN_EINVAL);
    size_t nb = 0;
    EXPECT(gnn_sampler_workspace_size(1000, 64, 10, &nb), GNN_OK);
    EXPECT(gnn_sampler_workspace_size(1000, 64, 0, &nb), GNN_EINVAL);
    EXPECT(gnn_update_fwd_workspace_size(8, 4, 1000, GNN_BF16, &nb), GNN_OK);
    EXPECT(gnn_update_fwd_workspace_size(8, 4, 4, GNN_F16, &nb), GNN_EUNSUPPORTED);
    EXPECT(gnn_update_bwd_workspace_size(0, 4, 4, GNN_BF16, &nb), GNN_EINVAL);
    EXPECT(gnn_update_bwd_workspace_size(1536, 1024, 26624, GNN_BF16, &nb), GNN_OK);
    EXPECT(gnn_softmax_ce_workspace_size(-1, &nb), GNN_EINVAL);

    /* pointers below are never dereferenced: every call fails validation */
    void *fake = (void *)(uintptr_t)(1u << 24);
    EXPECT(gnn_update_fwd(NULL, NULL, GNN_F32, 8, NULL, 4, NULL, NULL, NULL, 8, 0, GNN_F32, NULL, GNN_F32, NULL, 0, NULL),
           GNN_EINVAL);
    EXPECT(gnn_update_fwd(NULL, NULL, GNN_F16, 8, NULL, 4, NULL, NULL, NULL, 8, 0, GNN_F32, NULL, GNN_F32, NULL, 0, NULL),
           GNN_EUNSUPPORTED);
    EXPECT(gnn_update_fwd(fake, fake, GNN_BF16, 8, NULL, 4, fake, (const uint16_t *)((char *)fake + 2), NULL, 8, 1,
                          GNN_BF16, fake, GNN_BF16, NULL, 0, NULL),
           GNN_EINVAL);
    EXPECT(gnn_update_bwd(NULL, NULL, GNN_F32, 8, NULL, 4, NULL, NULL, 8, GNN_F32, NULL, NULL, NULL, NULL, 0, NULL),
           GNN_EINVAL);
    EXPECT(gnn_update_bwd(fake, NULL, GNN_F32, 8, NULL, 4, fake, fake, 8, GNN_F32, fake, NULL, NULL, fake, 0, NULL),
           GNN_ESIZE);
    /* the wide host-table layer needs more than the static scratch */
    EXPECT(gnn_update_bwd_noalloc(fake, fake, GNN_BF16, 768, NULL, 26624, fake, fake, 1024, GNN_BF16, fake, NULL,
                                  NULL, NULL),
           GNN_ESIZE);
    EXPECT(gnn_update_bwd_noalloc(NULL, NULL, GNN_F16, 8, NULL, 4, NULL, NULL, 8, GNN_F32, NULL, NULL, NULL, NULL),
           GNN_EUNSUPPORTED);
    EXPECT(gnn_gather_features(NULL, GNN_F32, GNN_LOC_DEVICE, 10, 4, 4, NULL, NULL, 3, NULL, GNN_F16, NULL),
           GNN_EUNSUPPORTED);
    EXPECT(gnn_gather_features(NULL, GNN_F32, 7, 10, 4, 4, NULL, NULL, 3, NULL, GNN_F32, NULL), GNN_EINVAL);
    EXPECT(gnn_gather_features(NULL, GNN_F32, GNN_LOC_DEVICE, 10, 4, 2, NULL, NULL, 3, NULL, GNN_F32, NULL),
           GNN_EINVAL);
    EXPECT(gnn_sgd(NULL, NULL, -1, 0.1f, NULL), GNN_EINVAL);
    EXPECT(gnn_aggregate_fwd(NULL, GNN_AGG_SAGE_MEAN, NULL, GNN_F32, 4, NULL, GNN_F32, NULL), GNN_EINVAL);
    EXPECT(gnn_softmax_ce(NULL, 4, 0, NULL, NULL, NULL, NULL, NULL, 0, NULL), GNN_EINVAL);
    gnn_block blk;
    memset(&blk, 0, sizeof(blk));
    blk.cap_dst = 4;
    blk.cap_src = 8;
    blk.cap_nnz = 8;
    EXPECT(gnn_aggregate_bwd(&blk, GNN_AGG_SAGE_MEAN, NULL, 4, NULL, GNN_F32, NULL, NULL), GNN_EINVAL);
    gnn_graph g = {10, 20, NULL, NULL};
    EXPECT(gnn_build_block(&g, NULL, NULL, NULL, 5, 0, 0, 1, 1, &blk, NULL, 0, NULL), GNN_EINVAL);

    /* model shapes, layouts, the two-stage and pipelined steps */
    const int dims[] = {100, 256, 47}, fan[] = {25, 10};
    gnn_model m = model(GNN_AGG_SAGE_MEAN, GNN_BF16, dims, fan, 2);
    gnn_step_layout lay;
    EXPECT(gnn_train_step_layout(&m, 2449029, 1024, &lay), GNN_OK);
    if (lay.total_bytes != lay.prep_bytes + lay.compute_bytes || lay.error == 0) return 1;
    EXPECT(gnn_train_step_workspace_size(&m, 2449029, 1024, &nb), GNN_OK);
    EXPECT(gnn_train_step_workspace_size(&m, 1000, 2000, &nb), GNN_EINVAL);
    const int bad_fan[] = {25, 0};
    gnn_model bad = model(GNN_AGG_SAGE_MEAN, GNN_BF16, dims, bad_fan, 2);
    EXPECT(gnn_train_step_workspace_size(&bad, 1000, 10, &nb), GNN_EINVAL);
    bad = model(GNN_AGG_SAGE_MEAN, GNN_F16, dims, fan, 2);
    EXPECT(gnn_train_step_workspace_size(&bad, 1000, 10, &nb), GNN_EUNSUPPORTED);
    const int sdims[] = {32, 16, 8}, sfan[] = {5, 5};
    gnn_model s = model(GNN_AGG_SAGE_MEAN, GNN_F32, sdims, sfan, 2);
    for (int l = 0; l < 2; ++l) s.w[l] = s.b[l] = s.dw[l] = s.db[l] = (float *)(uintptr_t)(1u << 20);
    EXPECT(gnn_train_step_layout(&s, 1000, 64, &lay), GNN_OK);
    EXPECT(gnn_step_prepare_workspace_init(&s, 1000, 64, fake, lay.prep_bytes - 256, NULL), GNN_ESIZE);
    EXPECT(gnn_step_compute(&s, 1000, fake, 64, 0.1f, NULL, NULL, fake, lay.prep_bytes, fake, lay.compute_bytes - 256,
                            NULL),
           GNN_ESIZE);
    gnn_graph g2 = {1000, 5000, (const int64_t *)fake, (const int64_t *)fake};
    EXPECT(gnn_step_prepare(&s, NULL, NULL, fake, GNN_F32, GNN_LOC_DEVICE, 32, fake, 64, 0, 0, fake, lay.prep_bytes,
                            NULL),
           GNN_EINVAL);
    void *slots[2] = {fake, (char *)fake + (1 << 22)};
    EXPECT(gnn_train_steps(&s, &g2, NULL, fake, GNN_F32, GNN_LOC_DEVICE, 32, fake, fake, 64, 0, 0, 3, 0.1f, NULL,
                           NULL, slots, 1, lay.prep_bytes, fake, lay.compute_bytes, NULL, NULL),
           GNN_EINVAL);
    EXPECT(gnn_train_steps(&s, &g2, NULL, fake, GNN_F32, GNN_LOC_DEVICE, 32, fake, fake, 64, 0, 0, 3, 0.1f, NULL,
                           NULL, slots, 9, lay.prep_bytes, fake, lay.compute_bytes, NULL, NULL),
           GNN_EINVAL);

    /* device error words: decode on the host */
    EXPECT(gnn_decode_device_errors(0), GNN_OK);
    EXPECT(gnn_decode_device_errors(GNN_DEVERR_WAIT | GNN_DEVERR_RANGE | 0x40), GNN_EDEVICE);
    if (strstr(gnn_last_error(), "unknown flags 0x40") == NULL) return 1;
    EXPECT(gnn_check_device_errors(NULL, NULL), GNN_EINVAL);
    EXPECT(gnn_debug_sampler_fault(-2, 1), GNN_EINVAL);
    EXPECT(gnn_debug_sampler_fault(-1, 0), GNN_OK);
    printf("abi driver: ok\n");
    return 0;
}
