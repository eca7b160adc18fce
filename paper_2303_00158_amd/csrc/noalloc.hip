// gnn_update_bwd_noalloc: the update backward with its scratch (the dW
// partial tiles of the split reduction) in a static device array instead of
// a caller workspace, for callers that cannot allocate device memory.
//
// The array lives in the library's code object, one copy per GPU, held from
// the first call on that GPU until the process ends.  Host code never passes
// the array's own name to a kernel: on the host that name is a stand-in, not
// a device address.  The first call on a device looks the copy's address up
// with hipGetSymbolAddress (with that device current) and every later call on
// that device reuses it.
#include <mutex>

#include "internal.h"

namespace gnn {

namespace {

// 32 MiB holds the dW partials of every layer up to K = 2,048 and n_out =
// 256 at any row count, and of wider layers while K x n_out x splits stays
// under the cap (gnn_update_bwd_workspace_size gives the need).
constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Device address of this device's copy of `scratch`, looked up once.
gnn_status scratch_on_current_device(void **out, const char *who) {
    int dev = -1;
    GNN_HIP(hipGetDevice(&dev));
    GNN_CHECK(dev >= 0 && dev < kMaxDevices, GNN_EUNSUPPORTED, "%s: device %d is beyond the %d supported", who, dev,
              kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return fail(GNN_EHIP, "%s: hipGetSymbolAddress of the static scratch failed on device %d: %s", who, dev,
                        hipGetErrorString(e));
        }
        GNN_CHECK(aligned(p, 256), GNN_EHIP, "%s: static scratch is not 256-byte aligned", who);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return GNN_OK;
}

}  // namespace

}  // namespace gnn

using namespace gnn;

extern "C" {

gnn_status gnn_update_bwd_noalloc(const void *a_self, const void *a_nbr, gnn_dtype adt, int64_t k_each,
                                  const int64_t *m_dev, int64_t cap_m, const float *w, const float *g,
                                  int64_t n_out, gnn_dtype gemm_dt, float *dw, float *db, float *d_a,
                                  gnn_stream s) {
    clear_error();
    const char *who = "gnn_update_bwd_noalloc";
    size_t need = 0;
    GNN_TRY(check_update_bwd(a_self, a_nbr, adt, k_each, m_dev, cap_m, w, g, n_out, gemm_dt, dw, db, d_a, &need, who));
    GNN_CHECK(need <= kScratchBytes, GNN_ESIZE,
              "%s: this shape needs %zu bytes of scratch; the static scratch holds %zu (use gnn_update_bwd with a "
              "workspace)",
              who, need, kScratchBytes);
    void *ws = nullptr;
    GNN_TRY(scratch_on_current_device(&ws, who));
    // Every split writes its whole partial tile before the reduction reads
    // it, so nothing in the scratch needs clearing between calls.
    return launch_update_bwd(a_self, a_nbr, adt, k_each, m_dev, cap_m, w, g, n_out, gemm_dt, dw, db, d_a, ws,
                             nullptr, nullptr, nullptr, 0.f, stream_of(s));
}

}  // extern "C"
