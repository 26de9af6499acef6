// gcn_aggregate_noalloc: the feature propagation of gcn_aggregate for callers
// that cannot allocate device memory (code under graph capture, tight serving
// loops).  Its scratch -- the merge-path row ranges and the partial sums of
// rows cut by wavefront boundaries, and with GCN_BF16 the bfloat16 copy of
// the gathered rows -- lives in one file-scope device array instead of a
// caller workspace.  The kernels are those of gcn_aggregate; they get the
// array's device address as their workspace argument.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.h"

namespace {

// One copy per GPU, held by the loaded library until the process ends.
static __device__ __align__(256) unsigned char scratch[GCN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_ptr[kMaxDevices];   // device address of `scratch` on each device, once known

// The address of this device's copy of `scratch`.  In host code the array's
// name is only a stand-in, so the address is asked of the runtime, once per
// device, with that device current.
int scratch_on(int dev, void **out) {
    if (dev < 0 || dev >= kMaxDevices) {
        gcn::set_error("gcn_aggregate_noalloc: device %d beyond the %d the library tracks", dev, kMaxDevices);
        return GCN_EUNSUPPORTED;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        int cur = -1;
        GCN_HIP_CHECK(hipGetDevice(&cur));
        if (cur != dev) GCN_HIP_CHECK(hipSetDevice(dev));
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess && e2 != hipSuccess) return gcn::hip_fail(e2, "hipSetDevice (restore)");
        }
        if (e != hipSuccess) return gcn::hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) {
            gcn::set_error("gcn_aggregate_noalloc: no device address for the scratch array");
            return GCN_EHIP;
        }
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return GCN_OK;
}

}  // namespace

extern "C" int gcn_aggregate_noalloc(const gcn_csr *A, const float *X, int32_t k, int32_t ldx, float *out,
                                     int32_t ldo, gcn_prec prec, void *stream) {
    if (!A) {
        gcn::set_error("gcn_aggregate_noalloc: null CSR");
        return GCN_EINVAL;
    }
    if (A->n_rows < 0 || A->n_cols < 0 || A->nnz < 0 || k < 0) {
        gcn::set_error("gcn_aggregate_noalloc: negative size");
        return GCN_ESHAPE;
    }
    if (A->n_rows == 0 || k == 0) return gcn_aggregate(A, X, k, ldx, out, ldo, prec, nullptr, 0, stream);
    const size_t need = gcn_aggregate_workspace_bytes(A->n_rows, A->n_cols, A->nnz, k, prec);
    if (need > (size_t)GCN_NOALLOC_SCRATCH_BYTES) {
        gcn::set_error("gcn_aggregate_noalloc: needs %zu bytes of scratch, more than its %zu-byte array "
                       "(use gcn_aggregate with a workspace)", need, (size_t)GCN_NOALLOC_SCRATCH_BYTES);
        return GCN_EUNSUPPORTED;
    }
    // the device the work goes to: the stream's, or the current one
    int dev = -1;
    if (stream) GCN_HIP_CHECK(hipStreamGetDevice((hipStream_t)stream, &dev));
    else GCN_HIP_CHECK(hipGetDevice(&dev));
    void *ptr = nullptr;
    int rc = scratch_on(dev, &ptr);
    if (rc) return rc;
    gcn::ProfSuppress quiet;   // no timing events: nothing is created on this path
    return gcn_aggregate(A, X, k, ldx, out, ldo, prec, ptr, (size_t)GCN_NOALLOC_SCRATCH_BYTES, stream);
}
