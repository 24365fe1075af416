// Allocation-free variant of the stored-CSR forward: the traversal's plan and partial states live
// in a fixed device array of this file instead of a caller-provided workspace, so the call makes no
// allocation of any kind (for callers that cannot allocate: code under stream capture, tight
// serving loops, harnesses that forbid allocation).
#include <mutex>

#include "csr_fwd.hpp"

using namespace tiga;

namespace {

// The fixed workspace: one copy per device, held from the first call on that device until the
// process ends.  In host code `scratch` names a host-side stand-in, never the device memory: its
// device address comes from hipGetSymbolAddress, once per device, and only that address is used.
constexpr size_t kScratchBytes = size_t{64} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device (set once)

int scratch_address(void **out) {
    int dev = -1;
    if (int rc = check_hip(hipGetDevice(&dev), "hipGetDevice")) return rc;
    if (dev < 0 || dev >= kMaxDevices) return fail(TIGA_EUNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        if (int rc = check_hip(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"))
            return rc;
        if (!p) return fail(TIGA_EDEVICE, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return TIGA_OK;
}

}  // namespace

extern "C" {

size_t tiga_mp_csr_fwd_noalloc_limit(void) { return kScratchBytes; }

int tiga_mp_csr_fwd_noalloc(const tiga_csr *rel, int32_t feat, const float *x_src, int msg, const float *w_edge,
                            int reducer, float *y, int32_t *argmax, void *stream) {
    {
        EntryScope scope;
        if (!rel) return fail(TIGA_EINVAL, "rel is NULL");
        if (feat < 1) return fail(TIGA_EINVAL, "feat must be >= 1 (got %d)", feat);
        if (reducer != TIGA_REDUCE_SUM && reducer != TIGA_REDUCE_MAX)
            return fail(TIGA_EINVAL, "unknown reducer %d", reducer);
        if (rel->num_dst < 0 || rel->num_edges < 0)
            return fail(TIGA_EINVAL, "negative relation size (num_dst %lld, num_edges %lld)",
                        (long long)rel->num_dst, (long long)rel->num_edges);
        const size_t need = tiga_mp_csr_fwd_workspace(rel, feat, reducer);
        if (need > kScratchBytes)
            return fail(TIGA_EUNSUPPORTED,
                        "the relation needs a %zu-byte workspace; the allocation-free forward holds %zu bytes "
                        "(use tiga_mp_csr_fwd with a caller-provided workspace)",
                        need, kScratchBytes);
    }
    void *ws = nullptr;
    if (int rc = scratch_address(&ws)) return rc;
    // every other check, and the launches, are those of the forward with a workspace; the plan
    // writes every word of the workspace it later reads, so nothing needs clearing between calls
    return tiga_mp_csr_fwd(rel, feat, x_src, msg, w_edge, reducer, y, argmax, ws, kScratchBytes, stream);
}

}  // extern "C"
