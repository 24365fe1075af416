// Error reporting, profiling events and small shared kernels.
#include "common.hpp"

#include <mutex>
#include <vector>

namespace tiga {

namespace {
thread_local char g_error[512] = "";
thread_local hipEvent_t g_prof_start = nullptr;
thread_local hipEvent_t g_prof_stop = nullptr;
thread_local bool g_prof_started = false;
}  // namespace

void set_error(const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
}

void clear_error() { g_error[0] = '\0'; }

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return code;
}

int check_hip(hipError_t err, const char *what) {
    if (err == hipSuccess) return TIGA_OK;
    return fail(TIGA_EDEVICE, "%s: %s", what, hipGetErrorString(err));
}

void prof_before(hipStream_t stream) {
    g_prof_started = false;
    if (g_prof_start && g_prof_stop) {
        if (hipEventRecord(g_prof_start, stream) == hipSuccess) g_prof_started = true;
    }
}

void prof_after(hipStream_t stream) {
    if (g_prof_started) (void)hipEventRecord(g_prof_stop, stream);
    g_prof_started = false;
    g_prof_start = nullptr;
    g_prof_stop = nullptr;
}

void prof_disarm() {
    g_prof_started = false;
    g_prof_start = nullptr;
    g_prof_stop = nullptr;
}

int device_cus() {
    static std::mutex mu;
    static std::vector<int> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    std::lock_guard<std::mutex> lk(mu);
    if (dev >= static_cast<int>(cache.size())) cache.resize(dev + 1, 0);
    if (cache[dev] == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        cache[dev] = cus;
    }
    return cache[dev];
}

int resident_blocks(const void *kernel, int block) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, block, 0) != hipSuccess || n < 1) n = 1;
    return n;
}

__global__ void fill_u32_kernel(uint32_t *p, uint32_t v, int64_t n) {
    int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (; i < n; i += stride) p[i] = v;
}

int fill_u32(void *p, uint32_t v, int64_t n, hipStream_t stream) {
    if (n <= 0) return TIGA_OK;
    int64_t blocks = ceil_div(n, 256);
    const int64_t cap = static_cast<int64_t>(device_cus()) * 16;
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                       static_cast<uint32_t *>(p), v, n);
    return check_launch("fill");
}

}  // namespace tiga

extern "C" {

const char *tiga_last_error(void) { return tiga::g_error; }

int tiga_mp_abi_version(void) { return TIGA_MP_ABI_VERSION; }

int tiga_mp_set_kernel_events(void *start, void *stop) {
    tiga::g_prof_start = static_cast<hipEvent_t>(start);
    tiga::g_prof_stop = static_cast<hipEvent_t>(stop);
    tiga::g_prof_started = false;
    return TIGA_OK;
}

}  // extern "C"
