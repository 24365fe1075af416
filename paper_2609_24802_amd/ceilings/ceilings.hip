// Hardware ceilings for the fused message-passing kernels on one MI355X.
//
// Measures, with HIP events (best of 3), on data resident in HBM:
//   stream_read   : 4 GiB read with 16-B non-temporal loads
//   stream_copy   : 4 GiB read + 4 GiB written
//   gather_64     : random 64-B rows (4 lanes x 16 B) from a 3.2 GB table,
//                   indices streamed from a 4 GB array (the CSR forward pattern)
//   gather_32, gather_128, gather_256 : the same with 32-, 128- and 256-B rows
//   gather_64 from a 64 MB table and from a 256 MB table (held in the
//                   last-level cache, so DRAM is not what limits them)
//   fma           : fp32 FMA chains (non-packed), 8 independent chains per lane
//   rsq, exp      : transcendental throughput (v_rsq_f32, v_exp_f32)
// and prints one JSON object.  Index arrays are filled on the device with a
// hash reduced modulo the table's row count, so every access is in bounds.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>

#define CHECK(x)                                                                             \
    do {                                                                                     \
        hipError_t e_ = (x);                                                                 \
        if (e_ != hipSuccess) {                                                              \
            fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            exit(1);                                                                         \
        }                                                                                    \
    } while (0)

typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

__device__ __forceinline__ uint32_t mix(uint64_t x) {
    x ^= x >> 33;
    x *= 0xff51afd7ed558ccdULL;
    x ^= x >> 33;
    x *= 0xc4ceb9fe1a85ec53ULL;
    x ^= x >> 33;
    return static_cast<uint32_t>(x);
}

__global__ void init_idx(int32_t *idx, int64_t n, uint32_t rows) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        idx[i] = static_cast<int32_t>(mix(static_cast<uint64_t>(i) + 12345) % rows);
}

__global__ void fill(f32x4 *p, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = f32x4{1.0f, 0.5f, 0.25f, static_cast<float>(i & 7)};
}

__global__ __launch_bounds__(256) void stream_read(const f32x4 *__restrict__ a, int64_t n, float *out) {
    f32x4 acc = {0, 0, 0, 0};
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        acc += __builtin_nontemporal_load(a + i);
    out[blockIdx.x * 256 + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

__global__ __launch_bounds__(256) void stream_copy(const f32x4 *__restrict__ a, f32x4 *__restrict__ b, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        __builtin_nontemporal_store(__builtin_nontemporal_load(a + i), b + i);
}

// LPR lanes of 16 B per row; U rows in flight per lane.  CASE only tells the measurements apart in
// a profiler's per-kernel tables (same code for every case).
template <int LPR, int CASE, int U = 4>
__global__ __launch_bounds__(256) void gather_rows(const int32_t *__restrict__ idx, const f32x4 *__restrict__ tab,
                                                   int64_t n, float *out) {
    constexpr int S = 64 / LPR;
    const int lane = threadIdx.x & 63;
    const int slot = lane / LPR, q = lane % LPR;
    const int64_t wave = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t nw = (int64_t)gridDim.x * 4;
    f32x4 acc = {0, 0, 0, 0};
    for (int64_t base = wave * S * U; base < n; base += nw * S * U) {
        int32_t c[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t e = base + u * S + slot;
            c[u] = e < n ? __builtin_nontemporal_load(idx + e) : 0;
        }
        f32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = tab[(int64_t)c[u] * LPR + q];
#pragma unroll
        for (int u = 0; u < U; ++u) acc += v[u];
    }
    out[blockIdx.x * 256 + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

constexpr int kIters = 4096;

__global__ __launch_bounds__(256) void fma_loop(float *out, float a) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = threadIdx.x * 1e-3f + k;
    for (int i = 0; i < kIters; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = fmaf(x[k], a, 0.5f);
    float s = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) s += x[k];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void rsq_loop(float *out, float a) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = 1.0f + threadIdx.x * 1e-3f + k;
    for (int i = 0; i < kIters; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = __builtin_amdgcn_rsqf(x[k] + a);
    float s = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) s += x[k];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void exp_loop(float *out, float a) {
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = -1e-3f * (threadIdx.x + k);
    for (int i = 0; i < kIters; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = __builtin_amdgcn_exp2f(x[k] * a);
    float s = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) s += x[k];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

template <class F>
float best_ms(F f) {
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    f();
    CHECK(hipDeviceSynchronize());
    float best = 1e30f;
    for (int r = 0; r < 3; ++r) {
        CHECK(hipEventRecord(a));
        f();
        CHECK(hipEventRecord(b));
        CHECK(hipEventSynchronize(b));
        float ms;
        CHECK(hipEventElapsedTime(&ms, a, b));
        if (ms < best) best = ms;
    }
    CHECK(hipEventDestroy(a));
    CHECK(hipEventDestroy(b));
    return best;
}

}  // namespace

int main() {
    hipDeviceProp_t p;
    CHECK(hipGetDeviceProperties(&p, 0));
    const int cus = p.multiProcessorCount;
    const int grid = cus * 8;
    const int64_t idx_n = 1000000000;         // 4 GB of indices
    const int64_t tab_bytes = 3200000000LL;   // 50M rows of 64 B
    int32_t *idx;
    f32x4 *tab, *cp;
    float *out;
    CHECK(hipMalloc(&idx, idx_n * 4));
    CHECK(hipMalloc(&tab, tab_bytes));
    CHECK(hipMalloc(&cp, idx_n * 4));
    CHECK(hipMalloc(&out, static_cast<size_t>(grid) * 256 * 4 * 64));
    hipLaunchKernelGGL(fill, dim3(grid), dim3(256), 0, 0, tab, tab_bytes / 16);
    CHECK(hipDeviceSynchronize());

    const int64_t n4 = idx_n / 4;  // float4 elements in 4 GB
    hipLaunchKernelGGL(fill, dim3(grid), dim3(256), 0, 0, reinterpret_cast<f32x4 *>(idx), n4);
    const float t_read = best_ms([&] {
        hipLaunchKernelGGL(stream_read, dim3(grid), dim3(256), 0, 0, reinterpret_cast<const f32x4 *>(idx), n4, out);
    });
    const float t_copy = best_ms([&] {
        hipLaunchKernelGGL(stream_copy, dim3(grid), dim3(256), 0, 0, reinterpret_cast<const f32x4 *>(idx), cp, n4);
    });

    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, idx_n, static_cast<uint32_t>(tab_bytes / 64));
    const float t_g64 = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<4, 64>), dim3(grid), dim3(256), 0, 0, idx, tab, idx_n, out);
    });
    // occupancy: the same 64-byte gathers with 1 row in flight per lane, and with 1/8, 1/4 and 1/2
    // of the grid (256 CUs x 8 blocks of 4 wavefronts), i.e. 1, 2 and 4 wavefronts per SIMD
    const float t_g64_u1 = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<4, 641, 1>), dim3(grid), dim3(256), 0, 0, idx, tab, idx_n, out);
    });
    float t_g64_grid[3];
    for (int k = 0; k < 3; ++k)
        t_g64_grid[k] = best_ms([&] {
            hipLaunchKernelGGL((gather_rows<4, 6400>), dim3(grid >> (3 - k)), dim3(256), 0, 0, idx, tab, idx_n, out);
        });
    const int64_t n128 = idx_n / 2;
    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, n128, static_cast<uint32_t>(tab_bytes / 128));
    const float t_g128 = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<8, 128>), dim3(grid), dim3(256), 0, 0, idx, tab, n128, out);
    });
    const int64_t n256 = idx_n / 4;
    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, n256, static_cast<uint32_t>(tab_bytes / 256));
    const float t_g256 = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<16, 256>), dim3(grid), dim3(256), 0, 0, idx, tab, n256, out);
    });
    const int64_t n32 = idx_n / 2;
    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, n32, static_cast<uint32_t>(tab_bytes / 32));
    const float t_g32 = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<2, 32>), dim3(grid), dim3(256), 0, 0, idx, tab, n32, out);
    });
    // 64-B rows from tables of 64 MB and 256 MB: these stay in the 256 MB last-level cache
    const int64_t nsm = idx_n / 2;
    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, nsm, static_cast<uint32_t>((64LL << 20) / 64));
    const float t_g64_64m = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<4, 6464>), dim3(grid), dim3(256), 0, 0, idx, tab, nsm, out);
    });
    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, nsm, static_cast<uint32_t>((256LL << 20) / 64));
    const float t_g64_256m = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<4, 64256>), dim3(grid), dim3(256), 0, 0, idx, tab, nsm, out);
    });
    // and from a 2 MB table, which every XCD's 4 MB L2 holds: no request leaves the XCD
    hipLaunchKernelGGL(init_idx, dim3(grid), dim3(256), 0, 0, idx, nsm, static_cast<uint32_t>((2LL << 20) / 64));
    const float t_g64_2m = best_ms([&] {
        hipLaunchKernelGGL((gather_rows<4, 642>), dim3(grid), dim3(256), 0, 0, idx, tab, nsm, out);
    });

    const int vgrid = cus * 64;
    const double lanes = static_cast<double>(vgrid) * 256;
    const float t_fma = best_ms([&] { hipLaunchKernelGGL(fma_loop, dim3(vgrid), dim3(256), 0, 0, out, 0.999f); });
    const float t_rsq = best_ms([&] { hipLaunchKernelGGL(rsq_loop, dim3(vgrid), dim3(256), 0, 0, out, 0.5f); });
    const float t_exp = best_ms([&] { hipLaunchKernelGGL(exp_loop, dim3(vgrid), dim3(256), 0, 0, out, 0.999f); });
    const double ops = lanes * kIters * 8;

    printf("{\"device\": \"%s\", \"cus\": %d, "
           "\"stream_read_gbs\": %.1f, \"stream_copy_gbs\": %.1f, "
           "\"gather64_rows_per_s\": %.4g, \"gather64_useful_gbs\": %.1f, "
           "\"gather128_rows_per_s\": %.4g, \"gather128_useful_gbs\": %.1f, "
           "\"gather32_rows_per_s\": %.4g, \"gather256_rows_per_s\": %.4g, \"gather256_useful_gbs\": %.1f, "
           "\"gather64_table2mb_rows_per_s\": %.4g, "
           "\"gather64_table64mb_rows_per_s\": %.4g, \"gather64_table256mb_rows_per_s\": %.4g, "
           "\"gather64_one_in_flight_rows_per_s\": %.4g, \"gather64_waves_per_simd_1_2_4_rows_per_s\": [%.4g, %.4g, %.4g], "
           "\"fma_fp32_tflops\": %.2f, \"rsq_per_s\": %.4g, \"exp_per_s\": %.4g}\n",
           p.gcnArchName, cus, idx_n * 4.0 / t_read / 1e6, idx_n * 8.0 / t_copy / 1e6, idx_n / (t_g64 * 1e-3),
           idx_n * 68.0 / t_g64 / 1e6, n128 / (t_g128 * 1e-3), n128 * 132.0 / t_g128 / 1e6,
           n32 / (t_g32 * 1e-3), n256 / (t_g256 * 1e-3), n256 * 260.0 / t_g256 / 1e6, nsm / (t_g64_2m * 1e-3),
           nsm / (t_g64_64m * 1e-3),
           nsm / (t_g64_256m * 1e-3), idx_n / (t_g64_u1 * 1e-3), idx_n / (t_g64_grid[0] * 1e-3),
           idx_n / (t_g64_grid[1] * 1e-3), idx_n / (t_g64_grid[2] * 1e-3),
           2.0 * ops / (t_fma * 1e-3) / 1e12, ops / (t_rsq * 1e-3), ops / (t_exp * 1e-3));
    CHECK(hipFree(idx));
    CHECK(hipFree(tab));
    CHECK(hipFree(cp));
    CHECK(hipFree(out));
    return 0;
}
