// Dense all-pairs relation without an edge array (Section 1 of the paper: a
// dense relation may need no edge array), softened inverse-square message:
//   y_i = sum_{j != i} q_j (p_j - p_i) (|p_j - p_i|^2 + eps^2)^(-3/2)
//
// VALU-bound.  Each thread owns one destination i; the j range is split into
// kSplit slices (grid.y) so that enough wavefronts are resident, and each
// slice is streamed through LDS in tiles of kTile (p_j, q_j) records.  The
// j = i term is exactly zero (zero displacement, eps > 0), so no branch is
// needed.  Summation is two-level (kInner terms per inner sum) and the slices
// are merged in a fixed order, so every output's serial run stays short.
#include "dense.hpp"

namespace tiga {
namespace dense {

namespace {

constexpr int kBlock = 256;
constexpr int kTile = 256;
constexpr int kInner = 64;

__global__ __launch_bounds__(kBlock) void pack_kernel(const float *__restrict__ pos, const float *__restrict__ q,
                                                      int64_t n, int64_t npad, float4 *__restrict__ pq) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < npad; i += stride) {
        // padding records carry zero charge: they contribute exactly zero
        pq[i] = i < n ? make_float4(pos[i * 3 + 0], pos[i * 3 + 1], pos[i * 3 + 2], q[i])
                      : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
}

__global__ __launch_bounds__(kBlock) void pairs_kernel(const float4 *__restrict__ pq, int64_t n, int64_t slice,
                                                       float eps2, float *__restrict__ part) {
    __shared__ float4 tile[kTile];
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    const float4 pi = pq[i < n ? i : 0];
    const int64_t j0 = static_cast<int64_t>(blockIdx.y) * slice;
    const int64_t j1 = j0 + slice;
    float ox = 0.0f, oy = 0.0f, oz = 0.0f;
    for (int64_t jt = j0; jt < j1; jt += kTile) {
        __syncthreads();
        tile[threadIdx.x] = pq[jt + threadIdx.x];
        __syncthreads();
#pragma unroll 1
        for (int jb = 0; jb < kTile; jb += kInner) {
            float ax = 0.0f, ay = 0.0f, az = 0.0f;
#pragma unroll 8
            for (int j = jb; j < jb + kInner; ++j) {
                const float4 pj = tile[j];
                const float dx = pj.x - pi.x;
                const float dy = pj.y - pi.y;
                const float dz = pj.z - pi.z;
                const float r2 = fmaf(dx, dx, fmaf(dy, dy, fmaf(dz, dz, eps2)));
                const float inv = __builtin_amdgcn_rsqf(r2);
                const float s = pj.w * (inv * inv * inv);
                ax = fmaf(s, dx, ax);
                ay = fmaf(s, dy, ay);
                az = fmaf(s, dz, az);
            }
            ox += ax;
            oy += ay;
            oz += az;
        }
    }
    if (i < n) {
        float *o = part + (static_cast<int64_t>(blockIdx.y) * n + i) * 3;
        o[0] = ox;
        o[1] = oy;
        o[2] = oz;
    }
}

__global__ __launch_bounds__(kBlock) void merge_kernel(const float *__restrict__ part, int64_t n, int nsplit,
                                                       float *__restrict__ y) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (k >= 3 * n) return;
    // pairwise tree over the slices (fixed order)
    float v[64];
    int m = nsplit;
    for (int s = 0; s < m; ++s) v[s] = part[static_cast<int64_t>(s) * 3 * n + k];
    while (m > 1) {
        const int h = (m + 1) / 2;
        for (int s = 0; s + h < m; ++s) v[s] += v[s + h];
        m = h;
    }
    y[k] = v[0];
}

struct Ws {
    float4 *pq;
    float *part;
};

int64_t padded(int64_t n) { return ceil_div(n > 0 ? n : 1, kTile) * kTile; }

int splits_for(int64_t n) {
    // enough wavefronts to fill the chip, at least one tile per slice, at most 64
    const int64_t tiles = padded(n) / kTile;
    int64_t want = ceil_div(static_cast<int64_t>(device_cus()) * 64, ceil_div(n, kBlock) * (kBlock / kWave));
    if (want < 1) want = 1;
    if (want > 64) want = 64;
    if (want > tiles) want = tiles;
    // slices must be whole tiles
    while (tiles % want) --want;
    return static_cast<int>(want);
}

Ws carve(Carve &c, int64_t n, int nsplit) {
    Ws w;
    w.pq = c.take<float4>(padded(n));
    w.part = c.take<float>(static_cast<size_t>(nsplit) * 3 * n);
    return w;
}

}  // namespace

size_t workspace_bytes(int64_t n) {
    Carve c(nullptr);
    carve(c, n, 64);
    return c.bytes();
}

int forward(int64_t n, const float *pos, const float *q, float eps, float *y, void *ws, hipStream_t stream) {
    const int nsplit = splits_for(n);
    Carve c(ws);
    Ws w = carve(c, n, nsplit);
    const int64_t npad = padded(n);
    int pb = static_cast<int>(ceil_div(npad, kBlock));
    hipLaunchKernelGGL(pack_kernel, dim3(pb), dim3(kBlock), 0, stream, pos, q, n, npad, w.pq);
    if (int rc = check_launch("dense pack")) return rc;
    const int64_t slice = npad / nsplit;
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)), static_cast<unsigned>(nsplit));
    prof_before(stream);
    hipLaunchKernelGGL(pairs_kernel, grid, dim3(kBlock), 0, stream, w.pq, n, slice, eps * eps, w.part);
    prof_after(stream);
    if (int rc = check_launch("dense pairs")) return rc;
    hipLaunchKernelGGL(merge_kernel, dim3(static_cast<unsigned>(ceil_div(3 * n, kBlock))), dim3(kBlock), 0, stream,
                       w.part, n, nsplit, y);
    return check_launch("dense merge");
}

}  // namespace dense
}  // namespace tiga
