// Generated radius relation (Section 4.9 of the paper): a uniform cell
// directory restricts candidates, an exact fp32 distance predicate accepts,
// and accepted messages are folded into registers without storing edges.
//
// Build (every call, stateless):
//   bounding box -> cell size h >= r (1 + 2^-10), at most n + 64 cells ->
//   cell id per point (fp64 coordinates) -> counts -> exclusive scan ->
//   scatter (counting sort) -> per-cell sort by point id (deterministic order)
//   -> cell-ordered records (p, id) and feature rows.
// Consume: one thread per destination point in cell order; the 27 neighbour
// cells are 9 contiguous runs of the cell-ordered arrays (x-adjacent cells are
// adjacent in memory).
#include "csr_bwd.hpp"
#include "radius.hpp"

namespace tiga {
namespace radius {

using csr::launch_excl_scan;
using csr::scan_ws_bytes;

namespace {

constexpr int kBlock = 256;

struct Params {
    double lo[3];
    double inv_h;
    int dim[3];
    int ncell;
};

__global__ __launch_bounds__(kBlock) void bbox_partial_kernel(const float *__restrict__ pos, int64_t n,
                                                              float *__restrict__ part) {
    float mn[3] = {__builtin_inff(), __builtin_inff(), __builtin_inff()};
    float mx[3] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            const float v = pos[i * 3 + a];
            mn[a] = fminf(mn[a], v);
            mx[a] = fmaxf(mx[a], v);
        }
    }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], shfl_xor_f(mn[a], m));
            mx[a] = fmaxf(mx[a], shfl_xor_f(mx[a], m));
        }
    __shared__ float sh[kBlock / kWave][6];
    const int wave = threadIdx.x / kWave;
    if (lane_id() == 0)
        for (int a = 0; a < 3; ++a) {
            sh[wave][a] = mn[a];
            sh[wave][3 + a] = mx[a];
        }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kBlock / kWave; ++w)
            for (int a = 0; a < 3; ++a) {
                sh[0][a] = fminf(sh[0][a], sh[w][a]);
                sh[0][3 + a] = fmaxf(sh[0][3 + a], sh[w][3 + a]);
            }
        for (int k = 0; k < 6; ++k) part[blockIdx.x * 6 + k] = sh[0][k];
    }
}

// One block: reduce the per-block boxes, then thread 0 picks the cell size and
// the grid dimensions.
__global__ __launch_bounds__(kBlock) void grid_params_kernel(const float *__restrict__ part, int nblocks, int64_t n,
                                                             float radius, int64_t max_cells,
                                                             Params *__restrict__ prm) {
    float mn[3] = {__builtin_inff(), __builtin_inff(), __builtin_inff()};
    float mx[3] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    for (int b = threadIdx.x; b < nblocks; b += blockDim.x)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], part[b * 6 + a]);
            mx[a] = fmaxf(mx[a], part[b * 6 + 3 + a]);
        }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], shfl_xor_f(mn[a], m));
            mx[a] = fmaxf(mx[a], shfl_xor_f(mx[a], m));
        }
    __shared__ float sh[kBlock / kWave][6];
    if (lane_id() == 0)
        for (int a = 0; a < 3; ++a) {
            sh[threadIdx.x / kWave][a] = mn[a];
            sh[threadIdx.x / kWave][3 + a] = mx[a];
        }
    __syncthreads();
    if (threadIdx.x != 0) return;
    double lo[3], hi[3];
    for (int a = 0; a < 3; ++a) {
        lo[a] = sh[0][a];
        hi[a] = sh[0][3 + a];
        for (int w = 1; w < kBlock / kWave; ++w) {
            lo[a] = fmin(lo[a], static_cast<double>(sh[w][a]));
            hi[a] = fmax(hi[a], static_cast<double>(sh[w][3 + a]));
        }
    }
    double ext[3], vol = 1.0;
    for (int a = 0; a < 3; ++a) {
        ext[a] = hi[a] - lo[a];
        if (!(ext[a] >= 0.0)) ext[a] = 0.0;
        vol *= ext[a];
    }
    // cells no smaller than the radius (with a relative margin that covers the
    // fp32 rounding of the predicate), and not much smaller than the mean
    // point spacing; grown until the directory has at most max_cells cells
    double h = static_cast<double>(radius) * (1.0 + 1.0 / 1024.0);
    const double spacing = cbrt(vol / static_cast<double>(n > 0 ? n : 1));
    if (spacing > h) h = spacing;
    int64_t d[3] = {1, 1, 1};
    bool fits = false;
    for (int it = 0; it < 200 && !fits; ++it) {
        int64_t cells = 1;
        for (int a = 0; a < 3; ++a) {
            const double t = floor(ext[a] / h) + 1.0;
            d[a] = t > 2e9 ? static_cast<int64_t>(2e9) : static_cast<int64_t>(t);
            cells = (cells > (int64_t{1} << 40)) ? cells : cells * d[a];
        }
        fits = cells <= max_cells;
        if (!fits) h *= 1.25;
    }
    if (!fits) {
        // unreachable for finite positions; one cell keeps the scan correct
        d[0] = d[1] = d[2] = 1;
        h = 1.0 + ext[0] + ext[1] + ext[2];
    }
    for (int a = 0; a < 3; ++a) {
        prm->lo[a] = lo[a];
        prm->dim[a] = static_cast<int>(d[a]);
    }
    prm->inv_h = 1.0 / h;
    prm->ncell = static_cast<int>(d[0] * d[1] * d[2]);
}

__device__ __forceinline__ int cell_axis(const Params &p, int a, float v) {
    double t = floor((static_cast<double>(v) - p.lo[a]) * p.inv_h);
    int c = static_cast<int>(t);
    if (t < 0.0) c = 0;
    if (c >= p.dim[a]) c = p.dim[a] - 1;
    return c;
}

__global__ __launch_bounds__(kBlock) void cell_count_kernel(const float *__restrict__ pos, int64_t n,
                                                            const Params *__restrict__ prm,
                                                            int32_t *__restrict__ cell,
                                                            unsigned long long *__restrict__ count) {
    const Params p = *prm;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int cx = cell_axis(p, 0, pos[i * 3 + 0]);
        const int cy = cell_axis(p, 1, pos[i * 3 + 1]);
        const int cz = cell_axis(p, 2, pos[i * 3 + 2]);
        const int c = (cz * p.dim[1] + cy) * p.dim[0] + cx;
        cell[i] = c;
        atomicAdd(&count[c], 1ull);
    }
}

__global__ __launch_bounds__(kBlock) void cell_scatter_kernel(const int32_t *__restrict__ cell, int64_t n,
                                                              const int64_t *__restrict__ start,
                                                              unsigned int *__restrict__ cursor,
                                                              int32_t *__restrict__ perm) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int c = cell[i];
        perm[start[c] + atomicAdd(&cursor[c], 1u)] = static_cast<int32_t>(i);
    }
}

// Sort the point ids of each cell ascending so that the candidate order (and
// hence every summation order) depends only on the input.  A wavefront per
// cell computes each element's rank; cells beyond kSortMax points keep the
// order of the scatter (still correct, not bit-reproducible).
constexpr int kSortMax = 4096;

__global__ __launch_bounds__(kBlock) void cell_sort_kernel(const int64_t *__restrict__ start,
                                                           const Params *__restrict__ prm,
                                                           const int32_t *__restrict__ perm_in,
                                                           int32_t *__restrict__ perm_out) {
    const int ncell = prm->ncell;
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t c = wave; c < ncell; c += nwaves) {
        const int64_t b = start[c], e = start[c + 1], d = e - b;
        if (d > kSortMax) {
            for (int64_t k = b + lane_id(); k < e; k += kWave) perm_out[k] = perm_in[k];
            continue;
        }
        for (int64_t k = b + lane_id(); k < e; k += kWave) {
            const int32_t v = perm_in[k];
            int64_t rank = 0;
            for (int64_t m = b; m < e; ++m) rank += perm_in[m] < v;
            perm_out[b + rank] = v;
        }
    }
}

// Cell-ordered records and feature rows (one thread per 16-byte unit when the
// width allows it, else per float).
__global__ __launch_bounds__(kBlock) void gather_records_kernel(const int32_t *__restrict__ perm, int64_t n,
                                                                const float *__restrict__ pos,
                                                                float4 *__restrict__ rec) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; s < n; s += stride) {
        const int32_t i = perm[s];
        rec[s] = make_float4(pos[i * 3 + 0], pos[i * 3 + 1], pos[i * 3 + 2], __int_as_float(i));
    }
}

// I is the index type of the (row, unit) enumeration: 32-bit division when the
// product fits, which is the common case.
template <int K, class I>
__global__ __launch_bounds__(kBlock) void gather_rows_kernel(const int32_t *__restrict__ perm, I total, I fu,
                                                             const float *__restrict__ a, const float *__restrict__ b,
                                                             float *__restrict__ as, float *__restrict__ bs) {
    const I stride = static_cast<I>(gridDim.x) * blockDim.x;
    for (I k = static_cast<I>(blockIdx.x) * blockDim.x + threadIdx.x; k < total; k += stride) {
        const I s = k / fu;
        const I u = k - s * fu;
        const int64_t src = static_cast<int64_t>(perm[s]) * fu + u;
        if (a) {
            const csr::Vec<K> v = csr::load_unit<K>(a, src);
            csr::store_unit<K>(as, static_cast<int64_t>(k), v.v);
        }
        if (b) {
            const csr::Vec<K> v = csr::load_unit<K>(b, src);
            csr::store_unit<K>(bs, static_cast<int64_t>(k), v.v);
        }
    }
}

template <int K>
int launch_gather_rows(const int32_t *perm, int64_t n, int64_t fu, const float *a, const float *b, float *as,
                       float *bs, hipStream_t stream);

// Exact membership test: direct fp32 differences, products and sums, each
// rounded once (no contraction), strict comparison with fp32(r*r).
__device__ __forceinline__ bool accept(float4 pi, float4 pj, float r2, float &d2) {
#pragma clang fp contract(off)
    const float dx = pj.x - pi.x;
    const float dy = pj.y - pi.y;
    const float dz = pj.z - pi.z;
    const float sx = dx * dx;
    const float sy = dy * dy;
    const float sz = dz * dz;
    d2 = (sx + sy) + sz;
    return d2 < r2;
}

// Visit the candidate runs of the point with record `pi`.
template <class F>
__device__ __forceinline__ void for_candidates(const Params &p, const int64_t *__restrict__ start, float4 pi,
                                               F &&body) {
    const int cx = cell_axis(p, 0, pi.x);
    const int cy = cell_axis(p, 1, pi.y);
    const int cz = cell_axis(p, 2, pi.z);
    const int x0 = cx > 0 ? cx - 1 : 0;
    const int x1 = cx + 1 < p.dim[0] ? cx + 1 : p.dim[0] - 1;
    for (int z = cz - 1; z <= cz + 1; ++z) {
        if (z < 0 || z >= p.dim[2]) continue;
        for (int y = cy - 1; y <= cy + 1; ++y) {
            if (y < 0 || y >= p.dim[1]) continue;
            const int rowc = (z * p.dim[1] + y) * p.dim[0];
            const int64_t b = start[rowc + x0];
            const int64_t e = start[rowc + x1 + 1];
            for (int64_t t = b; t < e; ++t) body(t);
        }
    }
}

// FB float4 units of features per pass (a feature block), scalar tail handled
// by the K = 1 instantiation.
template <int K, int NU>
__global__ __launch_bounds__(kBlock) void radius_fwd_kernel(const Params *__restrict__ prm,
                                                            const int64_t *__restrict__ start,
                                                            const float4 *__restrict__ rec,
                                                            const float *__restrict__ xs, int64_t n, int64_t fu,
                                                            float r2, float neg_inv_s2, float *__restrict__ y,
                                                            int32_t *__restrict__ count) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    for (int64_t fb = 0; fb < fu; fb += NU) {
        float acc[NU][K];
#pragma unroll
        for (int u = 0; u < NU; ++u)
#pragma unroll
            for (int k = 0; k < K; ++k) acc[u][k] = 0.0f;
        int cnt = 0;
        for_candidates(p, start, pi, [&](int64_t t) {
            const float4 pj = rec[t];
            float d2;
            if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) {
                ++cnt;
                const float kw = __expf(d2 * neg_inv_s2);
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    if (fb + u < fu) {
                        csr::Vec<K> xv = csr::load_unit<K>(xs, t * fu + fb + u);
#pragma unroll
                        for (int k = 0; k < K; ++k) acc[u][k] = fmaf(kw, xv.v[k], acc[u][k]);
                    }
                }
            }
        });
#pragma unroll
        for (int u = 0; u < NU; ++u)
            if (fb + u < fu) csr::store_unit<K>(y, static_cast<int64_t>(i) * fu + fb + u, acc[u]);
        if (fb == 0 && count) count[i] = cnt;
    }
}

// Backward: dx_i = sum k_ij dy_j and dp_i = sum (2 k_ij / sigma^2)(p_j - p_i)
// (<dy_i, x_j> + <dy_j, x_i>), one thread per destination point.
template <int K, int NU, bool DX, bool DP>
__global__ __launch_bounds__(kBlock) void radius_bwd_kernel(const Params *__restrict__ prm,
                                                            const int64_t *__restrict__ start,
                                                            const float4 *__restrict__ rec,
                                                            const float *__restrict__ xs,
                                                            const float *__restrict__ ys, int64_t n, int64_t fu,
                                                            float r2, float neg_inv_s2, float two_inv_s2,
                                                            float *__restrict__ dx, float *__restrict__ dp) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    float gp[3] = {0.0f, 0.0f, 0.0f};
    for (int64_t fb = 0; fb < fu; fb += NU) {
        float gi[NU][K], xi[NU][K], acc[NU][K];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            csr::Vec<K> a, b;
            if (fb + u < fu) {
                a = csr::load_unit<K>(ys, s * fu + fb + u);
                if (DP) {
                    b = csr::load_unit<K>(xs, s * fu + fb + u);
                } else {
#pragma unroll
                    for (int k = 0; k < K; ++k) b.v[k] = 0.0f;
                }
            } else {
#pragma unroll
                for (int k = 0; k < K; ++k) a.v[k] = b.v[k] = 0.0f;
            }
#pragma unroll
            for (int k = 0; k < K; ++k) {
                gi[u][k] = a.v[k];
                xi[u][k] = b.v[k];
                acc[u][k] = 0.0f;
            }
        }
        float blk[3] = {0.0f, 0.0f, 0.0f};
        for_candidates(p, start, pi, [&](int64_t t) {
            const float4 pj = rec[t];
            float d2;
            if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) {
                const float kw = __expf(d2 * neg_inv_s2);
                float dot = 0.0f;
#pragma unroll
                for (int u = 0; u < NU; ++u) {
                    if (fb + u < fu) {
                        csr::Vec<K> gj = csr::load_unit<K>(ys, t * fu + fb + u);
                        csr::Vec<K> xj;
                        if (DP) xj = csr::load_unit<K>(xs, t * fu + fb + u);
#pragma unroll
                        for (int k = 0; k < K; ++k) {
                            if (DX) acc[u][k] = fmaf(kw, gj.v[k], acc[u][k]);
                            if (DP) dot = fmaf(gi[u][k], xj.v[k], fmaf(gj.v[k], xi[u][k], dot));
                        }
                    }
                }
                if (DP) {
                    const float c = two_inv_s2 * kw * dot;
                    blk[0] = fmaf(c, pj.x - pi.x, blk[0]);
                    blk[1] = fmaf(c, pj.y - pi.y, blk[1]);
                    blk[2] = fmaf(c, pj.z - pi.z, blk[2]);
                }
            }
        });
        if (DX) {
#pragma unroll
            for (int u = 0; u < NU; ++u)
                if (fb + u < fu) csr::store_unit<K>(dx, static_cast<int64_t>(i) * fu + fb + u, acc[u]);
        }
        gp[0] += blk[0];
        gp[1] += blk[1];
        gp[2] += blk[2];
    }
    if (DP) {
        dp[static_cast<int64_t>(i) * 3 + 0] = gp[0];
        dp[static_cast<int64_t>(i) * 3 + 1] = gp[1];
        dp[static_cast<int64_t>(i) * 3 + 2] = gp[2];
    }
}

// ---------------------------------------------------------------------------
// Wave-cooperative consume (16-byte feature units).
//
// A wavefront owns 64 consecutive destinations in cell order.  Phase 1: each
// lane walks the candidate runs of its destination, tests them and appends the
// accepted (cell-ordered index, kernel weight) pairs to its column of an LDS
// list, until the list is nearly full or the runs are exhausted.  Phase 2: the
// wave splits into groups of LPR lanes; a group takes one destination at a
// time and reads each listed neighbour's feature row as LPR consecutive
// 16-byte units (one coalesced row per group), accumulating in registers.  The
// two phases alternate until every lane's runs are exhausted.  The summation
// order is the candidate order, so results are reproducible.
constexpr int kCap = 24;    // list entries per destination between flushes
constexpr int kStep = 8;    // candidates tested per step of a lane
constexpr int kBatch = 8;   // list entries whose rows are loaded together
constexpr int kBatchDp = 2; // the same when position gradients are formed (more live registers)

struct Cursor {
    int cx0, cx1, cy, cz;
    int k;  // next run (z, y) = (cz - 1 + k / 3, cy - 1 + k % 3)
    int32_t t, e;
};

// Load the bounds of the next non-empty run; false when none is left.
__device__ __forceinline__ bool next_run(const Params &p, const int64_t *__restrict__ start, Cursor &c) {
    while (c.k < 9) {
        const int z = c.cz - 1 + c.k / 3;
        const int y = c.cy - 1 + c.k % 3;
        ++c.k;
        if (z < 0 || z >= p.dim[2] || y < 0 || y >= p.dim[1]) continue;
        const int rowc = (z * p.dim[1] + y) * p.dim[0];
        c.t = static_cast<int32_t>(start[rowc + c.cx0]);
        c.e = static_cast<int32_t>(start[rowc + c.cx1 + 1]);
        if (c.t < c.e) return true;
    }
    c.t = c.e = 0;
    return false;
}

__device__ __forceinline__ bool open_cursor(const Params &p, const int64_t *__restrict__ start, float4 pi,
                                            Cursor &c) {
    const int cx = cell_axis(p, 0, pi.x);
    c.cy = cell_axis(p, 1, pi.y);
    c.cz = cell_axis(p, 2, pi.z);
    c.cx0 = cx > 0 ? cx - 1 : 0;
    c.cx1 = cx + 1 < p.dim[0] ? cx + 1 : p.dim[0] - 1;
    c.k = 0;
    return next_run(p, start, c);
}

// Phase 1 for one lane: append accepted candidates to its column until the
// column is full or the runs are exhausted; the cursor stops right after the
// last candidate taken.  Returns the number of entries written.
__device__ __forceinline__ int fill_list(const Params &p, const int64_t *__restrict__ start,
                                         const float4 *__restrict__ rec, float4 pi, int32_t i, float r2,
                                         float neg_inv_s2, Cursor &c, bool &live, float2 (*list)[kWave], int lane) {
    int m = 0;
    while (live && m < kCap) {
        float4 pj[kStep];
#pragma unroll
        for (int u = 0; u < kStep; ++u)
            pj[u] = c.t + u < c.e ? rec[c.t + u] : make_float4(0.0f, 0.0f, 0.0f, __int_as_float(i));
        int32_t next = c.t + kStep;
#pragma unroll
        for (int u = 0; u < kStep; ++u) {
            float d2;
            if (accept(pi, pj[u], r2, d2) && __float_as_int(pj[u].w) != i) {
                if (m < kCap) {
                    list[m][lane] = make_float2(__int_as_float(c.t + u), __expf(d2 * neg_inv_s2));
                    ++m;
                } else if (next > c.t + u) {
                    next = c.t + u;  // resume here after the flush
                }
            }
        }
        c.t = next;
        if (c.t >= c.e) live = next_run(p, start, c);
    }
    return m;
}

__device__ __forceinline__ void lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ f32x4 unit4(const float *__restrict__ base, int64_t unit) {
    return reinterpret_cast<const f32x4 *>(base)[unit];
}

// y_i = sum_j k_ij x_j over the radius relation; LPR lanes per row, UPL units
// per lane, feature blocks of LPR * UPL units.
template <int LPR, int UPL>
__global__ __launch_bounds__(kBlock) void radius_fwd_coop_kernel(const Params *__restrict__ prm,
                                                                 const int64_t *__restrict__ start,
                                                                 const float4 *__restrict__ rec,
                                                                 const float *__restrict__ xs, int64_t n, int64_t fu,
                                                                 float r2, float neg_inv_s2, float *__restrict__ y,
                                                                 int32_t *__restrict__ count) {
    constexpr int G = kWave / LPR;  // groups per wave
    constexpr int R = LPR;          // destinations per group
    __shared__ float2 lists[kBlock / kWave][kCap][kWave];
    const Params p = *prm;
    const int lane = lane_id(), wv = threadIdx.x / kWave;
    const int g = lane / LPR, q = lane % LPR;
    const int64_t s0 = (static_cast<int64_t>(xcd_block()) * (kBlock / kWave) + wv) * kWave;
    if (s0 >= n) return;
    const int64_t s = s0 + lane;
    const bool own = s < n;
    const float4 pi = own ? rec[s] : make_float4(0.0f, 0.0f, 0.0f, __int_as_float(-1));
    const int32_t i = __float_as_int(pi.w);
    for (int64_t fb = 0; fb < fu; fb += LPR * UPL) {
        f32x4 acc[R][UPL];
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < UPL; ++u) acc[r][u] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        Cursor c;
        bool live = own && open_cursor(p, start, pi, c);
        int cnt = 0;
        while (true) {
            const int m = fill_list(p, start, rec, pi, i, r2, neg_inv_s2, c, live, lists[wv], lane);
            cnt += m;
            lds_fence();
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int d = r * G + g;
                const int md = __shfl(m, d, kWave);
                for (int k0 = 0; k0 < md; k0 += kBatch) {
                    float2 en[kBatch];
#pragma unroll
                    for (int b = 0; b < kBatch; ++b)
                        en[b] = k0 + b < md ? lists[wv][k0 + b][d] : make_float2(0.0f, 0.0f);
                    f32x4 xv[kBatch][UPL];
#pragma unroll
                    for (int b = 0; b < kBatch; ++b) {
                        const int64_t row = static_cast<int64_t>(__float_as_int(en[b].x)) * fu + fb + q;
#pragma unroll
                        for (int u = 0; u < UPL; ++u)
                            xv[b][u] = (k0 + b < md && fb + q + u * LPR < fu) ? unit4(xs, row + u * LPR)
                                                                              : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                    }
#pragma unroll
                    for (int b = 0; b < kBatch; ++b)
#pragma unroll
                        for (int u = 0; u < UPL; ++u) acc[r][u] += en[b].y * xv[b][u];
                }
            }
            lds_fence();
            if (__ballot(live) == 0) break;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int d = r * G + g;
            const int32_t id = __shfl(i, d, kWave);
            if (s0 + d < n) {
#pragma unroll
                for (int u = 0; u < UPL; ++u) {
                    const int64_t unit = fb + q + u * LPR;
                    if (unit < fu) stg_stream(reinterpret_cast<f32x4 *>(y) + static_cast<int64_t>(id) * fu + unit,
                                              acc[r][u]);
                }
            }
        }
        if (fb == 0 && own && count) count[i] = cnt;
    }
}

// Backward with the same schedule: dx_i = sum_j k_ij dy_j and
// dp_i = sum_j (2 k_ij / sigma^2) (p_j - p_i) (<dy_i, x_j> + <dy_j, x_i>).
// Each lane accumulates dp from the part of the inner products its units
// cover; the LPR partial sums of a destination are added once at the end.
template <int LPR, int UPL, bool DX, bool DP>
__global__ __launch_bounds__(kBlock) void radius_bwd_coop_kernel(const Params *__restrict__ prm,
                                                                 const int64_t *__restrict__ start,
                                                                 const float4 *__restrict__ rec,
                                                                 const float *__restrict__ xs,
                                                                 const float *__restrict__ ys, int64_t n, int64_t fu,
                                                                 float r2, float neg_inv_s2, float two_inv_s2,
                                                                 float *__restrict__ dx, float *__restrict__ dp) {
    constexpr int G = kWave / LPR;
    constexpr int R = LPR;
    constexpr int B = DP ? kBatchDp : kBatch;
    __shared__ float2 lists[kBlock / kWave][kCap][kWave];
    const Params p = *prm;
    const int lane = lane_id(), wv = threadIdx.x / kWave;
    const int g = lane / LPR, q = lane % LPR;
    const int64_t s0 = (static_cast<int64_t>(xcd_block()) * (kBlock / kWave) + wv) * kWave;
    if (s0 >= n) return;
    const int64_t s = s0 + lane;
    const bool own = s < n;
    const float4 pi = own ? rec[s] : make_float4(0.0f, 0.0f, 0.0f, __int_as_float(-1));
    const int32_t i = __float_as_int(pi.w);
    float gp[R][3];
#pragma unroll
    for (int r = 0; r < R; ++r) gp[r][0] = gp[r][1] = gp[r][2] = 0.0f;
    for (int64_t fb = 0; fb < fu; fb += LPR * UPL) {
        f32x4 acc[R][UPL];
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < UPL; ++u) acc[r][u] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        Cursor c;
        bool live = own && open_cursor(p, start, pi, c);
        while (true) {
            const int m = fill_list(p, start, rec, pi, i, r2, neg_inv_s2, c, live, lists[wv], lane);
            lds_fence();
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int d = r * G + g;
                const int md = __shfl(m, d, kWave);
                if (md == 0) continue;
                const int64_t sd = s0 + d;
                f32x4 gi[UPL], xi[UPL];
                float4 pd;
                if (DP) {
                    pd = rec[sd];
#pragma unroll
                    for (int u = 0; u < UPL; ++u) {
                        const int64_t unit = fb + q + u * LPR;
                        const bool ok = unit < fu;
                        gi[u] = ok ? unit4(ys, sd * fu + unit) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                        xi[u] = ok ? unit4(xs, sd * fu + unit) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                    }
                }
                for (int k0 = 0; k0 < md; k0 += B) {
                    float2 en[B];
#pragma unroll
                    for (int b = 0; b < B; ++b) en[b] = k0 + b < md ? lists[wv][k0 + b][d] : make_float2(0.0f, 0.0f);
                    f32x4 gj[B][UPL], xj[B][UPL];
                    float4 pj[B];
#pragma unroll
                    for (int b = 0; b < B; ++b) {
                        const bool live_b = k0 + b < md;
                        const int64_t t = __float_as_int(en[b].x);
                        const int64_t row = t * fu + fb + q;
#pragma unroll
                        for (int u = 0; u < UPL; ++u) {
                            const bool ok = live_b && fb + q + u * LPR < fu;
                            gj[b][u] = ok ? unit4(ys, row + u * LPR) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                            if (DP) xj[b][u] = ok ? unit4(xs, row + u * LPR) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
                        }
                        if (DP) pj[b] = live_b ? rec[t] : pd;
                    }
#pragma unroll
                    for (int b = 0; b < B; ++b) {
                        float dot = 0.0f;
#pragma unroll
                        for (int u = 0; u < UPL; ++u) {
                            if (DX) acc[r][u] += en[b].y * gj[b][u];
                            if (DP) {
                                const f32x4 a = gi[u] * xj[b][u] + gj[b][u] * xi[u];
                                dot += (a.x + a.y) + (a.z + a.w);
                            }
                        }
                        if (DP) {
                            const float cc = two_inv_s2 * en[b].y * dot;
                            gp[r][0] = fmaf(cc, pj[b].x - pd.x, gp[r][0]);
                            gp[r][1] = fmaf(cc, pj[b].y - pd.y, gp[r][1]);
                            gp[r][2] = fmaf(cc, pj[b].z - pd.z, gp[r][2]);
                        }
                    }
                }
            }
            lds_fence();
            if (__ballot(live) == 0) break;
        }
        if (DX) {
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int d = r * G + g;
                const int32_t id = __shfl(i, d, kWave);
                if (s0 + d < n) {
#pragma unroll
                    for (int u = 0; u < UPL; ++u) {
                        const int64_t unit = fb + q + u * LPR;
                        if (unit < fu)
                            stg_stream(reinterpret_cast<f32x4 *>(dx) + static_cast<int64_t>(id) * fu + unit,
                                       acc[r][u]);
                    }
                }
            }
        }
    }
    if (DP) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
#pragma unroll
            for (int m = 1; m < LPR; m <<= 1)
#pragma unroll
                for (int a = 0; a < 3; ++a) gp[r][a] += shfl_xor_f(gp[r][a], m);
            const int d = r * G + g;
            const int32_t id = __shfl(i, d, kWave);
            if (q == 0 && s0 + d < n)
#pragma unroll
                for (int a = 0; a < 3; ++a) dp[static_cast<int64_t>(id) * 3 + a] = gp[r][a];
        }
    }
}

__global__ __launch_bounds__(kBlock) void neighbor_count_kernel(const Params *__restrict__ prm,
                                                                const int64_t *__restrict__ start,
                                                                const float4 *__restrict__ rec, int64_t n, float r2,
                                                                int64_t *__restrict__ cnt64,
                                                                int32_t *__restrict__ count) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    int c = 0;
    for_candidates(p, start, pi, [&](int64_t t) {
        const float4 pj = rec[t];
        float d2;
        if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) ++c;
    });
    cnt64[i] = c;
    if (count) count[i] = c;
}

__global__ __launch_bounds__(kBlock) void neighbor_fill_kernel(const Params *__restrict__ prm,
                                                               const int64_t *__restrict__ start,
                                                               const float4 *__restrict__ rec, int64_t n, float r2,
                                                               const int64_t *__restrict__ ptr,
                                                               int32_t *__restrict__ idx) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    const int64_t b = ptr[i];
    int64_t w = b;
    for_candidates(p, start, pi, [&](int64_t t) {
        const float4 pj = rec[t];
        float d2;
        const int32_t j = __float_as_int(pj.w);
        if (accept(pi, pj, r2, d2) && j != i) idx[w++] = j;
    });
    // insertion sort of this point's list (ascending ids)
    for (int64_t a = b + 1; a < w; ++a) {
        const int32_t v = idx[a];
        int64_t k = a - 1;
        while (k >= b && idx[k] > v) {
            idx[k + 1] = idx[k];
            --k;
        }
        idx[k + 1] = v;
    }
}

struct Ws {
    Params *prm;
    float *bbox;
    int32_t *cell;
    unsigned long long *count;  // ncell_max + 1, scanned in place into `start`
    unsigned int *cursor;
    int32_t *perm_a, *perm_b;
    float4 *rec;
    float *as, *bs;
    void *scan;
    int64_t max_cells;
    int bbox_blocks;
};

Ws carve(Carve &c, int64_t n, int64_t feat) {
    Ws w;
    w.max_cells = n + 64;
    w.bbox_blocks = 1024;
    w.prm = c.take<Params>(1);
    w.bbox = c.take<float>(6 * w.bbox_blocks);
    w.cell = c.take<int32_t>(n);
    w.count = c.take<unsigned long long>(w.max_cells + 1);
    w.cursor = c.take<unsigned int>(w.max_cells);
    w.perm_a = c.take<int32_t>(n);
    w.perm_b = c.take<int32_t>(n);
    w.rec = c.take<float4>(n);
    w.as = c.take<float>(n * feat);
    w.bs = c.take<float>(n * feat);
    w.scan = c.take<char>(scan_ws_bytes(w.max_cells + 1));
    return w;
}

int blocks_for(int64_t n) {
    int64_t b = ceil_div(n > 0 ? n : 1, kBlock);
    const int64_t cap = static_cast<int64_t>(device_cus()) * 32;
    return static_cast<int>(b < cap ? b : cap);
}

// Build the cell directory and the cell-ordered copies of `a` and `b`.
int build(int64_t n, const float *pos, float radius, const float *a, const float *b, int32_t feat, Ws &w,
          hipStream_t stream) {
    int nb = w.bbox_blocks;
    const int64_t need = ceil_div(n, kBlock);
    if (need < nb) nb = static_cast<int>(need);
    hipLaunchKernelGGL(bbox_partial_kernel, dim3(nb), dim3(kBlock), 0, stream, pos, n, w.bbox);
    if (int rc = check_launch("radius bbox")) return rc;
    hipLaunchKernelGGL(grid_params_kernel, dim3(1), dim3(kBlock), 0, stream, w.bbox, nb, n, radius, w.max_cells,
                       w.prm);
    if (int rc = check_launch("radius grid")) return rc;
    if (int rc = fill_u32(w.count, 0u, 2 * (w.max_cells + 1), stream)) return rc;
    if (int rc = fill_u32(w.cursor, 0u, w.max_cells, stream)) return rc;
    hipLaunchKernelGGL(cell_count_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, pos, n, w.prm, w.cell,
                       w.count);
    if (int rc = check_launch("radius cell count")) return rc;
    int64_t *start = reinterpret_cast<int64_t *>(w.count);
    if (int rc = launch_excl_scan(start, start, w.max_cells + 1, w.scan, stream)) return rc;
    hipLaunchKernelGGL(cell_scatter_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, w.cell, n, start,
                       w.cursor, w.perm_a);
    if (int rc = check_launch("radius scatter")) return rc;
    hipLaunchKernelGGL(cell_sort_kernel, dim3(blocks_for(w.max_cells * kWave)), dim3(kBlock), 0, stream, start, w.prm,
                       w.perm_a, w.perm_b);
    if (int rc = check_launch("radius cell sort")) return rc;
    hipLaunchKernelGGL(gather_records_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, w.perm_b, n, pos, w.rec);
    if (int rc = check_launch("radius records")) return rc;
    if (feat > 0 && (a || b)) {
        const bool vec = feat % 4 == 0 && (!a || aligned16(a)) && (!b || aligned16(b));
        if (vec) return launch_gather_rows<4>(w.perm_b, n, feat / 4, a, b, w.as, w.bs, stream);
        return launch_gather_rows<1>(w.perm_b, n, feat, a, b, w.as, w.bs, stream);
    }
    return TIGA_OK;
}

template <int K>
int launch_gather_rows(const int32_t *perm, int64_t n, int64_t fu, const float *a, const float *b, float *as,
                       float *bs, hipStream_t stream) {
    const int64_t total = n * fu;
    const dim3 grid(static_cast<unsigned>(blocks_for(total)));
    if (total < (int64_t{1} << 32) - kBlock * int64_t{65536})
        hipLaunchKernelGGL((gather_rows_kernel<K, uint32_t>), grid, dim3(kBlock), 0, stream, perm,
                           static_cast<uint32_t>(total), static_cast<uint32_t>(fu), a, b, as, bs);
    else
        hipLaunchKernelGGL((gather_rows_kernel<K, int64_t>), grid, dim3(kBlock), 0, stream, perm, total, fu, a, b, as,
                           bs);
    return check_launch("radius rows");
}

template <int K>
int fwd_units(int64_t fu, const Ws &w, const int64_t *start, int64_t n, float r2, float nis, float *y,
              int32_t *count, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
    prof_before(stream);
    if constexpr (K == 4) {
#define TIGA_RF(LPR, UPL)                                                                                    \
    hipLaunchKernelGGL((radius_fwd_coop_kernel<LPR, UPL>), grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, \
                       w.as, n, fu, r2, nis, y, count)
        if (fu <= 1) TIGA_RF(1, 1);
        else if (fu <= 2) TIGA_RF(2, 1);
        else if (fu <= 4) TIGA_RF(4, 1);
        else if (fu <= 8) TIGA_RF(8, 1);
        else TIGA_RF(8, 2);
#undef TIGA_RF
    } else {
#define TIGA_RF(NU)                                                                                            \
    hipLaunchKernelGGL((radius_fwd_kernel<K, NU>), grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, w.as, n, \
                       fu, r2, nis, y, count)
        if (fu <= 1) TIGA_RF(1);
        else if (fu <= 2) TIGA_RF(2);
        else if (fu <= 4) TIGA_RF(4);
        else if (fu <= 8) TIGA_RF(8);
        else TIGA_RF(16);
#undef TIGA_RF
    }
    prof_after(stream);
    return check_launch("radius forward");
}

template <int K, bool DX, bool DP>
int bwd_units(int64_t fu, const Ws &w, const int64_t *start, int64_t n, float r2, float nis, float tis, float *dx,
              float *dp, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
    prof_before(stream);
    if constexpr (K == 4) {
#define TIGA_RB(LPR, UPL)                                                                                     \
    hipLaunchKernelGGL((radius_bwd_coop_kernel<LPR, UPL, DX, DP>), grid, dim3(kBlock), 0, stream, w.prm, start, \
                       w.rec, w.bs, w.as, n, fu, r2, nis, tis, dx, dp)
        if (fu <= 1) TIGA_RB(1, 1);
        else if (fu <= 2) TIGA_RB(2, 1);
        else if (fu <= 4) TIGA_RB(4, 1);
        else if (fu <= 8) TIGA_RB(8, 1);
        else TIGA_RB(8, 2);
#undef TIGA_RB
    } else {
#define TIGA_RB(NU)                                                                                          \
    hipLaunchKernelGGL((radius_bwd_kernel<K, NU, DX, DP>), grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, \
                       w.bs, w.as, n, fu, r2, nis, tis, dx, dp)
        if (fu <= 1) TIGA_RB(1);
        else if (fu <= 2) TIGA_RB(2);
        else if (fu <= 4) TIGA_RB(4);
        else TIGA_RB(8);
#undef TIGA_RB
    }
    prof_after(stream);
    return check_launch("radius backward");
}

}  // namespace

size_t workspace_bytes(int64_t n, int64_t feat) {
    Carve c(nullptr);
    carve(c, n, feat);
    return c.bytes();
}

int forward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, float *y,
            int32_t *count, void *ws, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, feat);
    if (int rc = build(n, pos, radius, x, nullptr, feat, w, stream)) return rc;
    const int64_t *start = reinterpret_cast<const int64_t *>(w.count);
    const float r2 = radius * radius;
    const float nis = -1.0f / (sigma * sigma);
    const bool vec = feat % 4 == 0 && aligned16(y);
    if (vec) return fwd_units<4>(feat / 4, w, start, n, r2, nis, y, count, stream);
    return fwd_units<1>(feat, w, start, n, r2, nis, y, count, stream);
}

int backward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, const float *dy,
             float *dx, float *dpos, void *ws, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, feat);
    // as = cell-ordered dy, bs = cell-ordered x (only needed for dpos)
    if (int rc = build(n, pos, radius, dy, dpos ? x : nullptr, feat, w, stream)) return rc;
    const int64_t *start = reinterpret_cast<const int64_t *>(w.count);
    const float r2 = radius * radius;
    const float nis = -1.0f / (sigma * sigma);
    const float tis = 2.0f / (sigma * sigma);
    const bool vec = feat % 4 == 0 && (!dx || aligned16(dx));
    const int64_t fu = vec ? feat / 4 : feat;
#define TIGA_B(KK)                                                                          \
    if (dx && dpos) return bwd_units<KK, true, true>(fu, w, start, n, r2, nis, tis, dx, dpos, stream); \
    if (dx) return bwd_units<KK, true, false>(fu, w, start, n, r2, nis, tis, dx, dpos, stream);        \
    return bwd_units<KK, false, true>(fu, w, start, n, r2, nis, tis, dx, dpos, stream)
    if (vec) {
        TIGA_B(4);
    } else {
        TIGA_B(1);
    }
#undef TIGA_B
}

int neighbors(int64_t n, const float *pos, float radius, int32_t *count, int64_t *nbr_ptr, int32_t *nbr_idx,
              void *ws, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, 0);
    if (int rc = build(n, pos, radius, nullptr, nullptr, 0, w, stream)) return rc;
    const int64_t *start = reinterpret_cast<const int64_t *>(w.count);
    const float r2 = radius * radius;
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
    if (!nbr_idx) {
        // counts into nbr_ptr[0..n), then the exclusive scan in place
        hipLaunchKernelGGL(neighbor_count_kernel, grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, n, r2, nbr_ptr,
                           count);
        if (int rc = check_launch("radius neighbour count")) return rc;
        if (int rc = fill_u32(nbr_ptr + n, 0u, 2, stream)) return rc;
        if (int rc = launch_excl_scan(nbr_ptr, nbr_ptr, n + 1, w.scan, stream)) return rc;
    } else {
        hipLaunchKernelGGL(neighbor_fill_kernel, grid, dim3(kBlock), 0, stream, w.prm, start, w.rec, n, r2, nbr_ptr,
                           nbr_idx);
        if (int rc = check_launch("radius neighbour fill")) return rc;
    }
    return check_hip(hipStreamSynchronize(stream), "radius neighbours: synchronize");
}

}  // namespace radius
}  // namespace tiga
