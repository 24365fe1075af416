// Cell directory of the generated radius relation, shared by the kernels that consume it.
#pragma once

#include "common.hpp"

namespace tiga {
namespace radius {

// Uniform grid over the box of the finite coordinates: cells of size h >= r (1 + 2^-10) per axis.
struct Params {
    double lo[3];
    double inv_h;
    int dim[3];
    int ncell;
};

__device__ __forceinline__ int cell_axis(const Params &p, int a, float v) {
    double t = floor((static_cast<double>(v) - p.lo[a]) * p.inv_h);
    if (!(t >= 0.0)) t = 0.0;
    const double top = static_cast<double>(p.dim[a] - 1);
    if (t > top) t = top;
    return static_cast<int>(t);
}

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

// Visit the 9 runs [b, e) of cell-ordered positions that hold the 27 cells around the point with
// record `pi` (x-adjacent cells are adjacent in memory).
template <class F>
__device__ __forceinline__ void for_runs(const Params &p, const int64_t *__restrict__ start, float4 pi, F &&body) {
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
            body(start[rowc + x0], start[rowc + x1 + 1]);
        }
    }
}

// The built directory: grid parameters, ncell + 1 cell starts in cell order, and the cell-ordered
// records (x, y, z, point id as bits).  Device pointers into the caller's workspace.
struct Cells {
    const Params *prm;
    const int64_t *start;
    const float4 *rec;
};

// Workspace of a build over n points, and the build itself (enqueued on `stream`).
size_t cells_ws_bytes(int64_t n);
int build_cells(int64_t n, const float *pos, float radius, void *ws, Cells &out, hipStream_t stream);

}  // namespace radius
}  // namespace tiga
