// Degree-aware row plan (deterministic; no global atomics).
//
// count: per tile of kPlanTile rows, the number of chunk descriptors, partial
//        slots and split rows its medium/long rows need;
// scan:  exclusive prefix over tiles (one block), totals to PlanCounts;
// write: each tile recomputes its rows and writes descriptors at its offset.
// Within a tile, row (r, t) = tile_base + r * kBlock + t is visited in
// (r, t) order, so the descriptor order depends only on the topology.
#include "csr_common.hpp"

namespace tiga {
namespace csr {

namespace {

struct RowNeed {
    int64_t chunks, slots, splits;
};

__device__ __forceinline__ RowNeed row_need(const int64_t *__restrict__ ptr, int64_t row, int64_t nrows,
                                            int DS, int CH) {
    RowNeed r{0, 0, 0};
    if (row < nrows) {
        const int64_t d = ptr[row + 1] - ptr[row];
        if (d > DS) {
            r.chunks = (d + CH - 1) / CH;
            if (r.chunks > 1) {
                r.slots = r.chunks;
                r.splits = 1;
            }
        }
    }
    return r;
}

// Block-wide exclusive scan of three counters; returns block totals.
__device__ __forceinline__ RowNeed block_excl_scan3(RowNeed v, RowNeed &excl) {
    __shared__ int64_t sh[3][kWavesPerBlock];
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int64_t ic = wave_incl_scan(v.chunks);
    const int64_t is = wave_incl_scan(v.slots);
    const int64_t ip = wave_incl_scan(v.splits);
    if (lane == kWave - 1) {
        sh[0][wave] = ic;
        sh[1][wave] = is;
        sh[2][wave] = ip;
    }
    __syncthreads();
    int64_t oc = 0, os = 0, op = 0;
    RowNeed tot{0, 0, 0};
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
        if (w < wave) {
            oc += sh[0][w];
            os += sh[1][w];
            op += sh[2][w];
        }
        tot.chunks += sh[0][w];
        tot.slots += sh[1][w];
        tot.splits += sh[2][w];
    }
    __syncthreads();
    excl.chunks = oc + ic - v.chunks;
    excl.slots = os + is - v.slots;
    excl.splits = op + ip - v.splits;
    return tot;
}

__global__ __launch_bounds__(kBlock) void plan_count_kernel(const int64_t *__restrict__ ptr, int64_t nrows,
                                                            int DS, int CH, int64_t *__restrict__ tile_vals) {
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPlanTile;
    RowNeed acc{0, 0, 0};
#pragma unroll
    for (int r = 0; r < kPlanRowsPerThread; ++r) {
        RowNeed n = row_need(ptr, base + r * kBlock + threadIdx.x, nrows, DS, CH);
        acc.chunks += n.chunks;
        acc.slots += n.slots;
        acc.splits += n.splits;
    }
    RowNeed excl;
    RowNeed tot = block_excl_scan3(acc, excl);
    if (threadIdx.x == 0) {
        tile_vals[3 * blockIdx.x + 0] = tot.chunks;
        tile_vals[3 * blockIdx.x + 1] = tot.slots;
        tile_vals[3 * blockIdx.x + 2] = tot.splits;
    }
}

// One block: exclusive scan over the tiles, in place.
__global__ __launch_bounds__(kBlock) void plan_scan_kernel(int64_t *__restrict__ tile_vals, int64_t tiles,
                                                           PlanCounts *__restrict__ counts) {
    RowNeed carry{0, 0, 0};
    for (int64_t t0 = 0; t0 < tiles; t0 += kBlock) {
        const int64_t t = t0 + threadIdx.x;
        RowNeed v{0, 0, 0};
        if (t < tiles) {
            v.chunks = tile_vals[3 * t + 0];
            v.slots = tile_vals[3 * t + 1];
            v.splits = tile_vals[3 * t + 2];
        }
        RowNeed excl;
        RowNeed tot = block_excl_scan3(v, excl);
        if (t < tiles) {
            tile_vals[3 * t + 0] = carry.chunks + excl.chunks;
            tile_vals[3 * t + 1] = carry.slots + excl.slots;
            tile_vals[3 * t + 2] = carry.splits + excl.splits;
        }
        carry.chunks += tot.chunks;
        carry.slots += tot.slots;
        carry.splits += tot.splits;
    }
    if (threadIdx.x == 0) {
        counts->chunks = static_cast<unsigned long long>(carry.chunks);
        counts->slots = static_cast<unsigned long long>(carry.slots);
        counts->splits = static_cast<unsigned long long>(carry.splits);
        counts->pad = 0;
    }
}

__global__ __launch_bounds__(kBlock) void plan_write_kernel(const int64_t *__restrict__ ptr, int64_t nrows,
                                                            int DS, int CH,
                                                            const int64_t *__restrict__ tile_vals,
                                                            Desc *__restrict__ chunks, Desc *__restrict__ splits) {
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPlanTile;
    RowNeed run{tile_vals[3 * blockIdx.x + 0], tile_vals[3 * blockIdx.x + 1], tile_vals[3 * blockIdx.x + 2]};
    for (int r = 0; r < kPlanRowsPerThread; ++r) {
        const int64_t row = base + r * kBlock + threadIdx.x;
        RowNeed n = row_need(ptr, row, nrows, DS, CH);
        RowNeed excl;
        RowNeed tot = block_excl_scan3(n, excl);
        if (n.chunks > 0) {
            const int64_t c0 = run.chunks + excl.chunks;
            const int slot0 = n.slots ? static_cast<int>(run.slots + excl.slots) : -1;
            for (int64_t k = 0; k < n.chunks; ++k)
                chunks[c0 + k] = make_int4(static_cast<int>(row), static_cast<int>(k),
                                           slot0 >= 0 ? slot0 + static_cast<int>(k) : -1,
                                           static_cast<int>(n.chunks));
            if (n.splits)
                splits[run.splits + excl.splits] =
                    make_int4(static_cast<int>(row), slot0, static_cast<int>(n.chunks), 0);
        }
        run.chunks += tot.chunks;
        run.slots += tot.slots;
        run.splits += tot.splits;
    }
}

}  // namespace

int launch_plan(const int64_t *ptr, int64_t nrows, const Geom &g, const PlanBounds &b, const PlanWs &w,
                hipStream_t stream) {
    const unsigned tiles = static_cast<unsigned>(b.tiles);
    hipLaunchKernelGGL(plan_count_kernel, dim3(tiles), dim3(kBlock), 0, stream, ptr, nrows, g.DS, g.CH,
                       w.tile_vals);
    if (int rc = check_launch("plan count")) return rc;
    hipLaunchKernelGGL(plan_scan_kernel, dim3(1), dim3(kBlock), 0, stream, w.tile_vals, b.tiles, w.counts);
    if (int rc = check_launch("plan scan")) return rc;
    hipLaunchKernelGGL(plan_write_kernel, dim3(tiles), dim3(kBlock), 0, stream, ptr, nrows, g.DS, g.CH,
                       w.tile_vals, w.chunks, w.splits);
    return check_launch("plan write");
}

}  // namespace csr
}  // namespace tiga
