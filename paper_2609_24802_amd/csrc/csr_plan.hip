// Degree-aware row plan (deterministic; no global atomics).
//
// count: per tile of kPlanTile rows, the chunks of each class, partial slots
//        and split rows its non-short rows need;
// scan:  exclusive prefix over tiles (one block), totals to PlanCounts;
// write: each tile recomputes its rows and writes descriptors at its offsets,
//        in row order within each class; class c's descriptors follow those
//        of classes 0..c-1.
// Descriptor positions depend only on the topology.
#include "csr_common.hpp"

namespace tiga {
namespace csr {

namespace {

struct Need {
    int64_t v[kPlanVals];  // chunks per class, partial slots, split rows
};

// Chunks per class, partial slots and split rows needed by a row of degree deg.
__device__ __forceinline__ Need need_of(const Geom &g, int64_t deg) {
    Need r;
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) r.v[k] = 0;
    if (deg > g.DS) {
        const int64_t nch = (deg + g.CH - 1) / g.CH;
        const int64_t last = deg - (nch - 1) * g.CH;
        const int c = chunk_class(g, last);
        r.v[0] += nch - 1 + (c == 0);
        r.v[1] += (c == 1);
        r.v[2] += (c == 2);
        if (nch > 1) {
            r.v[kClasses] = nch;
            r.v[kClasses + 1] = 1;
        }
    }
    return r;
}

__device__ __forceinline__ Need row_need(const Geom &g, const int64_t *__restrict__ ptr, int64_t row, int64_t nrows,
                                         int64_t &e0, int64_t &deg) {
    e0 = 0;
    deg = 0;
    if (row < nrows) {
        e0 = ptr[row];
        deg = ptr[row + 1] - e0;
    }
    return need_of(g, deg);
}

// Block-wide exclusive scan of kPlanVals counters over BLOCK threads; returns
// the block totals.
template <int BLOCK = kBlock>
__device__ __forceinline__ Need block_excl_scan(const Need &v, Need &excl) {
    constexpr int W = BLOCK / kWave;
    __shared__ int64_t sh[kPlanVals][W];
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    Need inc, tot;
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) {
        inc.v[k] = wave_incl_scan(v.v[k]);
        if (lane == kWave - 1) sh[k][wave] = inc.v[k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) {
        int64_t off = 0, t = 0;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            if (w < wave) off += sh[k][w];
            t += sh[k][w];
        }
        excl.v[k] = off + inc.v[k] - v.v[k];
        tot.v[k] = t;
    }
    __syncthreads();
    return tot;
}

template <int L>
__global__ __launch_bounds__(kBlock) void plan_count_kernel(const int64_t *__restrict__ ptr, int64_t nrows,
                                                            int64_t *__restrict__ tile_vals) {
    constexpr Geom g = make_geom(L);  // compile-time chunk geometry: divisions by constants
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPlanTile;
    Need acc;
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) acc.v[k] = 0;
#pragma unroll
    for (int r = 0; r < kPlanRowsPerThread; ++r) {
        int64_t e0, deg;
        const Need n = row_need(g, ptr, base + r * kBlock + threadIdx.x, nrows, e0, deg);
#pragma unroll
        for (int k = 0; k < kPlanVals; ++k) acc.v[k] += n.v[k];
    }
    // block totals: wave sums, then thread 0 adds the waves
    __shared__ int64_t sh[kPlanVals][kWavesPerBlock];
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) {
        int64_t v = acc.v[k];
#pragma unroll
        for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
        if (lane_id() == 0) sh[k][threadIdx.x / kWave] = v;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int k = 0; k < kPlanVals; ++k) {
            int64_t t = 0;
#pragma unroll
            for (int w = 0; w < kWavesPerBlock; ++w) t += sh[k][w];
            tile_vals[kPlanVals * blockIdx.x + k] = t;
        }
    }
}

// One block of kScanBlock threads: exclusive scan over the tiles, in place,
// and the totals.  Each thread first sums a contiguous run of tiles, then one
// block scan combines the runs.
constexpr int kScanBlock = 1024;

__global__ __launch_bounds__(kScanBlock) void plan_scan_kernel(int64_t *__restrict__ tile_vals, int64_t tiles,
                                                               PlanCounts *__restrict__ counts) {
    const int64_t per = (tiles + kScanBlock - 1) / kScanBlock;
    const int64_t t0 = static_cast<int64_t>(threadIdx.x) * per;
    const int64_t t1 = t0 + per < tiles ? t0 + per : tiles;
    Need sum;
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) sum.v[k] = 0;
    // unrolled so that several tiles' loads are in flight at once
#pragma unroll 8
    for (int64_t t = t0; t < t1; ++t)
#pragma unroll
        for (int k = 0; k < kPlanVals; ++k) sum.v[k] += tile_vals[kPlanVals * t + k];
    Need excl;
    const Need tot = block_excl_scan<kScanBlock>(sum, excl);
#pragma unroll 8
    for (int64_t t = t0; t < t1; ++t)
#pragma unroll
        for (int k = 0; k < kPlanVals; ++k) {
            const int64_t v = tile_vals[kPlanVals * t + k];
            tile_vals[kPlanVals * t + k] = excl.v[k];
            excl.v[k] += v;
        }
    if (threadIdx.x == 0) {
        for (int c = 0; c < kClasses; ++c) counts->cls[c] = static_cast<unsigned long long>(tot.v[c]);
        counts->slots = static_cast<unsigned long long>(tot.v[kClasses]);
        counts->splits = static_cast<unsigned long long>(tot.v[kClasses + 1]);
        counts->pad[0] = counts->pad[1] = counts->pad[2] = 0;
    }
}

// Descriptors of a tile in row order: thread t owns the kPlanRowsPerThread
// consecutive rows base + t * kPlanRowsPerThread + r and writes them after the
// rows of threads 0..t-1, so consecutive descriptors of a class are rows in
// ascending order (a work item of several chunks writes neighbouring output
// rows).  The tile's row pointers are staged in LDS first (coalesced loads;
// one pad slot per 8 entries keeps the per-thread reads off a single bank).
__host__ __device__ constexpr int pad_ix(int i) { return i + (i >> 3); }

template <int L>
__global__ __launch_bounds__(kBlock) void plan_write_kernel(const int64_t *__restrict__ ptr, int64_t nrows,
                                                            const int64_t *__restrict__ tile_vals,
                                                            const PlanCounts *__restrict__ counts,
                                                            Desc *__restrict__ chunks, Split *__restrict__ splits) {
    constexpr Geom g = make_geom(L);
    __shared__ int64_t sptr[pad_ix(kPlanTile) + 1];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPlanTile;
    for (int i = threadIdx.x; i <= kPlanTile; i += kBlock) {
        const int64_t row = base + i;
        sptr[pad_ix(i)] = ptr[row < nrows ? row : nrows];
    }
    __syncthreads();
    int64_t cbase[kClasses];
    int64_t b = 0;
#pragma unroll
    for (int c = 0; c < kClasses; ++c) {
        cbase[c] = b;
        b += static_cast<int64_t>(counts->cls[c]);
    }
    int64_t e0[kPlanRowsPerThread], deg[kPlanRowsPerThread];
    Need mine;
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) mine.v[k] = 0;
#pragma unroll
    for (int r = 0; r < kPlanRowsPerThread; ++r) {
        const int i = threadIdx.x * kPlanRowsPerThread + r;
        const bool in = base + i < nrows;
        e0[r] = in ? sptr[pad_ix(i)] : 0;
        deg[r] = in ? sptr[pad_ix(i + 1)] - e0[r] : 0;
        const Need n = need_of(g, deg[r]);
#pragma unroll
        for (int k = 0; k < kPlanVals; ++k) mine.v[k] += n.v[k];
    }
    Need run;
    block_excl_scan(mine, run);
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) run.v[k] += tile_vals[kPlanVals * blockIdx.x + k];
#pragma unroll
    for (int r = 0; r < kPlanRowsPerThread; ++r) {
        if (deg[r] <= g.DS) continue;
        const int64_t row = base + threadIdx.x * kPlanRowsPerThread + r;
        const int64_t nch = (deg[r] + g.CH - 1) / g.CH;
        const int slot0 = nch > 1 ? static_cast<int>(run.v[kClasses]) : -1;
        for (int64_t k = 0; k < nch; ++k) {
            const int64_t len = (k + 1 < nch) ? g.CH : deg[r] - k * g.CH;
            const int c = (k + 1 < nch) ? 0 : chunk_class(g, len);
            Desc d;
            d.row = static_cast<int32_t>(row);
            d.slot = slot0 >= 0 ? slot0 + static_cast<int>(k) : -1;
            d.range = pack_range(e0[r] + k * g.CH, len);
            const int64_t pos = c == 0 ? cbase[0] + run.v[0] : (c == 1 ? cbase[1] + run.v[1] : cbase[2] + run.v[2]);
            chunks[pos] = d;
            run.v[0] += (c == 0);
            run.v[1] += (c == 1);
            run.v[2] += (c == 2);
        }
        if (nch > 1) {
            Split sp;
            sp.row = static_cast<int32_t>(row);
            sp.slot0 = slot0;
            sp.nch = static_cast<int32_t>(nch);
            sp.pad = 0;
            splits[run.v[kClasses + 1]] = sp;
            run.v[kClasses] += nch;
            run.v[kClasses + 1] += 1;
        }
    }
}

}  // namespace

namespace {
template <int L>
int launch_plan_t(const int64_t *ptr, int64_t nrows, const PlanBounds &b, const PlanWs &w, hipStream_t stream) {
    const unsigned tiles = static_cast<unsigned>(b.tiles);
    hipLaunchKernelGGL(plan_count_kernel<L>, dim3(tiles), dim3(kBlock), 0, stream, ptr, nrows, w.tile_vals);
    if (int rc = check_launch("plan count")) return rc;
    hipLaunchKernelGGL(plan_scan_kernel, dim3(1), dim3(kScanBlock), 0, stream, w.tile_vals, b.tiles, w.counts);
    if (int rc = check_launch("plan scan")) return rc;
    hipLaunchKernelGGL(plan_write_kernel<L>, dim3(tiles), dim3(kBlock), 0, stream, ptr, nrows, w.tile_vals, w.counts,
                       w.chunks, w.splits);
    return check_launch("plan write");
}
}  // namespace

int launch_plan(const int64_t *ptr, int64_t nrows, const Geom &g, const PlanBounds &b, const PlanWs &w,
                hipStream_t stream) {
    switch (g.L) {
        case 1: return launch_plan_t<1>(ptr, nrows, b, w, stream);
        case 2: return launch_plan_t<2>(ptr, nrows, b, w, stream);
        case 4: return launch_plan_t<4>(ptr, nrows, b, w, stream);
        case 8: return launch_plan_t<8>(ptr, nrows, b, w, stream);
        case 16: return launch_plan_t<16>(ptr, nrows, b, w, stream);
        case 32: return launch_plan_t<32>(ptr, nrows, b, w, stream);
        case 64: return launch_plan_t<64>(ptr, nrows, b, w, stream);
        default: return fail(TIGA_EINVAL, "internal: plan for %d lanes per edge", g.L);
    }
}

}  // namespace csr
}  // namespace tiga
