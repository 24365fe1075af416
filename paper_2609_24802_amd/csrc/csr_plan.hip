// Degree-aware row plan, one pass over the rows.
//
// init: clear the counters and record where classes 1 and 2 start in the
//       chunk array (each class has a region of its own capacity);
// plan: each block takes a tile of kPlanTile rows, scans the chunks of each
//       class, partial slots and split rows its rows need (block-local scan),
//       reserves those ranges with one atomic add per counter, and writes the
//       descriptors in row order within its ranges.
// Only rows longer than the short-row bound get descriptors; short rows are
// taken in natural order by the traversal itself.
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

__global__ void plan_init_kernel(PlanCounts *__restrict__ counts, int64_t off1, int64_t off2) {
    if (threadIdx.x < kPlanVals) counts->ctr[threadIdx.x].v = 0;
    if (threadIdx.x == 0) {
        counts->off[0] = static_cast<unsigned long long>(off1);
        counts->off[1] = static_cast<unsigned long long>(off2);
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
__global__ __launch_bounds__(kBlock) void plan_kernel(const int64_t *__restrict__ ptr, int64_t nrows,
                                                      PlanCounts *__restrict__ counts, Desc *__restrict__ chunks,
                                                      Split *__restrict__ splits) {
    constexpr Geom g = make_geom(L);
    __shared__ int64_t sptr[pad_ix(kPlanTile) + 1];
    __shared__ int64_t sbase[kPlanVals];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPlanTile;
    for (int i = threadIdx.x; i <= kPlanTile; i += kBlock) {
        const int64_t row = base + i;
        sptr[pad_ix(i)] = ptr[row < nrows ? row : nrows];
    }
    __syncthreads();
    const int64_t cbase[kClasses] = {0, static_cast<int64_t>(counts->off[0]), static_cast<int64_t>(counts->off[1])};
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
    const Need tot = block_excl_scan(mine, run);
    // one reservation per counter for the whole tile: thread k adds the tile's total of counter k
    // (vector atomics, all in flight together)
    if (threadIdx.x < kPlanVals) {
        int64_t t = 0;
#pragma unroll
        for (int k = 0; k < kPlanVals; ++k) t = threadIdx.x == k ? tot.v[k] : t;
        sbase[threadIdx.x] =
            t > 0 ? static_cast<int64_t>(atomicAdd(&counts->ctr[threadIdx.x].v, static_cast<unsigned long long>(t))) : 0;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPlanVals; ++k) run.v[k] += sbase[k];
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
    hipLaunchKernelGGL(plan_init_kernel, dim3(1), dim3(kWave), 0, stream, w.counts, b.cap[0], b.cap[0] + b.cap[1]);
    if (int rc = check_launch("plan init")) return rc;
    hipLaunchKernelGGL(plan_kernel<L>, dim3(static_cast<unsigned>(b.tiles)), dim3(kBlock), 0, stream, ptr, nrows,
                       w.counts, w.chunks, w.splits);
    return check_launch("plan");
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
