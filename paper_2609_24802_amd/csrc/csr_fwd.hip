// Fused CSR gather-reduce: forward aggregation (sum / max) and the transposed
// gather used by the deterministic backward.
#include "csr_fwd.hpp"

namespace tiga {
namespace csr {

namespace {

// Persistent traversal: work items are [chunk descriptors | short-row groups];
// each wavefront takes items it, it + nwaves, ...  Every wavefront leaves the
// loop once `it` passes the item count, so the grid always drains.
template <int K, int L, int RED, int WM>
__global__ __launch_bounds__(kBlock) void gather_reduce_kernel(Trav t, int64_t n_groups,
                                                               const Desc *__restrict__ chunks,
                                                               const PlanCounts *__restrict__ counts,
                                                               float *__restrict__ out,
                                                               int32_t *__restrict__ out_arg,
                                                               float *__restrict__ part_v,
                                                               int32_t *__restrict__ part_e) {
    constexpr Geom g = make_geom(L);
    using A = Acc<K, RED>;
    const int lane = lane_id();
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
    const int64_t n_chunks = static_cast<int64_t>(counts->chunks);
    const int64_t total = n_chunks + n_groups;
    const int l = lane % L;

    for (int64_t it = wave; it < total; it += nwaves) {
        if (it < n_chunks) {
            // one wavefront over up to CH edges of a medium or long row
            const Desc d = chunks[it];
            const int64_t row = d.x;
            const int64_t rb = t.ptr[row];
            const int64_t re = t.ptr[row + 1];
            const int64_t e0 = rb + static_cast<int64_t>(d.y) * g.CH;
            const int64_t e1 = (re < e0 + g.CH) ? re : e0 + g.CH;
            const int s = lane / L;
            for (int64_t fb = 0; fb < t.fu; fb += L) {
                const int64_t u = fb + l;
                const bool uok = u < t.fu;
                A acc;
                acc.init();
                run_edges<K, RED, WM, g.S>(t, e0, e1, s, u, uok, acc);
                reduce_lanes<L, kWave>(acc);
                if (s == 0 && uok) {
                    if (d.z < 0) {
                        acc.finalize();
                        store_unit<K>(out, row * t.fu + u, acc.v);
                        if constexpr (RED == RED_MAX) store_unit_i<K>(out_arg, row * t.fu + u, acc.e);
                    } else {
                        const int64_t slot = d.z;
                        store_unit<K>(part_v, slot * t.fu + u, acc.v);
                        if constexpr (RED == RED_MAX) store_unit_i<K>(part_e, slot * t.fu + u, acc.e);
                    }
                }
            }
        } else {
            // RPW short rows in natural order, one group of G lanes each
            const int64_t gi = it - n_chunks;
            const int grp = lane / g.G;
            const int s = (lane % g.G) / L;
            const int64_t row = gi * g.RPW + grp;
            int64_t e0 = 0, e1 = 0;
            bool mine = false;
            if (row < t.nrows) {
                e0 = t.ptr[row];
                e1 = t.ptr[row + 1];
                mine = (e1 - e0) <= g.DS;
            }
            if (!mine) e1 = e0;  // medium and long rows belong to chunk items
            for (int64_t fb = 0; fb < t.fu; fb += L) {
                const int64_t u = fb + l;
                const bool uok = u < t.fu;
                A acc;
                acc.init();
                run_edges<K, RED, WM, g.P>(t, e0, e1, s, u, uok, acc);
                reduce_lanes<L, g.G>(acc);
                if (mine && s == 0 && uok) {
                    acc.finalize();
                    store_unit<K>(out, row * t.fu + u, acc.v);
                    if constexpr (RED == RED_MAX) store_unit_i<K>(out_arg, row * t.fu + u, acc.e);
                }
            }
        }
    }
}

// Merge the partial states of split rows in chunk order: lane slot s folds
// chunks s, s + S, ..., then the slots are combined by a fixed shuffle tree.
template <int K, int L, int RED>
__global__ __launch_bounds__(kBlock) void merge_kernel(const Desc *__restrict__ splits,
                                                       const PlanCounts *__restrict__ counts, int64_t fu,
                                                       const float *__restrict__ part_v,
                                                       const int32_t *__restrict__ part_e,
                                                       float *__restrict__ out, int32_t *__restrict__ out_arg) {
    constexpr Geom g = make_geom(L);
    using A = Acc<K, RED>;
    const int lane = lane_id();
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
    const int64_t n_split = static_cast<int64_t>(counts->splits);
    const int s = lane / L;
    const int l = lane % L;
    for (int64_t it = wave; it < n_split; it += nwaves) {
        const Desc d = splits[it];
        const int64_t row = d.x;
        for (int64_t fb = 0; fb < fu; fb += L) {
            const int64_t u = fb + l;
            const bool uok = u < fu;
            A acc;
            acc.init();
            if (uok) {
                for (int c = s; c < d.z; c += g.S) {
                    const int64_t unit = (static_cast<int64_t>(d.y) + c) * fu + u;
                    Vec<K> p = load_unit<K>(part_v, unit);
                    int pe[K];
                    if constexpr (RED == RED_MAX) {
                        load_unit_i<K>(part_e, unit, pe);
                    } else {
#pragma unroll
                        for (int k = 0; k < K; ++k) pe[k] = 0;
                    }
                    acc.add_partial(p, pe);
                }
            }
            reduce_lanes<L, kWave>(acc);
            if (s == 0 && uok) {
                acc.finalize();
                store_unit<K>(out, row * fu + u, acc.v);
                if constexpr (RED == RED_MAX) store_unit_i<K>(out_arg, row * fu + u, acc.e);
            }
        }
    }
}

template <int K, int L, int RED, int WM>
int launch_traversal_t(const Trav &t, int64_t nedges, const PlanWs &w, const PlanBounds &b, float *out,
                       int32_t *out_arg, hipStream_t stream) {
    constexpr Geom g = make_geom(L);
    if (int rc = launch_plan(t.ptr, t.nrows, g, b, w, stream)) return rc;
    const int64_t n_groups = ceil_div(t.nrows, g.RPW);
    const int blocks = persistent_blocks(n_groups + b.max_chunks);
    prof_before(stream);
    hipLaunchKernelGGL((gather_reduce_kernel<K, L, RED, WM>), dim3(blocks), dim3(kBlock), 0, stream, t,
                       n_groups, w.chunks, w.counts, out, out_arg, w.part_v, w.part_e);
    prof_after(stream);
    if (int rc = check_launch("gather-reduce")) return rc;
    const int mblocks = persistent_blocks(b.max_splits, 4);
    hipLaunchKernelGGL((merge_kernel<K, L, RED>), dim3(mblocks), dim3(kBlock), 0, stream, w.splits, w.counts,
                       t.fu, w.part_v, w.part_e, out, out_arg);
    return check_launch("merge");
}

template <int K, int RED, int WM>
int dispatch_lanes(int L, const Trav &t, int64_t nedges, const PlanWs &w, const PlanBounds &b, float *out,
                   int32_t *out_arg, hipStream_t stream) {
    switch (L) {
        case 1: return launch_traversal_t<K, 1, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        case 2: return launch_traversal_t<K, 2, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        case 4: return launch_traversal_t<K, 4, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        case 8: return launch_traversal_t<K, 8, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        case 16: return launch_traversal_t<K, 16, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        case 32: return launch_traversal_t<K, 32, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        case 64: return launch_traversal_t<K, 64, RED, WM>(t, nedges, w, b, out, out_arg, stream);
        default: return fail(TIGA_EINVAL, "internal: lanes per edge %d", L);
    }
}

}  // namespace

Layout layout_for(int64_t feat, bool vec) {
    Layout lay;
    lay.K = vec ? 4 : 1;
    lay.fu = vec ? feat / 4 : feat;
    lay.L = lanes_for(lay.fu);
    lay.g = make_geom(lay.L);
    return lay;
}

size_t traversal_ws_bytes(int64_t nrows, int64_t nedges, int64_t feat, bool with_arg) {
    // the bound must hold for either unit width, so take the larger footprint
    size_t best = 0;
    for (int vec = 0; vec < 2; ++vec) {
        Layout lay = layout_for(feat, vec != 0 && feat % 4 == 0);
        Carve c(nullptr);
        carve_plan(c, plan_bounds(nrows, nedges, lay.g), feat, with_arg);
        if (c.bytes() > best) best = c.bytes();
    }
    return best;
}

int launch_traversal(const Trav &t, int64_t nedges, const Layout &lay, int red, int wm, void *ws, float *out,
                     int32_t *out_arg, hipStream_t stream) {
    if (t.nrows == 0) return TIGA_OK;
    const PlanBounds b = plan_bounds(t.nrows, nedges, lay.g);
    Carve c(ws);
    const PlanWs w = carve_plan(c, b, lay.fu * lay.K, red == RED_MAX);
#define TIGA_DISPATCH(KK, RR, WW) \
    if (lay.K == KK && red == RR && wm == WW) return dispatch_lanes<KK, RR, WW>(lay.L, t, nedges, w, b, out, out_arg, stream)
    TIGA_DISPATCH(4, RED_SUM, W_DIRECT);
    TIGA_DISPATCH(4, RED_SUM, W_NONE);
    TIGA_DISPATCH(4, RED_SUM, W_INDIRECT);
    TIGA_DISPATCH(4, RED_SUM, W_ROUTE);
    TIGA_DISPATCH(4, RED_MAX, W_DIRECT);
    TIGA_DISPATCH(4, RED_MAX, W_NONE);
    TIGA_DISPATCH(1, RED_SUM, W_DIRECT);
    TIGA_DISPATCH(1, RED_SUM, W_NONE);
    TIGA_DISPATCH(1, RED_SUM, W_INDIRECT);
    TIGA_DISPATCH(1, RED_SUM, W_ROUTE);
    TIGA_DISPATCH(1, RED_MAX, W_DIRECT);
    TIGA_DISPATCH(1, RED_MAX, W_NONE);
#undef TIGA_DISPATCH
    return fail(TIGA_EUNSUPPORTED, "internal: no traversal for reducer %d weight mode %d", red, wm);
}

}  // namespace csr
}  // namespace tiga
