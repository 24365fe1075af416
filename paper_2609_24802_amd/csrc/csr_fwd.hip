// Fused CSR gather-reduce: forward aggregation (sum / max) and the transposed
// gather used by the deterministic backward.
#include "csr_fwd.hpp"

namespace tiga {
namespace csr {

namespace {

// Relations at most this large take the single-launch direct traversal (no plan, no merge): their
// time is launch latency, which the plan's three extra launches and the merge would dominate.
constexpr int64_t kDirectEdges = int64_t{1} << 16;
constexpr int64_t kDirectRows = int64_t{1} << 16;

// Edge gradient of the backward, formed during the traversal of the reverse
// incidence: dw[e] = <x_j, dy[dst(e)]> for the source row j being folded
// (for max, only the units whose argmax is e are nonzero when they arrive).  Each lane holds one unit of x_j; the L lanes of an edge slot add
// their parts by a fixed shuffle tree and the slot's first lane writes dw[e].
// The row must fit one feature block (fu <= L).
template <int K, int L>
struct DwHook {
    float xj[K];
    float *__restrict__ dw;
    int l;
    template <int KK>
    __device__ __forceinline__ void edge(const Vec<KK> &g, int32_t e, bool ok) {
        float p = 0.0f;
#pragma unroll
        for (int k = 0; k < K; ++k) p = fmaf(xj[k], g.v[k], p);
#pragma unroll
        for (int m = 1; m < L; m <<= 1) p += shfl_xor_f(p, m);
        if (ok && l == 0) dw[e] = p;
    }
};

// Fold one chunk (or short row) per group, reduce the group's slots, and
// write the finalized output row or the chunk's partial state.  With DW the
// fold also forms the edge gradients (DwHook; x rows in hx, output hdw).
template <int K, int L, int RED, int WM, bool BUF, bool NT, bool DW = false>
struct GatherBody {
    const Trav &t;
    const Table<K, BUF, NT> &tab;
    const __amdgpu_buffer_rsrc_t &ars;
    float *__restrict__ out;
    int32_t *__restrict__ out_arg;
    float *__restrict__ part_v;
    int32_t *__restrict__ part_e;
    const float *__restrict__ hx;
    float *__restrict__ hdw;

    template <int GL>
    __device__ __forceinline__ void run(const Meta &m, int glane) {
        using A = Acc<K, RED>;
        const int s = glane / L;
        const int l = glane % L;
        for (int64_t fb = 0; fb < t.fu; fb += L) {
            const int64_t u = fb + l;
            const bool uok = u < t.fu;
            A acc;
            acc.init();
            if constexpr (DW) {
                DwHook<K, L> h;
                h.dw = hdw;
                h.l = l;
                const bool own = uok && m.n > 0;
                const Vec<K> xr = load_unit<K>(hx, own ? static_cast<int64_t>(m.row) * t.fu + u : 0);
#pragma unroll
                for (int k = 0; k < K; ++k) h.xj[k] = own ? xr.v[k] : 0.0f;
                run_edges<K, RED, WM, GL / L, BUF, NT>(t, tab, ars, m.e0, m.e0 + m.n, s, u, uok, acc, h);
            } else {
                run_edges<K, RED, WM, GL / L, BUF, NT>(t, tab, ars, m.e0, m.e0 + m.n, s, u, uok, acc);
            }
            reduce_lanes<L, GL>(acc);
            if (m.write && s == 0 && uok) {
                if (m.slot < 0) {
                    acc.finalize();
                    const int64_t unit = static_cast<int64_t>(m.row) * t.fu + u;
                    store_unit<K>(out, unit, acc.v);
                    if constexpr (RED == RED_MAX) store_unit_i<K>(out_arg, unit, acc.e);
                } else {
                    const int64_t unit = static_cast<int64_t>(m.slot) * t.fu + u;
                    store_unit<K>(part_v, unit, acc.v);
                    if constexpr (RED == RED_MAX) store_unit_i<K>(part_e, unit, acc.e);
                }
            }
        }
    }
};

template <int K, int L, int RED, int WM, bool BUF, bool NT, bool DW>
__global__ __launch_bounds__(kBlock) void gather_reduce_kernel(Trav t, int64_t n_groups,
                                                               const Desc *__restrict__ chunks,
                                                               const PlanCounts *__restrict__ counts,
                                                               float *__restrict__ out,
                                                               int32_t *__restrict__ out_arg,
                                                               float *__restrict__ part_v,
                                                               int32_t *__restrict__ part_e,
                                                               const float *__restrict__ hx,
                                                               float *__restrict__ hdw) {
    const Table<K, BUF, NT> tab(t.table, t.fu, t.table_bytes);
    // argmax table (max-routing gather only; otherwise an unused empty resource)
    const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(t.arg), 0, (BUF && WM == W_ROUTE) ? t.table_bytes : 0u, kBufWord3);
    GatherBody<K, L, RED, WM, BUF, NT, DW> body{t, tab, ars, out, out_arg, part_v, part_e, hx, hdw};
    const Items items = make_items(counts, n_groups);
    for_each_item<L>(items, chunks, t.ptr, t.nrows, body);
}

// Small relations (at most kDirectEdges edges and kDirectRows rows): no plan and no merge, one
// launch.  Wavefront w folds rows w, w + nwaves, ... with all 64 lanes, whatever their degree (a
// row of kDirectEdges edges is about a thousand 64-edge steps), and writes each finalized row.
template <int K, int L, int RED, int WM, bool BUF, bool NT, bool DW>
__global__ __launch_bounds__(kBlock) void direct_kernel(Trav t, float *__restrict__ out, int32_t *__restrict__ out_arg,
                                                        const float *__restrict__ hx, float *__restrict__ hdw) {
    const Table<K, BUF, NT> tab(t.table, t.fu, t.table_bytes);
    const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(t.arg), 0, (BUF && WM == W_ROUTE) ? t.table_bytes : 0u, kBufWord3);
    GatherBody<K, L, RED, WM, BUF, NT, DW> body{t, tab, ars, out, out_arg, nullptr, nullptr, hx, hdw};
    const int lane = lane_id();
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
    for (int64_t row = wave; row < t.nrows; row += nwaves) {
        const int64_t e0 = t.ptr[row];
        const Meta m{e0, static_cast<int32_t>(t.ptr[row + 1] - e0), static_cast<int32_t>(row), -1, 1};
        body.template run<kWave>(m, lane);
    }
}

// Merge the partial states of split rows in chunk order: lane slot s folds
// chunks s, s + S, ..., then the slots are combined by a fixed shuffle tree.
template <int K, int L, int RED>
__global__ __launch_bounds__(kBlock) void merge_kernel(const Split *__restrict__ splits,
                                                       const PlanCounts *__restrict__ counts, int64_t fu,
                                                       const float *__restrict__ part_v,
                                                       const int32_t *__restrict__ part_e,
                                                       float *__restrict__ out, int32_t *__restrict__ out_arg) {
    constexpr Geom g = make_geom(L);
    using A = Acc<K, RED>;
    const int lane = lane_id();
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
    const int64_t n_split = static_cast<int64_t>(counts->ctr[kCtrSplits].v);
    const int s = lane / L;
    const int l = lane % L;
    for (int64_t it = wave; it < n_split; it += nwaves) {
        const Split d = splits[it];
        const int64_t row = d.row;
        for (int64_t fb = 0; fb < fu; fb += L) {
            const int64_t u = fb + l;
            const bool uok = u < fu;
            A acc;
            acc.init();
            if (uok) {
                for (int c = s; c < d.nch; c += g.S) {
                    const int64_t unit = (static_cast<int64_t>(d.slot0) + c) * fu + u;
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

template <int K, int L, int RED, int WM, bool BUF, bool NT, bool DW>
int launch_gather_reduce(const Trav &t, int64_t n_groups, const PlanWs &w, const PlanBounds &b, float *out,
                         int32_t *out_arg, const EdgeGrad &eg, hipStream_t stream) {
    auto kern = gather_reduce_kernel<K, L, RED, WM, BUF, NT, DW>;
    static const int per_cu = resident_blocks(reinterpret_cast<const void *>(kern), kBlock);
    const int blocks = persistent_blocks(n_groups + b.max_chunks, per_cu);
    prof_before(stream);
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(kBlock), 0, stream, t, n_groups, w.chunks, w.counts, out, out_arg,
                       w.part_v, w.part_e, eg.x, eg.dw);
    prof_after(stream);
    return check_launch("gather-reduce");
}

template <int K, int L, int RED, int WM, bool BUF, bool NT, bool DW>
int launch_direct(const Trav &t, float *out, int32_t *out_arg, const EdgeGrad &eg, hipStream_t stream) {
    auto kern = direct_kernel<K, L, RED, WM, BUF, NT, DW>;
    static const int per_cu = resident_blocks(reinterpret_cast<const void *>(kern), kBlock);
    const int blocks = persistent_blocks(t.nrows, per_cu);
    prof_before(stream);
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(kBlock), 0, stream, t, out, out_arg, eg.x, eg.dw);
    prof_after(stream);
    return check_launch("direct gather-reduce");
}

template <int K, int L, int RED, int WM, bool DW>
int launch_traversal_t(const Trav &t, int64_t nedges, const PlanWs &w, const PlanBounds &b, float *out,
                       int32_t *out_arg, const EdgeGrad &eg, hipStream_t stream, bool direct) {
    constexpr Geom g = make_geom(L);
    if (direct) {
        if (!t.table_bytes) return launch_direct<K, L, RED, WM, false, true, DW>(t, out, out_arg, eg, stream);
        return launch_direct<K, L, RED, WM, true, false, DW>(t, out, out_arg, eg, stream);
    }
    if (int rc = launch_plan(t.ptr, t.nrows, g, b, w, stream)) return rc;
    const int64_t n_groups = ceil_div(t.nrows, g.RPW);
    int rc;
    if (!t.table_bytes)
        rc = launch_gather_reduce<K, L, RED, WM, false, true, DW>(t, n_groups, w, b, out, out_arg, eg, stream);
    else if (t.table_bytes > kStreamTableBytes)
        rc = launch_gather_reduce<K, L, RED, WM, true, true, DW>(t, n_groups, w, b, out, out_arg, eg, stream);
    else
        rc = launch_gather_reduce<K, L, RED, WM, true, false, DW>(t, n_groups, w, b, out, out_arg, eg, stream);
    if (rc) return rc;
    const int mblocks = persistent_blocks(b.max_splits, 4);
    hipLaunchKernelGGL((merge_kernel<K, L, RED>), dim3(mblocks), dim3(kBlock), 0, stream, w.splits, w.counts,
                       t.fu, w.part_v, w.part_e, out, out_arg);
    return check_launch("merge");
}

template <int K, int RED, int WM, bool DW = false>
int dispatch_lanes(int L, const Trav &t, int64_t nedges, const PlanWs &w, const PlanBounds &b, float *out,
                   int32_t *out_arg, const EdgeGrad &eg, hipStream_t stream, bool direct) {
    switch (L) {
        case 1: return launch_traversal_t<K, 1, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
        case 2: return launch_traversal_t<K, 2, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
        case 4: return launch_traversal_t<K, 4, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
        case 8: return launch_traversal_t<K, 8, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
        case 16: return launch_traversal_t<K, 16, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
        case 32: return launch_traversal_t<K, 32, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
        case 64: return launch_traversal_t<K, 64, RED, WM, DW>(t, nedges, w, b, out, out_arg, eg, stream, direct);
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

bool direct_traversal(int64_t nrows, int64_t nedges) { return nedges <= kDirectEdges && nrows <= kDirectRows; }

int launch_traversal(const Trav &t0, int64_t table_rows, int64_t nedges, const Layout &lay, int red, int wm, void *ws,
                     float *out, int32_t *out_arg, hipStream_t stream, bool direct, const EdgeGrad &eg) {
    if (t0.nrows == 0) return TIGA_OK;
    Trav t = t0;
    const int64_t tb = table_rows * lay.fu * lay.K * 4;
    t.table_bytes = (tb > 0 && tb < (int64_t{1} << 32)) ? static_cast<uint32_t>(tb) : 0u;
    const PlanBounds b = plan_bounds(t.nrows, nedges, lay.g);
    Carve c(ws);
    const PlanWs w = carve_plan(c, b, lay.fu * lay.K, red == RED_MAX);
    if (eg.dw) {
        // fused backward over the reverse incidence (sum: W_INDIRECT; max: the
        // argmax-routed W_ROUTE, whose unselected units reach the hook as zero)
        if (red != RED_SUM || (wm != W_INDIRECT && wm != W_ROUTE) || lay.fu > lay.L)
            return fail(TIGA_EUNSUPPORTED, "internal: fused edge gradients need a routed sum over one feature block");
        if (wm == W_INDIRECT) {
            if (lay.K == 4)
                return dispatch_lanes<4, RED_SUM, W_INDIRECT, true>(lay.L, t, nedges, w, b, out, out_arg, eg, stream, direct);
            return dispatch_lanes<1, RED_SUM, W_INDIRECT, true>(lay.L, t, nedges, w, b, out, out_arg, eg, stream, direct);
        }
        if (lay.K == 4)
            return dispatch_lanes<4, RED_SUM, W_ROUTE, true>(lay.L, t, nedges, w, b, out, out_arg, eg, stream, direct);
        return dispatch_lanes<1, RED_SUM, W_ROUTE, true>(lay.L, t, nedges, w, b, out, out_arg, eg, stream, direct);
    }
#define TIGA_DISPATCH(KK, RR, WW) \
    if (lay.K == KK && red == RR && wm == WW) return dispatch_lanes<KK, RR, WW>(lay.L, t, nedges, w, b, out, out_arg, eg, stream, direct)
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
