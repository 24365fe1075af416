// Vector-Jacobian products of the CSR aggregation (Section 5 of the paper):
//   sum: dx[j] = sum_{e: col[e]=j} w[e] dy[d(e)],  dw[e] = <x[col[e]], dy[d(e)]>
//   max: the same terms, restricted per (row, feature) to the argmax edge.
// dw is computed row-parallel on the forward relation (each edge is written
// once: deterministic).  dx either scatters with device atomics from the same
// pass, or is gathered over the reverse incidence (deterministic).
#include "csr_bwd.hpp"

namespace tiga {
namespace csr {

namespace {

struct EdgeT {
    const int64_t *__restrict__ ptr;
    const int32_t *__restrict__ col;
    const float *__restrict__ w;
    const float *__restrict__ x;
    const float *__restrict__ dy;
    const int32_t *__restrict__ arg;
    float *__restrict__ dx;
    float *__restrict__ dw;
    int64_t nrows;
    int64_t fu;
};

// Edges [e0, e1) of `row`; this lane is slot s (of SL) and unit u.
template <int K, int L, int RED, bool DW, bool DX, int SL>
__device__ __forceinline__ void edge_pass(const EdgeT &t, int64_t row, int64_t e0, int64_t e1, int s, int l,
                                          int64_t u, bool uok, bool first_block) {
    Vec<K> g;
    int ga[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        g.v[k] = 0.0f;
        ga[k] = -1;
    }
    if (uok && e1 > e0) {
        g = load_unit<K>(t.dy, row * t.fu + u);
        if constexpr (RED == RED_MAX) load_unit_i<K>(t.arg, row * t.fu + u, ga);
    }
    // dx is scattered lane-contiguously: atomic k of lane l adds to float f0 + k L of the source
    // row, f0 = (u - l) K + l. Over the L lanes and K atomics this covers exactly the K L floats of
    // units u - l .. u - l + L - 1, and each atomic instruction of an edge writes one contiguous
    // run of L floats instead of L floats spaced K apart.
    const int64_t nf = t.fu * K, f0 = (u - l) * K + l;
    float gt[K];
    int gat[K];
    bool fok[K];
    if constexpr (DX) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int64_t f = f0 + static_cast<int64_t>(k) * L;
            fok[k] = f < nf && e1 > e0;
            gt[k] = fok[k] ? t.dy[row * nf + f] : 0.0f;
            gat[k] = -1;
            if constexpr (RED == RED_MAX) gat[k] = fok[k] ? t.arg[row * nf + f] : -1;
        }
    }
    for (int64_t base = e0; base < e1; base += SL * kUnroll) {
        int32_t c[kUnroll];
        float wv[kUnroll];
        bool ok[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int64_t e = base + static_cast<int64_t>(r) * SL + s;
            ok[r] = e < e1;
            c[r] = ok[r] ? t.col[e] : 0;  // cached: neighbouring items share lines
            wv[r] = ok[r] ? (t.w ? t.w[e] : 1.0f) : 0.0f;
        }
        Vec<K> xv[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            if (DW && ok[r] && uok) {
                xv[r] = load_unit<K>(t.x, static_cast<int64_t>(c[r]) * t.fu + u);
            } else {
#pragma unroll
                for (int k = 0; k < K; ++k) xv[r].v[k] = 0.0f;
            }
        }
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int64_t e = base + static_cast<int64_t>(r) * SL + s;
            if constexpr (DX) {
                if (ok[r]) {
                    float *dst = t.dx + static_cast<int64_t>(c[r]) * nf + f0;
#pragma unroll
                    for (int k = 0; k < K; ++k)
                        if (fok[k] && (RED == RED_SUM || gat[k] == static_cast<int>(e)))
                            unsafeAtomicAdd(dst + k * L, wv[r] * gt[k]);
                }
            }
            if constexpr (DW) {
                float p = 0.0f;
#pragma unroll
                for (int k = 0; k < K; ++k)
                    if (RED == RED_SUM || ga[k] == static_cast<int>(e)) p = fmaf(xv[r].v[k], g.v[k], p);
#pragma unroll
                for (int m = 1; m < L; m <<= 1) p += shfl_xor_f(p, m);
                if (l == 0 && ok[r]) t.dw[e] = first_block ? p : t.dw[e] + p;
            }
        }
    }
}

template <int K, int L, int RED, bool DW, bool DX>
struct EdgeBody {
    const EdgeT &t;

    template <int GL>
    __device__ __forceinline__ void run(const Meta &m, int glane) {
        const int l = glane % L;
        for (int64_t fb = 0; fb < t.fu; fb += L) {
            const int64_t u = fb + l;
            edge_pass<K, L, RED, DW, DX, GL / L>(t, m.row, m.e0, m.e0 + m.n, glane / L, l, u, u < t.fu, fb == 0);
        }
    }

};

template <int K, int L, int RED, bool DW, bool DX>
__global__ __launch_bounds__(kBlock) void edge_kernel(EdgeT t, int64_t n_groups, const Desc *__restrict__ chunks,
                                                      const PlanCounts *__restrict__ counts) {
    EdgeBody<K, L, RED, DW, DX> body{t};
    const Items items = make_items(counts, n_groups);
    for_each_item<L>(items, chunks, t.ptr, t.nrows, body);
}

template <int K, int L, int RED, bool DW, bool DX>
int launch_edge_t(const EdgeT &t, int64_t nedges, void *ws, hipStream_t stream) {
    constexpr Geom g = make_geom(L);
    const PlanBounds b = plan_bounds(t.nrows, nedges, g);
    Carve c(ws);
    const PlanWs w = carve_plan(c, b, t.fu * K, false);
    if (int rc = launch_plan(t.ptr, t.nrows, g, b, w, stream)) return rc;
    const int64_t n_groups = ceil_div(t.nrows, g.RPW);
    auto kern = edge_kernel<K, L, RED, DW, DX>;
    static const int per_cu = resident_blocks(reinterpret_cast<const void *>(kern), kBlock);
    const int blocks = persistent_blocks(n_groups + b.max_chunks, per_cu);
    prof_before(stream);
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(kBlock), 0, stream, t, n_groups, w.chunks, w.counts);
    prof_after(stream);
    return check_launch("edge backward");
}

template <int K, int RED, bool DW, bool DX>
int edge_lanes(int L, const EdgeT &t, int64_t nedges, void *ws, hipStream_t stream) {
    switch (L) {
        case 1: return launch_edge_t<K, 1, RED, DW, DX>(t, nedges, ws, stream);
        case 2: return launch_edge_t<K, 2, RED, DW, DX>(t, nedges, ws, stream);
        case 4: return launch_edge_t<K, 4, RED, DW, DX>(t, nedges, ws, stream);
        case 8: return launch_edge_t<K, 8, RED, DW, DX>(t, nedges, ws, stream);
        case 16: return launch_edge_t<K, 16, RED, DW, DX>(t, nedges, ws, stream);
        case 32: return launch_edge_t<K, 32, RED, DW, DX>(t, nedges, ws, stream);
        case 64: return launch_edge_t<K, 64, RED, DW, DX>(t, nedges, ws, stream);
        default: return fail(TIGA_EINVAL, "internal: lanes per edge %d", L);
    }
}

template <int K, int RED>
int edge_flags(bool dw, bool dx, int L, const EdgeT &t, int64_t nedges, void *ws, hipStream_t stream) {
    if (dw && dx) return edge_lanes<K, RED, true, true>(L, t, nedges, ws, stream);
    if (dw) return edge_lanes<K, RED, true, false>(L, t, nedges, ws, stream);
    return edge_lanes<K, RED, false, true>(L, t, nedges, ws, stream);
}

// Workspace of the backward: the (weight, destination row) record of every edge (used with the
// reverse incidence), then the region the plan of either traversal takes.
struct BwdWs {
    int2 *rec;
    void *rest;
};

BwdWs carve_bwd(void *ws, int64_t num_edges) {
    Carve c(ws);
    BwdWs w;
    w.rec = c.take<int2>(num_edges);
    w.rest = ws ? static_cast<char *>(ws) + c.bytes() : nullptr;
    return w;
}

size_t bwd_rows_bytes(int64_t num_edges) {
    Carve c(nullptr);
    c.take<int2>(num_edges);
    return c.bytes();
}

}  // namespace

size_t bwd_ws_bytes(int64_t num_dst, int64_t num_src, int64_t num_edges, int64_t feat) {
    size_t a = traversal_ws_bytes(num_dst, num_edges, feat, false);
    size_t b = traversal_ws_bytes(num_src, num_edges, feat, false);
    return bwd_rows_bytes(num_edges) + (a > b ? a : b);
}

int launch_bwd(const BwdArgs &a, void *ws_all, hipStream_t stream) {
    const tiga_csr *rel = a.rel;
    const BwdWs bw = carve_bwd(ws_all, rel->num_edges);
    void *ws = bw.rest;
    const bool vec = a.feat % 4 == 0 && aligned16(a.dy) && (!a.dx || aligned16(a.dx)) &&
                     (!a.dw || !a.x || aligned16(a.x)) && (!a.arg || aligned16(a.arg));
    const Layout lay = layout_for(a.feat, vec);
    const bool atomic_dx = a.dx && !a.rev;
    if (atomic_dx) {
        if (int rc = fill_u32(a.dx, 0u, rel->num_src * static_cast<int64_t>(a.feat), stream)) return rc;
    }
    // With the reverse incidence and both gradients: one traversal of the
    // reverse incidence gathers each dy row once and forms dx_j and dw_e
    // together (x_j is the source's own row), when the row fits one feature
    // block.  Otherwise dw comes from the row-parallel edge kernel.
    const bool fused = a.rev && a.dx && a.dw && a.x && lay.fu <= lay.L;
    if ((a.dw || atomic_dx) && !fused && rel->num_dst > 0) {
        EdgeT t{rel->row_ptr, rel->col_idx, a.w, a.x, a.dy, a.arg, atomic_dx ? a.dx : nullptr, a.dw,
                rel->num_dst, lay.fu};
        int rc;
        if (lay.K == 4)
            rc = a.red == RED_MAX ? edge_flags<4, RED_MAX>(a.dw != nullptr, atomic_dx, lay.L, t, rel->num_edges, ws, stream)
                                  : edge_flags<4, RED_SUM>(a.dw != nullptr, atomic_dx, lay.L, t, rel->num_edges, ws, stream);
        else
            rc = a.red == RED_MAX ? edge_flags<1, RED_MAX>(a.dw != nullptr, atomic_dx, lay.L, t, rel->num_edges, ws, stream)
                                  : edge_flags<1, RED_SUM>(a.dw != nullptr, atomic_dx, lay.L, t, rel->num_edges, ws, stream);
        if (rc) return rc;
    }
    if (a.dx && a.rev && rel->num_src > 0) {
        // the reverse incidence carries forward edge ids only: each traversed slot reads its edge's
        // (weight, destination row) record, built here from row_ptr and w in one streaming pass
        if (int rc = launch_edge_records(rel, a.w, bw.rec, stream)) return rc;
        Trav t{a.rev->src_ptr, nullptr, nullptr, a.rev->edge_id, a.dy, rel->num_src, lay.fu, a.arg, 0u,
               rel->num_edges, bw.rec};
        const int wm = a.red == RED_MAX ? W_ROUTE : W_INDIRECT;
        EdgeGrad eg;
        if (fused) {
            eg.x = a.x;
            eg.dw = a.dw;
        }
        if (int rc = launch_traversal(t, rel->num_dst, rel->num_edges, lay, RED_SUM, wm, ws, a.dx, nullptr, stream,
                                      direct_traversal(rel->num_src, rel->num_edges), eg))
            return rc;
    }
    return TIGA_OK;
}

}  // namespace csr
}  // namespace tiga
