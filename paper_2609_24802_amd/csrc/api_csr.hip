// C ABI of the stored-CSR entry points: argument checks and dispatch.
#include "csr_bwd.hpp"
#include "csr_fwd.hpp"

using namespace tiga;
using namespace tiga::csr;

namespace {

int check_csr_meta(const tiga_csr *rel) {
    if (!rel) return fail(TIGA_EINVAL, "rel is NULL");
    if (rel->num_dst < 0 || rel->num_src < 0 || rel->num_edges < 0)
        return fail(TIGA_EINVAL, "negative relation size (num_dst %lld, num_src %lld, num_edges %lld)",
                    (long long)rel->num_dst, (long long)rel->num_src, (long long)rel->num_edges);
    if (rel->num_dst > INT32_MAX - 1)
        return fail(TIGA_EUNSUPPORTED, "num_dst %lld exceeds 2^31 - 2", (long long)rel->num_dst);
    if (rel->num_src > static_cast<int64_t>(INT32_MAX) + 1)
        return fail(TIGA_EUNSUPPORTED, "num_src %lld exceeds the int32 source-id range",
                    (long long)rel->num_src);
    if (rel->num_dst > 0 && !rel->row_ptr) return fail(TIGA_EINVAL, "row_ptr is NULL");
    if (rel->num_edges > 0 && !rel->col_idx) return fail(TIGA_EINVAL, "col_idx is NULL");
    if (rel->num_edges > 0 && rel->num_dst == 0)
        return fail(TIGA_EINVAL, "num_edges %lld > 0 with no destination rows", (long long)rel->num_edges);
    if (rel->num_edges > 0 && rel->num_src == 0)
        return fail(TIGA_EINVAL, "num_edges %lld > 0 with no source entities", (long long)rel->num_edges);
    return TIGA_OK;
}

int check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (ws_bytes < need)
        return fail(TIGA_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, need);
    if (need > 0 && !ws) return fail(TIGA_EINVAL, "ws is NULL");
    if (ws && (reinterpret_cast<uintptr_t>(ws) & 255u))
        return fail(TIGA_EINVAL, "ws must be 256-byte aligned");
    return TIGA_OK;
}

int check_common(const tiga_csr *rel, int32_t feat, int msg, const float *w_edge, int reducer) {
    if (int rc = check_csr_meta(rel)) return rc;
    if (feat < 1) return fail(TIGA_EINVAL, "feat must be >= 1 (got %d)", feat);
    if (reducer != TIGA_REDUCE_SUM && reducer != TIGA_REDUCE_MAX)
        return fail(TIGA_EINVAL, "unknown reducer %d", reducer);
    if (msg != TIGA_MSG_SRC && msg != TIGA_MSG_EDGE_SCALED_SRC) return fail(TIGA_EINVAL, "unknown message %d", msg);
    if (msg == TIGA_MSG_SRC && w_edge) return fail(TIGA_EINVAL, "w_edge must be NULL for TIGA_MSG_SRC");
    if (msg == TIGA_MSG_EDGE_SCALED_SRC && !w_edge && rel->num_edges > 0)
        return fail(TIGA_EINVAL, "w_edge is required for TIGA_MSG_EDGE_SCALED_SRC");
    if (reducer == TIGA_REDUCE_MAX && rel->num_edges > INT32_MAX)
        return fail(TIGA_EUNSUPPORTED, "max reducer needs num_edges < 2^31 (argmax is int32)");
    return TIGA_OK;
}

}  // namespace

extern "C" {

size_t tiga_mp_csr_fwd_paged_workspace(int32_t feat, int reducer, int64_t page_edges) {
    if (feat < 1 || page_edges < 1 || page_edges > INT32_MAX) return 0;
    if (reducer != TIGA_REDUCE_SUM && reducer != TIGA_REDUCE_MAX) return 0;
    return paged_ws_bytes(page_edges, feat, reducer == TIGA_REDUCE_MAX);
}

int tiga_mp_csr_fwd_paged(const tiga_csr *rel_host, int32_t feat, const float *x_src, int msg, const float *w_host,
                          int reducer, float *y, int32_t *argmax, int64_t page_edges, void *ws, size_t ws_bytes,
                          void *stream) {
    EntryScope scope;
    if (int rc = check_common(rel_host, feat, msg, w_host, reducer)) return rc;
    if (page_edges < 1 || page_edges > INT32_MAX) return fail(TIGA_EINVAL, "page_edges must be in [1, 2^31)");
    if (rel_host->num_dst == 0) return TIGA_OK;
    if (!y) return fail(TIGA_EINVAL, "y is NULL");
    if (rel_host->num_edges > 0 && !x_src) return fail(TIGA_EINVAL, "x_src is NULL");
    if (reducer == TIGA_REDUCE_MAX && !argmax) return fail(TIGA_EINVAL, "argmax is required for the max reducer");
    if (reducer == TIGA_REDUCE_SUM && argmax) return fail(TIGA_EINVAL, "argmax must be NULL for the sum reducer");
    // host-side metadata checks: the relation's ends, and no row longer than a page
    const int64_t *rp = rel_host->row_ptr;
    if (rp[0] != 0 || rp[rel_host->num_dst] != rel_host->num_edges)
        return fail(TIGA_EGRAPH, "row_ptr must start at 0 and end at num_edges");
    for (int64_t i = 0; i < rel_host->num_dst; ++i) {
        const int64_t d = rp[i + 1] - rp[i];
        if (d < 0) return fail(TIGA_EGRAPH, "row_ptr decreases at row %lld", (long long)i);
        if (d > page_edges)
            return fail(TIGA_EUNSUPPORTED, "row %lld has %lld edges, more than page_edges %lld", (long long)i,
                        (long long)d, (long long)page_edges);
    }
    const size_t need = paged_ws_bytes(page_edges, feat, reducer == TIGA_REDUCE_MAX);
    if (int rc = check_ws(ws, ws_bytes, need)) return rc;
    return launch_paged_fwd(rel_host, feat, x_src, msg == TIGA_MSG_EDGE_SCALED_SRC ? w_host : nullptr,
                            reducer == TIGA_REDUCE_MAX ? RED_MAX : RED_SUM, y, argmax, page_edges, ws,
                            static_cast<hipStream_t>(stream));
}

size_t tiga_mp_csr_fwd_workspace(const tiga_csr *rel, int32_t feat, int reducer) {
    if (!rel || feat < 1 || rel->num_dst < 0 || rel->num_edges < 0) return 0;
    if (reducer != TIGA_REDUCE_SUM && reducer != TIGA_REDUCE_MAX) return 0;
    return traversal_ws_bytes(rel->num_dst, rel->num_edges, feat, reducer == TIGA_REDUCE_MAX);
}

int tiga_mp_csr_fwd(const tiga_csr *rel, int32_t feat, const float *x_src, int msg, const float *w_edge,
                    int reducer, float *y, int32_t *argmax, void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_common(rel, feat, msg, w_edge, reducer)) return rc;
    if (rel->num_dst == 0) return TIGA_OK;
    if (!y) return fail(TIGA_EINVAL, "y is NULL");
    if (rel->num_edges > 0 && !x_src) return fail(TIGA_EINVAL, "x_src is NULL");
    if (reducer == TIGA_REDUCE_MAX && !argmax) return fail(TIGA_EINVAL, "argmax is required for the max reducer");
    if (reducer == TIGA_REDUCE_SUM && argmax) return fail(TIGA_EINVAL, "argmax must be NULL for the sum reducer");
    const size_t need = tiga_mp_csr_fwd_workspace(rel, feat, reducer);
    if (int rc = check_ws(ws, ws_bytes, need)) return rc;
    const bool vec = feat % 4 == 0 && aligned16(x_src) && aligned16(y) && (!argmax || aligned16(argmax));
    const Layout lay = layout_for(feat, vec);
    Trav t{rel->row_ptr, rel->col_idx, w_edge, nullptr, x_src, rel->num_dst, lay.fu, nullptr, 0u, rel->num_edges};
    const int wm = msg == TIGA_MSG_EDGE_SCALED_SRC ? W_DIRECT : W_NONE;
    return launch_traversal(t, rel->num_src, rel->num_edges, lay, reducer == TIGA_REDUCE_MAX ? RED_MAX : RED_SUM, wm, ws, y,
                            argmax, static_cast<hipStream_t>(stream), direct_traversal(rel->num_dst, rel->num_edges));
}

size_t tiga_mp_csr_bwd_workspace(const tiga_csr *rel, int32_t feat, int reducer) {
    if (!rel || feat < 1 || rel->num_dst < 0 || rel->num_src < 0 || rel->num_edges < 0) return 0;
    if (reducer != TIGA_REDUCE_SUM && reducer != TIGA_REDUCE_MAX) return 0;
    return bwd_ws_bytes(rel->num_dst, rel->num_src, rel->num_edges, feat);
}

int tiga_mp_csr_bwd(const tiga_csr *rel, const tiga_csr_t *rev, int32_t feat, const float *x_src, int msg,
                    const float *w_edge, int reducer, const int32_t *argmax, const float *dy, float *dx,
                    float *dw, void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_common(rel, feat, msg, w_edge, reducer)) return rc;
    if (dw && msg != TIGA_MSG_EDGE_SCALED_SRC)
        return fail(TIGA_EINVAL, "dw requires TIGA_MSG_EDGE_SCALED_SRC");
    if (!dx && !dw) return TIGA_OK;
    if (reducer == TIGA_REDUCE_MAX && !argmax && rel->num_dst > 0)
        return fail(TIGA_EINVAL, "argmax is required for the max reducer");
    if (!dy && rel->num_dst > 0) return fail(TIGA_EINVAL, "dy is NULL");
    if (dw && rel->num_edges > 0 && !x_src) return fail(TIGA_EINVAL, "x_src is NULL (needed for dw)");
    if (rev) {
        if (rel->num_edges > INT32_MAX)
            return fail(TIGA_EUNSUPPORTED, "reverse incidence needs num_edges < 2^31");
        if (rel->num_src > 0 && !rev->src_ptr) return fail(TIGA_EINVAL, "rev->src_ptr is NULL");
        if (rel->num_edges > 0 && !rev->edge_id) return fail(TIGA_EINVAL, "rev->edge_id is NULL");
    }
    const size_t need = tiga_mp_csr_bwd_workspace(rel, feat, reducer);
    if (int rc = check_ws(ws, ws_bytes, need)) return rc;
    BwdArgs a{rel, rev, feat, x_src, msg == TIGA_MSG_EDGE_SCALED_SRC ? w_edge : nullptr,
              reducer == TIGA_REDUCE_MAX ? RED_MAX : RED_SUM, argmax, dy, dx, dw};
    return launch_bwd(a, ws, static_cast<hipStream_t>(stream));
}

size_t tiga_csr_transpose_workspace(const tiga_csr *rel) {
    if (!rel || rel->num_dst < 0 || rel->num_src < 0 || rel->num_edges < 0) return 0;
    return transpose_ws_bytes(rel->num_dst, rel->num_src, rel->num_edges);
}

int tiga_csr_transpose(const tiga_csr *rel, int64_t *src_ptr, int32_t *edge_id, void *ws, size_t ws_bytes,
                       void *stream) {
    EntryScope scope;
    if (int rc = check_csr_meta(rel)) return rc;
    if (rel->num_edges > INT32_MAX) return fail(TIGA_EUNSUPPORTED, "transpose needs num_edges < 2^31");
    if (!src_ptr) return fail(TIGA_EINVAL, "src_ptr is NULL");
    if (rel->num_edges > 0 && !edge_id) return fail(TIGA_EINVAL, "edge_id is NULL");
    const size_t need = tiga_csr_transpose_workspace(rel);
    if (int rc = check_ws(ws, ws_bytes, need)) return rc;
    return launch_transpose(rel, src_ptr, edge_id, ws, static_cast<hipStream_t>(stream));
}

int tiga_csr_validate(const tiga_csr *rel, int level, void *stream) {
    EntryScope scope;
    if (level != 1 && level != 2) return fail(TIGA_EINVAL, "validation level must be 1 or 2 (got %d)", level);
    if (int rc = check_csr_meta(rel)) return rc == TIGA_EINVAL ? TIGA_EGRAPH : rc;
    if (level == 1) return TIGA_OK;
    return launch_validate(rel, static_cast<hipStream_t>(stream));
}

}  // extern "C"
