// C ABI of the generated radius relation and the dense all-pairs relation.
#include "dense.hpp"
#include "edgenn.hpp"
#include "knn.hpp"
#include "radius.hpp"

using namespace tiga;

namespace {

int check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (ws_bytes < need)
        return fail(TIGA_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, need);
    if (need > 0 && !ws) return fail(TIGA_EINVAL, "ws is NULL");
    if (ws && (reinterpret_cast<uintptr_t>(ws) & 255u)) return fail(TIGA_EINVAL, "ws must be 256-byte aligned");
    return TIGA_OK;
}

int check_points(int64_t n, const float *pos) {
    if (n < 0) return fail(TIGA_EINVAL, "n must be >= 0 (got %lld)", (long long)n);
    if (n > INT32_MAX - 64) return fail(TIGA_EUNSUPPORTED, "n %lld exceeds the int32 point-id range", (long long)n);
    if (n > 0 && !pos) return fail(TIGA_EINVAL, "pos is NULL");
    return TIGA_OK;
}

int check_radius(float radius, float sigma) {
    if (!(radius > 0.0f) || !(radius < 3.0e38f)) return fail(TIGA_EINVAL, "radius must be finite and > 0");
    if (!(sigma > 0.0f) || !(sigma < 3.0e38f)) return fail(TIGA_EINVAL, "sigma must be finite and > 0");
    // the kernels scale by -log2(e) / sigma^2 and 2 / sigma^2 in fp32: both must be finite, or a
    // coincident pair (d2 = 0) would get weight exp2(0 * -inf) = NaN
    const float two_inv_s2 = 2.0f / (sigma * sigma);
    if (!(two_inv_s2 <= 3.4028234e38f))
        return fail(TIGA_EINVAL, "sigma %g is too small: 2 / sigma^2 overflows fp32 (sigma must be >= 7.7e-20)",
                    (double)sigma);
    return TIGA_OK;
}

}  // namespace

extern "C" {

size_t tiga_mp_radius_workspace(int64_t n, int32_t feat) {
    if (n < 0 || feat < 0) return 0;
    return radius::workspace_bytes(n, feat);
}

int tiga_mp_radius_fwd(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma,
                       int reducer, float *y, int32_t *count, void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (feat < 0) return fail(TIGA_EINVAL, "feat must be >= 0 (got %d)", feat);
    if (reducer == TIGA_REDUCE_MAX) return fail(TIGA_EUNSUPPORTED, "the radius relation supports the sum reducer only");
    if (reducer != TIGA_REDUCE_SUM) return fail(TIGA_EINVAL, "unknown reducer %d", reducer);
    if (int rc = check_radius(radius, sigma)) return rc;
    if (feat == 0 && !count) return fail(TIGA_EINVAL, "feat 0 computes counts only: count is required");
    if (n == 0) return TIGA_OK;
    if (feat > 0 && (!x || !y)) return fail(TIGA_EINVAL, "x and y are required");
    if (int rc = check_ws(ws, ws_bytes, radius::workspace_bytes(n, feat))) return rc;
    return radius::forward(n, feat, pos, x, radius, sigma, y, count, ws, static_cast<hipStream_t>(stream));
}

int tiga_mp_radius_bwd(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma,
                       const float *dy, float *dx, float *dpos, void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (feat < 1) return fail(TIGA_EINVAL, "feat must be >= 1 (got %d)", feat);
    if (int rc = check_radius(radius, sigma)) return rc;
    if (n == 0 || (!dx && !dpos)) return TIGA_OK;
    if (!dy) return fail(TIGA_EINVAL, "dy is NULL");
    if (dpos && !x) return fail(TIGA_EINVAL, "x is required for dpos");
    if (int rc = check_ws(ws, ws_bytes, radius::workspace_bytes(n, feat))) return rc;
    return radius::backward(n, feat, pos, x, radius, sigma, dy, dx, dpos, ws, static_cast<hipStream_t>(stream));
}

int tiga_radius_neighbors(int64_t n, const float *pos, float radius, const int64_t *nbr_ptr, int32_t *nbr_idx,
                          void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (int rc = check_radius(radius, 1.0f)) return rc;
    if (n == 0) return TIGA_OK;
    if (!nbr_ptr) return fail(TIGA_EINVAL, "nbr_ptr is NULL");
    if (!nbr_idx) return fail(TIGA_EINVAL, "nbr_idx is NULL");
    if (int rc = check_ws(ws, ws_bytes, radius::workspace_bytes(n, 0))) return rc;
    return radius::neighbors(n, pos, radius, nbr_ptr, nbr_idx, ws, static_cast<hipStream_t>(stream));
}

size_t tiga_mp_dense_workspace(int64_t n) {
    if (n < 0) return 0;
    return dense::workspace_bytes(n);
}

int tiga_mp_dense_fwd(int64_t n, const float *pos, const float *q, float eps, int reducer, float *y, void *ws,
                      size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (reducer == TIGA_REDUCE_MAX) return fail(TIGA_EUNSUPPORTED, "the dense relation supports the sum reducer only");
    if (reducer != TIGA_REDUCE_SUM) return fail(TIGA_EINVAL, "unknown reducer %d", reducer);
    if (!(eps > 0.0f) || !(eps < 3.0e38f)) return fail(TIGA_EINVAL, "eps must be finite and > 0");
    // the message is formed with the fp32 constant eps * eps: it must be a finite normal number, or the
    // zero-displacement self term (0 * rsq(0)^3) would not vanish
    const float eps2 = eps * eps;
    if (!(eps2 >= 1.17549435e-38f) || !(eps2 < 3.0e38f))
        return fail(TIGA_EINVAL, "eps * eps (%g) must be a finite normal fp32 number", static_cast<double>(eps2));
    if (n == 0) return TIGA_OK;
    if (!q || !y) return fail(TIGA_EINVAL, "q and y are required");
    if (int rc = check_ws(ws, ws_bytes, dense::workspace_bytes(n))) return rc;
    return dense::forward(n, pos, q, eps, y, ws, static_cast<hipStream_t>(stream));
}

namespace {

// The edge-MLP path's shared cell directory holds up to 8 n + 64 cells, indexed by int32 keys.
int check_shared_cells(int64_t n) {
    if (8 * n + 64 > INT32_MAX)
        return fail(TIGA_EUNSUPPORTED, "n %lld: the cell directory of the edge MLP needs 8 n + 64 < 2^31",
                    (long long)n);
    return TIGA_OK;
}

int check_net(int32_t feat, int32_t hidden, int32_t out) {
    if (feat < 0 || hidden < 1 || out < 1) return fail(TIGA_EINVAL, "need feat >= 0, hidden >= 1, out >= 1");
    if (feat > edgenn::kMaxFeat || hidden > edgenn::kMaxHidden || out > edgenn::kMaxOut)
        return fail(TIGA_EUNSUPPORTED, "edge MLP widths feat %d, hidden %d, out %d exceed %d, %d, %d", feat, hidden,
                    out, edgenn::kMaxFeat, edgenn::kMaxHidden, edgenn::kMaxOut);
    return TIGA_OK;
}

}  // namespace

size_t tiga_mp_edgenn_workspace(int64_t n, int32_t feat, int32_t hidden, int32_t out) {
    if (n < 0 || feat < 0 || hidden < 1 || out < 1) return 0;
    return edgenn::workspace_bytes(n, edgenn::Net{feat, hidden, out, nullptr, nullptr, nullptr, nullptr});
}

int tiga_mp_edgenn_fwd(int64_t n, int32_t feat, int32_t hidden, int32_t out, const float *pos, const float *x,
                       float radius, const float *W1, const float *b1, const float *W2, const float *b2, float *y,
                       void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (int rc = check_shared_cells(n)) return rc;
    if (int rc = check_net(feat, hidden, out)) return rc;
    if (int rc = check_radius(radius, 1.0f)) return rc;
    if (n == 0) return TIGA_OK;
    if (!W1 || !b1 || !W2 || !b2 || !y || (feat > 0 && !x)) return fail(TIGA_EINVAL, "a required array is NULL");
    const edgenn::Net net{feat, hidden, out, W1, b1, W2, b2};
    if (int rc = check_ws(ws, ws_bytes, edgenn::workspace_bytes(n, net))) return rc;
    return edgenn::forward(n, pos, x, radius, net, y, ws, static_cast<hipStream_t>(stream));
}

int tiga_mp_edgenn_bwd(int64_t n, int32_t feat, int32_t hidden, int32_t out, const float *pos, const float *x,
                       float radius, const float *W1, const float *b1, const float *W2, const float *b2,
                       const float *dy, float *dx, float *dpos, float *dW1, float *db1, float *dW2, float *db2,
                       void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (int rc = check_shared_cells(n)) return rc;
    if (int rc = check_net(feat, hidden, out)) return rc;
    if (int rc = check_radius(radius, 1.0f)) return rc;
    if (n == 0) {
        // no messages: the parameter gradients are zero
        hipStream_t s = static_cast<hipStream_t>(stream);
        const int64_t D = 3 + feat;
        if (dW1) if (int rc = fill_u32(dW1, 0u, hidden * D, s)) return rc;
        if (db1) if (int rc = fill_u32(db1, 0u, hidden, s)) return rc;
        if (dW2) if (int rc = fill_u32(dW2, 0u, static_cast<int64_t>(out) * hidden, s)) return rc;
        if (db2) if (int rc = fill_u32(db2, 0u, out, s)) return rc;
        return TIGA_OK;
    }
    if (!W1 || !b1 || !W2 || !b2 || !dy || (feat > 0 && !x)) return fail(TIGA_EINVAL, "a required array is NULL");
    const edgenn::Net net{feat, hidden, out, W1, b1, W2, b2};
    if (int rc = check_ws(ws, ws_bytes, edgenn::workspace_bytes(n, net))) return rc;
    return edgenn::backward(n, pos, x, radius, net, dy, edgenn::Grads{dx, dpos, dW1, db1, dW2, db2}, ws,
                            static_cast<hipStream_t>(stream));
}

size_t tiga_mp_knn_workspace(int64_t n) {
    if (n < 0) return 0;
    return knn::workspace_bytes(n);
}

int tiga_mp_knn_fwd(int64_t n, int32_t feat, const float *pos, const float *x, int32_t k, int reducer, float *y,
                    int32_t *nbr, void *ws, size_t ws_bytes, void *stream) {
    EntryScope scope;
    if (int rc = check_points(n, pos)) return rc;
    if (reducer == TIGA_REDUCE_MAX) return fail(TIGA_EUNSUPPORTED, "the kNN relation supports the sum reducer only");
    if (reducer != TIGA_REDUCE_SUM) return fail(TIGA_EINVAL, "unknown reducer %d", reducer);
    if (k < 0) return fail(TIGA_EINVAL, "k must be >= 0 (got %d)", k);
    if (k > knn::kMaxK) return fail(TIGA_EUNSUPPORTED, "k = %d exceeds the supported %d", k, knn::kMaxK);
    if (feat < 0) return fail(TIGA_EINVAL, "feat must be >= 0");
    if (n == 0) return TIGA_OK;
    if (feat > 0 && (!x || !y)) return fail(TIGA_EINVAL, "x and y are required when feat > 0");
    if (int rc = check_ws(ws, ws_bytes, knn::workspace_bytes(n))) return rc;
    return knn::forward(n, feat, pos, x, k, y, nbr, ws, static_cast<hipStream_t>(stream));
}

}  // extern "C"
