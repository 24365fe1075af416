/*
 * tiga_mp.h -- C ABI of the MI355X (gfx950) fused message-passing library.
 *
 * Fused message passing (Tiga, "Compiling Graph Message Passing at Scale"):
 * for every destination entity the library traverses a relation, forms one
 * message per (source, destination) pair and folds it into the reducer state
 * immediately, so neither the edge list of a generated relation nor any
 * per-edge message array is ever stored (Section 3.1 message/update equation;
 * Section 4.2 on fused row traversal versus materialized E*F messages).
 *
 * Three relations are supported:
 *   - a stored destination-major CSR graph (Sections 3.1 and 4.3),
 *   - a radius relation generated from positions through a cell directory
 *     (Section 4.9),
 *   - the dense all-pairs relation, which needs no edge array (Section 1).
 * Reverse mode (Section 5, vector-Jacobian products) is provided for the CSR
 * and radius relations.
 *
 * Conventions shared by every entry point
 *   - Arrays are DEVICE pointers unless a comment says otherwise.  The caller
 *     owns every buffer, including the workspace `ws` of `ws_bytes` bytes
 *     (size it with the matching *_workspace query; it must be 256-byte
 *     aligned).  The library keeps no pointer after the call returns.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is the
 *     null stream).  Calls return before the work completes; a device fault
 *     surfaces at the caller's next synchronization.  Only
 *     tiga_csr_validate(level 2) and tiga_radius_neighbors synchronize.
 *   - Outputs are overwritten, never accumulated into.
 *   - fp32 features are row-major [rows, feat].  A 16-byte aligned feature
 *     array with feat % 4 == 0 takes the vector path; any other width works
 *     through the scalar path.
 *   - Arguments are checked on the host before anything is enqueued.  On
 *     error the call returns a negative status, enqueues nothing, and
 *     tiga_last_error() describes the problem.  There is no silent fallback:
 *     unsupported combinations return TIGA_EUNSUPPORTED (the paper requires
 *     explicit diagnosis rather than a substituted route, Sections 4.1 and 4.8).
 *   - The library holds no global mutable state other than the per-thread
 *     error string and the per-thread profiling events; calls are reentrant.
 */
#ifndef TIGA_MP_H
#define TIGA_MP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TIGA_MP_ABI_VERSION 2

/* Status codes. */
enum tiga_status {
    TIGA_OK = 0,
    TIGA_EINVAL = -1,       /* bad argument (NULL, negative size, misaligned ws) */
    TIGA_EGRAPH = -2,       /* the relation violates CSR invariants (validation) */
    TIGA_EUNSUPPORTED = -3, /* valid request this library does not implement */
    TIGA_EWORKSPACE = -4,   /* ws_bytes smaller than the workspace query */
    TIGA_EDEVICE = -5       /* a HIP call failed */
};

/* Reducers (Section 3.1: identity, lift, combine, finalize).
 *   SUM: identity 0; an empty row finalizes to 0.
 *   MAX: identity -inf; ties keep the lowest edge position; an empty row
 *        finalizes to value 0 with argmax -1. */
enum tiga_reducer { TIGA_REDUCE_SUM = 0, TIGA_REDUCE_MAX = 1 };

/* Messages over a stored CSR relation (edge function of Section 3.1). */
enum tiga_csr_msg {
    TIGA_MSG_SRC = 0,             /* m_e = x[s(e)]          (w_edge must be NULL) */
    TIGA_MSG_EDGE_SCALED_SRC = 1  /* m_e = w[e] * x[s(e)]   (w_edge required)     */
};

/* Destination-major CSR relation (Sections 3.1, 4.3).  Destination row i owns
 * edge positions [row_ptr[i], row_ptr[i+1]); the edge position indexes edge
 * fields and col_idx[e] is the source id.  Duplicates and self edges are
 * ordinary separate edges; num_src may differ from num_dst.
 *   row_ptr: int64 [num_dst + 1], row_ptr[0] == 0, non-decreasing,
 *            row_ptr[num_dst] == num_edges.
 *   col_idx: int32 [num_edges], each in [0, num_src).
 * The struct itself lives in HOST memory; the two arrays on the device. */
typedef struct {
    int64_t num_dst;
    int64_t num_src;
    int64_t num_edges;
    const int64_t *row_ptr;
    const int32_t *col_idx;
} tiga_csr;

/* Reverse incidence of a tiga_csr (the transposed relation; Section 4.6
 * notes that source gradients accumulate over reverse incidence).
 *   src_ptr: int64 [num_src + 1]; source j owns slots [src_ptr[j], src_ptr[j+1]).
 *   edge_id: int32 [num_edges]; the forward edge position of each slot,
 *            ascending within a source (a stable transpose).
 * Built by tiga_csr_transpose; valid only for the unchanged topology (a
 * topology snapshot is fixed for derivatives, Section 3.2).  The struct lives
 * in HOST memory, the two arrays on the device. */
typedef struct {
    const int64_t *src_ptr;
    const int32_t *edge_id;
} tiga_csr_t;

/* ---------------------------------------------------------------- errors */

/* Message describing the last failure on the calling thread ("" if none).
 * Valid until the next library call on that thread.  Host pointer. */
const char *tiga_last_error(void);

/* TIGA_MP_ABI_VERSION of the built library. */
int tiga_mp_abi_version(void);

/* ------------------------------------------------------------ stored CSR */

/* Workspace bytes for tiga_mp_csr_fwd on this relation shape (0 on error). */
size_t tiga_mp_csr_fwd_workspace(const tiga_csr *rel, int32_t feat, int reducer);

/* Forward fused aggregation over a stored CSR relation (Section 3.1 equation,
 * Section 4.3 destination-major traversal, Section 4.4 bounded neighbour tiles
 * with a degree guard and a split of high-degree rows into partial states
 * merged afterwards):
 *   SUM: y[i,f] = sum_{e in row i} m_e[f]
 *   MAX: y[i,f] = max_{e in row i} m_e[f], argmax[i,f] = that e (lowest on ties)
 * with m_e = x_src[col[e], :] or w_edge[e] * x_src[col[e], :] (one fp32
 * multiply, so MAX values are exact products).
 *   x_src:  fp32 [num_src, feat];  w_edge: fp32 [num_edges] or NULL (see msg)
 *   y:      fp32 [num_dst, feat], overwritten
 *   argmax: int32 [num_dst, feat] for MAX (required), NULL for SUM
 * SUM results are deterministic (fixed reduction tree) but not bit-identical
 * to a serial sum; MAX results are exact.  MAX requires num_edges < 2^31.
 * Errors: TIGA_EINVAL, TIGA_EUNSUPPORTED, TIGA_EWORKSPACE, TIGA_EDEVICE. */
int tiga_mp_csr_fwd(const tiga_csr *rel, int32_t feat, const float *x_src, int msg,
                    const float *w_edge, int reducer, float *y, int32_t *argmax,
                    void *ws, size_t ws_bytes, void *stream);

/* Allocation-free tiga_mp_csr_fwd, for callers that cannot allocate device
 * memory (work under stream capture, tight serving loops, harnesses that
 * forbid allocation).  Same arguments, results and errors as tiga_mp_csr_fwd
 * without the workspace: the library keeps a fixed device array of
 * tiga_mp_csr_fwd_noalloc_limit() bytes (64 MiB) per device, taken from its
 * code object when this entry point is first called on that device and held
 * until the process ends.  A relation whose tiga_mp_csr_fwd_workspace exceeds
 * the limit is rejected with TIGA_EUNSUPPORTED before anything is enqueued.
 * The call makes no allocation (no hipMalloc, hipFree or allocating library
 * routine).  Every call on a device uses that device's one array: calls that
 * overlap on one device (other streams, other threads) race and must be
 * serialized by the caller; calls in order on one stream are safe.  The
 * device is the current device, and `stream` must belong to it. */
size_t tiga_mp_csr_fwd_noalloc_limit(void);
int tiga_mp_csr_fwd_noalloc(const tiga_csr *rel, int32_t feat, const float *x_src, int msg,
                            const float *w_edge, int reducer, float *y, int32_t *argmax,
                            void *stream);

/* Workspace bytes for tiga_mp_csr_fwd_paged with pages of at most page_edges
 * edges (0 on error).  Independent of the relation's size. */
size_t tiga_mp_csr_fwd_paged_workspace(int32_t feat, int reducer, int64_t page_edges);

/* tiga_mp_csr_fwd for a relation kept in HOST memory (Section 6, storage and
 * memory: the relation stays in a persistent store, one destination-row page
 * at a time is staged, and the kernel runs with a bounded device working set;
 * the output stays in device memory).
 *   rel_host: row_ptr and col_idx are HOST pointers (pinned memory lets the
 *             copies run asynchronously); w_host likewise (or NULL, see msg).
 *   x_src, y, argmax: DEVICE pointers, as in tiga_mp_csr_fwd.
 * Pages hold whole destination rows and at most page_edges edges; each page's
 * slices are copied on `stream` into the workspace and reduced there, so the
 * device working set is fixed by page_edges.  Results equal tiga_mp_csr_fwd's
 * (argmax holds global edge positions).  The host reads rel_host->row_ptr
 * during the call (to cut pages and to reject a row longer than page_edges
 * with TIGA_EUNSUPPORTED, or a row_ptr that does not run from 0 to num_edges
 * without decreasing with TIGA_EGRAPH); the host arrays must stay valid until
 * the stream has run the copies.
 * Errors: as tiga_mp_csr_fwd, plus TIGA_EGRAPH. */
int tiga_mp_csr_fwd_paged(const tiga_csr *rel_host, int32_t feat, const float *x_src, int msg,
                          const float *w_host, int reducer, float *y, int32_t *argmax, int64_t page_edges,
                          void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes for tiga_mp_csr_bwd (0 on error). */
size_t tiga_mp_csr_bwd_workspace(const tiga_csr *rel, int32_t feat, int reducer);

/* Vector-Jacobian product of tiga_mp_csr_fwd (Section 5 weighted-sum adjoint):
 *   SUM: dx[j,f] = sum_{e: col[e]=j} w[e] dy[d(e),f];  dw[e] = sum_f x[col[e],f] dy[d(e),f]
 *   MAX: the same terms restricted to the selected edge e* = argmax[i,f] of
 *        each (i,f); argmax is the forward's output (required for MAX).
 * (w = 1 under TIGA_MSG_SRC.)  dx: fp32 [num_src, feat]; dw: fp32 [num_edges];
 * either may be NULL (skipped) and each is overwritten.  dw requires
 * TIGA_MSG_EDGE_SCALED_SRC.
 * rev == NULL: dx accumulates with device fp32 atomics: no set-up, summation
 *   order not fixed, and bound by the atomics (at feat = 64 a little over twice
 *   the time of the gather mode).
 * rev != NULL: dx is gathered over the reverse incidence (deterministic); build
 *   it once per topology with tiga_csr_transpose.  The destination row of
 *   each reverse slot is derived during the call from row_ptr and edge_id
 *   (into the workspace).
 * Errors: as tiga_mp_csr_fwd. */
int tiga_mp_csr_bwd(const tiga_csr *rel, const tiga_csr_t *rev, int32_t feat,
                    const float *x_src, int msg, const float *w_edge, int reducer,
                    const int32_t *argmax, const float *dy, float *dx, float *dw,
                    void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes for tiga_csr_transpose (0 on error). */
size_t tiga_csr_transpose_workspace(const tiga_csr *rel);

/* Build the reverse incidence (see tiga_csr_t) with a stable sort by source:
 * within a source, edge ids ascend.  Topology set-up: build once per
 * unchanged topology.  src_ptr int64 [num_src+1] and edge_id int32
 * [num_edges], both overwritten.  Requires num_edges < 2^31. */
int tiga_csr_transpose(const tiga_csr *rel, int64_t *src_ptr, int32_t *edge_id,
                       void *ws, size_t ws_bytes, void *stream);

/* CSR validation (the paper's validate="full" and basic modes, Section 6.3):
 *   level 1: host-only metadata checks (sizes, pointers); enqueues nothing.
 *   level 2: additionally scans the device arrays: row_ptr[0] == 0,
 *            non-decreasing, row_ptr[num_dst] == num_edges, every col_idx in
 *            [0, num_src).  Synchronizes `stream`.
 * Returns TIGA_OK or TIGA_EGRAPH (the first violation is described by
 * tiga_last_error()). */
int tiga_csr_validate(const tiga_csr *rel, int level, void *stream);

/* -------------------------------------------------- generated radius relation */

/* Workspace bytes for tiga_mp_radius_fwd / _bwd / tiga_radius_neighbors on n
 * points with feat features (0 on error). */
size_t tiga_mp_radius_workspace(int64_t n, int32_t feat);

/* Forward over the radius relation generated from positions (Section 4.9:
 * a cell directory restricts candidates, an exact distance predicate accepts,
 * messages are consumed without storing accepted edges):
 *   N(i) = { j != i : d2(i,j) < fl(radius*radius) },
 *   d2   = fl(fl(fl(dx*dx) + fl(dy*dy)) + fl(dz*dz)), dx = fl(p_j.x - p_i.x), ...
 *   y_i  = sum_{j in N(i)} exp(-|p_i - p_j|^2 / sigma^2) x_j
 *   count_i = |N(i)|
 * The cell directory is rebuilt on every call (stateless).
 *   pos: fp32 [n, 3]; x: fp32 [n, feat]; y: fp32 [n, feat] (input order);
 *   count: int32 [n] or NULL.  reducer must be TIGA_REDUCE_SUM.
 *   feat == 0 computes the counts only (x and y may be NULL; count required):
 *   the first phase of tiga_radius_neighbors.
 * Requires n < 2^31, radius finite and > 0, sigma > 0 with 2 / sigma^2 finite
 * in fp32 (sigma >= 7.7e-20; TIGA_EINVAL otherwise).  A point with a non-finite
 * coordinate has no neighbours (every d2 involving it compares false). */
int tiga_mp_radius_fwd(int64_t n, int32_t feat, const float *pos, const float *x,
                       float radius, float sigma, int reducer, float *y, int32_t *count,
                       void *ws, size_t ws_bytes, void *stream);

/* VJP of tiga_mp_radius_fwd with membership held fixed (Section 5: radius
 * cutoff membership is discrete and not differentiated):
 *   dx_i = sum_{j in N(i)} k_ij dy_j
 *   dpos_i = sum_{j in N(i)} (2 k_ij / sigma^2) (p_j - p_i) (<dy_i, x_j> + <dy_j, x_i>)
 * with k_ij = exp(-|p_i - p_j|^2 / sigma^2).  dx: fp32 [n, feat] or NULL;
 * dpos: fp32 [n, 3] or NULL (x is only read when dpos is requested).
 * The same requirements as tiga_mp_radius_fwd. */
int tiga_mp_radius_bwd(int64_t n, int32_t feat, const float *pos, const float *x,
                       float radius, float sigma, const float *dy, float *dx, float *dpos,
                       void *ws, size_t ws_bytes, void *stream);

/* Accepted neighbour lists of the radius relation, ascending per point (the
 * relation a fused call consumes, exported for exact checking; the paper
 * resolves a generated relation to CSR for inspection, Section 4.9).  Two
 * phases: the counts come from tiga_mp_radius_fwd (feat 0 computes only
 * them), the caller forms nbr_ptr int64 [n+1] as their exclusive prefix sum,
 * and this call fills nbr_idx int32 [nbr_ptr[n]].
 *   nbr_ptr: device, read only.  Each point's list is written only inside its
 *            span [nbr_ptr[i], nbr_ptr[i+1]); if a span differs from that
 *            point's count the call returns TIGA_EINVAL (nothing is written
 *            outside the spans, the lists are then incomplete).
 * Synchronizes `stream`.  Not on the fused path: for tests and inspection. */
int tiga_radius_neighbors(int64_t n, const float *pos, float radius, const int64_t *nbr_ptr,
                          int32_t *nbr_idx, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------- dense all-pairs relation */

/* Workspace bytes for tiga_mp_dense_fwd (0 on error). */
size_t tiga_mp_dense_workspace(int64_t n);

/* Dense all-pairs relation without an edge array (Section 1), softened
 * inverse-square message, sum reducer:
 *   y_i = sum_{j != i} q_j (p_j - p_i) / (|p_j - p_i|^2 + eps^2)^(3/2)
 * pos: fp32 [n, 3]; q: fp32 [n]; y: fp32 [n, 3].  reducer must be SUM.
 * Requires n < 2^31 and eps > 0. */
int tiga_mp_dense_fwd(int64_t n, const float *pos, const float *q, float eps, int reducer,
                      float *y, void *ws, size_t ws_bytes, void *stream);

/* ----------------------------------------------- generated exact kNN relation */

/* Workspace bytes for tiga_mp_knn_fwd on n points (0 on error). */
size_t tiga_mp_knn_workspace(int64_t n);

/* Forward over the exact k-nearest-neighbour relation generated from positions
 * (Section 4.9, generated relations: candidate tiles are scanned for each query
 * with a padded top-k state keyed by squared distance and source index; no
 * adjacency is stored), with the neighbour-sum message of the exact-kNN
 * workload of Section 7:
 *   S_i  = the k sources j != i with the smallest keys (d2_ij, j), compared
 *          lexicographically (a distance tie keeps the lower index); a source
 *          whose d2 is not finite is never selected, so S_i may hold fewer
 *          than k sources;
 *   d2   = fl(fl(fl(dx*dx) + fl(dy*dy)) + fl(dz*dz)), dx = fl(p_j.x - p_i.x), ...
 *   y_i  = sum_{j in S_i} x_j      (fp32; terms in key order, added sequentially
 *          above 16,384 points and by a fixed pairwise tree at or below)
 *   nbr[i][t] = the t-th selected source in key order, -1 past |S_i|.
 * The relation is rebuilt on every call (stateless).
 *   pos: fp32 [n, 3]; x: fp32 [n, feat] (NULL if feat == 0); y: fp32 [n, feat]
 *   (NULL if feat == 0); nbr: int32 [n, k] or NULL.  reducer must be
 *   TIGA_REDUCE_SUM.  Requires 0 <= k <= 32 (TIGA_EUNSUPPORTED above 32) and
 *   n < 2^31 - 64.  Selection is exact: it equals a full scan of all pairs.
 * Errors: TIGA_EINVAL, TIGA_EUNSUPPORTED, TIGA_EWORKSPACE, TIGA_EDEVICE. */
int tiga_mp_knn_fwd(int64_t n, int32_t feat, const float *pos, const float *x, int32_t k, int reducer, float *y,
                    int32_t *nbr, void *ws, size_t ws_bytes, void *stream);

/* -------------------------------- edge-local MLP message on the radius relation */

/* Workspace bytes for tiga_mp_edgenn_fwd / _bwd (0 on error). */
size_t tiga_mp_edgenn_workspace(int64_t n, int32_t feat, int32_t hidden, int32_t out);

/* Edge-local neural-network message summed over the generated radius relation
 * (appendix "A differentiable EdgeNN example"; the relation as in
 * tiga_mp_radius_fwd: j != i and the fp32 squared distance strictly below
 * fl(radius*radius)):
 *   in_ij = [p_j - p_i ; x_j]  (3 + feat values; fp32 differences)
 *   y_i   = sum_{j in N(i)} ( W2 max(W1 in_ij + b1, 0) + b2 )
 * (the final bias is part of every message; an empty row gives 0).  No edge,
 * message or hidden activation is stored.
 *   pos fp32 [n, 3]; x fp32 [n, feat] (NULL if feat == 0);
 *   W1 [hidden, 3 + feat], b1 [hidden], W2 [out, hidden], b2 [out] fp32
 *   row-major; y fp32 [n, out], overwritten.
 * Requires 0 <= feat <= 64, 1 <= hidden <= 64, 1 <= out <= 8
 * (TIGA_EUNSUPPORTED beyond), radius finite and > 0, n < 2^31 - 64.
 * Errors: TIGA_EINVAL, TIGA_EUNSUPPORTED, TIGA_EWORKSPACE, TIGA_EDEVICE. */
int tiga_mp_edgenn_fwd(int64_t n, int32_t feat, int32_t hidden, int32_t out, const float *pos, const float *x,
                       float radius, const float *W1, const float *b1, const float *W2, const float *b2, float *y,
                       void *ws, size_t ws_bytes, void *stream);

/* Vector-Jacobian product of tiga_mp_edgenn_fwd with the relation held fixed
 * (Section 5: radius membership is discrete and not differentiated); hidden
 * activations are recomputed, never stored.  For L = sum_i <dy_i, y_i>:
 *   dx [n, feat], dpos [n, 3], dW1 [hidden, 3 + feat], db1 [hidden],
 *   dW2 [out, hidden], db2 [out]   (fp32; each may be NULL; overwritten).
 * The derivative of max(a, 0) at a = 0 is 0.  Deterministic: fixed
 * summation orders for every output.  Arguments and errors as the forward. */
int tiga_mp_edgenn_bwd(int64_t n, int32_t feat, int32_t hidden, int32_t out, const float *pos, const float *x,
                       float radius, const float *W1, const float *b1, const float *W2, const float *b2,
                       const float *dy, float *dx, float *dpos, float *dW1, float *db1, float *dW2, float *db2,
                       void *ws, size_t ws_bytes, void *stream);

/* ------------------------------- online-softmax reducer (streaming attention) */

/* 16-bit input types of the attention path. */
enum tiga_dtype { TIGA_DT_F16 = 0 /* IEEE binary16 */, TIGA_DT_BF16 = 1 /* bfloat16 */ };

/* Implicit relations of the attention path (no edge array). */
enum tiga_relation {
    TIGA_REL_TRIANGULAR = 0, /* N(i) = {0, ..., i}: causal, the diagonal included */
    TIGA_REL_DENSE = 1       /* N(i) = {0, ..., n-1} */
};

/* Online-softmax reducer over an implicit triangular or dense relation: the
 * streaming attention forward (appendix "Causal attention as message
 * passing"; reducer state of Section 5.2: running maximum, mass and
 * accumulator, combined by rescaling into a common maximum).  Per head h and
 * destination i, with the message (score, value) of source j:
 *   s_ij = scale * <q_i, k_j>,
 *   y_i  = sum_{j in N(i)} exp(s_ij) v_j / sum_{j in N(i)} exp(s_ij),
 *   lse_i = log sum_{j in N(i)} exp(s_ij).
 * No score or weight array is stored.
 *   q, k, v: [heads, n, width] head-major, 16-bit (dtype), 16-byte aligned
 *            (a permuted view of a contiguous (heads, n, width) allocation
 *            is the paper's logical (n, heads, width) tensor).
 *   y:       [heads, n, width] of dtype, overwritten (rounded to nearest even).
 *   lse:     fp32 [heads, n] or NULL.
 * Scores, weights and sums are fp32 (products of the 16-bit inputs are exact);
 * the weights enter both the value product and the mass rounded to dtype, so
 * y is an exactly normalized combination of the values and lse carries up to
 * one unit roundoff of dtype (2^-11 binary16, 2^-8 bfloat16) of absolute
 * error from that rounding.  Every row
 * is nonempty under both relations.  Requires width 64 or 128
 * (TIGA_EUNSUPPORTED otherwise), n < 2^31, heads * n < 2^40, scale finite and
 * > 0.  n == 0 or heads == 0 enqueues nothing.  Needs no workspace.
 * Errors: TIGA_EINVAL, TIGA_EUNSUPPORTED, TIGA_EDEVICE. */
int tiga_mp_attention_fwd(int64_t n, int32_t heads, int32_t width, int dtype, const void *q, const void *k,
                          const void *v, float scale, int relation, void *y, float *lse, void *stream);

/* ------------------------------------------------------------- profiling */

/* Profiling aid.  Arms the calling thread so that its next entry-point call
 * records hipEvent `start` on its stream immediately before, and `stop`
 * immediately after, the launch of that call's dominant kernel (the one that
 * streams the edges or pairs).  The events (hipEvent_t passed as void*) stay
 * owned by the caller and must live until that call returns.  The arming is
 * consumed by that one call; a call without a fused kernel (transpose,
 * validation, neighbour lists) records nothing and drops it.  Passing NULL for
 * both disarms.  Returns TIGA_OK. */
int tiga_mp_set_kernel_events(void *start, void *stop);

#ifdef __cplusplus
}
#endif

#endif /* TIGA_MP_H */
