// Host interface of the CSR gather-reduce traversal.
#pragma once

#include "csr_common.hpp"

namespace tiga {
namespace csr {

struct Layout {
    int K;       // floats per unit (4: float4 path, 1: scalar path)
    int64_t fu;  // units per feature row
    int L;       // lanes per edge
    Geom g;
};

Layout layout_for(int64_t feat, bool vec);

// Workspace bytes for one traversal over (nrows, nedges) with `feat` features.
size_t traversal_ws_bytes(int64_t nrows, int64_t nedges, int64_t feat, bool with_arg);

// Optional edge gradients formed during a traversal of the reverse incidence
// (sum backward): dw[eid[e]] = <x[row], table[idx[e]]> for every folded edge.
struct EdgeGrad {
    const float *x = nullptr;  // [nrows, feat] rows of the traversal's own rows
    float *dw = nullptr;       // [nedges], indexed by eid
};

// Enqueue plan + gather-reduce + merge: out[i, :] = reduce_{e in row i} w(e) * table[idx[e], :].
// `table_rows` is the row count of t.table (and t.arg); tables below 4 GiB are
// read through buffer resources.  With eg.dw the traversal must be a sum with
// W_INDIRECT or W_ROUTE weights over one feature block (fu <= L).
// Whether a relation of nrows rows and nedges edges takes the single-launch direct traversal (no
// plan, no merge).  The direct traversal folds each row with all 64 lanes of a wavefront, the
// planned one with a lane group sized by the row's degree class, so the two differ in rounding.
bool direct_traversal(int64_t nrows, int64_t nedges);

// `direct` chooses the traversal (callers pass direct_traversal() of the relation the result must
// agree with bit for bit: a page of a relation takes the whole relation's choice).
int launch_traversal(const Trav &t, int64_t table_rows, int64_t nedges, const Layout &lay, int red, int wm, void *ws,
                     float *out, int32_t *out_arg, hipStream_t stream, bool direct,
                     const EdgeGrad &eg = EdgeGrad{});

// Paged forward: rel's row_ptr and col_idx and w_host live in host memory; pages of whole rows
// with at most page_edges edges are staged through the workspace (see csr_paged.hip).
size_t paged_ws_bytes(int64_t page_edges, int64_t feat, bool with_arg);
int launch_paged_fwd(const tiga_csr *rel, int32_t feat, const float *x_src, const float *w_host, int red, float *y,
                     int32_t *argmax, int64_t page_edges, void *ws, hipStream_t stream);

}  // namespace csr
}  // namespace tiga
