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

// Enqueue plan + gather-reduce + merge: out[i, :] = reduce_{e in row i} w(e) * table[idx[e], :].
// `table_rows` is the row count of t.table (and t.arg); tables below 4 GiB are
// read through buffer resources.
int launch_traversal(const Trav &t, int64_t table_rows, int64_t nedges, const Layout &lay, int red, int wm, void *ws,
                     float *out, int32_t *out_arg, hipStream_t stream);

}  // namespace csr
}  // namespace tiga
