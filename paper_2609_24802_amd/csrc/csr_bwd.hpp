// Host interface of the CSR vector-Jacobian products, the stable transpose and
// full validation.
#pragma once

#include "csr_fwd.hpp"

namespace tiga {
namespace csr {

struct BwdArgs {
    const tiga_csr *rel;
    const tiga_csr_t *rev;  // null: atomic dx
    int32_t feat;
    const float *x;         // [num_src, feat]
    const float *w;         // [num_edges] or null (unweighted message)
    int red;
    const int32_t *arg;     // [num_dst, feat] (max)
    const float *dy;        // [num_dst, feat]
    float *dx;              // [num_src, feat] or null
    float *dw;              // [num_edges] or null
};

size_t bwd_ws_bytes(int64_t num_dst, int64_t num_src, int64_t num_edges, int64_t feat);
int launch_bwd(const BwdArgs &a, void *ws, hipStream_t stream);

size_t transpose_ws_bytes(int64_t num_dst, int64_t num_src, int64_t num_edges);
int launch_transpose(const tiga_csr *rel, int64_t *src_ptr, int32_t *edge_id, void *ws, hipStream_t stream);

// Per forward edge e: rec[e] = (bits of w[e] (1.0 when w is null), the destination row of e), the
// 8-byte record the traversal of the reverse incidence reads through edge ids.  [num_edges].
int launch_edge_records(const tiga_csr *rel, const float *w, int2 *rec, hipStream_t stream);

int launch_validate(const tiga_csr *rel, hipStream_t stream);

// Stable sort of n keys in [0, key_limit): sorted keys to keys_out, the input
// position of each to idx_out (ascending within equal keys), and
// ptr[j] = first sorted position with key >= j for j in [0, key_limit] (ptr may be null:
// then only the sort runs).
size_t sort_keys_ws_bytes(int64_t n);
int launch_sort_keys(const int32_t *keys, int64_t n, int64_t key_limit, int32_t *keys_out, int32_t *idx_out,
                     int64_t *ptr, void *ws, hipStream_t stream);

// Device-wide exclusive prefix sum of n int64 values (in may equal out).
size_t scan_ws_bytes(int64_t n);
int launch_excl_scan(const int64_t *in, int64_t *out, int64_t n, void *ws, hipStream_t stream);

}  // namespace csr
}  // namespace tiga
