// Paged forward over a stored CSR relation whose arrays stay in host memory (Section 6, storage
// and memory: the relation lives in a persistent store, one destination-row page at a time is
// staged, and the kernel runs with a bounded device working set; the output stays in device
// memory).  Each page holds whole destination rows and at most page_edges edges: its row_ptr,
// col_idx and w slices are copied to a device staging area on the caller's stream, row_ptr is
// rebased to the page's first edge, and the resident gather-reduce runs on the page, writing its
// rows of y (and argmax, shifted back to global edge positions).
#include "csr_fwd.hpp"

namespace tiga {
namespace csr {

namespace {

__global__ __launch_bounds__(kBlock) void rebase_kernel(int64_t *__restrict__ rp, int64_t n, int64_t base) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < n) rp[i] -= base;
}

__global__ __launch_bounds__(kBlock) void shift_arg_kernel(int32_t *__restrict__ arg, int64_t n, int32_t base) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < n && arg[i] >= 0) arg[i] += base;
}

struct PagedWs {
    int64_t *rp;
    int32_t *col;
    float *w;
    void *trav;
};

PagedWs carve_paged(Carve &c, int64_t page_edges, int64_t feat, bool with_arg) {
    PagedWs p;
    p.rp = c.take<int64_t>(page_edges + 1);
    p.col = c.take<int32_t>(page_edges);
    p.w = c.take<float>(page_edges);
    p.trav = c.take<char>(traversal_ws_bytes(page_edges, page_edges, feat, with_arg));
    return p;
}

}  // namespace

size_t paged_ws_bytes(int64_t page_edges, int64_t feat, bool with_arg) {
    Carve c(nullptr);
    carve_paged(c, page_edges, feat, with_arg);
    return c.bytes();
}

int launch_paged_fwd(const tiga_csr *rel, int32_t feat, const float *x_src, const float *w_host, int red, float *y,
                     int32_t *argmax, int64_t page_edges, void *ws, hipStream_t stream) {
    Carve c(ws);
    const PagedWs p = carve_paged(c, page_edges, feat, red == RED_MAX);
    const int64_t *rp = rel->row_ptr;   // host
    const bool vec = feat % 4 == 0 && aligned16(x_src) && aligned16(y) && (!argmax || aligned16(argmax));
    const Layout lay = layout_for(feat, vec);
    const int wm = w_host ? W_DIRECT : W_NONE;
    int64_t r0 = 0;
    while (r0 < rel->num_dst) {
        // whole rows, at most page_edges edges and page_edges rows
        const int64_t e0 = rp[r0];
        int64_t r1 = r0;
        while (r1 < rel->num_dst && r1 - r0 < page_edges && rp[r1 + 1] - e0 <= page_edges) ++r1;
        const int64_t rows = r1 - r0, edges = rp[r1] - e0;
        if (int rc = check_hip(hipMemcpyAsync(p.rp, rp + r0, (rows + 1) * sizeof(int64_t), hipMemcpyHostToDevice,
                                              stream), "paged: row_ptr copy"))
            return rc;
        if (edges > 0) {
            if (int rc = check_hip(hipMemcpyAsync(p.col, rel->col_idx + e0, edges * sizeof(int32_t),
                                                  hipMemcpyHostToDevice, stream), "paged: col_idx copy"))
                return rc;
            if (w_host)
                if (int rc = check_hip(hipMemcpyAsync(p.w, w_host + e0, edges * sizeof(float), hipMemcpyHostToDevice,
                                                      stream), "paged: w copy"))
                    return rc;
        }
        hipLaunchKernelGGL(rebase_kernel, dim3(static_cast<unsigned>(ceil_div(rows + 1, kBlock))), dim3(kBlock), 0,
                           stream, p.rp, rows + 1, e0);
        if (int rc = check_launch("paged: rebase")) return rc;
        Trav t{p.rp, p.col, w_host ? p.w : nullptr, nullptr, x_src, rows, lay.fu, nullptr, 0u, edges};
        int32_t *arg = argmax ? argmax + r0 * feat : nullptr;
        // every page takes the traversal the whole relation would take, so that each row is folded
        // in the same order as by the resident forward
        if (int rc = launch_traversal(t, rel->num_src, edges, lay, red, wm, p.trav, y + r0 * feat, arg, stream,
                                      direct_traversal(rel->num_dst, rel->num_edges)))
            return rc;
        if (arg && e0 > 0) {
            hipLaunchKernelGGL(shift_arg_kernel, dim3(static_cast<unsigned>(ceil_div(rows * feat, kBlock))),
                               dim3(kBlock), 0, stream, arg, rows * feat, static_cast<int32_t>(e0));
            if (int rc = check_launch("paged: argmax shift")) return rc;
        }
        r0 = r1;
    }
    return TIGA_OK;
}

}  // namespace csr
}  // namespace tiga
