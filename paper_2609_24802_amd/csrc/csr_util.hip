// Topology utilities: device exclusive scan, the stable CSR transpose (an LSD
// radix sort of edge positions keyed by source id) and full validation.
#include "csr_bwd.hpp"

namespace tiga {
namespace csr {

namespace {

constexpr int kScanItems = 8;
constexpr int kScanTile = kBlock * kScanItems;

// Block-wide exclusive scan of one int64 per thread; returns the block total.
__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t &excl) {
    __shared__ int64_t sh[kWavesPerBlock];
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int64_t inc = wave_incl_scan(v);
    if (lane == kWave - 1) sh[wave] = inc;
    __syncthreads();
    int64_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
        if (w < wave) off += sh[w];
        tot += sh[w];
    }
    __syncthreads();
    excl = off + inc - v;
    return tot;
}

__global__ __launch_bounds__(kBlock) void scan_reduce_kernel(const int64_t *__restrict__ in, int64_t n,
                                                             int64_t *__restrict__ partial) {
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile;
    int64_t s = 0;
#pragma unroll
    for (int r = 0; r < kScanItems; ++r) {
        const int64_t i = base + r * kBlock + threadIdx.x;
        if (i < n) s += in[i];
    }
    int64_t excl;
    const int64_t tot = block_excl_scan(s, excl);
    if (threadIdx.x == 0) partial[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void scan_partials_kernel(int64_t *__restrict__ partial, int64_t n) {
    int64_t carry = 0;
    for (int64_t b = 0; b < n; b += kBlock) {
        const int64_t i = b + threadIdx.x;
        const int64_t v = i < n ? partial[i] : 0;
        int64_t excl;
        const int64_t tot = block_excl_scan(v, excl);
        if (i < n) partial[i] = carry + excl;
        carry += tot;
    }
}

// One block of 1024 threads scans a short array in one pass (8 consecutive
// elements per thread, all loads in flight together): one launch instead of
// three, for the sorts of small point sets and graphs, which spend more on
// launches than on their scans.  In place is allowed: every element is read
// before the block's scan and written after it.
constexpr int kSmallThreads = 1024;
constexpr int kSmallItems = 8;
constexpr int64_t kScanSmall = static_cast<int64_t>(kSmallThreads) * kSmallItems;

__global__ __launch_bounds__(kSmallThreads) void scan_small_kernel(const int64_t *in, int64_t *out, int64_t n) {
    __shared__ int64_t wsum[kSmallThreads / kWave];
    const int64_t base = static_cast<int64_t>(threadIdx.x) * kSmallItems;
    int64_t v[kSmallItems];
    int64_t s = 0;
#pragma unroll
    for (int r = 0; r < kSmallItems; ++r) {
        v[r] = (base + r < n) ? in[base + r] : 0;
        s += v[r];
    }
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const int64_t inc = wave_incl_scan(s);
    if (lane == kWave - 1) wsum[wave] = inc;
    __syncthreads();
    int64_t run = inc - s;
    for (int w = 0; w < wave; ++w) run += wsum[w];
#pragma unroll
    for (int r = 0; r < kSmallItems; ++r) {
        if (base + r < n) out[base + r] = run;
        run += v[r];
    }
}

// Each thread scans kScanItems consecutive elements of the tile.
__global__ __launch_bounds__(kBlock) void scan_down_kernel(const int64_t *in, int64_t *out, int64_t n,
                                                           const int64_t *__restrict__ partial) {
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile + threadIdx.x * kScanItems;
    int64_t v[kScanItems];
    int64_t s = 0;
#pragma unroll
    for (int r = 0; r < kScanItems; ++r) {
        v[r] = (base + r < n) ? in[base + r] : 0;
        s += v[r];
    }
    int64_t excl;
    block_excl_scan(s, excl);
    int64_t run = partial[blockIdx.x] + excl;
#pragma unroll
    for (int r = 0; r < kScanItems; ++r) {
        if (base + r < n) out[base + r] = run;
        run += v[r];
    }
}

// ---------------------------------------------------------------- radix sort

constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;
constexpr int kSortItems = 8;
constexpr int kSortTile = kBlock * kSortItems;

__global__ __launch_bounds__(kBlock) void radix_hist_kernel(const int32_t *__restrict__ keys, int64_t n, int shift,
                                                            int64_t nblocks, int64_t *__restrict__ counts) {
    __shared__ int hist[kRadix];
    hist[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortTile;
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t i = base + r * kBlock + threadIdx.x;
        if (i < n) atomicAdd(&hist[(static_cast<uint32_t>(keys[i]) >> shift) & (kRadix - 1)], 1);
    }
    __syncthreads();
    // digit-major layout: all blocks of digit 0, then digit 1, ...
    counts[static_cast<int64_t>(threadIdx.x) * nblocks + blockIdx.x] = hist[threadIdx.x];
}

// Stable scatter through LDS.  The tile's elements are ranked in (round, wave,
// lane) order, which is their input order, and placed in LDS grouped by digit;
// the block then writes each digit's run of the tile with consecutive lanes on
// consecutive addresses (a tile of 2048 elements holds about 8 per digit, so the
// stores come in runs instead of one element per digit and round).  The second
// payload is optional (null in and out).
__global__ __launch_bounds__(kBlock) void radix_scatter_kernel(
    const int32_t *__restrict__ keys_in, const int32_t *__restrict__ v0_in, const int32_t *__restrict__ v1_in,
    int32_t *__restrict__ keys_out, int32_t *__restrict__ v0_out, int32_t *__restrict__ v1_out, int64_t n,
    int shift, int64_t nblocks, const int64_t *__restrict__ offsets, int iota_v0) {
    __shared__ int64_t run[kRadix];   // output position of this tile's first element of each digit
    __shared__ int first[kRadix];     // LDS slot of this tile's first element of each digit
    __shared__ int fill[kRadix];      // digit counts, then elements of each digit placed so far
    __shared__ int wsum[kWavesPerBlock];
    __shared__ int wcnt[kWavesPerBlock][kRadix];
    __shared__ int32_t sk[kSortTile], sa[kSortTile], sb[kSortTile];
    const int t = threadIdx.x;
    const int lane = lane_id();
    const int wave = t / kWave;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortTile;
    const int total = static_cast<int>(n - base < kSortTile ? n - base : kSortTile);
    run[t] = offsets[static_cast<int64_t>(t) * nblocks + blockIdx.x];
    fill[t] = 0;
    __syncthreads();
    int32_t key[kSortItems], a[kSortItems], b[kSortItems];
    int digit[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int j = r * kBlock + t;
        key[r] = a[r] = b[r] = 0;
        digit[r] = 0;
        if (j < total) {
            const int64_t i = base + j;
            key[r] = keys_in[i];
            a[r] = iota_v0 ? static_cast<int32_t>(i) : v0_in[i];
            b[r] = v1_in ? v1_in[i] : 0;
            digit[r] = (static_cast<uint32_t>(key[r]) >> shift) & (kRadix - 1);
            atomicAdd(&fill[digit[r]], 1);
        }
    }
    __syncthreads();
    // exclusive scan of the tile's digit counts, thread t = digit t
    const int cnt = fill[t];
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int v = __shfl_up(incl, o);
        if (lane >= o) incl += v;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += wsum[w];
    first[t] = before + incl - cnt;
    fill[t] = 0;
    for (int r = 0; r < kSortItems; ++r) {
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) wcnt[w][t] = 0;
        __syncthreads();
        const bool valid = r * kBlock + t < total;
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < kRadixBits; ++bit) {
            const uint64_t m = __ballot((digit[r] >> bit) & 1);
            peers &= ((digit[r] >> bit) & 1) ? m : ~m;
        }
        const int rank = __popcll(peers & lt_mask);
        if (valid && rank == 0) wcnt[wave][digit[r]] = __popcll(peers);
        __syncthreads();
        if (valid) {
            const int d = digit[r];
            int slot = first[d] + fill[d] + rank;
            for (int w = 0; w < wave; ++w) slot += wcnt[w][d];
            sk[slot] = key[r];
            sa[slot] = a[r];
            sb[slot] = b[r];
        }
        __syncthreads();
        int add = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) add += wcnt[w][t];
        fill[t] += add;
    }
    __syncthreads();
    for (int slot = t; slot < total; slot += kBlock) {
        const int32_t k = sk[slot];
        const int d = (static_cast<uint32_t>(k) >> shift) & (kRadix - 1);
        const int64_t pos = run[d] + (slot - first[d]);
        if (pos < n) {
            keys_out[pos] = k;
            v0_out[pos] = sa[slot];
            if (v1_out) v1_out[pos] = sb[slot];
        }
    }
}

// dst id of every edge position (row expansion of row_ptr).
__global__ __launch_bounds__(kBlock) void expand_rows_kernel(const int64_t *__restrict__ row_ptr, int64_t nrows,
                                                             int32_t *__restrict__ dst) {
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
    for (int64_t row = wave; row < nrows; row += nwaves) {
        const int64_t e1 = row_ptr[row + 1];
        for (int64_t e = row_ptr[row] + lane_id(); e < e1; e += kWave) dst[e] = static_cast<int32_t>(row);
    }
}

// rec[e] = (bits of w[e], or of 1.0 without weights; the destination row of e) for every edge of the
// rows [x * kRecRows, (x + 1) * kRecRows) of tile x = blockIdx.x, shared by the kRecParts blocks
// blockIdx.y of the tile (a tile holding hub rows has far more edges than the others).  The tile's row
// pointers are staged in LDS; thread t of part y takes edges y * kBlock + t, then every
// kBlock * kRecParts-th (coalesced reads of w, coalesced 8-byte writes), and finds its row by binary
// search in LDS, so a long row costs its edges, not a serial walk.
constexpr int kRecRows = 2048;
constexpr int kRecParts = 16;

__global__ __launch_bounds__(kBlock) void edge_records_kernel(const int64_t *__restrict__ row_ptr, int64_t nrows,
                                                              const float *__restrict__ w, int2 *__restrict__ rec) {
    __shared__ int64_t sp[kRecRows + 1];
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kRecRows;
    const int nr = static_cast<int>(nrows - r0 < kRecRows ? nrows - r0 : kRecRows);
    for (int i = threadIdx.x; i <= nr; i += kBlock) sp[i] = row_ptr[r0 + i];
    __syncthreads();
    const int64_t e0 = sp[0], e1 = sp[nr];
    for (int64_t e = e0 + blockIdx.y * kBlock + threadIdx.x; e < e1; e += kBlock * kRecParts) {
        // the last row i of the tile with sp[i] <= e (rows are nonempty there: sp[i] <= e < sp[i+1])
        int lo = 0, hi = nr - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (sp[mid] <= e) lo = mid;
            else hi = mid - 1;
        }
        rec[e] = make_int2(__float_as_int(w ? w[e] : 1.0f), static_cast<int32_t>(r0 + lo));
    }
}

// ptr[j] = first sorted position with key >= j, for j in [0, nkeys]: one
// binary search per j, so long runs of absent keys cost no serial work.
__global__ __launch_bounds__(kBlock) void ptr_from_sorted_kernel(const int32_t *__restrict__ sorted, int64_t n,
                                                                 int64_t nkeys, int64_t *__restrict__ ptr) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; j <= nkeys; j += stride) {
        int64_t lo = 0, hi = n;
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo) / 2;
            if (static_cast<int64_t>(sorted[mid]) < j) lo = mid + 1;
            else hi = mid;
        }
        ptr[j] = lo;
    }
}

// ---------------------------------------------------------------- validation

struct Violations {
    unsigned long long first_row;    // first i with row_ptr[i] > row_ptr[i+1]
    unsigned long long first_col;    // first e with col out of range
    long long rp0, rpn;              // row_ptr[0], row_ptr[num_dst]
};

__global__ __launch_bounds__(kBlock) void validate_kernel(const int64_t *__restrict__ row_ptr,
                                                          const int32_t *__restrict__ col, int64_t nrows,
                                                          int64_t nedges, int64_t nsrc, Violations *v) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (tid == 0) {
        v->rp0 = row_ptr[0];
        v->rpn = row_ptr[nrows];
    }
    for (int64_t i = tid; i < nrows; i += stride)
        if (row_ptr[i] > row_ptr[i + 1]) atomicMin(&v->first_row, static_cast<unsigned long long>(i));
    for (int64_t e = tid; e < nedges; e += stride) {
        const int32_t c = col[e];
        if (c < 0 || c >= nsrc) atomicMin(&v->first_col, static_cast<unsigned long long>(e));
    }
}

__global__ void validate_init_kernel(Violations *v) {
    v->first_row = ~0ull;
    v->first_col = ~0ull;
    v->rp0 = 0;
    v->rpn = 0;
}

}  // namespace

size_t scan_ws_bytes(int64_t n) {
    Carve c(nullptr);
    c.take<int64_t>(ceil_div(n > 0 ? n : 1, kScanTile));
    return c.bytes();
}

int launch_excl_scan(const int64_t *in, int64_t *out, int64_t n, void *ws, hipStream_t stream) {
    if (n <= 0) return TIGA_OK;
    if (n <= kScanSmall) {
        hipLaunchKernelGGL(scan_small_kernel, dim3(1), dim3(kSmallThreads), 0, stream, in, out, n);
        return check_launch("scan (one block)");
    }
    const int64_t blocks = ceil_div(n, kScanTile);
    Carve c(ws);
    int64_t *partial = c.take<int64_t>(blocks);
    hipLaunchKernelGGL(scan_reduce_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0, stream, in, n, partial);
    if (int rc = check_launch("scan reduce")) return rc;
    hipLaunchKernelGGL(scan_partials_kernel, dim3(1), dim3(kBlock), 0, stream, partial, blocks);
    if (int rc = check_launch("scan partials")) return rc;
    hipLaunchKernelGGL(scan_down_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0, stream, in, out, n,
                       partial);
    return check_launch("scan down");
}

namespace {
struct SortWs {
    int32_t *k[2], *a[2], *b[2];
    int64_t *counts;
    void *scan;
};

SortWs carve_sort(Carve &c, int64_t n, bool payload) {
    SortWs s;
    const int64_t nb = ceil_div(n > 0 ? n : 1, kSortTile);
    for (int i = 0; i < 2; ++i) {
        s.k[i] = c.take<int32_t>(n);
        s.a[i] = c.take<int32_t>(n);
        s.b[i] = payload ? c.take<int32_t>(n) : nullptr;
    }
    s.counts = c.take<int64_t>(nb * kRadix);
    s.scan = c.take<char>(scan_ws_bytes(nb * kRadix));
    return s;
}

// Stable LSD radix sort of n keys in [0, key_limit), 8 bits per pass.  Carries
// the input position of every key (to idx_out) and optionally one payload
// (pay -> pay_out).  The sorted keys go to keys_out when given; *sorted points
// at them in any case.
int radix_sort(const int32_t *keys, const int32_t *pay, int64_t n, int64_t key_limit, int32_t *keys_out,
               int32_t *idx_out, int32_t *pay_out, const SortWs &s, const int32_t **sorted, hipStream_t stream) {
    int bits = 1;
    while (bits < 31 && (int64_t{1} << bits) < key_limit) ++bits;
    const int passes = (bits + kRadixBits - 1) / kRadixBits;
    const int64_t nb = ceil_div(n, kSortTile);
    const int32_t *kin = keys, *ain = nullptr, *bin = pay;
    for (int p = 0; p < passes; ++p) {
        const int shift = p * kRadixBits;
        hipLaunchKernelGGL(radix_hist_kernel, dim3(static_cast<unsigned>(nb)), dim3(kBlock), 0, stream, kin, n, shift,
                           nb, s.counts);
        if (int rc = check_launch("radix histogram")) return rc;
        if (int rc = launch_excl_scan(s.counts, s.counts, nb * kRadix, s.scan, stream)) return rc;
        // ping-pong through the workspace; the last pass writes the caller's arrays
        const bool last = p == passes - 1;
        const int buf = p & 1;
        int32_t *ko = last && keys_out ? keys_out : s.k[buf];
        int32_t *ao = last ? idx_out : s.a[buf];
        int32_t *bo = pay ? (last ? pay_out : s.b[buf]) : nullptr;
        hipLaunchKernelGGL(radix_scatter_kernel, dim3(static_cast<unsigned>(nb)), dim3(kBlock), 0, stream, kin, ain,
                           bin, ko, ao, bo, n, shift, nb, s.counts, p == 0 ? 1 : 0);
        if (int rc = check_launch("radix scatter")) return rc;
        kin = ko;
        ain = ao;
        bin = bo;
    }
    *sorted = kin;
    return TIGA_OK;
}

int ptr_from_sorted(const int32_t *sorted, int64_t n, int64_t nkeys, int64_t *ptr, hipStream_t stream) {
    const int pb = persistent_blocks(ceil_div(nkeys + 1, kWave), 8);
    hipLaunchKernelGGL(ptr_from_sorted_kernel, dim3(pb), dim3(kBlock), 0, stream, sorted, n, nkeys, ptr);
    return check_launch("pointers from sorted keys");
}
}  // namespace

size_t transpose_ws_bytes(int64_t num_dst, int64_t num_src, int64_t num_edges) {
    (void)num_dst;
    (void)num_src;
    Carve c(nullptr);
    carve_sort(c, num_edges, false);
    return c.bytes();
}

int launch_transpose(const tiga_csr *rel, int64_t *src_ptr, int32_t *edge_id, void *ws, hipStream_t stream) {
    const int64_t n = rel->num_edges;
    Carve c(ws);
    SortWs s = carve_sort(c, n, false);
    if (n == 0) return fill_u32(src_ptr, 0u, 2 * (rel->num_src + 1), stream);
    const int32_t *sorted = nullptr;
    if (int rc = radix_sort(rel->col_idx, nullptr, n, rel->num_src, nullptr, edge_id, nullptr, s, &sorted, stream))
        return rc;
    return ptr_from_sorted(sorted, n, rel->num_src, src_ptr, stream);
}

int launch_edge_records(const tiga_csr *rel, const float *w, int2 *rec, hipStream_t stream) {
    if (rel->num_edges == 0 || rel->num_dst == 0) return TIGA_OK;
    const int64_t tiles = ceil_div(rel->num_dst, kRecRows);
    hipLaunchKernelGGL(edge_records_kernel, dim3(static_cast<unsigned>(tiles), kRecParts), dim3(kBlock), 0, stream,
                       rel->row_ptr, rel->num_dst, w, rec);
    return check_launch("edge records");
}

size_t sort_keys_ws_bytes(int64_t n) {
    Carve c(nullptr);
    carve_sort(c, n, false);
    return c.bytes();
}

int launch_sort_keys(const int32_t *keys, int64_t n, int64_t key_limit, int32_t *keys_out, int32_t *idx_out,
                     int64_t *ptr, void *ws, hipStream_t stream) {
    Carve c(ws);
    SortWs s = carve_sort(c, n, false);
    const int32_t *sorted = nullptr;
    if (n > 0)
        if (int rc = radix_sort(keys, nullptr, n, key_limit, keys_out, idx_out, nullptr, s, &sorted, stream)) return rc;
    if (!ptr) return TIGA_OK;
    return ptr_from_sorted(n > 0 ? sorted : keys_out, n, key_limit, ptr, stream);
}

int launch_validate(const tiga_csr *rel, hipStream_t stream) {
    Violations *dv = nullptr;
    if (int rc = check_hip(hipMalloc(&dv, sizeof(Violations)), "validate: hipMalloc")) return rc;
    Violations hv{};
    int rc = TIGA_OK;
    hipLaunchKernelGGL(validate_init_kernel, dim3(1), dim3(1), 0, stream, dv);
    rc = check_launch("validate init");
    if (!rc) {
        const int blocks = persistent_blocks(ceil_div(rel->num_dst + rel->num_edges, kWave), 8);
        hipLaunchKernelGGL(validate_kernel, dim3(blocks), dim3(kBlock), 0, stream, rel->row_ptr, rel->col_idx,
                           rel->num_dst, rel->num_edges, rel->num_src, dv);
        rc = check_launch("validate");
    }
    if (!rc) rc = check_hip(hipMemcpyAsync(&hv, dv, sizeof hv, hipMemcpyDeviceToHost, stream), "validate: copy");
    if (!rc) rc = check_hip(hipStreamSynchronize(stream), "validate: synchronize");
    (void)hipFree(dv);
    if (rc) return rc;
    if (hv.rp0 != 0) return fail(TIGA_EGRAPH, "row_ptr[0] = %lld, expected 0", hv.rp0);
    if (hv.first_row != ~0ull)
        return fail(TIGA_EGRAPH, "row_ptr decreases at row %llu (row_ptr[i] > row_ptr[i+1])", hv.first_row);
    if (hv.rpn != rel->num_edges)
        return fail(TIGA_EGRAPH, "row_ptr[num_dst] = %lld, expected num_edges = %lld", hv.rpn,
                    (long long)rel->num_edges);
    if (hv.first_col != ~0ull)
        return fail(TIGA_EGRAPH, "col_idx[%llu] is outside [0, %lld)", hv.first_col, (long long)rel->num_src);
    return TIGA_OK;
}

}  // namespace csr
}  // namespace tiga
