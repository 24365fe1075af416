// Generated radius relation (Section 4.9 of the paper): a uniform cell
// directory restricts candidates, an exact fp32 distance predicate accepts,
// and accepted messages are folded into registers without storing edges.
//
// Build (every call, stateless):
//   bounding box -> cell size h >= r (1 + 2^-10), at most n + 64 cells ->
//   cell id per point (fp64 coordinates) -> stable radix sort of the cell ids
//   (ascending point ids within a cell: a deterministic order) -> cell
//   boundaries -> cell-ordered records (p, id) and feature rows.
// Consume: one wavefront per destination cell; the 27 neighbour cells are 9
// contiguous runs of the cell-ordered arrays (x-adjacent cells are adjacent
// in memory).
#include "csr_bwd.hpp"
#include "radius.hpp"
#include "radius_cells.hpp"

namespace tiga {
namespace radius {

using csr::launch_excl_scan;
using csr::scan_ws_bytes;

namespace {

constexpr int kBlock = 256;


__global__ __launch_bounds__(kBlock) void bbox_partial_kernel(const float *__restrict__ pos, int64_t n,
                                                              float *__restrict__ part) {
    float mn[3] = {__builtin_inff(), __builtin_inff(), __builtin_inff()};
    float mx[3] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            // the box covers finite coordinates only; a non-finite one is
            // never within the radius of anything and lands in a border cell
            const float v = pos[i * 3 + a];
            if (__builtin_isfinite(v)) {
                mn[a] = fminf(mn[a], v);
                mx[a] = fmaxf(mx[a], v);
            }
        }
    }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], shfl_xor_f(mn[a], m));
            mx[a] = fmaxf(mx[a], shfl_xor_f(mx[a], m));
        }
    __shared__ float sh[kBlock / kWave][6];
    const int wave = threadIdx.x / kWave;
    if (lane_id() == 0)
        for (int a = 0; a < 3; ++a) {
            sh[wave][a] = mn[a];
            sh[wave][3 + a] = mx[a];
        }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kBlock / kWave; ++w)
            for (int a = 0; a < 3; ++a) {
                sh[0][a] = fminf(sh[0][a], sh[w][a]);
                sh[0][3 + a] = fmaxf(sh[0][3 + a], sh[w][3 + a]);
            }
        for (int k = 0; k < 6; ++k) part[blockIdx.x * 6 + k] = sh[0][k];
    }
}

// One block: reduce the per-block boxes, then thread 0 picks the cell size and
// the grid dimensions.
__global__ __launch_bounds__(kBlock) void grid_params_kernel(const float *__restrict__ part, int nblocks, int64_t n,
                                                             float radius, int64_t max_cells, double spacing_scale,
                                                             Params *__restrict__ prm) {
    float mn[3] = {__builtin_inff(), __builtin_inff(), __builtin_inff()};
    float mx[3] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    for (int b = threadIdx.x; b < nblocks; b += blockDim.x)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], part[b * 6 + a]);
            mx[a] = fmaxf(mx[a], part[b * 6 + 3 + a]);
        }
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1)
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            mn[a] = fminf(mn[a], shfl_xor_f(mn[a], m));
            mx[a] = fmaxf(mx[a], shfl_xor_f(mx[a], m));
        }
    __shared__ float sh[kBlock / kWave][6];
    if (lane_id() == 0)
        for (int a = 0; a < 3; ++a) {
            sh[threadIdx.x / kWave][a] = mn[a];
            sh[threadIdx.x / kWave][3 + a] = mx[a];
        }
    __syncthreads();
    if (threadIdx.x != 0) return;
    double lo[3], hi[3];
    for (int a = 0; a < 3; ++a) {
        lo[a] = sh[0][a];
        hi[a] = sh[0][3 + a];
        for (int w = 1; w < kBlock / kWave; ++w) {
            lo[a] = fmin(lo[a], static_cast<double>(sh[w][a]));
            hi[a] = fmax(hi[a], static_cast<double>(sh[w][3 + a]));
        }
    }
    double ext[3], vol = 1.0;
    for (int a = 0; a < 3; ++a) {
        ext[a] = hi[a] - lo[a];
        if (!(ext[a] >= 0.0)) ext[a] = 0.0;
        vol *= ext[a];
    }
    // cells no smaller than the radius (with a relative margin that covers the
    // fp32 rounding of the predicate), and not much smaller than the mean
    // point spacing; grown until the directory has at most max_cells cells
    double h = static_cast<double>(radius) * (1.0 + 1.0 / 1024.0);
    const double spacing = spacing_scale * cbrt(vol / static_cast<double>(n > 0 ? n : 1));
    if (spacing > h) h = spacing;
    int64_t d[3] = {1, 1, 1};
    bool fits = false;
    for (int it = 0; it < 200 && !fits; ++it) {
        double cells = 1.0;  // in double: the product of three capped extents cannot overflow
        for (int a = 0; a < 3; ++a) {
            const double t = floor(ext[a] / h) + 1.0;
            d[a] = t > 2e9 ? static_cast<int64_t>(2e9) : static_cast<int64_t>(t);
            cells *= static_cast<double>(d[a]);
        }
        fits = cells <= static_cast<double>(max_cells);
        if (!fits) h *= 1.25;
    }
    if (!fits) {
        // unreachable for finite positions; one cell keeps the scan correct
        d[0] = d[1] = d[2] = 1;
        h = 1.0 + ext[0] + ext[1] + ext[2];
    }
    for (int a = 0; a < 3; ++a) {
        prm->lo[a] = lo[a];
        prm->dim[a] = static_cast<int>(d[a]);
    }
    prm->inv_h = 1.0 / h;
    prm->ncell = static_cast<int>(d[0] * d[1] * d[2]);
}

// Cell coordinate along axis a, clamped to [0, dim - 1] before conversion
// (NaN and -inf go to 0, +inf to the last cell).

// Cell id of every point (z-major, x fastest).
__global__ __launch_bounds__(kBlock) void cell_key_kernel(const float *__restrict__ pos, int64_t n,
                                                          const Params *__restrict__ prm, int32_t *__restrict__ cell) {
    const Params p = *prm;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int cx = cell_axis(p, 0, pos[i * 3 + 0]);
        const int cy = cell_axis(p, 1, pos[i * 3 + 1]);
        const int cz = cell_axis(p, 2, pos[i * 3 + 2]);
        cell[i] = (cz * p.dim[1] + cy) * p.dim[0] + cx;
    }
}

// Cell-ordered records (position, point id).
__global__ __launch_bounds__(kBlock) void gather_records_kernel(const int32_t *__restrict__ perm, int64_t n,
                                                                const float *__restrict__ pos,
                                                                float4 *__restrict__ rec) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; s < n; s += stride) {
        const int32_t i = perm[s];
        rec[s] = make_float4(pos[i * 3 + 0], pos[i * 3 + 1], pos[i * 3 + 2], __int_as_float(i));
    }
}




// ---------------------------------------------------------------------------
// Consume: one wavefront per destination cell.
//
// Every point of a cell has the same candidate set, the 27 cells around it
// (9 runs of the cell-ordered arrays), so the run bounds are wave-uniform.
// Phase 1: the wave loads 64 candidates at a time (one per lane, coalesced)
// and tests them against each destination of the cell in turn (up to kDch
// destinations per pass); the accepted lanes of a destination append
// (point id, kernel weight) to that destination's LDS list in candidate order
// (ballot + prefix count).  Phase 2 (a flush, when a list would overflow and
// at the end of the pass): lane groups of LPR lanes read each listed
// neighbour's feature row in place (caller's layout, no reordered copy) as
// LPR consecutive units, one destination per group; when the cell has few
// destinations, S groups share a destination (interleaved entries) and are
// combined by a fixed shuffle tree.  Every summation order depends only on the
// input.
constexpr int kDch = 8;      // destinations per pass over a cell's candidates
constexpr int kCapC = 64;    // list entries per destination between flushes
constexpr int kBatch = 6;    // list entries whose rows are loaded together
constexpr int kBatchDp = 2;  // the same when position gradients are formed

static_assert(kCapC >= kWave, "one candidate chunk may add a wave's worth of entries after a flush");
typedef float2 CellList[kDch][kCapC + 1];  // +1: groups reading different lists hit different banks

__device__ __forceinline__ void lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Visit order: the cell grid is cut into bricks of 8 x 8 x 8 cells (thinner at
// the far faces), walked brick by brick (x-, then y-, then z-major; cells within
// a brick the same way); order[t] is the t-th cell.  Each XCD (blockIdx.x % 8)
// owns one contiguous eighth of that order, so the cells in flight on an XCD
// form a compact block whose neighbour rows stay in that XCD's L2 (a run of
// whole x-rows of cells would touch three full z-planes of rows per pass).
//
// Dealing: cell costs vary (Poisson occupancy), and a fixed cells-to-waves
// split leaves the last waves running long after the rest, so cells are taken
// as waves finish.  An XCD has 4 counters (one 256-byte line each); counter k
// serves its waves w = k (mod 4) with the cells k (mod 4) of its share.  Each
// such wave takes its class's cells w' and W' + w' (w' = w / 4, W' waves in
// the class, at least 1 since the grid has at least 8 blocks of 4 waves), then
// the next one from the counter.  Increments of one counter are serialized
// where it lives: a single counter per XCD capped the rate at which cells were
// handed out, four spread the increments while the cells in flight stay one
// compact run of the order.  A wave knows its next cell one cell ahead (the
// counter is read, and the next cell's id loaded, while the current one runs),
// so neither latency is exposed.
constexpr float kLog2e = 1.44269504088896341f;
constexpr int kBrickLog = 3;
constexpr int kBrick = 1 << kBrickLog;
constexpr int kSchedStride = 64;  // uint32 per counter: one 256-byte line each
constexpr int kCtrPerXcd = 4;     // counters per XCD: counter k hands out the cells k (mod 4)

// Next value of this wave's XCD counter (one lane's atomic, broadcast).
__device__ __forceinline__ int64_t take_visit(uint32_t *__restrict__ sched, int k) {
    uint32_t v = 0;
    if (lane_id() == 0) v = atomicAdd(sched + ((blockIdx.x % kXcds) * kCtrPerXcd + k) * kSchedStride, 1u);
    return __builtin_amdgcn_readfirstlane(v);
}

// order[rank(c)] = c for every cell c: the rank counts the cells of the whole
// slabs, brick rows and bricks before c's, then c's place inside its brick.
// Also clears the XCD counters of the consuming kernel that follows.
__global__ __launch_bounds__(kBlock) void visit_order_kernel(const Params *__restrict__ prm,
                                                            int32_t *__restrict__ order,
                                                            uint32_t *__restrict__ sched) {
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < kXcds * kCtrPerXcd * kSchedStride; i += kBlock) sched[i] = 0u;
    const Params p = *prm;
    const int64_t X = p.dim[0], Y = p.dim[1], Z = p.dim[2];
    for (int64_t c = blockIdx.x * static_cast<int64_t>(kBlock) + threadIdx.x; c < p.ncell;
         c += static_cast<int64_t>(gridDim.x) * kBlock) {
        const int64_t cx = c % X, cy = (c / X) % Y, cz = c / (X * Y);
        const int64_t x0 = cx & ~static_cast<int64_t>(kBrick - 1), y0 = cy & ~static_cast<int64_t>(kBrick - 1),
                      z0 = cz & ~static_cast<int64_t>(kBrick - 1);
        const int64_t h = Z - z0 < kBrick ? Z - z0 : kBrick;
        const int64_t wy = Y - y0 < kBrick ? Y - y0 : kBrick;
        const int64_t wx = X - x0 < kBrick ? X - x0 : kBrick;
        const int64_t rank = z0 * X * Y + y0 * h * X + x0 * h * wy + (cz - z0) * wy * wx + (cy - y0) * wx + (cx - x0);
        order[rank] = static_cast<int32_t>(c);
    }
}

// Split factor for a flush over dn destinations with G groups: the largest
// power of two S with S * dn <= G (1 when dn > G / 2).
__device__ __forceinline__ int split_for(int dn, int groups) {
    int s = 1;
    while (2 * s * dn <= groups) s *= 2;
    return s;
}

template <int K>
__device__ __forceinline__ void load_k(const float *__restrict__ base, int64_t unit, bool ok, float (&v)[K]) {
    if (ok) {
        const csr::Vec<K> t = csr::load_unit<K>(base, unit);
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = t.v[k];
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = 0.0f;
    }
}

// Write (first flush of a pass) or accumulate (later flushes) one unit.
template <int K>
__device__ __forceinline__ void put_k(float *__restrict__ base, int64_t unit, const float (&v)[K], bool first) {
    if (first) {
        csr::store_unit<K>(base, unit, v);
    } else {
        const csr::Vec<K> o = csr::load_unit<K>(base, unit);
        float s[K];
#pragma unroll
        for (int k = 0; k < K; ++k) s[k] = o.v[k] + v[k];
        csr::store_unit<K>(base, unit, s);
    }
}

// v[lane] = val (val and lane wave-uniform): one v_writelane_b32 (the lane
// select is taken from m0, which does not count against the one-scalar-operand
// limit).
__device__ __forceinline__ void set_lane(int &v, int lane, int val) {
    asm("v_writelane_b32 %0, %1, %2" : "+v"(v) : "s"(val), "{m0}"(lane));
}

// Candidate positions of a cell: the 3 x 3 (z, y) rows of its neighbourhood,
// each one run of up to 3 cells that is contiguous in cell order, laid end to
// end.  Lane k < 9 loads run k's bounds (one round trip for all nine); the runs
// are then turned, window by window, into an LDS table that maps each candidate
// position to its cell-ordered record index, so a chunk of 64 candidates is
// decoded by one LDS read per lane.
constexpr int kWin = 256;  // candidate positions per table window
typedef int32_t CandTable[kWin];

struct CellRuns {
    int32_t pos;    // lane k < 9: first position of run k
    int32_t len;    // lane k < 9: its length
    int32_t off;    // lane k < 9: record index - position within run k
    int32_t total;  // number of candidates (uniform)
};

__device__ __forceinline__ CellRuns cell_runs(const Params &p, const int64_t *__restrict__ start, int cx, int cy,
                                              int cz) {
    const int lane = lane_id();
    const int x0 = cx > 0 ? cx - 1 : 0;
    const int x1 = cx + 1 < p.dim[0] ? cx + 1 : p.dim[0] - 1;
    int64_t s0 = 0;
    int32_t len = 0;
    if (lane < 9) {
        const int z = cz - 1 + lane / 3;
        const int y = cy - 1 + lane % 3;
        if (z >= 0 && z < p.dim[2] && y >= 0 && y < p.dim[1]) {
            const int64_t rowc = (static_cast<int64_t>(z) * p.dim[1] + y) * p.dim[0];
            s0 = start[rowc + x0];
            len = static_cast<int32_t>(start[rowc + x1 + 1] - s0);
        }
    }
    // exclusive prefix of the lengths over lanes 0..8
    int32_t pos = 0, total = 0;
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        const int32_t l = __builtin_amdgcn_readlane(len, k);
        pos = lane == k ? total : pos;
        total += l;
    }
    return CellRuns{pos, len, static_cast<int32_t>(s0) - pos, total};
}

// Table entries of positions [w0, min(w0 + kWin, total)).
__device__ __forceinline__ void fill_candidates(const CellRuns &r, int32_t w0, CandTable &tab) {
    const int lane = lane_id();
    const int32_t lo_l = r.pos > w0 ? r.pos : w0;
    const int32_t hi_l = r.pos + r.len < w0 + kWin ? r.pos + r.len : w0 + kWin;
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        const int32_t lo = __builtin_amdgcn_readlane(lo_l, k), hi = __builtin_amdgcn_readlane(hi_l, k);
        if (lo >= hi) continue;
        const int32_t off = __builtin_amdgcn_readlane(r.off, k);
        for (int32_t q = lo + lane; q < hi; q += kWave) tab[q - w0] = q + off;
    }
}

// Phase 1 over every cell of this wave; `flush(cnt, dn, d0, id, first)` runs
// phase 2 for the destinations d0 .. d0 + dn - 1 (lane d holds the list
// length `cnt` and point id `id` of destination d).  Weights are
// exp2(d2 * nis_log2e), nis_log2e = -log2(e) / sigma^2.
template <class Flush>
__device__ __forceinline__ void cell_consume(const Params &p, const int32_t *__restrict__ order,
                                             uint32_t *__restrict__ sched, const int64_t *__restrict__ start,
                                             const float4 *__restrict__ rec, float r2, float nis_log2e,
                                             CellList &list, CandTable &tab, int32_t *__restrict__ count,
                                             Flush &&flush) {
    const int lane = lane_id();
    const int64_t lo = static_cast<int64_t>(p.ncell) * (blockIdx.x % kXcds) / kXcds;
    const int64_t hi = static_cast<int64_t>(p.ncell) * (blockIdx.x % kXcds + 1) / kXcds;
    // waves per XCD and this wave's index among them (uniform)
    const int64_t nw = static_cast<int64_t>(gridDim.x / kXcds) * (kBlock / kWave);
    const int64_t lw = static_cast<int64_t>(blockIdx.x / kXcds) * (kBlock / kWave) +
                       uniform(static_cast<int>(threadIdx.x / kWave));
    // counter k = lw mod 4 serves the nwk waves of that residue; its i-th cell is lo + k + 4 i
    // (every XCD has at least 4 waves, so every residue is served)
    const int k = static_cast<int>(lw % kCtrPerXcd);
    const int64_t nwk = (nw - k + kCtrPerXcd - 1) / kCtrPerXcd, lwk = lw / kCtrPerXcd;
    int64_t t = lo + k + kCtrPerXcd * lwk, t1 = lo + k + kCtrPerXcd * (nwk + lwk), t2 = hi;
    int64_t c = t < hi ? order[t] : 0, c1 = 0;
    for (; t < hi; t = t1, c = c1, t1 = t2) {
        // the cell after this one: its id now, and the counter for the one after that
        c1 = t1 < hi ? order[t1] : 0;
        t2 = t1 < hi ? lo + k + kCtrPerXcd * (2 * nwk + take_visit(sched, k)) : hi;
        const int64_t ds = start[c], de = start[c + 1];
        if (ds == de) continue;
        const int cx = static_cast<int>(c % p.dim[0]);
        const int cy = static_cast<int>((c / p.dim[0]) % p.dim[1]);
        const int cz = static_cast<int>(c / (static_cast<int64_t>(p.dim[0]) * p.dim[1]));
        const CellRuns runs = cell_runs(p, start, cx, cy, cz);
        const int32_t total = runs.total;
        fill_candidates(runs, 0, tab);
        // the destinations' own positions, which the test must skip: record
        // d0 + d sits in run 4 (the cell's own row), at position d0 + d - off_4
        const int32_t ds_pos = static_cast<int32_t>(ds) - __builtin_amdgcn_readlane(runs.off, 4);
        for (int64_t d0 = ds; d0 < de; d0 += kDch) {
            const int dn = static_cast<int>(de - d0 < kDch ? de - d0 : kDch);
            const int32_t idl = lane < dn ? __float_as_int(rec[d0 + lane].w) : -1;
            const int32_t self0 = ds_pos + static_cast<int32_t>(d0 - ds);
            int cnt = 0, tot = 0;
            bool first = true;
            for (int32_t w0 = 0; w0 < total; w0 += kWin) {
                // window 0 of a cell with at most kWin candidates is filled once per cell
                if (w0 > 0 || (d0 > ds && total > kWin)) {
                    lds_fence();
                    fill_candidates(runs, w0, tab);
                }
                lds_fence();
                const int32_t w1 = total < w0 + kWin ? total : w0 + kWin;
                for (int32_t c0 = w0; c0 < w1; c0 += kWave) {
                    const int32_t pos = c0 + lane;
                    // lanes past the end test a point at +inf, which no destination accepts
                    const float4 pj = pos < w1 ? rec[tab[pos - w0]]
                                               : make_float4(__int_as_float(0x7f800000), __int_as_float(0x7f800000),
                                                             __int_as_float(0x7f800000), __int_as_float(-1));
                    for (int d = 0; d < dn; ++d) {
                        const float4 pd = rec[d0 + d];  // uniform address: a scalar load
                        float d2;
                        // pos - c0 == self only on the destination's own lane; each
                        // compare is balloted on its own so that both masks come straight
                        // from the compares
                        const bool near = accept(pd, pj, r2, d2);
                        const bool other = lane != self0 + d - c0;
                        const uint64_t mask = __builtin_amdgcn_ballot_w64(near) & __builtin_amdgcn_ballot_w64(other);
                        if (mask == 0) continue;
                        const int nnew = __popcll(mask);
                        int cd = __builtin_amdgcn_readlane(cnt, d);
                        if (cd + nnew > kCapC) {
                            tot += cnt;
                            flush(cnt, dn, d0, idl, first);
                            first = false;
                            cnt = 0;
                            cd = 0;
                        }
                        if (near & other) {
                            const int pfx = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                                                      __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0));
                            // (point id, weight)
                            list[d][cd + pfx] = make_float2(pj.w, __builtin_amdgcn_exp2f(d2 * nis_log2e));
                        }
                        set_lane(cnt, d, cd + nnew);
                    }
                }
            }
            tot += cnt;
            flush(cnt, dn, d0, idl, first);
            if (count && lane < dn) count[idl] = tot;
        }
    }
}

// y_i = sum_j k_ij x_j; K floats per unit, LPR lanes per row, UPL units per
// lane per feature block. The pair loop is latency-bound, so the one-unit
// forms are held to 72 registers (7 waves per SIMD instead of 6); the few
// values this spills cost less than the extra wave gains. The two-unit form
// would spill dozens and keeps its registers.
template <int K, int LPR, int UPL>
__global__ __launch_bounds__(kBlock, UPL == 1 ? 7 : 1) void radius_fwd_cell_kernel(const Params *__restrict__ prm,
                                                                 const int32_t *__restrict__ order,
                                                                 uint32_t *__restrict__ sched,
                                                                 const int64_t *__restrict__ start,
                                                                 const float4 *__restrict__ rec,
                                                                 const float *__restrict__ xs, int64_t fu, float r2,
                                                                 float nis_log2e, float *__restrict__ y,
                                                                 int32_t *__restrict__ count) {
    constexpr int G = kWave / LPR;
    __shared__ CellList lists[kBlock / kWave];
    __shared__ CandTable tabs[kBlock / kWave];
    const Params p = *prm;
    const int wv = uniform(static_cast<int>(threadIdx.x / kWave));
    CellList &list = lists[wv];
    const int lane = lane_id(), g = lane / LPR, q = lane % LPR;
    const uint32_t ufu = static_cast<uint32_t>(fu);  // n * fu < 2^32 (checked by the host)
    auto flush = [&](int cnt, int dn, int64_t, int32_t idl, bool first) {
        lds_fence();
        const int S = split_for(dn, G);
        const int D = G / S;
        const int slot = g % D, sp = g / D;
        for (int r0 = 0; r0 < dn; r0 += D) {
            const int d = r0 + slot;
            const bool dv = d < dn;
            // every lane takes part in the shuffles: a lane outside the exec
            // mask would read as zero
            const int mds = __shfl(cnt, dv ? d : 0, kWave);
            const int md = dv ? mds : 0;
            const int32_t id = __shfl(idl, dv ? d : 0, kWave);
            if (!first && __ballot(md > 0) == 0) continue;
            for (int64_t fb = 0; fb < fu; fb += LPR * UPL) {
                const uint32_t ufb = static_cast<uint32_t>(fb);
                float acc[UPL][K];
#pragma unroll
                for (int u = 0; u < UPL; ++u)
#pragma unroll
                    for (int k = 0; k < K; ++k) acc[u][k] = 0.0f;
                // units past the row end (fu not a multiple of LPR) load the
                // last unit instead; their sums are never stored
                uint32_t uc[UPL];
#pragma unroll
                for (int u = 0; u < UPL; ++u) {
                    const uint32_t unit = ufb + q + u * LPR;
                    uc[u] = unit < ufu ? unit : ufu - 1;
                }
                // FULL: all kBatch entries exist, no per-entry masks
                auto batch = [&](int k0, auto full) __attribute__((always_inline)) {
                    constexpr bool FULL = decltype(full)::value;
                    float2 en[kBatch];
#pragma unroll
                    for (int b = 0; b < kBatch; ++b)
                        en[b] = FULL || k0 + b * S < md ? list[d][k0 + b * S] : make_float2(0.0f, 0.0f);
                    float xv[kBatch][UPL][K];
#pragma unroll
                    for (int b = 0; b < kBatch; ++b) {
                        const uint32_t row = static_cast<uint32_t>(__float_as_int(en[b].x)) * ufu;
#pragma unroll
                        for (int u = 0; u < UPL; ++u) load_k<K>(xs, row + uc[u], FULL || k0 + b * S < md, xv[b][u]);
                    }
#pragma unroll
                    for (int b = 0; b < kBatch; ++b)
#pragma unroll
                        for (int u = 0; u < UPL; ++u)
#pragma unroll
                            for (int k = 0; k < K; ++k) acc[u][k] = fmaf(en[b].y, xv[b][u][k], acc[u][k]);
                };
                int k0 = sp;
                for (; k0 + (kBatch - 1) * S < md; k0 += S * kBatch) batch(k0, std::true_type{});
                if (k0 < md) batch(k0, std::false_type{});
                for (int o = D * LPR; o < kWave; o <<= 1)
#pragma unroll
                    for (int u = 0; u < UPL; ++u)
#pragma unroll
                        for (int k = 0; k < K; ++k) acc[u][k] += shfl_xor_f(acc[u][k], o);
                if (sp == 0 && dv) {
#pragma unroll
                    for (int u = 0; u < UPL; ++u) {
                        const int64_t unit = fb + q + u * LPR;
                        if (unit < fu) put_k<K>(y, static_cast<int64_t>(id) * fu + unit, acc[u], first);
                    }
                }
            }
        }
        lds_fence();
    };
    cell_consume(p, order, sched, start, rec, r2, nis_log2e, list, tabs[wv], count, flush);
}

struct Pos3 {
    float x, y, z;
};

// Backward on the same schedule: dx_i = sum_j k_ij dy_j and
// dp_i = sum_j (2 k_ij / sigma^2) (p_j - p_i) (<dy_i, x_j> + <dy_j, x_i>).
// Each lane forms the part of the inner products its units cover; the parts
// of a destination are added by the shuffle tree once per flush.
template <int K, int LPR, int UPL, bool DX, bool DP>
__global__ __launch_bounds__(kBlock, DP ? 5 : 6) void radius_bwd_cell_kernel(const Params *__restrict__ prm,
                                                                 const int32_t *__restrict__ order,
                                                                 uint32_t *__restrict__ sched,
                                                                 const int64_t *__restrict__ start,
                                                                 const float4 *__restrict__ rec,
                                                                 const float *__restrict__ pos,
                                                                 const float *__restrict__ xs,
                                                                 const float *__restrict__ ys, int64_t fu, float r2,
                                                                 float nis_log2e, float two_inv_s2,
                                                                 float *__restrict__ dx, float *__restrict__ dp) {
    constexpr int G = kWave / LPR;
    constexpr int B = DP ? kBatchDp : kBatch;
    __shared__ CellList lists[kBlock / kWave];
    __shared__ CandTable tabs[kBlock / kWave];
    const Params p = *prm;
    const int wv = uniform(static_cast<int>(threadIdx.x / kWave));
    CellList &list = lists[wv];
    const int lane = lane_id(), g = lane / LPR, q = lane % LPR;
    const uint32_t ufu = static_cast<uint32_t>(fu);  // n * fu < 2^32 (checked by the host)
    auto flush = [&](int cnt, int dn, int64_t d0, int32_t idl, bool first) {
        lds_fence();
        const int S = split_for(dn, G);
        const int D = G / S;
        const int slot = g % D, sp = g / D;
        for (int r0 = 0; r0 < dn; r0 += D) {
            const int d = r0 + slot;
            const bool dv = d < dn;
            // every lane takes part in the shuffles: a lane outside the exec
            // mask would read as zero
            const int mds = __shfl(cnt, dv ? d : 0, kWave);
            const int md = dv ? mds : 0;
            const int32_t id = __shfl(idl, dv ? d : 0, kWave);
            if (!first && __ballot(md > 0) == 0) continue;
            const int64_t sd = d0 + (dv ? d : 0);
            const float4 pd = DP ? rec[sd] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);  // sd is a valid point
            float gp[3] = {0.0f, 0.0f, 0.0f};
            for (int64_t fb = 0; fb < fu; fb += LPR * UPL) {
                const uint32_t ufb = static_cast<uint32_t>(fb);
                float acc[UPL][K], gi[UPL][K], xi[UPL][K];
#pragma unroll
                for (int u = 0; u < UPL; ++u) {
                    const int64_t unit = fb + q + u * LPR;
                    const bool ok = DP && dv && unit < fu;
                    const int64_t at = ok ? static_cast<int64_t>(id) * fu + unit : 0;
                    const csr::Vec<K> a = csr::load_unit<K>(ys, at);
                    const csr::Vec<K> c = csr::load_unit<K>(xs, at);
#pragma unroll
                    for (int k = 0; k < K; ++k) {
                        gi[u][k] = ok ? a.v[k] : 0.0f;
                        xi[u][k] = ok ? c.v[k] : 0.0f;
                        acc[u][k] = 0.0f;
                    }
                }
                // units past the row end (fu not a multiple of LPR) load the
                // last unit instead and take no part in the inner products
                uint32_t uc[UPL];
                bool uok[UPL];
#pragma unroll
                for (int u = 0; u < UPL; ++u) {
                    const uint32_t unit = ufb + q + u * LPR;
                    uok[u] = unit < ufu;
                    uc[u] = uok[u] ? unit : ufu - 1;
                }
                auto batch = [&](int k0, auto full) __attribute__((always_inline)) {
                    constexpr bool FULL = decltype(full)::value;
                    float2 en[B];
#pragma unroll
                    for (int b = 0; b < B; ++b)
                        en[b] = FULL || k0 + b * S < md ? list[d][k0 + b * S] : make_float2(0.0f, 0.0f);
                    float gj[B][UPL][K], xj[B][UPL][K];
                    f32x4 pj[B];
#pragma unroll
                    for (int b = 0; b < B; ++b) {
                        const bool live = FULL || k0 + b * S < md;
                        const uint32_t t = static_cast<uint32_t>(__float_as_int(en[b].x));  // point id
#pragma unroll
                        for (int u = 0; u < UPL; ++u) {
                            load_k<K>(ys, t * ufu + uc[u], live, gj[b][u]);
                            if (DP) load_k<K>(xs, t * ufu + uc[u], live, xj[b][u]);
                        }
                        if (DP) {
                            // t is a valid point id for every entry (0 past the list end);
                            // one 12-byte load
                            const Pos3 v = *reinterpret_cast<const Pos3 *>(pos + t * 3);
                            pj[b] = live ? f32x4{v.x, v.y, v.z, 0.0f} : f32x4{pd.x, pd.y, pd.z, pd.w};
                        }
                    }
#pragma unroll
                    for (int b = 0; b < B; ++b) {
                        float dot = 0.0f;
#pragma unroll
                        for (int u = 0; u < UPL; ++u) {
                            float du = 0.0f;
#pragma unroll
                            for (int k = 0; k < K; ++k) {
                                if (DX) acc[u][k] = fmaf(en[b].y, gj[b][u][k], acc[u][k]);
                                if (DP) du = fmaf(gi[u][k], xj[b][u][k], fmaf(gj[b][u][k], xi[u][k], du));
                            }
                            dot += uok[u] ? du : 0.0f;
                        }
                        if (DP) {
                            const float cc = two_inv_s2 * en[b].y * dot;
                            gp[0] = fmaf(cc, pj[b].x - pd.x, gp[0]);
                            gp[1] = fmaf(cc, pj[b].y - pd.y, gp[1]);
                            gp[2] = fmaf(cc, pj[b].z - pd.z, gp[2]);
                        }
                    }
                };
                int k0 = sp;
                for (; k0 + (B - 1) * S < md; k0 += S * B) batch(k0, std::true_type{});
                if (k0 < md) batch(k0, std::false_type{});
                if (DX) {
                    for (int o = D * LPR; o < kWave; o <<= 1)
#pragma unroll
                        for (int u = 0; u < UPL; ++u)
#pragma unroll
                            for (int k = 0; k < K; ++k) acc[u][k] += shfl_xor_f(acc[u][k], o);
                    if (sp == 0 && dv) {
#pragma unroll
                        for (int u = 0; u < UPL; ++u) {
                            const int64_t unit = fb + q + u * LPR;
                            if (unit < fu) put_k<K>(dx, static_cast<int64_t>(id) * fu + unit, acc[u], first);
                        }
                    }
                }
            }
            if (DP) {
#pragma unroll
                for (int o = 1; o < LPR; o <<= 1)
#pragma unroll
                    for (int a = 0; a < 3; ++a) gp[a] += shfl_xor_f(gp[a], o);
                for (int o = D * LPR; o < kWave; o <<= 1)
#pragma unroll
                    for (int a = 0; a < 3; ++a) gp[a] += shfl_xor_f(gp[a], o);
                if (sp == 0 && q == 0 && dv) {
                    float *o = dp + static_cast<int64_t>(id) * 3;
#pragma unroll
                    for (int a = 0; a < 3; ++a) o[a] = first ? gp[a] : o[a] + gp[a];
                }
            }
        }
        lds_fence();
    };
    cell_consume(p, order, sched, start, rec, r2, nis_log2e, list, tabs[wv], nullptr, flush);
}

__global__ __launch_bounds__(kBlock) void neighbor_count_kernel(const Params *__restrict__ prm,
                                                                const int64_t *__restrict__ start,
                                                                const float4 *__restrict__ rec, int64_t n, float r2,
                                                                int32_t *__restrict__ count) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    int c = 0;
    for_candidates(p, start, pi, [&](int64_t t) {
        const float4 pj = rec[t];
        float d2;
        if (accept(pi, pj, r2, d2) && __float_as_int(pj.w) != i) ++c;
    });
    count[i] = c;
}

__global__ __launch_bounds__(kBlock) void neighbor_fill_kernel(const Params *__restrict__ prm,
                                                               const int64_t *__restrict__ start,
                                                               const float4 *__restrict__ rec, int64_t n, float r2,
                                                               const int64_t *__restrict__ ptr,
                                                               int32_t *__restrict__ idx,
                                                               uint32_t *__restrict__ mismatch) {
    const Params p = *prm;
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const float4 pi = rec[s];
    const int32_t i = __float_as_int(pi.w);
    // writes stay inside the caller's span [ptr[i], ptr[i+1]); a span that is not the point's
    // neighbour count is reported, never overrun
    const int64_t b = ptr[i];
    const int64_t e = ptr[i + 1];
    int64_t w = b;
    for_candidates(p, start, pi, [&](int64_t t) {
        const float4 pj = rec[t];
        float d2;
        const int32_t j = __float_as_int(pj.w);
        if (accept(pi, pj, r2, d2) && j != i) {
            if (w < e) idx[w] = j;
            ++w;
        }
    });
    if (w != e) atomicOr(mismatch, 1u);
    if (w > e) w = e;
    // insertion sort of this point's list (ascending ids)
    for (int64_t a = b + 1; a < w; ++a) {
        const int32_t v = idx[a];
        int64_t k = a - 1;
        while (k >= b && idx[k] > v) {
            idx[k + 1] = idx[k];
            --k;
        }
        idx[k + 1] = v;
    }
}

struct Ws {
    Params *prm;
    float *bbox;
    int32_t *cell, *cell_sorted;
    int32_t *perm_b;  // point id at each cell-ordered position
    int64_t *start;   // max_cells + 1 cell boundaries in cell order
    int32_t *order;   // max_cells: the cell visit order of the consuming kernels
    uint32_t *sched;  // the consuming kernels' per-XCD cell counters
    float4 *rec;
    void *sort;
    void *scan;
    uint32_t *flag;
    int64_t max_cells;
    int bbox_blocks;
};

// cells_per_point bounds the directory (max_cells = cells_per_point * n + 64): 1 for volume
// clouds; more for callers whose points lie on surfaces, where the volume-based spacing floor
// overestimates the point spacing.
Ws carve(Carve &c, int64_t n, int64_t cells_per_point = 1) {
    Ws w;
    w.max_cells = cells_per_point * n + 64;
    w.bbox_blocks = 1024;
    w.prm = c.take<Params>(1);
    w.bbox = c.take<float>(6 * w.bbox_blocks);
    w.cell = c.take<int32_t>(n);
    w.cell_sorted = c.take<int32_t>(n);
    w.perm_b = c.take<int32_t>(n);
    w.start = c.take<int64_t>(w.max_cells + 1);
    w.order = c.take<int32_t>(w.max_cells);
    w.sched = c.take<uint32_t>(kXcds * kCtrPerXcd * kSchedStride);
    w.rec = c.take<float4>(n);
    w.sort = c.take<char>(csr::sort_keys_ws_bytes(n));
    w.scan = c.take<char>(scan_ws_bytes(n + 1));
    w.flag = c.take<uint32_t>(1);
    return w;
}

int blocks_for(int64_t n) {
    int64_t b = ceil_div(n > 0 ? n : 1, kBlock);
    const int64_t cap = static_cast<int64_t>(device_cus()) * 32;
    return static_cast<int>(b < cap ? b : cap);
}

// Build the cell directory and the cell-ordered records.
int build(int64_t n, const float *pos, float radius, Ws &w, hipStream_t stream, double spacing_scale = 1.0) {
    int nb = w.bbox_blocks;
    const int64_t need = ceil_div(n, kBlock);
    if (need < nb) nb = static_cast<int>(need);
    hipLaunchKernelGGL(bbox_partial_kernel, dim3(nb), dim3(kBlock), 0, stream, pos, n, w.bbox);
    if (int rc = check_launch("radius bbox")) return rc;
    hipLaunchKernelGGL(grid_params_kernel, dim3(1), dim3(kBlock), 0, stream, w.bbox, nb, n, radius, w.max_cells,
                       spacing_scale, w.prm);
    if (int rc = check_launch("radius grid")) return rc;
    // cell-ordered positions: a stable sort by cell keeps ascending point ids
    // within a cell, so every candidate order depends only on the input
    hipLaunchKernelGGL(cell_key_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, pos, n, w.prm, w.cell);
    if (int rc = check_launch("radius cell keys")) return rc;
    if (int rc = csr::launch_sort_keys(w.cell, n, w.max_cells, w.cell_sorted, w.perm_b, w.start, w.sort, stream))
        return rc;
    hipLaunchKernelGGL(gather_records_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, stream, w.perm_b, n, pos, w.rec);
    return check_launch("radius records");
}

// The cell visit order and cleared counters of the consuming kernels (after build).
int visit_order(const Ws &w, hipStream_t stream) {
    hipLaunchKernelGGL(visit_order_kernel, dim3(blocks_for(w.max_cells)), dim3(kBlock), 0, stream, w.prm, w.order,
                       w.sched);
    return check_launch("radius visit order");
}

// Persistent grid for the cell kernels: a multiple of 8 blocks (one share
// per XCD), as many as stay resident.
int cell_grid(const void *kernel) {
    int64_t blocks = static_cast<int64_t>(resident_blocks(kernel, kBlock)) * device_cus();
    blocks = blocks / kXcds * kXcds;
    return static_cast<int>(blocks < kXcds ? kXcds : blocks);
}

template <int K, int LPR, int UPL>
int fwd_cell(int64_t fu, const Ws &w, const float *x, float r2, float nis, float *y, int32_t *count,
             hipStream_t stream) {
    const void *kern = reinterpret_cast<const void *>(&radius_fwd_cell_kernel<K, LPR, UPL>);
    static const int grid = cell_grid(kern);
    prof_before(stream);
    hipLaunchKernelGGL((radius_fwd_cell_kernel<K, LPR, UPL>), dim3(grid), dim3(kBlock), 0, stream, w.prm, w.order,
                       w.sched, w.start, w.rec, x, fu, r2, nis, y, count);
    prof_after(stream);
    return check_launch("radius forward");
}

// Lanes per row: the smallest power of two covering the row's units, at most
// 8 (with two units per lane beyond that); wider rows loop over feature blocks.
template <int K>
int fwd_units(int64_t fu, const Ws &w, const float *x, float r2, float nis, float *y, int32_t *count,
              hipStream_t stream) {
    if (fu <= 1) return fwd_cell<K, 1, 1>(fu, w, x, r2, nis, y, count, stream);
    if (fu <= 2) return fwd_cell<K, 2, 1>(fu, w, x, r2, nis, y, count, stream);
    if (fu <= 4) return fwd_cell<K, 4, 1>(fu, w, x, r2, nis, y, count, stream);
    if (fu <= 8) return fwd_cell<K, 8, 1>(fu, w, x, r2, nis, y, count, stream);
    return fwd_cell<K, 8, 2>(fu, w, x, r2, nis, y, count, stream);
}

struct BwdIo {
    const float *pos, *x, *dy;
    float *dx, *dp;
};

template <int K, int LPR, int UPL, bool DX, bool DP>
int bwd_cell(int64_t fu, const Ws &w, const BwdIo &io, float r2, float nis, float tis, hipStream_t stream) {
    const void *kern = reinterpret_cast<const void *>(&radius_bwd_cell_kernel<K, LPR, UPL, DX, DP>);
    static const int grid = cell_grid(kern);
    prof_before(stream);
    hipLaunchKernelGGL((radius_bwd_cell_kernel<K, LPR, UPL, DX, DP>), dim3(grid), dim3(kBlock), 0, stream, w.prm,
                       w.order, w.sched, w.start, w.rec, io.pos, io.x, io.dy, fu, r2, nis, tis, io.dx, io.dp);
    prof_after(stream);
    return check_launch("radius backward");
}

template <int K, bool DX, bool DP>
int bwd_units(int64_t fu, const Ws &w, const BwdIo &io, float r2, float nis, float tis, hipStream_t stream) {
    if (fu <= 1) return bwd_cell<K, 1, 1, DX, DP>(fu, w, io, r2, nis, tis, stream);
    if (fu <= 2) return bwd_cell<K, 2, 1, DX, DP>(fu, w, io, r2, nis, tis, stream);
    if (fu <= 4) return bwd_cell<K, 4, 1, DX, DP>(fu, w, io, r2, nis, tis, stream);
    if (fu <= 8) return bwd_cell<K, 8, 1, DX, DP>(fu, w, io, r2, nis, tis, stream);
    return bwd_cell<K, 8, 2, DX, DP>(fu, w, io, r2, nis, tis, stream);
}

// The consume kernels index feature units with 32-bit arithmetic.
int check_units(int64_t n, int64_t fu) {
    if (static_cast<uint64_t>(n) * static_cast<uint64_t>(fu) >= (uint64_t{1} << 32))
        return fail(TIGA_EUNSUPPORTED, "radius: n * feature units (%lld * %lld) reaches 2^32",
                    static_cast<long long>(n), static_cast<long long>(fu));
    return TIGA_OK;
}

}  // namespace

size_t workspace_bytes(int64_t n, int64_t feat) {
    (void)feat;  // feature rows are read in place
    Carve c(nullptr);
    carve(c, n);
    return c.bytes();
}

int forward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, float *y,
            int32_t *count, void *ws, hipStream_t stream) {
    if (feat == 0) {
        // no features: the relation's counts only
        Carve c(ws);
        Ws w = carve(c, n);
        if (int rc = build(n, pos, radius, w, stream)) return rc;
        hipLaunchKernelGGL(neighbor_count_kernel, dim3(static_cast<unsigned>(ceil_div(n, kBlock))), dim3(kBlock), 0,
                           stream, w.prm, w.start, w.rec, n, radius * radius, count);
        return check_launch("radius counts");
    }
    // 16-byte units when every row starts on a 16-byte boundary
    const bool vec = feat % 4 == 0 && aligned16(x) && aligned16(y);
    const int64_t fu = vec ? feat / 4 : feat;
    if (int rc = check_units(n, fu)) return rc;
    Carve c(ws);
    Ws w = carve(c, n);
    if (int rc = build(n, pos, radius, w, stream)) return rc;
    if (int rc = visit_order(w, stream)) return rc;
    const float r2 = radius * radius;
    const float nis = -1.0f / (sigma * sigma) * kLog2e;  // weights are exp2(d2 * nis)
    if (vec) return fwd_units<4>(fu, w, x, r2, nis, y, count, stream);
    return fwd_units<1>(fu, w, x, r2, nis, y, count, stream);
}

int backward(int64_t n, int32_t feat, const float *pos, const float *x, float radius, float sigma, const float *dy,
             float *dx, float *dpos, void *ws, hipStream_t stream) {
    const bool vec = feat % 4 == 0 && aligned16(dy) && (!dpos || aligned16(x)) && (!dx || aligned16(dx));
    const int64_t fu = vec ? feat / 4 : feat;
    if (int rc = check_units(n, fu)) return rc;
    Carve c(ws);
    Ws w = carve(c, n);
    if (int rc = build(n, pos, radius, w, stream)) return rc;
    if (int rc = visit_order(w, stream)) return rc;
    const float r2 = radius * radius;
    const float nis = -1.0f / (sigma * sigma) * kLog2e;  // weights are exp2(d2 * nis)
    const float tis = 2.0f / (sigma * sigma);
    const BwdIo io{pos, x, dy, dx, dpos};
#define TIGA_B(KK)                                                                  \
    if (dx && dpos) return bwd_units<KK, true, true>(fu, w, io, r2, nis, tis, stream); \
    if (dx) return bwd_units<KK, true, false>(fu, w, io, r2, nis, tis, stream);        \
    return bwd_units<KK, false, true>(fu, w, io, r2, nis, tis, stream)
    if (vec) {
        TIGA_B(4);
    } else {
        TIGA_B(1);
    }
#undef TIGA_B
}

// The shared directory (edge-MLP messages): up to 8 cells per point and half the volume-based
// spacing floor, so that surface clouds get cells near the radius.
constexpr int64_t kSharedCellsPerPoint = 8;
constexpr double kSharedSpacingScale = 0.5;

size_t cells_ws_bytes(int64_t n) {
    Carve c(nullptr);
    carve(c, n, kSharedCellsPerPoint);
    return c.bytes();
}

int build_cells(int64_t n, const float *pos, float radius, void *ws, Cells &out, hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n, kSharedCellsPerPoint);
    if (int rc = build(n, pos, radius, w, stream, kSharedSpacingScale)) return rc;
    out.prm = w.prm;
    out.start = w.start;
    out.rec = w.rec;
    return TIGA_OK;
}

int neighbors(int64_t n, const float *pos, float radius, const int64_t *nbr_ptr, int32_t *nbr_idx, void *ws,
              hipStream_t stream) {
    Carve c(ws);
    Ws w = carve(c, n);
    if (int rc = build(n, pos, radius, w, stream)) return rc;
    if (int rc = fill_u32(w.flag, 0u, 1, stream)) return rc;
    const dim3 grid(static_cast<unsigned>(ceil_div(n, kBlock)));
    hipLaunchKernelGGL(neighbor_fill_kernel, grid, dim3(kBlock), 0, stream, w.prm, w.start, w.rec, n, radius * radius,
                       nbr_ptr, nbr_idx, w.flag);
    if (int rc = check_launch("radius neighbour fill")) return rc;
    uint32_t mismatch = 0;
    if (int rc = check_hip(hipMemcpyAsync(&mismatch, w.flag, sizeof mismatch, hipMemcpyDeviceToHost, stream),
                           "radius neighbours: copy"))
        return rc;
    if (int rc = check_hip(hipStreamSynchronize(stream), "radius neighbours: synchronize")) return rc;
    if (mismatch)
        return fail(TIGA_EINVAL, "nbr_ptr is not the exclusive prefix of the relation's neighbour counts "
                                 "(spans were filled without overrun, the lists are incomplete)");
    return TIGA_OK;
}

}  // namespace radius
}  // namespace tiga
