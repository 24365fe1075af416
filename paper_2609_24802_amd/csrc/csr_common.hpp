// Degree-aware traversal of a destination-major CSR relation on gfx950.
//
// Rows are split by degree (Section 4.4 of the paper: a bounded neighbour
// tile needs a degree guard; a high-degree row needs explicit partial states
// and a legal merge):
//   short rows (deg <= DS): taken in their natural order, one group of G lanes
//                           per row, RPW rows per wavefront (no plan entry);
//   other rows:             cut into chunks of at most CH edges.  A chunk is
//                           processed by a group of 64, 32 or 16 lanes chosen
//                           by its length (its "class"), so a wavefront holds
//                           one long chunk or several short ones.  A row of
//                           several chunks writes partial states that a merge
//                           kernel combines in chunk order.
// Chunk descriptors come from a one-pass plan: each block of rows scans its
// own rows' needs and reserves its descriptor range with one atomic add per
// class; each descriptor carries its edge range, so a work item needs no
// dependent row-pointer load.  Where a block's range lands depends on timing,
// but every chunk's reduction and every split row's merge (in chunk order)
// do not, so results are deterministic.
//
// Lane layout: a feature row is FU "units" (float4 when the vector path
// applies, else float).  L lanes (a power of two >= FU, at most 64) cover one
// edge's units, so a group of GL lanes holds GL / L edge slots.  Each lane
// accumulates its slot's edges serially (kUnroll edges in flight), then the
// slots of a group are reduced with cross-lane shuffles.
#pragma once

#include "common.hpp"

namespace tiga {
namespace csr {

enum { RED_SUM = 0, RED_MAX = 1 };
// Edge weight of a traversal: none (1), w[e], w[eid[e]], or the max-routing
// message of the transposed backward (w[eid[e]] where argmax selects the edge).
enum { W_NONE = 0, W_DIRECT = 1, W_INDIRECT = 2, W_ROUTE = 3 };

constexpr int kUnroll = 4;
constexpr int kBlock = 256;        // threads per block of the traversal kernels
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kPlanRowsPerThread = 8;
constexpr int kPlanTile = kBlock * kPlanRowsPerThread;
constexpr int kClasses = 3;        // chunk groups of 64, 32 and 16 lanes
constexpr int kPlanVals = kClasses + 2;  // per tile: chunks of each class, partial slots, split rows

__host__ __device__ constexpr int class_lanes(int c) { return c == 0 ? 64 : (c == 1 ? 32 : 16); }

struct Geom {
    int L;    // lanes per edge
    int S;    // edge slots per wavefront
    int P;    // edge slots per short-row group
    int G;    // lanes per short-row group
    int RPW;  // short rows per wavefront
    int DS;   // short-row degree bound
    int CH;   // chunk length (edges)
    int nclass;           // chunk classes whose group holds at least one edge
    int cap[kClasses];    // longest chunk of each class (about four steps of its group)
};

__host__ __device__ constexpr Geom make_geom(int L) {
    const int P = L >= 8 ? 1 : 8 / L;
    const int nclass = L <= 16 ? 3 : (L <= 32 ? 2 : 1);
    return Geom{L,
                kWave / L,
                P,
                L >= 8 ? L : 8,
                kWave / (L >= 8 ? L : 8),
                2 * P * kUnroll,
                (kWave / L) * kUnroll * 16,
                nclass,
                {(kWave / L) * kUnroll * 16, 4 * (32 / L > 0 ? 32 / L : 1) * kUnroll,
                 4 * (16 / L > 0 ? 16 / L : 1) * kUnroll}};
}

// Class of a chunk of n edges: the narrowest group that finishes it in about
// four steps.
__host__ __device__ constexpr int chunk_class(const Geom &g, int64_t n) {
    return (g.nclass > 2 && n <= g.cap[2]) ? 2 : ((g.nclass > 1 && n <= g.cap[1]) ? 1 : 0);
}

// Chunk descriptor: destination row, partial slot (-1 when the row is one
// chunk and writes its output directly) and the edge range packed as
// (first edge << 24) | length.
struct alignas(16) Desc {
    int32_t row;
    int32_t slot;
    uint64_t range;
};
constexpr int kRangeBits = 24;
__host__ __device__ inline uint64_t pack_range(int64_t e0, int64_t n) {
    return (static_cast<uint64_t>(e0) << kRangeBits) | static_cast<uint64_t>(n);
}

// Split row: row, first partial slot, chunk count.
struct alignas(16) Split {
    int32_t row;
    int32_t slot0;
    int32_t nch;
    int32_t pad;
};

// Written by the plan: chunks of each class, partial slots and split rows
// reserved so far (atomic counters, cleared by the plan's first kernel), and
// the first descriptor of classes 1 and 2 (class c's descriptors live in their
// own region of the chunk array, sized by PlanBounds::cap).
// Each counter sits on a cache line of its own (k < kClasses: chunks of class k; then partial
// slots, then split rows), so that the tiles' reservations on different counters proceed in
// parallel in different L2 channels.
struct alignas(256) PlanCounter {
    unsigned long long v;
};
enum { kCtrSlots = kClasses, kCtrSplits = kClasses + 1 };
struct PlanCounts {
    PlanCounter ctr[kPlanVals];
    unsigned long long off[2];
};

struct PlanBounds {
    int64_t tiles, cap[kClasses], max_chunks, max_slots, max_splits;
};

// Capacities: a chunk of class c holds more than lo_c edges (class 0: a full
// chunk, or a last chunk longer than the class-1 bound; class c > 0: a last
// chunk longer than the next class's bound, or than the short-row bound), and
// every class-1 or class-2 chunk ends a distinct row.
inline PlanBounds plan_bounds(int64_t nrows, int64_t nedges, const Geom &g) {
    PlanBounds b;
    b.tiles = ceil_div(nrows > 0 ? nrows : 1, kPlanTile);
    for (int c = 0; c < kClasses; ++c) {
        int64_t cap = 0;
        if (c < g.nclass) {
            const int64_t lo = c + 1 < g.nclass ? g.cap[c + 1] : g.DS;
            cap = nedges / (lo + 1);
            if (c > 0 && cap > nrows) cap = nrows;
            cap += 1;
        }
        b.cap[c] = cap;
    }
    b.max_chunks = b.cap[0] + b.cap[1] + b.cap[2];
    b.max_splits = nedges / (g.CH + 1) + 1;
    b.max_slots = 2 * (nedges / g.CH) + 2;
    return b;
}

// Workspace layout of a plan; `feat` partial floats (and int32 edge ids for
// max) per slot.
struct PlanWs {
    PlanCounts *counts;
    Desc *chunks;  // class 0 at [0, cap0), class 1 at [cap0, cap0 + cap1), class 2 after
    Split *splits;
    float *part_v;
    int32_t *part_e;
};

inline PlanWs carve_plan(Carve &c, const PlanBounds &b, int64_t feat, bool with_arg) {
    PlanWs w;
    w.counts = c.take<PlanCounts>(1);
    w.chunks = c.take<Desc>(b.max_chunks);
    w.splits = c.take<Split>(b.max_splits);
    w.part_v = c.take<float>(b.max_slots * feat);
    w.part_e = with_arg ? c.take<int32_t>(b.max_slots * feat) : nullptr;
    return w;
}

// Enqueue the plan (two kernels: clear the counters, then one pass over the rows) for rows
// [0, nrows) of `ptr`.
int launch_plan(const int64_t *ptr, int64_t nrows, const Geom &g, const PlanBounds &b,
                const PlanWs &w, hipStream_t stream);

// Lanes-per-edge for `fu` feature units.
inline int lanes_for(int64_t fu) {
    int L = 1;
    while (L < fu && L < kWave) L <<= 1;
    return L;
}

// Number of persistent blocks for a traversal kernel with `items_bound` work
// items (one wavefront each).
inline int persistent_blocks(int64_t items_bound, int blocks_per_cu = 8) {
    int64_t cap = static_cast<int64_t>(device_cus()) * blocks_per_cu;
    int64_t need = ceil_div(items_bound > 0 ? items_bound : 1, kWavesPerBlock);
    return static_cast<int>(need < cap ? need : cap);
}

// ------------------------------------------------------------------ device

template <int K>
struct Vec {
    float v[K];
};

template <int K>
__device__ __forceinline__ Vec<K> load_unit(const float *__restrict__ base, int64_t unit) {
    Vec<K> r;
    if constexpr (K == 4) {
        const f32x4 t = reinterpret_cast<const f32x4 *>(base)[unit];
        r.v[0] = t.x;
        r.v[1] = t.y;
        r.v[2] = t.z;
        r.v[3] = t.w;
    } else {
        r.v[0] = base[unit];
    }
    return r;
}

template <int K>
__device__ __forceinline__ void store_unit(float *__restrict__ base, int64_t unit, const float (&v)[K]) {
    if constexpr (K == 4) {
        stg_stream(reinterpret_cast<f32x4 *>(base) + unit, f32x4{v[0], v[1], v[2], v[3]});
    } else {
        stg_stream(base + unit, v[0]);
    }
}

template <int K>
__device__ __forceinline__ void store_unit_i(int32_t *__restrict__ base, int64_t unit, const int (&v)[K]) {
    if constexpr (K == 4) {
        stg_stream(reinterpret_cast<i32x4 *>(base) + unit, i32x4{v[0], v[1], v[2], v[3]});
    } else {
        stg_stream(base + unit, v[0]);
    }
}

template <int K>
__device__ __forceinline__ void load_unit_i(const int32_t *__restrict__ base, int64_t unit, int (&out)[K]) {
    if constexpr (K == 4) {
        const i32x4 t = reinterpret_cast<const i32x4 *>(base)[unit];
        out[0] = t.x;
        out[1] = t.y;
        out[2] = t.z;
        out[3] = t.w;
    } else {
        out[0] = base[unit];
    }
}

constexpr int kNoEdge = 0x7fffffff;

// Reducer state (Section 3.1: identity, combine, finalize).
template <int K, int RED>
struct Acc;

template <int K>
struct Acc<K, RED_SUM> {
    float v[K];
    __device__ __forceinline__ void init() {
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = 0.0f;
    }
    // fold one weighted message w * x (fused multiply-add; order is free)
    __device__ __forceinline__ void add(float w, const Vec<K> &x, int64_t, bool) {
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] = fmaf(w, x.v[k], v[k]);
    }
    __device__ __forceinline__ void add_partial(const Vec<K> &p, const int (&)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] += p.v[k];
    }
    __device__ __forceinline__ void shfl_combine(int m) {
#pragma unroll
        for (int k = 0; k < K; ++k) v[k] += shfl_xor_f(v[k], m);
    }
    __device__ __forceinline__ void finalize() {}
};

template <int K>
struct Acc<K, RED_MAX> {
    float v[K];
    int e[K];
    __device__ __forceinline__ void init() {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            v[k] = -__builtin_inff();
            e[k] = kNoEdge;
        }
    }
    // message = one fp32 product; strict '>' keeps the earliest edge of a lane
    __device__ __forceinline__ void add(float w, const Vec<K> &x, int64_t edge, bool ok) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const float m = w * x.v[k];
            const bool take = ok && (m > v[k] || e[k] == kNoEdge);
            v[k] = take ? m : v[k];
            e[k] = take ? static_cast<int>(edge) : e[k];
        }
    }
    __device__ __forceinline__ void take(float ov, int oe, int k) {
        // (ov, oe) wins if larger, or equal with a lower edge position
        if (oe != kNoEdge && (e[k] == kNoEdge || ov > v[k] || (ov == v[k] && oe < e[k]))) {
            v[k] = ov;
            e[k] = oe;
        }
    }
    __device__ __forceinline__ void add_partial(const Vec<K> &p, const int (&pe)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) take(p.v[k], pe[k], k);
    }
    __device__ __forceinline__ void shfl_combine(int m) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            float ov = shfl_xor_f(v[k], m);
            int oe = shfl_xor_i(e[k], m);
            take(ov, oe, k);
        }
    }
    __device__ __forceinline__ void finalize() {
#pragma unroll
        for (int k = 0; k < K; ++k)
            if (e[k] == kNoEdge) {
                v[k] = 0.0f;
                e[k] = -1;
            }
    }
};

// Reduce across the lanes at xor distances FROM, 2*FROM, ..., < TO.
template <int FROM, int TO, class A>
__device__ __forceinline__ void reduce_lanes(A &acc) {
#pragma unroll
    for (int m = FROM; m < TO; m <<= 1) acc.shfl_combine(m);
}

// Inputs of one traversal: the relation (ptr/idx), the per-edge weight and the
// gathered table.
struct Trav {
    const int64_t *__restrict__ ptr;   // [nrows + 1]
    const int32_t *__restrict__ idx;   // [nedges] gathered row of `table`
    const float *__restrict__ w;       // weights (direct or through eid) or null
    const int32_t *__restrict__ eid;   // indirection for W_INDIRECT / W_ROUTE
    const float *__restrict__ table;   // [*, feat]
    int64_t nrows;
    int64_t fu;                        // feature units per row
    const int32_t *__restrict__ arg;   // [*, feat] selected edges (W_ROUTE only)
    uint32_t table_bytes;              // byte size of `table` (and `arg`) when below 4 GiB, else 0
    int64_t nedges;                    // edges of the relation (idx, w and eid have this many)
    // W_INDIRECT / W_ROUTE: per forward edge, (weight bits, gathered row) in one 8-byte record read
    // through eid (then idx and w are unused): one random request yields both
    const int2 *__restrict__ wrow = nullptr;
};

// Row gathers from the feature table.  Tables below 4 GiB go through a buffer
// resource: 32-bit byte offsets (fewer address registers) and a load outside
// the table returns zero rather than faulting.  Larger tables use 64-bit
// global loads.  Either way the load carries the non-temporal hint: a
// random row is rarely reused before it would be evicted.
constexpr int kBufWord3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9)
constexpr int kPolicyNT = 2;
// Tables above this size are streamed with the non-temporal hint; smaller ones
// stay eligible for the caches (a table that fits the 256 MB last-level cache
// is re-read from it).
constexpr int64_t kStreamTableBytes = int64_t{1} << 30;

template <int K, bool BUF, bool NT = true>
struct Table {
    __amdgpu_buffer_rsrc_t rs;
    const float *base;
    uint32_t row_bytes;
    __device__ __forceinline__ Table(const float *p, int64_t fu, uint32_t bytes) : base(p) {
        row_bytes = static_cast<uint32_t>(fu * K * 4);
        if constexpr (BUF) rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), 0, bytes, kBufWord3);
    }
    __device__ __forceinline__ Vec<K> load(int32_t row, int64_t u, int64_t fu) const {
        Vec<K> r;
        if constexpr (BUF) {
            const int off = static_cast<int>(static_cast<uint32_t>(row) * row_bytes + static_cast<uint32_t>(u) * (K * 4));
            if constexpr (K == 4) {
                const f32x4 t =
                    __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, NT ? kPolicyNT : 0));
                r.v[0] = t.x;
                r.v[1] = t.y;
                r.v[2] = t.z;
                r.v[3] = t.w;
            } else {
                r.v[0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, NT ? kPolicyNT : 0));
            }
        } else {
            // callers pass a valid row; padding units read the row's first unit
            const int64_t unit = static_cast<int64_t>(row) * fu + (u < fu ? u : 0);
            if constexpr (K == 4) {
                const f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(base) + unit);
                r.v[0] = t.x;
                r.v[1] = t.y;
                r.v[2] = t.z;
                r.v[3] = t.w;
            } else {
                r.v[0] = __builtin_nontemporal_load(base + unit);
            }
        }
        return r;
    }
    // the same row of an int32 table with identical shape (argmax)
    __device__ __forceinline__ void load_i(const int32_t *ib, const __amdgpu_buffer_rsrc_t &irs, int32_t row,
                                           int64_t u, int64_t fu, int (&out)[K]) const {
        if constexpr (BUF) {
            const int off = static_cast<int>(static_cast<uint32_t>(row) * row_bytes + static_cast<uint32_t>(u) * (K * 4));
            if constexpr (K == 4) {
                const i32x4 t = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(irs, off, 0, 0));
                out[0] = t.x;
                out[1] = t.y;
                out[2] = t.z;
                out[3] = t.w;
            } else {
                out[0] = __builtin_bit_cast(int, __builtin_amdgcn_raw_buffer_load_b32(irs, off, 0, 0));
            }
        } else {
            load_unit_i<K>(ib, static_cast<int64_t>(row) * fu + (u < fu ? u : 0), out);
        }
    }
};

// Fold the edges [e0, e1) of one row into `acc`; this lane is slot `s` of SL
// slots and covers feature unit `u` (`uok` false for padding lanes).  The
// lane issues kUnroll independent row gathers per step; latency is hidden by
// the other resident wavefronts.  Offsets inside the row are 32-bit (a row
// piece is at most one chunk of edges).  Lanes past the row's end issue no
// loads at all (their exec bit is off).
// Per-edge side computation of a traversal, called with each gathered unit
// (zero for lanes past the row end) before it is weighted.  The default does
// nothing.
struct NoEdgeHook {
    template <int K>
    __device__ __forceinline__ void edge(const Vec<K> &, int32_t, bool) {}
};

template <int K, int RED, int WM, int SL, bool BUF, bool NT, class A, class H = NoEdgeHook>
__device__ __forceinline__ void run_edges(const Trav &t, const Table<K, BUF, NT> &tab,
                                          const __amdgpu_buffer_rsrc_t &ars, int64_t e0, int64_t e1, int s,
                                          int64_t u, bool uok, A &acc, H &&hook = H{}) {
    constexpr int STEP = SL * kUnroll;
    const int n = static_cast<int>(e1 - e0);
    constexpr bool VIA_EID = WM == W_INDIRECT || WM == W_ROUTE;
    const int32_t *__restrict__ colr = VIA_EID ? nullptr : t.idx + e0;
    const float *__restrict__ wr = WM == W_DIRECT ? t.w + e0 : nullptr;
    const int32_t *__restrict__ er = VIA_EID ? t.eid + e0 : nullptr;
    for (int k0 = 0; k0 < n; k0 += STEP) {
        int32_t c[kUnroll];
        int32_t ee[kUnroll];
        float wv[kUnroll];
        bool ok[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int k = k0 + r * SL + s;
            ok[r] = k < n;
            // ids and weights take ordinary (cached) loads: neighbouring work
            // items share their cache lines, which the non-temporal hint would
            // let go back to HBM between the items
            ee[r] = 0;
            if constexpr (WM == W_INDIRECT || WM == W_ROUTE) {
                ee[r] = ok[r] ? er[k] : 0;
                const int2 pr = ok[r] ? t.wrow[ee[r]] : make_int2(0, 0);
                c[r] = pr.y;
                wv[r] = __int_as_float(pr.x);
            } else {
                c[r] = ok[r] ? colr[k] : 0;
                if constexpr (WM == W_DIRECT) {
                    wv[r] = ok[r] ? wr[k] : 0.0f;
                } else {
                    wv[r] = ok[r] ? 1.0f : 0.0f;
                }
            }
        }
        Vec<K> xv[kUnroll];
        int sel[kUnroll][K];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            if (ok[r] && uok) {
                xv[r] = tab.load(c[r], u, t.fu);
                if constexpr (WM == W_ROUTE) tab.load_i(t.arg, ars, c[r], u, t.fu, sel[r]);
            } else {
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    xv[r].v[k] = 0.0f;
                    sel[r][k] = -1;
                }
            }
        }
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const bool live = ok[r] && uok;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                bool keep = live;
                if constexpr (WM == W_ROUTE) keep = keep && sel[r][k] == ee[r];
                xv[r].v[k] = keep ? xv[r].v[k] : 0.0f;
            }
            hook.template edge<K>(xv[r], ee[r], ok[r]);
            acc.add(wv[r], xv[r], e0 + k0 + r * SL + s, live);
        }
    }
}

// Work items of one traversal, in this order: class-0 chunks (one per
// wavefront), pairs of class-1 chunks, quadruples of class-2 chunks, then
// groups of RPW short rows in natural order.
struct Items {
    int64_t n0, n1, n2;      // chunks of each class
    int64_t b1, b2;          // first descriptor of classes 1 and 2 (class 0 starts at 0)
    int64_t s1, s2, s3;      // first item of classes 1, 2 and of the short-row groups
    int64_t total;
};

__device__ __forceinline__ Items make_items(const PlanCounts *__restrict__ pc, int64_t n_groups) {
    Items it;
    it.n0 = static_cast<int64_t>(pc->ctr[0].v);
    it.n1 = static_cast<int64_t>(pc->ctr[1].v);
    it.n2 = static_cast<int64_t>(pc->ctr[2].v);
    it.b1 = static_cast<int64_t>(pc->off[0]);
    it.b2 = static_cast<int64_t>(pc->off[1]);
    it.s1 = it.n0;
    it.s2 = it.s1 + (it.n1 + 1) / 2;
    it.s3 = it.s2 + (it.n2 + 3) / 4;
    it.total = it.s3 + n_groups;
    return it;
}

// What one group needs to process its part of a work item: the edge range,
// the output row, the partial slot (-1: write the output row) and whether it
// writes at all (padding groups and skipped rows do not).
struct Meta {
    int64_t e0;
    int32_t n;
    int32_t row;
    int32_t slot;
    int32_t write;
};

// Metadata of item `it` for this lane (class-c chunk items and short-row
// groups; see Items).  Geometry: L lanes per edge.
template <int L>
__device__ __forceinline__ Meta load_meta(const Items &items, const Desc *__restrict__ chunks,
                                          const int64_t *__restrict__ ptr, int64_t nrows, int64_t it, int lane) {
    constexpr Geom g = make_geom(L);
    Meta m{0, 0, 0, -1, 0};
    if (it >= items.total) return m;
    int64_t j = -1, nj = 0;
    if (it < items.s1) {
        j = it;
        nj = items.n0;
    } else if (it < items.s2) {
        const int64_t k = (it - items.s1) * 2 + lane / 32;
        j = items.b1 + k;
        nj = items.b1 + items.n1;
    } else if (it < items.s3) {
        const int64_t k = (it - items.s2) * 4 + lane / 16;
        j = items.b2 + k;
        nj = items.b2 + items.n2;
    } else {
        const int64_t row = (it - items.s3) * g.RPW + lane / g.G;
        if (row < nrows) {
            const int64_t e0 = ptr[row];
            const int64_t d = ptr[row + 1] - e0;
            if (d <= g.DS) {
                m.e0 = e0;
                m.n = static_cast<int32_t>(d);
                m.row = static_cast<int32_t>(row);
                m.write = 1;
            }
        }
        return m;
    }
    if (j < nj) {
        const Desc d = chunks[j];
        m.e0 = static_cast<int64_t>(d.range >> kRangeBits);
        m.n = static_cast<int32_t>(d.range & ((1u << kRangeBits) - 1));
        m.row = d.row;
        m.slot = d.slot;
        m.write = 1;
    }
    return m;
}

// Persistent loop: wavefront w takes items w, w + nwaves, ...; every
// wavefront leaves once it passes the item count, so the grid drains.  The
// next item's metadata is loaded before the current item is processed, so its
// latency hides behind the current item's gathers.
// Body provides  template <int GL> run(const Meta&, int lane_in_group).
template <int L, class Body>
__device__ __forceinline__ void for_each_item(const Items &items, const Desc *__restrict__ chunks,
                                              const int64_t *__restrict__ ptr, int64_t nrows, Body &body) {
    constexpr Geom g = make_geom(L);
    const int lane = lane_id();
    const int64_t wave = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
    Meta cur = load_meta<L>(items, chunks, ptr, nrows, wave, lane);
    for (int64_t it = wave; it < items.total; it += nwaves) {
        const Meta nxt = load_meta<L>(items, chunks, ptr, nrows, it + nwaves, lane);
        if (it < items.s1) {
            body.template run<64>(cur, lane);
        } else if (it < items.s2) {
            if constexpr (32 >= L) body.template run<32>(cur, lane % 32);
        } else if (it < items.s3) {
            if constexpr (16 >= L) body.template run<16>(cur, lane % 16);
        } else {
            body.template run<g.G>(cur, lane % g.G);
        }
        cur = nxt;
    }
}

}  // namespace csr
}  // namespace tiga
