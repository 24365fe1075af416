// Degree-aware traversal of a destination-major CSR relation on gfx950.
//
// The relation's rows are split into three classes by degree (Section 4.4 of
// the paper: a bounded neighbour tile needs a degree guard; a high-degree row
// needs explicit partial states and a legal merge):
//   short rows  (deg <= DS): one group of G lanes per row, rows taken in their
//                            natural order, RPW rows per wavefront;
//   medium rows (DS < deg <= CH): one wavefront per row;
//   long rows   (deg > CH): split into chunks of CH edges, one wavefront per
//                           chunk, each producing a partial state that a
//                           merge kernel combines in a fixed order.
// Medium and long rows are both described by chunk descriptors, produced by a
// deterministic plan (count per tile, scan, write) without global atomics.
//
// Lane layout: a feature row is FU "units" (float4 when the vector path
// applies, else float).  L lanes (a power of two >= FU, at most 64) cover one
// edge's units, so a wavefront holds S = 64 / L edge slots.  Each lane
// accumulates its slot's edges serially (kUnroll edges in flight), then the
// slots of a row are reduced with cross-lane shuffles.
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

struct Geom {
    int L;    // lanes per edge
    int S;    // edge slots per wavefront
    int P;    // edge slots per short-row group
    int G;    // lanes per short-row group
    int RPW;  // short rows per wavefront
    int DS;   // short-row degree bound
    int CH;   // chunk length (edges) for medium and long rows
};

__host__ __device__ constexpr Geom make_geom(int L) {
    return Geom{L,
                kWave / L,
                L >= 8 ? 1 : 8 / L,
                L >= 8 ? L : 8,
                kWave / (L >= 8 ? L : 8),
                2 * (L >= 8 ? 1 : 8 / L) * kUnroll,
                (kWave / L) * kUnroll * 16};
}

// Chunk descriptor: row, chunk index within the row, partial slot (-1 when
// the row is a single chunk and writes its output directly), chunks in row.
// Split descriptor: row, first partial slot, chunk count, unused.
using Desc = int4;

// Counters written by the plan: [0] chunks, [1] partial slots, [2] split rows.
struct PlanCounts {
    unsigned long long chunks, slots, splits, pad;
};

struct PlanBounds {
    int64_t tiles, max_chunks, max_slots, max_splits;
};

inline PlanBounds plan_bounds(int64_t nrows, int64_t nedges, const Geom &g) {
    PlanBounds b;
    b.tiles = ceil_div(nrows > 0 ? nrows : 1, kPlanTile);
    int64_t long_rows = nedges / (g.DS + 1);
    if (long_rows > nrows) long_rows = nrows;
    b.max_chunks = long_rows + nedges / g.CH + 1;
    b.max_splits = nedges / (g.CH + 1) + 1;
    b.max_slots = 2 * (nedges / g.CH) + 2;
    return b;
}

// Workspace layout of a plan; `feat` partial floats (and int32 edge ids for
// max) per slot.
struct PlanWs {
    PlanCounts *counts;
    int64_t *tile_vals;  // 3 per tile: chunks, slots, splits (count, then offset)
    Desc *chunks;
    Desc *splits;
    float *part_v;
    int32_t *part_e;
};

inline PlanWs carve_plan(Carve &c, const PlanBounds &b, int64_t feat, bool with_arg) {
    PlanWs w;
    w.counts = c.take<PlanCounts>(1);
    w.tile_vals = c.take<int64_t>(3 * b.tiles);
    w.chunks = c.take<Desc>(b.max_chunks);
    w.splits = c.take<Desc>(b.max_splits);
    w.part_v = c.take<float>(b.max_slots * feat);
    w.part_e = with_arg ? c.take<int32_t>(b.max_slots * feat) : nullptr;
    return w;
}

// Enqueue the plan (three kernels) for rows [0, nrows) of `ptr`.
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
        if (!ok) return;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            float m = w * x.v[k];
            if (m > v[k] || e[k] == kNoEdge) {
                v[k] = m;
                e[k] = static_cast<int>(edge);
            }
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
};

// Fold the edges [e0, e1) of one row into `acc`; this lane is slot `s` of SL
// slots and covers feature unit `u` (`uok` false for padding lanes).
template <int K, int RED, int WM, int SL, class A>
__device__ __forceinline__ void run_edges(const Trav &t, int64_t e0, int64_t e1, int s, int64_t u,
                                          bool uok, A &acc) {
    constexpr int STEP = SL * kUnroll;
    int32_t c[kUnroll];
    int32_t ee[kUnroll];
    float wv[kUnroll];
    auto fetch = [&](int64_t b, int32_t(&cc)[kUnroll], int32_t(&ei)[kUnroll], float(&ww)[kUnroll]) {
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int64_t e = b + static_cast<int64_t>(r) * SL + s;
            const bool ok = e < e1;
            cc[r] = ok ? ldg_stream(t.idx + e) : -1;
            ei[r] = 0;
            if constexpr (WM == W_DIRECT) {
                ww[r] = ok ? ldg_stream(t.w + e) : 0.0f;
            } else if constexpr (WM == W_INDIRECT || WM == W_ROUTE) {
                ei[r] = ok ? ldg_stream(t.eid + e) : 0;
                ww[r] = ok ? (t.w ? t.w[ei[r]] : 1.0f) : 0.0f;
            } else {
                ww[r] = ok ? 1.0f : 0.0f;
            }
        }
    };
    int64_t base = e0;
    if (base < e1) fetch(base, c, ee, wv);
    for (; base < e1; base += STEP) {
        Vec<K> xv[kUnroll];
        int sel[kUnroll][K];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            if (c[r] >= 0 && uok) {
                const int64_t unit = static_cast<int64_t>(c[r]) * t.fu + u;
                xv[r] = load_unit<K>(t.table, unit);
                if constexpr (WM == W_ROUTE) load_unit_i<K>(t.arg, unit, sel[r]);
            } else {
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    xv[r].v[k] = 0.0f;
                    sel[r][k] = -1;
                }
            }
        }
        int32_t cn[kUnroll];
        int32_t en[kUnroll];
        float wn[kUnroll];
        const int64_t nb = base + STEP;
        if (nb < e1) {
            fetch(nb, cn, en, wn);
        } else {
#pragma unroll
            for (int r = 0; r < kUnroll; ++r) {
                cn[r] = -1;
                en[r] = 0;
                wn[r] = 0.0f;
            }
        }
        if constexpr (WM == W_ROUTE) {
            // only the (row, feature) entries whose argmax is this edge receive its message
#pragma unroll
            for (int r = 0; r < kUnroll; ++r)
#pragma unroll
                for (int k = 0; k < K; ++k)
                    if (sel[r][k] != ee[r]) xv[r].v[k] = 0.0f;
        }
#pragma unroll
        for (int r = 0; r < kUnroll; ++r)
            acc.add(wv[r], xv[r], base + static_cast<int64_t>(r) * SL + s, c[r] >= 0);
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            c[r] = cn[r];
            ee[r] = en[r];
            wv[r] = wn[r];
        }
    }
}

}  // namespace csr
}  // namespace tiga
