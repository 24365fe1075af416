// Generated exact kNN relation with a fused neighbour sum (Section 4.9, generated relations: one
// program scans candidate tiles for its queries, keeps a power-of-two padded top-k state keyed by
// (squared distance, source index), and consumes the selected sources without storing adjacency;
// the exact-kNN workload of Section 7 is a neighbour sum with k = 16).
//   S_i = the k sources j != i with the smallest keys (d2_ij, j), d2 finite,
//   d2  = fl(fl(fl(dx*dx) + fl(dy*dy)) + fl(dz*dz)), dx = fl(p_j.x - p_i.x), ...
//   y_i = sum_{j in S_i} x_j
//
// MI355X design:
//  - Build: points are ordered along a 30-bit Morton curve (box of the finite coordinates, radix
//    sort) into records (x, y, z, original index), cut into tiles of 64; each tile gets the box of
//    its finite members, and each group of 32 tiles a box too.  A block of 4 wavefronts owns one
//    tile of queries, compact in space.
//  - A key is one 64-bit integer, (bits of d2) << 32 | index: d2 >= 0, so the float bits order
//    like the values, and one unsigned compare gives the lexicographic order with the index as the
//    tie-break.  Keys of non-finite distances are >= the bits of +inf and never enter the state.
//  - Candidates arrive through scalar loads (the tile being scanned is uniform over the wavefront).
//    Each lane keeps its KP smallest keys sorted in registers (KP = k rounded up to a power of two,
//    the padded state; the test against the KP-th key is conservative for k < KP).
//  - Candidate tiles are visited nearest-index first (the query tile, then the rest of its group of
//    32 tiles outward along the curve, then the other groups nearest-first), which tightens every
//    lane's state early.  A group or a tile is skipped only when, for every lane, a lower bound of
//    the squared distance from the lane's query to the box, reduced by a relative 1e-6 that covers
//    the fp32 roundings of the bound and of d2, exceeds that lane's retained KP-th distance: then
//    none of its keys can enter any lane's state, so the skip is exact.  (A per-lane bound stays
//    tight where the curve jumps and a tile of queries spans a wide box.)  (The paper skips only the sort of such a tile; on this chip the distance
//    evaluation is the cost, so the bound is taken before it.)
#include "knn.hpp"

#include "csr_bwd.hpp"

namespace tiga {
namespace knn {

namespace {

constexpr int kBlock = 256;
constexpr int kTile = 64;                                 // records per tile = queries per wavefront
constexpr int kBits = 10;                                 // Morton bits per axis
constexpr uint64_t kNone = 0x7f80000000000000ull;         // key (+inf, 0): above every finite key
constexpr int kPartials = 1024;
constexpr int kGroup = 32;                                // tiles per group (the coarse skip level)
constexpr int kSplit = 4;                                 // wavefronts sharing one tile of queries

typedef float f4 __attribute__((ext_vector_type(4)));

struct Ws {
    float *part;        // [kPartials][6] box partials
    float *box;         // [8]: lo xyz, hi xyz
    int32_t *key, *key_sorted, *perm;
    void *sort;
    f4 *rec;            // [ntile * kTile] Morton-ordered (x, y, z, original index)
    f4 *tlo, *thi;      // [ntile] box of each tile's finite records
    f4 *slo, *shi;      // [ntile * kTile / 8] box of each run of 8 records (one candidate step)
    f4 *glo, *ghi;      // [ngroup] box of each group of kGroup tiles
};

Ws carve(Carve &c, int64_t n) {
    const int64_t ntile = ceil_div(n, kTile);
    Ws w;
    w.part = c.take<float>(kPartials * 6);
    w.box = c.take<float>(8);
    w.key = c.take<int32_t>(n);
    w.key_sorted = c.take<int32_t>(n);
    w.perm = c.take<int32_t>(n);
    w.sort = c.take<char>(csr::sort_keys_ws_bytes(n));
    w.rec = c.take<f4>(ntile * kTile);
    w.tlo = c.take<f4>(ntile);
    w.thi = c.take<f4>(ntile);
    w.slo = c.take<f4>(ntile * (kTile / 8));
    w.shi = c.take<f4>(ntile * (kTile / 8));
    w.glo = c.take<f4>(ceil_div(ntile, kGroup));
    w.ghi = c.take<f4>(ceil_div(ntile, kGroup));
    return w;
}

__device__ __forceinline__ bool finite3(float a, float b, float c) {
    return __builtin_isfinite(a) && __builtin_isfinite(b) && __builtin_isfinite(c);
}

__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) v = fminf(v, __shfl_xor(v, m, kWave));
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) v = fmaxf(v, __shfl_xor(v, m, kWave));
    return v;
}

// ---- build

// Box of the finite points: per-block partials (min xyz, max xyz).
__global__ __launch_bounds__(kBlock) void box_partial_kernel(const float *__restrict__ pos, int64_t n,
                                                             float *__restrict__ part) {
    __shared__ float red[kBlock / kWave][6];
    float v[6] = {__builtin_inff(), __builtin_inff(), __builtin_inff(),
                  -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride) {
        const float a = pos[i * 3], b = pos[i * 3 + 1], c = pos[i * 3 + 2];
        if (!finite3(a, b, c)) continue;
        v[0] = fminf(v[0], a), v[1] = fminf(v[1], b), v[2] = fminf(v[2], c);
        v[3] = fmaxf(v[3], a), v[4] = fmaxf(v[4], b), v[5] = fmaxf(v[5], c);
    }
#pragma unroll
    for (int a = 0; a < 3; ++a) v[a] = wave_min(v[a]);
#pragma unroll
    for (int a = 3; a < 6; ++a) v[a] = wave_max(v[a]);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0)
        for (int a = 0; a < 6; ++a) red[w][a] = v[a];
    __syncthreads();
    if (threadIdx.x < 6) {
        float r = red[0][threadIdx.x];
        for (int q = 1; q < kBlock / kWave; ++q)
            r = threadIdx.x < 3 ? fminf(r, red[q][threadIdx.x]) : fmaxf(r, red[q][threadIdx.x]);
        part[blockIdx.x * 6 + threadIdx.x] = r;
    }
}

__global__ __launch_bounds__(kWave) void box_final_kernel(const float *__restrict__ part, int np,
                                                          float *__restrict__ box) {
    float v[6] = {__builtin_inff(), __builtin_inff(), __builtin_inff(),
                  -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
    for (int p = lane_id(); p < np; p += kWave)
        for (int a = 0; a < 6; ++a) v[a] = a < 3 ? fminf(v[a], part[p * 6 + a]) : fmaxf(v[a], part[p * 6 + a]);
#pragma unroll
    for (int a = 0; a < 3; ++a) v[a] = wave_min(v[a]);
#pragma unroll
    for (int a = 3; a < 6; ++a) v[a] = wave_max(v[a]);
    if (lane_id() == 0)
        for (int a = 0; a < 6; ++a) box[a] = v[a];
}

__device__ __forceinline__ uint32_t spread3(uint32_t v) {
    v &= 0x3ffu;
    v = (v | (v << 16)) & 0x030000ffu;
    v = (v | (v << 8)) & 0x0300f00fu;
    v = (v | (v << 4)) & 0x030c30c3u;
    v = (v | (v << 2)) & 0x09249249u;
    return v;
}

// Morton key of every point (non-finite points: the last key).
__global__ __launch_bounds__(kBlock) void morton_kernel(const float *__restrict__ pos, int64_t n,
                                                        const float *__restrict__ box, int32_t *__restrict__ key) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i >= n) return;
    const float p[3] = {pos[i * 3], pos[i * 3 + 1], pos[i * 3 + 2]};
    if (!finite3(p[0], p[1], p[2])) {
        key[i] = (1 << (3 * kBits)) - 1;
        return;
    }
    uint32_t q[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
        const float ext = box[3 + a] - box[a];
        float t = ext > 0.0f ? (p[a] - box[a]) / ext * static_cast<float>(1 << kBits) : 0.0f;
        t = fminf(fmaxf(t, 0.0f), static_cast<float>((1 << kBits) - 1));
        q[a] = static_cast<uint32_t>(t);
    }
    key[i] = static_cast<int32_t>(spread3(q[0]) | (spread3(q[1]) << 1) | (spread3(q[2]) << 2));
}

// Records in curve order; the tail of the last tile is padding that no query selects.
__global__ __launch_bounds__(kBlock) void records_kernel(const float *__restrict__ pos, const int32_t *__restrict__ perm,
                                                         int64_t n, int64_t npad, f4 *__restrict__ rec) {
    const int64_t s = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (s >= npad) return;
    if (s < n) {
        const int64_t j = perm[s];
        rec[s] = f4{pos[j * 3], pos[j * 3 + 1], pos[j * 3 + 2], __int_as_float(static_cast<int32_t>(j))};
    } else {
        rec[s] = f4{__builtin_inff(), __builtin_inff(), __builtin_inff(), __int_as_float(-1)};
    }
}

// Box of each run of 8 records and of each tile, over the finite records (empty: lo = +inf,
// hi = -inf).  The 8-record boxes are reduced first; the tile box continues from them.
__global__ __launch_bounds__(kBlock) void tile_box_kernel(const f4 *__restrict__ rec, int64_t ntile,
                                                          f4 *__restrict__ tlo, f4 *__restrict__ thi,
                                                          f4 *__restrict__ slo, f4 *__restrict__ shi) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave;
    if (t >= ntile) return;
    const int lane = lane_id();
    const f4 r = rec[t * kTile + lane];
    const bool ok = finite3(r.x, r.y, r.z);
    const float inf = __builtin_inff();
    float lo[3] = {ok ? r.x : inf, ok ? r.y : inf, ok ? r.z : inf};
    float hi[3] = {ok ? r.x : -inf, ok ? r.y : -inf, ok ? r.z : -inf};
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) {
#pragma unroll
        for (int a = 0; a < 3; ++a) {
            lo[a] = fminf(lo[a], __shfl_xor(lo[a], m, kWave));
            hi[a] = fmaxf(hi[a], __shfl_xor(hi[a], m, kWave));
        }
        if (m == 4 && lane % 8 == 0) {
            slo[t * (kTile / 8) + lane / 8] = f4{lo[0], lo[1], lo[2], 0.0f};
            shi[t * (kTile / 8) + lane / 8] = f4{hi[0], hi[1], hi[2], 0.0f};
        }
    }
    if (lane == 0) {
        tlo[t] = f4{lo[0], lo[1], lo[2], 0.0f};
        thi[t] = f4{hi[0], hi[1], hi[2], 0.0f};
    }
}

// Box of each group of kGroup consecutive tiles.
__global__ __launch_bounds__(kBlock) void group_box_kernel(const f4 *__restrict__ tlo, const f4 *__restrict__ thi,
                                                           int64_t ntile, int64_t ngroup, f4 *__restrict__ glo,
                                                           f4 *__restrict__ ghi) {
    const int64_t g = static_cast<int64_t>(blockIdx.x) * (kBlock / kWave) + threadIdx.x / kWave;
    if (g >= ngroup) return;
    const int64_t t = g * kGroup + lane_id();
    const bool ok = lane_id() < kGroup && t < ntile;
    const float inf = __builtin_inff();
    const f4 lo = ok ? tlo[t] : f4{inf, inf, inf, 0.0f};
    const f4 hi = ok ? thi[t] : f4{-inf, -inf, -inf, 0.0f};
    const float lx = wave_min(lo.x), ly = wave_min(lo.y), lz = wave_min(lo.z);
    const float hx = wave_max(hi.x), hy = wave_max(hi.y), hz = wave_max(hi.z);
    if (lane_id() == 0) {
        glo[g] = f4{lx, ly, lz, 0.0f};
        ghi[g] = f4{hx, hy, hz, 0.0f};
    }
}

// ---- select and consume

__device__ __forceinline__ float sqdist(f4 pi, f4 pj) {
#pragma clang fp contract(off)
    const float dx = pj.x - pi.x, dy = pj.y - pi.y, dz = pj.z - pi.z;
    const float sx = dx * dx, sy = dy * dy, sz = dz * dz;
    const float s = sx + sy;
    return s + sz;
}

// Insert key nk (below kd[KP-1]) into the ascending state; equal keys cannot occur (indices differ).
template <int KP>
__device__ __forceinline__ void insert(uint64_t (&kd)[KP], uint64_t nk) {
#pragma unroll
    for (int t = KP - 1; t > 0; --t) {
        const bool up = nk < kd[t - 1];
        kd[t] = up ? kd[t - 1] : (nk < kd[t] ? nk : kd[t]);
    }
    kd[0] = nk < kd[0] ? nk : kd[0];
}

// Squared distance from a point to a box from per-axis gaps, in fp32: within 4 roundings
// (relative 2^-24 each) of the exact value, so with the skip margin below it bounds every computed
// d2 from that point to a record in the box (whose own fp32 evaluation is within 5 roundings of
// exact).  An empty box (lo = +inf, hi = -inf) gives +inf.
__device__ __forceinline__ float box_gap2(f4 p, f4 lo, f4 hi) {
#pragma clang fp contract(off)
    const float gx = fmaxf(fmaxf(lo.x - p.x, p.x - hi.x), 0.0f);
    const float gy = fmaxf(fmaxf(lo.y - p.y, p.y - hi.y), 0.0f);
    const float gz = fmaxf(fmaxf(lo.z - p.z, p.z - hi.z), 0.0f);
    return (gx * gx + gy * gy) + gz * gz;
}

constexpr float kSkipMargin = 1.0f - 1e-6f;   // > 9 roundings of 2^-24

// The KP smallest keys of two ascending states A (in place) and B: min(A[t], B[KP-1-t]) keeps
// exactly them as a bitonic sequence, which log2(KP) half-cleaner stages sort.
template <int KP>
__device__ __forceinline__ void merge_state(uint64_t (&a)[KP], const uint64_t (&b)[KP]) {
#pragma unroll
    for (int t = 0; t < KP; ++t) a[t] = b[KP - 1 - t] < a[t] ? b[KP - 1 - t] : a[t];
#pragma unroll
    for (int h = KP / 2; h >= 1; h /= 2)
#pragma unroll
        for (int t = 0; t < KP; ++t)
            if ((t & h) == 0) {
                const uint64_t lo = a[t + h] < a[t] ? a[t + h] : a[t];
                const uint64_t hi = a[t + h] < a[t] ? a[t] : a[t + h];
                a[t] = lo;
                a[t + h] = hi;
            }
}

// One block of kSplit wavefronts per query tile.  The candidate tiles, in visiting order, are
// dealt round-robin to the wavefronts; each keeps its own padded state, publishes every lane's
// KP-th distance in LDS (it only decreases, so a stale read is merely less tight), and rejects a
// candidate only if it is strictly farther than the tightest published KP-th distance of its
// lane, because then KP keys of the union already precede it.  Wavefront 0 merges the states.
template <int KP>
__global__ __launch_bounds__(kSplit * kWave) void select_kernel(const f4 *__restrict__ rec, const f4 *__restrict__ tlo,
                                                                const f4 *__restrict__ thi, const f4 *__restrict__ slo,
                                                                const f4 *__restrict__ shi, const f4 *__restrict__ glo,
                                                                const f4 *__restrict__ ghi, int ntile, int k, int feat,
                                                                const float *__restrict__ x, float *__restrict__ y,
                                                                int32_t *__restrict__ nbr) {
    __shared__ float shthr[kSplit][kWave];
    __shared__ uint64_t shkey[kSplit - 1][KP][kWave];
    const int qt = static_cast<int>(xcd_block());
    const int w = uniform(static_cast<int>(threadIdx.x) / kWave);
    const int lane = lane_id();
    const f4 me = rec[static_cast<int64_t>(qt) * kTile + lane];
    const int qid = __float_as_int(me.w);
    const bool live = qid >= 0 && finite3(me.x, me.y, me.z);
    uint64_t kd[KP];
#pragma unroll
    for (int t = 0; t < KP; ++t) kd[t] = kNone;
    // this lane's retained KP-th distance (+inf until its state is full; -inf for lanes without a
    // live query, which never need a candidate)
    float thr = live ? __builtin_inff() : -__builtin_inff();
    shthr[w][lane] = thr;
    __syncthreads();
    float tight = thr;   // min over the wavefronts' published values
    auto refresh = [&]() __attribute__((always_inline)) {
        float v = thr;
#pragma unroll
        for (int o = 0; o < kSplit; ++o)
            v = fminf(v, __hip_atomic_load(&shthr[o][lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
        tight = v;
    };
    // a box can be skipped when no lane could take anything from it
    auto needed = [&](f4 lo, f4 hi) __attribute__((always_inline)) {
        return __any(box_gap2(me, lo, hi) * kSkipMargin <= tight);
    };

    // scan one candidate tile (after its box test, except for the query tile itself)
    auto scan = [&](int t) __attribute__((always_inline)) {
        refresh();
        if (t != qt && !needed(tlo[t], thi[t])) return;
        const f4 *tr = rec + static_cast<int64_t>(t) * kTile;
        // keys above every key of distance `tight` are out (ties in distance are kept)
        const uint64_t cap = (static_cast<uint64_t>(__float_as_uint(tight)) << 32) | 0xffffffffull;
        bool changed = false;
        for (int c0 = 0; c0 < kTile; c0 += 8) {
            // a run of 8 records whose box no lane could take anything from is skipped (the
            // query tile too: its query is excluded by index, and its runs skip like any other)
            const int64_t sb = static_cast<int64_t>(t) * (kTile / 8) + c0 / 8;
            if (!needed(slo[sb], shi[sb])) continue;
            float d2[8];
            bool any = false;
            // a distance above the lane's tight bound cannot enter (ties go on to the key test)
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                d2[u] = sqdist(me, tr[c0 + u]);   // uniform address: a scalar load
                any |= d2[u] <= tight;
            }
            if (!__any(any)) continue;
            const uint64_t lim = kd[KP - 1] < cap ? kd[KP - 1] : cap;
            uint64_t nk[8];
            bool take = false;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const uint32_t cid = static_cast<uint32_t>(__float_as_int(tr[c0 + u].w));
                nk[u] = (static_cast<uint64_t>(__float_as_uint(d2[u])) << 32) | cid;
                if (t == qt) nk[u] = static_cast<int>(cid) == qid ? ~0ull : nk[u];   // the query itself
                nk[u] = nk[u] < lim ? nk[u] : ~0ull;
                take |= nk[u] != ~0ull;
            }
            if (__any(take)) {
                changed = true;
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (nk[u] < kd[KP - 1]) insert<KP>(kd, nk[u]);
            }
        }
        if (changed && live && kd[KP - 1] < kNone) {
            thr = __uint_as_float(static_cast<uint32_t>(kd[KP - 1] >> 32));
            __hip_atomic_store(&shthr[w][lane], thr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
    };

    // visiting order: the query tile, then the rest of its group outward along the curve, then the
    // other groups nearest-first, each behind its group box test; position p goes to wavefront
    // p % kSplit (positions count every tile, skipped or not, so all wavefronts agree on them)
    const int ngroup = (ntile + kGroup - 1) / kGroup;
    const int qg = qt / kGroup;
    const int g0 = qg * kGroup, g1 = g0 + kGroup < ntile ? g0 + kGroup : ntile;
    int p = 0;
    if (w == 0) scan(qt);
    ++p;
    for (int step = 1; step < 2 * kGroup; ++step) {
        const int t = (step & 1) ? qt - (step + 1) / 2 : qt + step / 2;
        if (t < g0 || t >= g1) continue;
        if (p % kSplit == w) scan(t);
        ++p;
    }
    for (int step = 1; step < 2 * ngroup; ++step) {
        const int g = (step & 1) ? qg - (step + 1) / 2 : qg + step / 2;
        if (g < 0 || g >= ngroup) continue;
        const int t0 = g * kGroup, t1 = t0 + kGroup < ntile ? t0 + kGroup : ntile;
        const int pg = p;
        p += t1 - t0;
        refresh();
        if (!needed(glo[g], ghi[g])) continue;
        // this wavefront's tiles of the group: positions pg + (t - t0) congruent to w
        for (int t = t0 + ((w - pg) % kSplit + kSplit) % kSplit; t < t1; t += kSplit) scan(t);
    }

    // merge the states into wavefront 0
    if (w > 0)
#pragma unroll
        for (int t = 0; t < KP; ++t) shkey[w - 1][t][lane] = kd[t];
    __syncthreads();
    if (w != 0 || qid < 0) return;
#pragma unroll
    for (int o = 0; o < kSplit - 1; ++o) {
        uint64_t other[KP];
#pragma unroll
        for (int t = 0; t < KP; ++t) other[t] = shkey[o][t][lane];
        merge_state<KP>(kd, other);
    }

    // the first k entries of the padded state, in key order (-1: fewer than k finite candidates)
    int32_t sel[KP];
#pragma unroll
    for (int t = 0; t < KP; ++t)
        sel[t] = t < k && kd[t] < kNone ? static_cast<int32_t>(static_cast<uint32_t>(kd[t])) : -1;
    if (nbr) {
#pragma unroll
        for (int t = 0; t < KP; ++t)
            if (t < k) nbr[static_cast<int64_t>(qid) * k + t] = sel[t];
    }
    for (int f = 0; f < feat; ++f) {
        float acc = 0.0f;
#pragma unroll
        for (int t = 0; t < KP; ++t)
            if (sel[t] >= 0) acc += x[static_cast<int64_t>(sel[t]) * feat + f];
        y[static_cast<int64_t>(qid) * feat + f] = acc;
    }
}

// ---- small relations: one wavefront per query, no build

// At or below this many points every query scans every point and no relation is built (box,
// Morton keys, sort, records, boxes): the build's launches and the tiled select's short dependent
// chains cost more there than the quadratic distance work.
constexpr int64_t kBruteMax = 16384;
constexpr int kBruteWaves = 4;   // queries per block

// 64-bit lane shift: lane t receives lane t - 1's value (lane 0 its own).
__device__ __forceinline__ uint64_t shift_up(uint64_t v) {
    const int src = lane_id() > 0 ? lane_id() - 1 : 0;
    const uint32_t lo = __builtin_amdgcn_ds_bpermute(src * 4, static_cast<int>(static_cast<uint32_t>(v)));
    const uint32_t hi = __builtin_amdgcn_ds_bpermute(src * 4, static_cast<int>(static_cast<uint32_t>(v >> 32)));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v)), l);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v >> 32)), l);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Wavefront w of block b takes query q = kBruteWaves b + w; its lanes scan the points 64 at a
// time in input order, with the fp32 distance and the (distance, index) key of the tiled select.
// The query's KP smallest keys are kept one per lane (lanes 0..KP-1, ascending); a step's keys
// below the current KP-th key are found by one ballot and inserted one at a time (each lane takes
// its left neighbour's key or the new one: the same rule as the register state of the tiled
// select), so the list is exact whatever the order of the scan.
template <int KP>
__global__ __launch_bounds__(kBruteWaves * kWave) void brute_kernel(const float *__restrict__ pos, int64_t n, int k,
                                                                    int feat, const float *__restrict__ x,
                                                                    float *__restrict__ y, int32_t *__restrict__ nbr) {
    const int lane = lane_id();
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kBruteWaves + uniform(static_cast<int>(threadIdx.x) / kWave);
    if (q >= n) return;
    const f4 me = f4{pos[q * 3], pos[q * 3 + 1], pos[q * 3 + 2], 0.0f};   // uniform: scalar loads
    uint64_t L = kNone;                                                      // lane t < KP: the t-th key
    if (finite3(me.x, me.y, me.z)) {
        uint64_t thr = kNone;                                                // the KP-th key (uniform)
        // candidates of the next step are loaded before the current step is tested
        int64_t j = lane;
        f4 pj = j < n ? f4{pos[j * 3], pos[j * 3 + 1], pos[j * 3 + 2], 0.0f} : f4{0.0f, 0.0f, 0.0f, 0.0f};
        for (int64_t c0 = 0; c0 < n; c0 += kWave) {
            const f4 cur = pj;
            const int64_t jc = c0 + lane;
            j = jc + kWave;
            if (j < n) pj = f4{pos[j * 3], pos[j * 3 + 1], pos[j * 3 + 2], 0.0f};
            const float d2 = sqdist(me, cur);
            uint64_t key = (static_cast<uint64_t>(__float_as_uint(d2)) << 32) | static_cast<uint32_t>(jc);
            key = (jc >= n || jc == q) ? ~0ull : key;   // past the end, or the query itself
            uint64_t mask = __builtin_amdgcn_ballot_w64(key < thr);
            while (mask) {
                const int b = __builtin_ctzll(mask);
                mask &= mask - 1;
                const uint64_t nk = readlane64(key, b);
                if (nk >= thr) continue;   // the list moved below it meanwhile
                const uint64_t left = shift_up(L);
                const uint64_t up = lane == 0 ? nk : (nk < left ? left : nk);
                L = lane < KP ? (nk < L ? up : L) : L;
                thr = readlane64(L, KP - 1);
            }
        }
    }
    const bool has = lane < k && L < kNone;
    const int32_t sel = has ? static_cast<int32_t>(static_cast<uint32_t>(L)) : -1;
    if (nbr && lane < k) nbr[q * k + lane] = sel;
    for (int f = 0; f < feat; ++f) {
        float v = has ? x[static_cast<int64_t>(sel) * feat + f] : 0.0f;
        // fixed shuffle tree over the lanes (the selected rows in key order, then zeros)
#pragma unroll
        for (int o = kWave / 2; o >= 1; o /= 2) v += __shfl_xor(v, o);
        if (lane == 0) y[q * feat + f] = v;
    }
}

template <int KP>
int launch_brute(int64_t n, int k, int feat, const float *pos, const float *x, float *y, int32_t *nbr,
                 hipStream_t stream) {
    prof_before(stream);
    hipLaunchKernelGGL(brute_kernel<KP>, dim3(static_cast<unsigned>(ceil_div(n, kBruteWaves))),
                       dim3(kBruteWaves * kWave), 0, stream, pos, n, k, feat, x, y, nbr);
    prof_after(stream);
    return check_launch("kNN brute force");
}

template <int KP>
int launch_select(const Ws &w, int64_t ntile, int k, int feat, const float *x, float *y, int32_t *nbr,
                  hipStream_t stream) {
    prof_before(stream);
    hipLaunchKernelGGL(select_kernel<KP>, dim3(static_cast<unsigned>(ntile)), dim3(kSplit * kWave), 0, stream, w.rec, w.tlo, w.thi, w.slo, w.shi, w.glo, w.ghi,
                       static_cast<int>(ntile), k, feat, x, y, nbr);
    prof_after(stream);
    return check_launch("kNN select");
}

}  // namespace

size_t workspace_bytes(int64_t n) {
    Carve c(nullptr);
    carve(c, n);
    return c.bytes();
}

int forward(int64_t n, int32_t feat, const float *pos, const float *x, int32_t k, float *y, int32_t *nbr, void *ws,
            hipStream_t stream) {
    const int kp = k <= 1 ? 1 : k <= 2 ? 2 : k <= 4 ? 4 : k <= 8 ? 8 : k <= 16 ? 16 : 32;
    if (n <= kBruteMax) {
        switch (kp) {
            case 1: return launch_brute<1>(n, k, feat, pos, x, y, nbr, stream);
            case 2: return launch_brute<2>(n, k, feat, pos, x, y, nbr, stream);
            case 4: return launch_brute<4>(n, k, feat, pos, x, y, nbr, stream);
            case 8: return launch_brute<8>(n, k, feat, pos, x, y, nbr, stream);
            case 16: return launch_brute<16>(n, k, feat, pos, x, y, nbr, stream);
            default: return launch_brute<32>(n, k, feat, pos, x, y, nbr, stream);
        }
    }
    Carve c(ws);
    Ws w = carve(c, n);
    const int64_t ntile = ceil_div(n, kTile);
    {
        const int np = static_cast<int>(ceil_div(n, kBlock) < kPartials ? ceil_div(n, kBlock) : kPartials);
        hipLaunchKernelGGL(box_partial_kernel, dim3(np), dim3(kBlock), 0, stream, pos, n, w.part);
        if (int rc = check_launch("kNN box")) return rc;
        hipLaunchKernelGGL(box_final_kernel, dim3(1), dim3(kWave), 0, stream, w.part, np, w.box);
        if (int rc = check_launch("kNN box")) return rc;
        hipLaunchKernelGGL(morton_kernel, dim3(static_cast<unsigned>(ceil_div(n, kBlock))), dim3(kBlock), 0, stream,
                           pos, n, w.box, w.key);
        if (int rc = check_launch("kNN keys")) return rc;
        if (int rc = csr::launch_sort_keys(w.key, n, int64_t{1} << (3 * kBits), w.key_sorted, w.perm, nullptr, w.sort,
                                           stream))
            return rc;
    }
    hipLaunchKernelGGL(records_kernel, dim3(static_cast<unsigned>(ceil_div(ntile * kTile, kBlock))), dim3(kBlock), 0,
                       stream, pos, w.perm, n, ntile * kTile, w.rec);
    if (int rc = check_launch("kNN records")) return rc;
    hipLaunchKernelGGL(tile_box_kernel, dim3(static_cast<unsigned>(ceil_div(ntile, kBlock / kWave))), dim3(kBlock), 0,
                       stream, w.rec, ntile, w.tlo, w.thi, w.slo, w.shi);
    if (int rc = check_launch("kNN tile boxes")) return rc;
    const int64_t ngroup = ceil_div(ntile, kGroup);
    hipLaunchKernelGGL(group_box_kernel, dim3(static_cast<unsigned>(ceil_div(ngroup, kBlock / kWave))), dim3(kBlock), 0,
                       stream, w.tlo, w.thi, ntile, ngroup, w.glo, w.ghi);
    if (int rc = check_launch("kNN group boxes")) return rc;
    switch (kp) {
        case 1: return launch_select<1>(w, ntile, k, feat, x, y, nbr, stream);
        case 2: return launch_select<2>(w, ntile, k, feat, x, y, nbr, stream);
        case 4: return launch_select<4>(w, ntile, k, feat, x, y, nbr, stream);
        case 8: return launch_select<8>(w, ntile, k, feat, x, y, nbr, stream);
        case 16: return launch_select<16>(w, ntile, k, feat, x, y, nbr, stream);
        default: return launch_select<32>(w, ntile, k, feat, x, y, nbr, stream);
    }
}

}  // namespace knn
}  // namespace tiga
