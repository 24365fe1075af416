// Edge-local MLP message over the generated radius relation, with its vector-Jacobian product
// (appendix "A differentiable EdgeNN example"; Section 5 for the VJP with the relation held fixed):
//   in_ij = [p_j - p_i ; x_j],  m_ij = W2 ReLU(W1 in_ij + b1) + b2,  y_i = sum_{j in N(i)} m_ij
// with N(i) the radius relation (j != i, fp32 squared distance strictly below fl(r*r)).
//
// MI355X design: a persistent grid of wavefronts walks the cell-ordered points, one point per
// wavefront at a time.  Lanes are (neighbour slot, hidden unit): HP lanes per neighbour (HP >= the
// hidden width, a power of two), 64 / HP neighbours per step.  Each lane keeps its row of W1 and
// its column of W2 in registers, so a message costs one lane 3 + F multiply-adds for its hidden
// unit and `out` for its share of the output; the output is summed over hidden units and
// neighbours by one wave reduction per point.  No edge, message or activation is stored.
//
// The VJP uses the symmetry of the radius relation (j in N(i) iff i in N(j)).  At point k, with
// neighbour l, a lane recomputes its hidden unit for both directed messages:
//   l -> k (k the destination, cotangent dy_k): the parameter gradients, and -W1[:, 0:3]^T da for
//     the position of k; every directed pair is the "l -> k" pair of exactly one point, so the
//     parameter gradients count each message once;
//   k -> l (k the source, cotangent dy_l): W1^T da gives the feature gradient of k and +W1[:, 0:3]^T
//     da its position gradient.
// The input gradients are W1^T times per-lane sums of da, so they need one wave reduction per point
// and no atomics.  Parameter gradients are summed in registers across a wavefront's points, written
// as one partial per wavefront, and reduced in a fixed order (deterministic).
#include "edgenn.hpp"

#include "radius_cells.hpp"

namespace tiga {
namespace edgenn {

using radius::Cells;
using radius::Params;

namespace {

constexpr int kBlock = 256;
constexpr int kMaxBlocks = 1024;                       // persistent grid cap
constexpr int kMaxWaves = kMaxBlocks * (kBlock / kWave);

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 1; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

// Sum over the lanes that hold the same hidden unit (the SL = 64 / HP neighbour slots).
template <int HP>
__device__ __forceinline__ float slot_sum(float v) {
#pragma unroll
    for (int m = HP; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
    return v;
}

int64_t param_count(const Net &net) {
    const int64_t D = 3 + net.feat;
    return net.hidden * D + net.hidden + net.out * net.hidden + net.out;
}

// The lane's weights: row h of W1, b1[h], column h of W2 (zero for h >= hidden).
template <int FP>
struct LaneNet {
    float w1[3 + FP];
    float bh;
    float w2[kMaxOut];
    __device__ __forceinline__ void load(const Net &net, int h) {
        const bool hv = h < net.hidden;
        const int D = 3 + net.feat;
#pragma unroll
        for (int c = 0; c < 3 + FP; ++c) w1[c] = hv && c < D ? net.W1[h * D + c] : 0.0f;
        bh = hv ? net.b1[h] : 0.0f;
#pragma unroll
        for (int o = 0; o < kMaxOut; ++o) w2[o] = hv && o < net.out ? net.W2[o * net.hidden + h] : 0.0f;
    }
};

template <int FP>
__device__ __forceinline__ void load_row(const float *__restrict__ x, int64_t j, int F, float (&v)[FP]) {
    const float *r = x + j * F;
#pragma unroll
    for (int c = 0; c < FP; ++c) v[c] = c < F ? r[c] : 0.0f;
}

template <int HP, int FP>
__global__ __launch_bounds__(kBlock) void fwd_kernel(const Params *__restrict__ prm, const int64_t *__restrict__ start,
                                                     const float4 *__restrict__ rec, int64_t n, float r2,
                                                     const float *__restrict__ x, Net net, float *__restrict__ y) {
    constexpr int SL = kWave / HP;
    const Params p = *prm;
    const int lane = lane_id(), slot = lane / HP, h = lane % HP;
    LaneNet<FP> L;
    L.load(net, h);
    const int F = net.feat, O = net.out;
    const int64_t nw = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t s = uniform(static_cast<int>(xcd_block() * (kBlock / kWave) + threadIdx.x / kWave)); s < n; s += nw) {
        const float4 pi = rec[s];
        const int32_t i = __float_as_int(pi.w);
        float acc[kMaxOut] = {};
        float cnt = 0.0f;
        radius::for_runs(p, start, pi, [&](int64_t b, int64_t e) {
            for (int64_t t0 = b; t0 < e; t0 += SL) {
                const int64_t t = t0 + slot;
                const float4 pj = rec[t < e ? t : b];
                float d2;
                const int32_t j = __float_as_int(pj.w);
                if (t < e && radius::accept(pi, pj, r2, d2) && j != i) {
#pragma clang fp contract(off)
                    const float dx = pj.x - pi.x, dy = pj.y - pi.y, dz = pj.z - pi.z;
                    float xj[FP];
                    load_row<FP>(x, j, F, xj);
                    float a = L.bh + L.w1[0] * dx + L.w1[1] * dy + L.w1[2] * dz;
#pragma unroll
                    for (int c = 0; c < FP; ++c) a += L.w1[3 + c] * xj[c];
                    const float r = fmaxf(a, 0.0f);
#pragma unroll
                    for (int o = 0; o < kMaxOut; ++o) acc[o] += L.w2[o] * r;
                    cnt += h == 0 ? 1.0f : 0.0f;
                }
            }
        });
        const float deg = wave_sum(cnt);
#pragma unroll
        for (int o = 0; o < kMaxOut; ++o) {
            const float v = wave_sum(acc[o]);
            if (o < O && lane == 0) y[static_cast<int64_t>(i) * O + o] = v + deg * net.b2[o];
        }
    }
}

// At feature width 32 the kernel is held to 168 registers (3 waves per SIMD instead of 2 at 179);
// the 8 values this spills cost less than the third wave gains. Other widths keep their registers.
template <int HP, int FP>
__global__ __launch_bounds__(kBlock, FP == 32 ? 3 : 1) void bwd_kernel(const Params *__restrict__ prm, const int64_t *__restrict__ start,
                                                     const float4 *__restrict__ rec, int64_t n, float r2,
                                                     const float *__restrict__ x, Net net, const float *__restrict__ dyv,
                                                     float *__restrict__ dxo, float *__restrict__ dpo,
                                                     float *__restrict__ part, int64_t P) {
    constexpr int SL = kWave / HP;
    const Params p = *prm;
    const int lane = lane_id(), slot = lane / HP, h = lane % HP;
    LaneNet<FP> L;
    L.load(net, h);
    const int F = net.feat, O = net.out, H = net.hidden, D = 3 + F;
    float gW1[3 + FP] = {}, gb1 = 0.0f, gW2[kMaxOut] = {}, gb2[kMaxOut] = {};
    const int64_t wv = uniform(static_cast<int>(xcd_block() * (kBlock / kWave) + threadIdx.x / kWave));
    const int64_t nw = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t s = wv; s < n; s += nw) {
        const float4 pi = rec[s];
        const int32_t i = __float_as_int(pi.w);
        float dyk[kMaxOut];
#pragma unroll
        for (int o = 0; o < kMaxOut; ++o) dyk[o] = o < O ? dyv[static_cast<int64_t>(i) * O + o] : 0.0f;
        float dhk = 0.0f;   // this lane's (W2^T dy_k)[h]
#pragma unroll
        for (int o = 0; o < kMaxOut; ++o) dhk += L.w2[o] * dyk[o];
        float xi[FP];
        load_row<FP>(x, i, F, xi);
        float ck = L.bh;    // the k -> l pre-activation without its displacement part
#pragma unroll
        for (int c = 0; c < FP; ++c) ck += L.w1[3 + c] * xi[c];
        float S = 0.0f, T = 0.0f, cnt = 0.0f;
        radius::for_runs(p, start, pi, [&](int64_t b, int64_t e) {
            for (int64_t t0 = b; t0 < e; t0 += SL) {
                const int64_t t = t0 + slot;
                const float4 pj = rec[t < e ? t : b];
                float d2;
                const int32_t j = __float_as_int(pj.w);
                if (t < e && radius::accept(pi, pj, r2, d2) && j != i) {
#pragma clang fp contract(off)
                    const float dx = pj.x - pi.x, dy = pj.y - pi.y, dz = pj.z - pi.z;
                    const float wd = L.w1[0] * dx + L.w1[1] * dy + L.w1[2] * dz;
                    // l -> k: input [d; x_l], cotangent dy_k
                    float xj[FP];
                    load_row<FP>(x, j, F, xj);
                    float a = L.bh + wd;
#pragma unroll
                    for (int c = 0; c < FP; ++c) a += L.w1[3 + c] * xj[c];
                    const float r = fmaxf(a, 0.0f);
#pragma unroll
                    for (int o = 0; o < kMaxOut; ++o) gW2[o] += dyk[o] * r;
                    const float da = a > 0.0f ? dhk : 0.0f;
                    gW1[0] += da * dx;
                    gW1[1] += da * dy;
                    gW1[2] += da * dz;
#pragma unroll
                    for (int c = 0; c < FP; ++c) gW1[3 + c] += da * xj[c];
                    gb1 += da;
                    T += da;
                    // k -> l: input [-d; x_k], cotangent dy_l
                    float dhl = 0.0f;
#pragma unroll
                    for (int o = 0; o < kMaxOut; ++o)
                        dhl += L.w2[o] * (o < O ? dyv[static_cast<int64_t>(j) * O + o] : 0.0f);
                    S += ck - wd > 0.0f ? dhl : 0.0f;
                    cnt += h == 0 ? 1.0f : 0.0f;
                }
            }
        });
        // input gradients of point i: W1^T times the lane sums of da (over hidden units and slots)
        if (dxo)
            for (int c = 0; c < F; ++c) {
                float w = 0.0f;
#pragma unroll
                for (int q = 0; q < FP; ++q) w = q == c ? L.w1[3 + q] : w;
                const float v = wave_sum(w * S);
                if (lane == 0) dxo[static_cast<int64_t>(i) * F + c] = v;
            }
        if (dpo) {
#pragma unroll
            for (int a = 0; a < 3; ++a) {
                const float v = wave_sum(L.w1[a] * (S - T));
                if (lane == 0) dpo[static_cast<int64_t>(i) * 3 + a] = v;
            }
        }
        // every message into i carries b2: db2 += deg(i) dy_i
        const float deg = wave_sum(cnt);
#pragma unroll
        for (int o = 0; o < kMaxOut; ++o) gb2[o] += deg * dyk[o];
    }
    if (!part) return;
    // this wavefront's parameter-gradient partial: [dW1 | db1 | dW2 | db2]
    float *pw = part + wv * P;
#pragma unroll
    for (int c = 0; c < 3 + FP; ++c) {
        const float v = slot_sum<HP>(gW1[c]);
        if (slot == 0 && h < H && c < D) pw[h * D + c] = v;
    }
    {
        const float v = slot_sum<HP>(gb1);
        if (slot == 0 && h < H) pw[H * D + h] = v;
    }
#pragma unroll
    for (int o = 0; o < kMaxOut; ++o) {
        const float v = slot_sum<HP>(gW2[o]);
        if (slot == 0 && h < H && o < O) pw[H * D + H + o * H + h] = v;
    }
    if (lane == 0)
        for (int o = 0; o < O; ++o) pw[H * D + H + O * H + o] = gb2[o];
}

// Sum the per-wavefront partials into the parameter gradients in two fixed-order stages: each of
// kGroups groups of wavefronts per parameter (consecutive wavefronts, in order), then the groups;
// 64 x 64 balances the two stages' serial sums for 4096 partials.
constexpr int kGroups = 64;

__global__ __launch_bounds__(kWave) void reduce_groups_kernel(const float *__restrict__ part, int64_t nw, int64_t P,
                                                              float *__restrict__ grp) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kWave + threadIdx.x;
    if (q >= P) return;
    const int64_t per = (nw + kGroups - 1) / kGroups;
    const int64_t w0 = blockIdx.y * per, w1 = w0 + per < nw ? w0 + per : nw;
    float s = 0.0f;
    for (int64_t w = w0; w < w1; ++w) s += part[w * P + q];
    grp[static_cast<int64_t>(blockIdx.y) * P + q] = s;
}

__global__ __launch_bounds__(kBlock) void reduce_params_kernel(const float *__restrict__ grp, int64_t P, Net net,
                                                               Grads g) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (q >= P) return;
    float s = 0.0f;
    for (int gi = 0; gi < kGroups; ++gi) s += grp[gi * P + q];
    const int64_t D = 3 + net.feat, H = net.hidden, O = net.out;
    if (q < H * D) {
        if (g.dW1) g.dW1[q] = s;
    } else if (q < H * D + H) {
        if (g.db1) g.db1[q - H * D] = s;
    } else if (q < H * D + H + O * H) {
        if (g.dW2) g.dW2[q - H * D - H] = s;
    } else if (g.db2) {
        g.db2[q - H * D - H - O * H] = s;
    }
}

int grid_blocks(int64_t n) {
    const int64_t b = ceil_div(n, kBlock / kWave);
    return static_cast<int>(b < kMaxBlocks ? b : kMaxBlocks);
}

template <int HP, int FP>
int launch_fwd(int64_t n, const Cells &cl, float r2, const float *x, const Net &net, float *y, hipStream_t stream) {
    // the forward keeps no per-wavefront partials, so its grid is as large as stays resident
    // (more wavefronts in flight hide the dependent record and row loads of each point)
    static const int per_cu = resident_blocks(reinterpret_cast<const void *>(&fwd_kernel<HP, FP>), kBlock);
    const int64_t cap = static_cast<int64_t>(device_cus()) * per_cu;
    const int64_t need = ceil_div(n, kBlock / kWave);
    const int blocks = static_cast<int>(need < cap ? need : cap);
    prof_before(stream);
    hipLaunchKernelGGL((fwd_kernel<HP, FP>), dim3(blocks), dim3(kBlock), 0, stream, cl.prm, cl.start, cl.rec,
                       n, r2, x, net, y);
    prof_after(stream);
    return check_launch("edge MLP forward");
}

template <int HP, int FP>
int launch_bwd(int64_t n, const Cells &cl, float r2, const float *x, const Net &net, const float *dy, const Grads &g,
               float *part, float *grp, hipStream_t stream) {
    const int blocks = grid_blocks(n);
    const int64_t P = param_count(net);
    const bool params = g.dW1 || g.db1 || g.dW2 || g.db2;
    prof_before(stream);
    hipLaunchKernelGGL((bwd_kernel<HP, FP>), dim3(blocks), dim3(kBlock), 0, stream, cl.prm, cl.start, cl.rec, n, r2,
                       x, net, dy, g.dx, g.dpos, params ? part : nullptr, P);
    prof_after(stream);
    if (int rc = check_launch("edge MLP backward")) return rc;
    if (!params) return TIGA_OK;
    hipLaunchKernelGGL(reduce_groups_kernel, dim3(static_cast<unsigned>(ceil_div(P, kWave)), kGroups), dim3(kWave), 0,
                       stream, part, static_cast<int64_t>(blocks) * (kBlock / kWave), P, grp);
    if (int rc = check_launch("edge MLP parameter reduction")) return rc;
    hipLaunchKernelGGL(reduce_params_kernel, dim3(static_cast<unsigned>(ceil_div(P, kBlock))), dim3(kBlock), 0,
                       stream, grp, P, net, g);
    return check_launch("edge MLP parameter reduction");
}

template <int HP, class Fn>
int by_feat(int F, Fn &&fn) {
    if (F <= 8) return fn(std::integral_constant<int, 8>{});
    if (F <= 16) return fn(std::integral_constant<int, 16>{});
    if (F <= 32) return fn(std::integral_constant<int, 32>{});
    return fn(std::integral_constant<int, 64>{});
}

template <class Fn>
int dispatch(const Net &net, Fn &&fn) {
    if (net.hidden <= 16)
        return by_feat<16>(net.feat, [&](auto fp) { return fn(std::integral_constant<int, 16>{}, fp); });
    if (net.hidden <= 32)
        return by_feat<32>(net.feat, [&](auto fp) { return fn(std::integral_constant<int, 32>{}, fp); });
    return by_feat<64>(net.feat, [&](auto fp) { return fn(std::integral_constant<int, 64>{}, fp); });
}

}  // namespace

size_t workspace_bytes(int64_t n, const Net &net) {
    Carve c(nullptr);
    c.take<char>(radius::cells_ws_bytes(n));
    c.take<float>(static_cast<size_t>(kMaxWaves) * param_count(net));
    c.take<float>(static_cast<size_t>(kGroups) * param_count(net));
    return c.bytes();
}

int forward(int64_t n, const float *pos, const float *x, float radius, const Net &net, float *y, void *ws,
            hipStream_t stream) {
    Carve c(ws);
    void *cws = c.take<char>(radius::cells_ws_bytes(n));
    Cells cl;
    if (int rc = radius::build_cells(n, pos, radius, cws, cl, stream)) return rc;
    const float r2 = radius * radius;
    return dispatch(net, [&](auto hp, auto fp) {
        return launch_fwd<decltype(hp)::value, decltype(fp)::value>(n, cl, r2, x, net, y, stream);
    });
}

int backward(int64_t n, const float *pos, const float *x, float radius, const Net &net, const float *dy,
             const Grads &g, void *ws, hipStream_t stream) {
    Carve c(ws);
    void *cws = c.take<char>(radius::cells_ws_bytes(n));
    float *part = c.take<float>(static_cast<size_t>(kMaxWaves) * param_count(net));
    float *grp = c.take<float>(static_cast<size_t>(kGroups) * param_count(net));
    Cells cl;
    if (int rc = radius::build_cells(n, pos, radius, cws, cl, stream)) return rc;
    const float r2 = radius * radius;
    return dispatch(net, [&](auto hp, auto fp) {
        return launch_bwd<decltype(hp)::value, decltype(fp)::value>(n, cl, r2, x, net, dy, g, part, grp, stream);
    });
}

}  // namespace edgenn
}  // namespace tiga
