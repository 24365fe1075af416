// Online-softmax reducer over an implicit triangular or dense relation: the streaming attention
// forward of the appendix "Causal attention as message passing", with the reducer state of
// Section 4.8 (running maximum m, mass l, accumulator o; two states combine by rescaling into the
// common maximum).  For head h and destination i:
//   s_ij = scale * <q_i, k_j>,  y_i = sum_{j in N(i)} exp(s_ij) v_j / sum_{j in N(i)} exp(s_ij)
// with N(i) = {0..i} (triangular, diagonal included) or {0..n-1} (dense).  No score or weight
// array is stored: scores live in registers for one 64-key tile.
//
// MI355X design (gfx950, MFMA 16x16x32 with fp32 accumulation):
//  - A block of 4 wavefronts owns 128 consecutive queries of one head (32 per wavefront) and
//    streams the keys in tiles of 64 through LDS, double-buffered with one barrier per tile.  K is
//    stored row-major (key, width); V is stored transposed (width, key) as it is written, so both
//    products read 8- or 16-byte runs.
//  - Scores are formed transposed, S^T = K Q^T (A = K from LDS, B = Q^T held in registers), so a
//    lane's scores all belong to one query (column = lane % 16).  The running maximum, mass and
//    rescale are then lane-local except for one cross-lane max per tile over the four lanes that
//    share a query.
//  - The exponentiated scores feed the second product O^T += V^T P^T straight from the
//    accumulator registers: a lane of the S^T accumulator holds keys 4g..4g+3 (g = lane / 16) of a
//    16-key block, and the B operand of a 32-deep MFMA wants 8 keys per lane.  The key slots
//    8g + j are therefore bound to keys {4g + j} (j < 4) of the first and {16 + 4g + j - 4} (j >= 4)
//    of the second 16-key block, and the V^T operand reads its keys in the same order; a
//    contraction does not depend on the order of its terms.
//  - The mass l is summed by the matrix core too: an all-ones A operand against the weights'
//    B operand gives, in every row, the sum over the chunk's keys for each query, from the same
//    rounded weights as the numerator (so y is an exactly normalized combination of the values).
//  - Scores are kept in the log2 domain (scale * log2 e folded into one multiply-add), and the
//    accumulator is rescaled only when a tile raises some query's maximum by more than 8 (a
//    factor 256): any reference point m gives the same y = sum 2^(t - m) v / sum 2^(t - m), and
//    2^(t - m) <= 256 stays far inside the range of the weights' 16-bit type.
//  - Causal blocks are scheduled heaviest first, and each XCD takes a contiguous range of
//    (head, query tile) tasks, so the K/V tiles of a head are shared in that XCD's L2.
#include "attention.hpp"

namespace tiga {
namespace attention {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;
constexpr int kQW = 32;                // queries per wavefront
constexpr int kBM = kWaves * kQW;      // queries per block
constexpr int kBN = 64;                // keys per tile
constexpr float kLazy = 8.0f;          // rescale threshold in the log2 domain
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef __bf16 b8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef __bf16 b2 __attribute__((ext_vector_type(2)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef __bf16 b4 __attribute__((ext_vector_type(4)));

// The 16-bit input type: MFMA and the packed fp32 -> 16-bit conversion (round to nearest even).
struct F16 {
    static __device__ __forceinline__ f4 mma(u4 a, u4 b, f4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8, a), __builtin_bit_cast(h8, b), c, 0, 0, 0);
    }
    static __device__ __forceinline__ uint32_t pack(float a, float b) {
        return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2{a, b}), h2));
    }
    static __device__ __forceinline__ u4 ones() { return u4{0x3c003c00u, 0x3c003c00u, 0x3c003c00u, 0x3c003c00u}; }
};
struct BF16 {
    static __device__ __forceinline__ f4 mma(u4 a, u4 b, f4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8, a), __builtin_bit_cast(b8, b), c, 0, 0, 0);
    }
    static __device__ __forceinline__ uint32_t pack(float a, float b) {
        return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2{a, b}), b2));
    }
    static __device__ __forceinline__ u4 ones() { return u4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u}; }
};

template <int D>
struct Geo {
    static constexpr int KS = D + 8;                     // K row stride in LDS (16-bit units)
    static constexpr int VS = kBN + 4;                   // V^T row stride in LDS
    static constexpr int CH = D / 32;                    // 32-deep chunks of the score product
    static constexpr int DB = D / 16;                    // 16-wide blocks of the output
    static constexpr int RPT = kBN * D / 8 / kThreads;   // 16-byte K chunks per thread per tile
    static constexpr int CPR = D / 8;                    // 16-byte chunks per row
    static constexpr int KPT = kBN / (kThreads / CPR);   // V keys per thread per tile
    static constexpr int NKG = kBN / KPT;                // V key groups per tile
    static_assert(RPT >= 1 && KPT >= 1 && (KPT == 2 || KPT == 4), "tile shape");
    static constexpr int LDS_K = kBN * KS;               // per buffer, 16-bit units
    static constexpr int LDS_V = D * VS;
};

// Maximum over the four lanes l, l^16, l^32, l^48 (the lanes that share a query column), with
// the gfx950 lane swaps (VALU, no LDS round trip): each swap returns, per lane, its own value and
// its partner's.
__device__ __forceinline__ float max_over_column(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ uint32_t lo16(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ __forceinline__ uint32_t hi16(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

__device__ __forceinline__ uint32_t word(const u4 &v, int i) { return v[i]; }

// Tile staging: global loads into registers (kr: K rows, vr: V rows), then stores into one LDS
// buffer (K row-major, V transposed).
template <int D>
__device__ __forceinline__ void stage_load(u4 (&kr)[Geo<D>::RPT], u4 (&vr)[Geo<D>::KPT],
                                           const u4 *__restrict__ kh, const u4 *__restrict__ vh, int64_t k0,
                                           int64_t n, int tid) {
    using G = Geo<D>;
    // one uniform tile base and per-thread 32-bit offsets
    const u4 *kt = kh + k0 * G::CPR;
    const u4 *vtl = vh + k0 * G::CPR;
    // consecutive threads take consecutive V key groups, so that one transposed row of the LDS
    // store is written by neighbouring lanes (contiguous, no bank conflicts)
    const int kg = tid % G::NKG, dg = tid / G::NKG;
    if (k0 + kBN <= n) {
#pragma unroll
        for (int r = 0; r < G::RPT; ++r) kr[r] = kt[tid + r * kThreads];
#pragma unroll
        for (int r = 0; r < G::KPT; ++r) vr[r] = vtl[(kg * G::KPT + r) * G::CPR + dg];
    } else {
        // keys past n read the last row instead: their scores are masked to -inf, so their
        // weights are exactly 0 and the (finite) row contributes nothing
        const int last = static_cast<int>(n - 1 - k0);     // tile-relative index of key n-1
#pragma unroll
        for (int r = 0; r < G::RPT; ++r) {
            const int idx = tid + r * kThreads;
            const int key = idx / G::CPR < last ? idx / G::CPR : last;
            kr[r] = kt[key * G::CPR + idx % G::CPR];
        }
#pragma unroll
        for (int r = 0; r < G::KPT; ++r) {
            const int key = kg * G::KPT + r < last ? kg * G::KPT + r : last;
            vr[r] = vtl[key * G::CPR + dg];
        }
    }
}

template <int D>
__device__ __forceinline__ void stage_store(const u4 (&kr)[Geo<D>::RPT], const u4 (&vr)[Geo<D>::KPT],
                                            uint16_t *ks, uint16_t *vt, int tid) {
    using G = Geo<D>;
#pragma unroll
    for (int r = 0; r < G::RPT; ++r) {
        const int idx = tid + r * kThreads;
        *reinterpret_cast<u4 *>(ks + (idx / G::CPR) * G::KS + (idx % G::CPR) * 8) = kr[r];
    }
    const int kg = tid % G::NKG, dg = tid / G::NKG;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        uint16_t *dst = vt + (dg * 8 + j) * G::VS + kg * G::KPT;
        const int w = j / 2;
        if constexpr (G::KPT == 4) {
            u2 p;
            p.x = (j & 1) ? hi16(word(vr[0], w), word(vr[1], w)) : lo16(word(vr[0], w), word(vr[1], w));
            p.y = (j & 1) ? hi16(word(vr[2], w), word(vr[3], w)) : lo16(word(vr[2], w), word(vr[3], w));
            *reinterpret_cast<u2 *>(dst) = p;
        } else {
            *reinterpret_cast<uint32_t *>(dst) =
                (j & 1) ? hi16(word(vr[0], w), word(vr[1], w)) : lo16(word(vr[0], w), word(vr[1], w));
        }
    }
}

// Task order: each XCD takes a contiguous range of tasks; within a head, causal query tiles run
// heaviest (last) first.
__device__ __forceinline__ void task_of(int ntq, bool causal, int &head, int &qt) {
    const int t = static_cast<int>(xcd_block());
    head = t / ntq;
    const int r = t % ntq;
    qt = causal ? ntq - 1 - r : r;
}

template <class T, int D, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(const u4 *__restrict__ q, const u4 *__restrict__ k,
                                                            const u4 *__restrict__ v, int64_t n, int ntq,
                                                            float c, uint16_t *__restrict__ y, float *__restrict__ lse) {
    using G = Geo<D>;
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * (G::LDS_K + G::LDS_V)];
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = uniform(tid / kWave);
    const int col = lane & 15, g = lane >> 4;

    int head, qt;
    task_of(ntq, CAUSAL, head, qt);
    const int64_t hb = static_cast<int64_t>(head) * n;               // first row of this head
    const u4 *qh = q + hb * G::CPR;
    const u4 *kh = k + hb * G::CPR;
    const u4 *vh = v + hb * G::CPR;
    const int64_t q0 = static_cast<int64_t>(qt) * kBM;
    const int64_t qw0 = q0 + w * kQW;                                 // this wavefront's first query

    // Q^T operands: query column `col` of block qb, width slots 8g..8g+7 of chunk ch.
    u4 qreg[2][G::CH];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        int64_t row = qw0 + qb * 16 + col;
        row = row < n ? row : n - 1;
#pragma unroll
        for (int ch = 0; ch < G::CH; ++ch) qreg[qb][ch] = qh[row * G::CPR + ch * 4 + g];
    }

    f4 o[G::DB][2];
#pragma unroll
    for (int db = 0; db < G::DB; ++db)
        for (int qb = 0; qb < 2; ++qb) o[db][qb] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    float m[2] = {-__builtin_inff(), -__builtin_inff()};
    // mass: an all-ones A operand sums P^T over the keys of a chunk for every query column, so
    // the denominator uses the same rounded weights as the numerator
    f4 l[2] = {f4{0.0f, 0.0f, 0.0f, 0.0f}, f4{0.0f, 0.0f, 0.0f, 0.0f}};
    const u4 ones = T::ones();

    const int64_t kend = CAUSAL ? (q0 + kBM < n ? q0 + kBM : n) : n;  // keys this block needs
    const int ntk = static_cast<int>((kend + kBN - 1) / kBN);

    u4 kr[G::RPT], vr[G::KPT];
    stage_load<D>(kr, vr, kh, vh, 0, n, tid);
    stage_store<D>(kr, vr, lds, lds + 2 * G::LDS_K, tid);
    __syncthreads();

    for (int kt = 0; kt < ntk; ++kt) {
        const int buf = kt & 1;
        const int64_t k0 = static_cast<int64_t>(kt) * kBN;
        // prefetch the next tile (the last iteration reloads its own tile into the idle buffer)
        stage_load<D>(kr, vr, kh, vh, kt + 1 < ntk ? k0 + kBN : k0, n, tid);

        const uint16_t *ks = lds + buf * G::LDS_K;
        const uint16_t *vt = lds + 2 * G::LDS_K + buf * G::LDS_V;
        // a wavefront whose queries all precede the tile has nothing to add from it
        if (!CAUSAL || k0 <= qw0 + kQW - 1) {
            // ---- S^T = K Q^T for 4 blocks of 16 keys x 2 blocks of 16 queries
            f4 s[4][2];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
                for (int qb = 0; qb < 2; ++qb) s[kb][qb] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int ch = 0; ch < G::CH; ++ch) {
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const u4 a = *reinterpret_cast<const u4 *>(ks + (kb * 16 + col) * G::KS + ch * 32 + g * 8);
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb) s[kb][qb] = T::mma(a, qreg[qb][ch], s[kb][qb]);
                }
            }
            // ---- relation: keys past n, and (triangular) keys after the query
            const bool edge = k0 + kBN > n || (CAUSAL && k0 + kBN - 1 > qw0);
            if (edge) {
                // in tile-relative 32-bit units: key kb*16 + 4g + i is admissible iff it is below
                // nk = n - k0 and (triangular) not after the query at offset qw0 - k0 + 16 qb + col
                const int nk = static_cast<int>(n - k0 < kBN ? n - k0 : kBN);
                const int qr = static_cast<int>(CAUSAL ? qw0 - k0 : 0) + col;
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
                    const int lim = CAUSAL ? (qr + qb * 16 + 1 < nk ? qr + qb * 16 + 1 : nk) : nk;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const int kj = kb * 16 + g * 4 + i;
                            s[kb][qb][i] = kj < lim ? s[kb][qb][i] : -__builtin_inff();
                        }
                }
            }
            // ---- online-softmax state update (Section 4.8), log2 domain
            u4 pb[2][2];   // [key chunk][query block]: B operands of the second product
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                float mt = s[0][qb][0];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) mt = fmaxf(mt, s[kb][qb][i]);
                mt = max_over_column(mt);
                mt *= c;
                if (__any(mt > m[qb] + kLazy)) {
                    const float mn = fmaxf(m[qb], mt);
                    const float alpha = __builtin_amdgcn_exp2f(m[qb] - mn);
                    m[qb] = mn;
                    l[qb] *= alpha;
#pragma unroll
                    for (int db = 0; db < G::DB; ++db) o[db][qb] *= alpha;
                }
                float p[4][4];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        p[kb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][qb][i], c, -m[qb]));
                    }
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    pb[kc][qb].x = T::pack(p[2 * kc][0], p[2 * kc][1]);
                    pb[kc][qb].y = T::pack(p[2 * kc][2], p[2 * kc][3]);
                    pb[kc][qb].z = T::pack(p[2 * kc + 1][0], p[2 * kc + 1][1]);
                    pb[kc][qb].w = T::pack(p[2 * kc + 1][2], p[2 * kc + 1][3]);
                }
            }
            // ---- O^T += V^T P^T
#pragma unroll
            for (int db = 0; db < G::DB; ++db) {
#pragma unroll
                for (int kc = 0; kc < 2; ++kc) {
                    const uint16_t *row = vt + (db * 16 + col) * G::VS + kc * 32 + g * 4;
                    const u2 lo = *reinterpret_cast<const u2 *>(row);
                    const u2 hi = *reinterpret_cast<const u2 *>(row + 16);
                    const u4 a = u4{lo.x, lo.y, hi.x, hi.y};
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb) o[db][qb] = T::mma(a, pb[kc][qb], o[db][qb]);
                }
            }
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) l[qb] = T::mma(ones, pb[kc][qb], l[qb]);
        }
        stage_store<D>(kr, vr, lds + (buf ^ 1) * G::LDS_K, lds + 2 * G::LDS_K + (buf ^ 1) * G::LDS_V, tid);
        __syncthreads();
    }

    // ---- finalize: total mass over the four lanes of a query, divide, store
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float lt = l[qb][0];          // every row of the mass block holds the full sum
        const float inv = 1.0f / lt;
        const int64_t qi = qw0 + qb * 16 + col;
        if (qi < n) {
            uint16_t *yr = y + (hb + qi) * D;
#pragma unroll
            for (int db = 0; db < G::DB; ++db) {
                const f4 r = o[db][qb] * inv;
                u2 out;
                out.x = T::pack(r[0], r[1]);
                out.y = T::pack(r[2], r[3]);
                *reinterpret_cast<u2 *>(yr + db * 16 + g * 4) = out;
            }
            if (lse && g == 0) lse[hb + qi] = (m[qb] + __log2f(lt)) * kLn2;
        }
    }
}

template <class T, int D, bool CAUSAL>
int launch(int64_t n, int heads, const void *q, const void *k, const void *v, float scale, void *y, float *lse,
           hipStream_t stream) {
    const int64_t ntq = ceil_div(n, kBM);
    const int64_t blocks = ntq * heads;
    if (blocks > 0x7fffffff) return fail(TIGA_EUNSUPPORTED, "attention: too many query tiles (%lld)", (long long)blocks);
    prof_before(stream);
    hipLaunchKernelGGL((attn_fwd_kernel<T, D, CAUSAL>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, stream,
                       static_cast<const u4 *>(q), static_cast<const u4 *>(k), static_cast<const u4 *>(v), n,
                       static_cast<int>(ntq), scale * kLog2e, static_cast<uint16_t *>(y), lse);
    prof_after(stream);
    return check_launch("attention forward");
}

template <class T, int D>
int launch_rel(int64_t n, int heads, const void *q, const void *k, const void *v, float scale, int relation, void *y,
               float *lse, hipStream_t stream) {
    return relation == TIGA_REL_TRIANGULAR ? launch<T, D, true>(n, heads, q, k, v, scale, y, lse, stream)
                                           : launch<T, D, false>(n, heads, q, k, v, scale, y, lse, stream);
}

template <class T>
int launch_width(int64_t n, int heads, int width, const void *q, const void *k, const void *v, float scale,
                 int relation, void *y, float *lse, hipStream_t stream) {
    if (width == 64) return launch_rel<T, 64>(n, heads, q, k, v, scale, relation, y, lse, stream);
    return launch_rel<T, 128>(n, heads, q, k, v, scale, relation, y, lse, stream);
}

}  // namespace

int forward(int64_t n, int32_t heads, int32_t width, int dtype, const void *q, const void *k, const void *v,
            float scale, int relation, void *y, float *lse, hipStream_t stream) {
    return dtype == TIGA_DT_F16 ? launch_width<F16>(n, heads, width, q, k, v, scale, relation, y, lse, stream)
                                : launch_width<BF16>(n, heads, width, q, k, v, scale, relation, y, lse, stream);
}

}  // namespace attention
}  // namespace tiga
