// Online-softmax reducer over an implicit triangular or dense relation: the streaming attention
// forward of the appendix "Causal attention as message passing", with the reducer state of
// Section 5.2 (running maximum m, mass l, accumulator o; two states combine by rescaling into the
// common maximum).  For head h and destination i:
//   s_ij = scale * <q_i, k_j>,  y_i = sum_{j in N(i)} exp(s_ij) v_j / sum_{j in N(i)} exp(s_ij)
// with N(i) = {0..i} (triangular, diagonal included) or {0..n-1} (dense).  No score or weight
// array is stored: scores live in registers for one key tile.
//
// MI355X design (gfx950, MFMA 16x16x32 with fp32 accumulation):
//  - A block of 4 wavefronts owns 128 consecutive queries of one head (32 per wavefront) and
//    streams the keys in tiles of 64 (width 128) or 128 (width 64) through LDS, double-buffered
//    with one barrier per tile.
//  - Scores are formed transposed, S^T = K Q^T (A = K from LDS, B = Q^T held in registers), so a
//    lane's scores all belong to one query (column = lane % 16).  The reference point, mass and
//    rescale are then lane-local; only the exact path's column maximum crosses lanes (the four
//    lanes that share a query).
//  - The exponentiated scores feed the second product O^T += V^T P^T straight from the
//    accumulator registers: a lane of the S^T accumulator holds keys 4g..4g+3 (g = lane / 16) of a
//    16-key block, and the B operand of a 32-deep MFMA wants 8 keys per lane.  The key slots
//    8g + j are therefore bound to keys {4g + j} (j < 4) of the first and {16 + 4g + j - 4} (j >= 4)
//    of the second 16-key block, and the V^T operand reads its keys in the same order; a
//    contraction does not depend on the order of its terms.
//  - The mass l is summed by the matrix core too: an all-ones A operand against the weights'
//    B operand gives, in every row, the sum over the chunk's keys for each query, from the same
//    rounded weights as the numerator (so y is an exactly normalized combination of the values).
//  - Scores are kept in the log2 domain (scale * log2 e folded into one multiply-add).  Any
//    reference point m gives the same y = sum 2^(t - m) v / sum 2^(t - m), so m is moved only
//    when it must be: each tile's weights are formed against the current m and the tile's mass
//    (from the matrix core) is checked; while it stays at most 2^12 for every query, every weight
//    is at most 2^12, far inside the range of the weights' 16-bit type, and no maximum is taken.
//    Otherwise (and always on the first tile, where m = -inf) the tile takes the exact path:
//    column maximum, rescale of the accumulator and the mass, weights formed again.
//  - K and V tiles go from global memory straight into LDS (16-byte direct loads, no staging
//    registers), in unpadded rows with XOR swizzles that keep the operand reads free of bank
//    conflicts; the V^T operand is read from the row-major V tile by the gfx950 transposing
//    LDS read, so V is never transposed by the VALU.
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
constexpr float kMassCap = 4096.0f;    // largest tile mass (and so weight) of the fast path
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
    static constexpr int CPR = D / 8;                    // 16-byte chunks per row
    static constexpr int RB = 2 * D;                     // bytes per row
    static constexpr int R = 256 / RB;                   // rows per 256-byte bank window (1 or 2)
    static constexpr int NB = D / 16;                    // 32-byte blocks per row
    static constexpr int CH = D / 32;                    // 32-deep chunks of the score product
    static constexpr int DB = D / 16;                    // 16-wide blocks of the output
    static constexpr int BN = D == 64 ? 128 : 64;        // keys per tile (registers allow 128 at width 64)
    static constexpr int KB = BN / 16;                   // 16-key blocks of the score product
    static constexpr int KC = BN / 32;                   // 32-key chunks of the value product
    static constexpr int TILE = BN * RB;                 // bytes of one K or V tile in LDS
    static constexpr int LPW = TILE / 1024 / kWaves;     // 1-KB direct loads per wavefront, tile and operand
    static_assert(LPW >= 1 && TILE % (1024 * kWaves) == 0, "tile shape");
    static constexpr int LDS = 4 * TILE;                 // two buffers of (K, V)
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

// LDS layouts (no padding; XOR swizzles keep the operand reads free of bank conflicts):
//  - K tile, row-major (key, width): the 16-byte chunk c of key row k sits at chunk
//    c ^ ((k / R) % CPR).  The score product reads 16 consecutive keys at one chunk, which then
//    fall into 16 distinct 16-byte bank groups of a 256-byte window.
//  - V tile, row-major (key, width): the 32-byte block b of key row k sits at block
//    b ^ ((k / R) % NB).  The transposing read of the value product takes 4 consecutive keys x
//    16 widths per 16 lanes, 8 keys per half wavefront: 8 distinct 32-byte bank groups.
// Both are filled by direct global -> LDS loads: lane t of a load writes bytes [16 t, 16 t + 16)
// of a 1-KB LDS run, so each lane fetches the global chunk whose swizzled place that is.
template <int D>
__device__ __forceinline__ int k_chunk(int k, int pc) { using G = Geo<D>; return pc ^ ((k / G::R) % G::CPR); }
template <int D>
__device__ __forceinline__ int v_chunk(int k, int pc) {
    using G = Geo<D>;
    return (((pc >> 1) ^ ((k / G::R) % G::NB)) << 1) | (pc & 1);
}

// 16 bytes per lane from global memory straight into LDS: lane t writes bytes [16 t, 16 t + 16)
// of the 1-KB run at `run` (a wavefront-uniform LDS address).
__device__ __forceinline__ void lds_load16(const void *src, uint8_t *run) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)run, 16, 0, 0);
}

// gfx950 transposing LDS read of 16-bit data: within each group of 16 lanes, lane i receives, in
// slot j, element i % 4 of the 8 bytes addressed by lane 4 j + i / 4 of its group.  Issued as
// inline assembly: the compiler cannot tell these reads from the direct loads of the next tile
// (which write the other LDS buffer) and would otherwise wait for those loads before every tile's
// value product.  The caller orders the data with lgkm_wait; the tile itself is complete once
// the barrier at the top of the tile has passed.
template <int OFF>
__device__ __forceinline__ u2 lds_read_tr16(uint32_t addr) {
    u2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}
// Wait until at most N LDS operations of this wavefront are outstanding (they complete in order),
// tied to the registers the waited-for reads wrote.
template <int N>
__device__ __forceinline__ void lgkm_wait(u4 &a, u4 &b) {
    asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "i"(N));
}
// Plain 16-byte LDS read, issued as inline assembly like the transposing read (same reason).
template <int OFF>
__device__ __forceinline__ u4 lds_read_b128(uint32_t addr) {
    u4 r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}
template <int N>
__device__ __forceinline__ void lgkm_wait1(u4 &a) {
    asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(a) : "i"(N));
}
template <int N>
__device__ __forceinline__ void lgkm_wait(u4 &a, u4 &b, u4 &c, u4 &d) {
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : "i"(N));
}
// 32-bit LDS address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const uint8_t *p) {
    return (uint32_t)(size_t)(const __attribute__((address_space(3))) uint8_t *)p;
}

// Issue the direct loads of the K and V tile starting at key k0 into one LDS buffer.  ko / vo
// hold this lane's global chunk offsets (row * CPR + chunk) for a full tile.
template <int D>
__device__ __forceinline__ void stage_kv(const u4 *__restrict__ kh, const u4 *__restrict__ vh, int64_t k0, int64_t n,
                                          const int *ko, const int *vo, uint8_t *kl,
                                          uint8_t *vl, int w, int lane) {
    using G = Geo<D>;
    const u4 *kt = kh + k0 * G::CPR;
    const u4 *vt = vh + k0 * G::CPR;
    if (k0 + G::BN <= n) {
#pragma unroll
        for (int r = 0; r < G::LPW; ++r) {
            const int run = (w * G::LPW + r) * 1024;
            lds_load16(kt + ko[r], kl + run);
            lds_load16(vt + vo[r], vl + run);
        }
    } else {
        // keys past n read the last row instead: their scores are masked to -inf, so their
        // weights are exactly 0 and the (finite) row contributes nothing
        const int last = static_cast<int>(n - 1 - k0);
#pragma unroll
        for (int r = 0; r < G::LPW; ++r) {
            const int run = (w * G::LPW + r) * 1024;
            const int k = (run + 16 * lane) / G::RB;
            const int pc = ((run + 16 * lane) % G::RB) / 16;
            const int key = k < last ? k : last;
            lds_load16(kt + key * G::CPR + k_chunk<D>(k, pc), kl + run);
            lds_load16(vt + key * G::CPR + v_chunk<D>(k, pc), vl + run);
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

template <class T, int D>
struct State {
    f4 o[Geo<D>::DB][2];
    float m[2];
    f4 l[2];
};

// V^T operands of one 16-wide output block for both 32-key chunks: 8 keys per lane, in the key
// slot order of the weights (keys 4g..4g+3 and 16+4g..16+4g+3 of the chunk).  VOFF is the byte
// offset of the V tile in LDS, addr this lane's address of the block within it.
template <int D, int VOFF>
__device__ __forceinline__ void read_vt(uint32_t addr, u4 *a) {
    using G = Geo<D>;
    const u2 l0 = lds_read_tr16<VOFF>(addr);
    const u2 h0 = lds_read_tr16<VOFF + 16 * G::RB>(addr);
    const u2 l1 = lds_read_tr16<VOFF + 32 * G::RB>(addr);
    const u2 h1 = lds_read_tr16<VOFF + 48 * G::RB>(addr);
    a[0] = u4{l0.x, l0.y, h0.x, h0.y};
    a[1] = u4{l1.x, l1.y, h1.x, h1.y};
    if constexpr (G::KC == 4) {
        const u2 l2 = lds_read_tr16<VOFF + 64 * G::RB>(addr);
        const u2 h2 = lds_read_tr16<VOFF + 80 * G::RB>(addr);
        const u2 l3 = lds_read_tr16<VOFF + 96 * G::RB>(addr);
        const u2 h3 = lds_read_tr16<VOFF + 112 * G::RB>(addr);
        a[2] = u4{l2.x, l2.y, h2.x, h2.y};
        a[3] = u4{l3.x, l3.y, h3.x, h3.y};
    }
}

// Weights 2^(c s - m) of query block qb, packed as the B operands of the value product: key
// chunk kc takes keys 32 kc + {4g..4g+3, 16+4g..16+4g+3}.
template <class T, int KB>
__device__ __forceinline__ void weights(const f4 (*s)[2], int qb, float c, float m, u4 (*pb)[2]) {
    float p[KB][4];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) p[kb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][qb][i], c, -m));
#pragma unroll
    for (int kc = 0; kc < KB / 2; ++kc)
        pb[kc][qb] = u4{T::pack(p[2 * kc][0], p[2 * kc][1]), T::pack(p[2 * kc][2], p[2 * kc][3]),
                        T::pack(p[2 * kc + 1][0], p[2 * kc + 1][1]), T::pack(p[2 * kc + 1][2], p[2 * kc + 1][3])};
}

// Mass of query block qb over the tile: l + the sum of its weights, by MFMAs against an all-ones
// A operand (every row of the result holds the sum for the block's query of that column).
template <class T, int KC>
__device__ __forceinline__ f4 mass(const u4 (*pb)[2], int qb, u4 ones, f4 l) {
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) l = T::mma(ones, pb[kc][qb], l);
    return l;
}

// Step R of the score product S^T = K Q^T: K operand R (chunk R / KB, key block R % KB) is
// consumed by the two query blocks, and the read of operand R + 4 is issued into its registers;
// at most 4 reads are in flight.  kaddr[ch] is this lane's LDS address of chunk ch in key block 0.
template <class T, int D, int KOFF, int R>
__device__ __forceinline__ void score_step(f4 (*s)[2], u4 (&ka)[4], const u4 *qreg, const uint32_t *kaddr) {
    using G = Geo<D>;
    constexpr int NR = G::KB * G::CH;
    if constexpr (R < NR) {
        constexpr int ch = R / G::KB, kb = R % G::KB, left = NR - 1 - R;
        lgkm_wait1<(left < 3 ? left : 3)>(ka[R % 4]);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
            s[kb][qb] = T::mma(ka[R % 4], qreg[qb * G::CH + ch], ch == 0 ? f4{0.0f, 0.0f, 0.0f, 0.0f} : s[kb][qb]);
        if constexpr (R + 4 < NR)
            ka[R % 4] = lds_read_b128<KOFF + (R + 4) % G::KB * 16 * G::RB>(kaddr[(R + 4) / G::KB]);
        score_step<T, D, KOFF, R + 1>(s, ka, qreg, kaddr);
    }
}

// S^T = K Q^T of one tile for KB blocks of 16 keys x 2 blocks of 16 queries (the K operands read in
// a rolling window of 4), with the relation applied: keys past n and (triangular) keys after the
// query get -inf.
template <class T, int D, bool CAUSAL, int KOFF>
__device__ __forceinline__ void scores_of(f4 (*s)[2], const u4 (&qreg)[2][Geo<D>::CH], const uint32_t *kaddr,
                                          int64_t k0, int64_t n, int64_t qw0, int col, int g) {
    using G = Geo<D>;
    u4 ka[4];
    ka[0] = lds_read_b128<KOFF + 0 * 16 * G::RB>(kaddr[0]);
    ka[1] = lds_read_b128<KOFF + 1 * 16 * G::RB>(kaddr[0]);
    ka[2] = lds_read_b128<KOFF + 2 * 16 * G::RB>(kaddr[0]);
    ka[3] = lds_read_b128<KOFF + 3 * 16 * G::RB>(kaddr[0]);
    score_step<T, D, KOFF, 0>(s, ka, &qreg[0][0], kaddr);
    const bool edge = k0 + G::BN > n || (CAUSAL && k0 + G::BN - 1 > qw0);
    if (edge) {
        const int nk = static_cast<int>(n - k0 < G::BN ? n - k0 : G::BN);
        const int qr = static_cast<int>(CAUSAL ? qw0 - k0 : 0) + col;
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const int lim = CAUSAL ? (qr + qb * 16 + 1 < nk ? qr + qb * 16 + 1 : nk) : nk;
            // key kb*16 + 4g + i is admissible iff kb*16 + i < lim - 4g (constants on the left)
            const int rel = lim - g * 4;
#pragma unroll
            for (int kb = 0; kb < G::KB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) s[kb][qb][i] = kb * 16 + i < rel ? s[kb][qb][i] : -__builtin_inff();
        }
    }
}

// Online-softmax state update of one tile (Section 5.2), log2 domain, producing the weights pb.
// Fast path: the weights are formed against the current reference point m and the mass of the
// tile (an MFMA against an all-ones operand) is checked: a tile mass of at most 2^12 for every
// query bounds every weight by 2^12, far inside the 16-bit range.  A larger, infinite or NaN mass
// (the first tile, where m = -inf, always) sends the wavefront to the exact path, which takes the
// tile's column maximum, rescales (o, l) to the new reference point and forms the weights again
// before any value product uses them.
template <class T, int D>
__device__ __forceinline__ void softmax_of(State<T, D> &st, const f4 (*s)[2], u4 (*pb)[2], float c, u4 ones) {
    using G = Geo<D>;
    f4 ln[2];
    // the weights are the VALU stretch of the tile: issued at raised priority, so that the
    // other wavefront of the SIMD keeps the matrix core busy meanwhile rather than competing
    // for the issue slots
    __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        weights<T, G::KB>(s, qb, c, st.m[qb], pb);
        ln[qb] = mass<T, G::KC>(pb, qb, ones, st.l[qb]);
    }
    const bool fast = ln[0][0] - st.l[0][0] <= kMassCap && ln[1][0] - st.l[1][0] <= kMassCap;
    if (!__all(fast)) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            float mt = s[0][qb][0];
#pragma unroll
            for (int kb = 0; kb < G::KB; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) mt = fmaxf(mt, s[kb][qb][i]);
            mt = max_over_column(mt) * c;
            if (mt > st.m[qb]) {
                const float alpha = __builtin_amdgcn_exp2f(st.m[qb] - mt);
                st.m[qb] = mt;
                st.l[qb] *= alpha;
#pragma unroll
                for (int db = 0; db < G::DB; ++db) st.o[db][qb] *= alpha;
            }
            weights<T, G::KB>(s, qb, c, st.m[qb], pb);
            ln[qb] = mass<T, G::KC>(pb, qb, ones, st.l[qb]);
        }
    }
    st.l[0] = ln[0];
    st.l[1] = ln[1];
    __builtin_amdgcn_s_setprio(0);
}

// O^T += V^T P^T of one tile; the V^T operand comes from the row-major V tile by transposing
// reads, the operands of block db + 1 being read while the products of block db run.
template <class T, int D, int VOFF>
__device__ __forceinline__ void values_of(State<T, D> &st, const u4 (*pb)[2], const uint32_t *vr) {
    using G = Geo<D>;
    u4 va[G::KC], vn[G::KC];
    read_vt<D, VOFF>(vr[0], va);
#pragma unroll
    for (int db = 0; db < G::DB; ++db) {
        if (db + 1 < G::DB) read_vt<D, VOFF>(vr[db + 1], vn);
        if constexpr (G::KC == 2) {
            if (db + 1 < G::DB) lgkm_wait<4>(va[0], va[1]);
            else lgkm_wait<0>(va[0], va[1]);
        } else {
            if (db + 1 < G::DB) lgkm_wait<8>(va[0], va[1], va[2], va[3]);
            else lgkm_wait<0>(va[0], va[1], va[2], va[3]);
        }
#pragma unroll
        for (int kc = 0; kc < G::KC; ++kc)
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) st.o[db][qb] = T::mma(va[kc], pb[kc][qb], st.o[db][qb]);
#pragma unroll
        for (int kc = 0; kc < G::KC; ++kc) va[kc] = vn[kc];
    }
}

// One key tile: scores, relation mask, online-softmax update, value and mass products.
// kaddr[ch] / vr[db] are this lane's LDS addresses of K chunk ch (key block 0) and of V^T output
// block db within a tile; KOFF / VOFF are the byte offsets of the tile's K and V buffers.
template <class T, int D, bool CAUSAL, int KOFF, int VOFF>
__device__ __forceinline__ void tile_step(State<T, D> &st, const u4 (&qreg)[2][Geo<D>::CH], const uint32_t *kaddr,
                                          const uint32_t *vr,
                                          int64_t k0, int64_t n, int64_t qw0, float c, int col, int g, u4 ones) {
    using G = Geo<D>;
    f4 s[G::KB][2];
    u4 pb[G::KC][2];   // [key chunk][query block]: B operands of the second product
    scores_of<T, D, CAUSAL, KOFF>(s, qreg, kaddr, k0, n, qw0, col, g);
    softmax_of<T, D>(st, s, pb, c, ones);
    values_of<T, D, VOFF>(st, pb, vr);
}

template <class T, int D, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(const u4 *__restrict__ q, const u4 *__restrict__ k,
                                                            const u4 *__restrict__ v, int64_t n, int ntq,
                                                            float c, uint16_t *__restrict__ y, float *__restrict__ lse) {
    using G = Geo<D>;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[G::LDS];
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

    // direct-load chunk offsets of this lane (full tiles)
    int ko[G::LPW], vo[G::LPW];
#pragma unroll
    for (int r = 0; r < G::LPW; ++r) {
        const int b = (w * G::LPW + r) * 1024 + 16 * lane;
        const int kk = b / G::RB, pc = (b % G::RB) / 16;
        ko[r] = kk * G::CPR + k_chunk<D>(kk, pc);
        vo[r] = kk * G::CPR + v_chunk<D>(kk, pc);
    }
    // operand read addresses of this lane within a tile
    uint32_t kr[G::CH];
    uint32_t vr[G::DB];
#pragma unroll
    for (int ch = 0; ch < G::CH; ++ch) kr[ch] = lds_addr(lds) + col * G::RB + 16 * k_chunk<D>(col, ch * 4 + g);
    {
        const int s = lane & 15;
        const int row = 4 * g + s / 4;           // key row of this lane's address (plus 16 / 32 steps)
        const int sw = (row / G::R) % G::NB;
#pragma unroll
        for (int db = 0; db < G::DB; ++db) vr[db] = lds_addr(lds) + row * G::RB + 32 * (db ^ sw) + 8 * (s % 4);
    }

    State<T, D> st;
#pragma unroll
    for (int db = 0; db < G::DB; ++db)
        for (int qb = 0; qb < 2; ++qb) st.o[db][qb] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    st.m[0] = st.m[1] = -__builtin_inff();
    // mass: an all-ones A operand sums P^T over the keys of a chunk for every query column, so
    // the denominator uses the same rounded weights as the numerator
    st.l[0] = st.l[1] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const u4 ones = T::ones();

    const int64_t kend = CAUSAL ? (q0 + kBM < n ? q0 + kBM : n) : n;  // keys this block needs
    const int ntk = static_cast<int>((kend + G::BN - 1) / G::BN);

    // last key any query of this wavefront admits (dense: every key; kept as a run-time bound in
    // both cases, which also keeps the two relations on one instruction schedule)
    const int64_t klast = CAUSAL ? qw0 + kQW - 1 : n;
    uint8_t *const l0 = lds;
    uint8_t *const l1 = lds + 2 * G::TILE;
    stage_kv<D>(kh, vh, 0, n, ko, vo, l0, l0 + G::TILE, w, lane);
    for (int kt = 0; kt < ntk; kt += 2) {
        // buffer 0 holds tile kt; prefetch tile kt + 1 into buffer 1
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        const int64_t k0 = static_cast<int64_t>(kt) * G::BN;
        if (kt + 1 < ntk) stage_kv<D>(kh, vh, k0 + G::BN, n, ko, vo, l1, l1 + G::TILE, w, lane);
        // a wavefront whose queries all precede the tile has nothing to add from it
        if (k0 <= klast)
            tile_step<T, D, CAUSAL, 0, G::TILE>(st, qreg, kr, vr, k0, n, qw0, c, col, g, ones);
        if (kt + 1 >= ntk) break;
        __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (kt + 2 < ntk) stage_kv<D>(kh, vh, k0 + 2 * G::BN, n, ko, vo, l0, l0 + G::TILE, w, lane);
        if (k0 + G::BN <= klast)
            tile_step<T, D, CAUSAL, 2 * G::TILE, 3 * G::TILE>(st, qreg, kr, vr, k0 + G::BN, n, qw0, c, col, g, ones);
    }

    // ---- finalize: total mass over the four lanes of a query, divide, store
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float lt = st.l[qb][0];       // every row of the mass block holds the full sum
        const float inv = 1.0f / lt;
        const int64_t qi = qw0 + qb * 16 + col;
        if (qi < n) {
            uint16_t *yr = y + (hb + qi) * D;
#pragma unroll
            for (int db = 0; db < G::DB; ++db) {
                const f4 r = st.o[db][qb] * inv;
                u2 out;
                out.x = T::pack(r[0], r[1]);
                out.y = T::pack(r[2], r[3]);
                *reinterpret_cast<u2 *>(yr + db * 16 + g * 4) = out;
            }
            if (lse && g == 0) lse[hb + qi] = (st.m[qb] + __log2f(lt)) * kLn2;
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
