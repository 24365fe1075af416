// Shared host and device infrastructure of the gfx950 message-passing library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstddef>
#include <cstdint>
#include <cstdio>

#include "tiga_mp.h"

namespace tiga {

constexpr int kWave = 64;

// ---------------------------------------------------------------- host side

// Per-thread error message (the only mutable library state besides the
// per-thread profiling events).
void set_error(const char *fmt, ...);
void clear_error();

// Return `code` after recording a formatted message.
int fail(int code, const char *fmt, ...);

// Profiling hook: record the armed start event (if any) on `stream`, and after
// the dominant launch the stop event; then disarm.
void prof_before(hipStream_t stream);
void prof_after(hipStream_t stream);
void prof_disarm();

// Scope of one C entry-point call: clears the thread's error message on entry
// and drops any kernel-event arming on exit, so an arming lasts exactly one
// call whether or not that call launched a timed kernel.
struct EntryScope {
    EntryScope() { clear_error(); }
    ~EntryScope() { prof_disarm(); }
    EntryScope(const EntryScope &) = delete;
    EntryScope &operator=(const EntryScope &) = delete;
};

// Check the result of a launch or HIP call; return TIGA_EDEVICE on failure.
int check_hip(hipError_t err, const char *what);
inline int check_launch(const char *what) { return check_hip(hipGetLastError(), what); }

// Number of compute units of the current device (cached per device).
int device_cus();

// Blocks of `block` threads of `kernel` that fit on one compute unit (>= 1).
int resident_blocks(const void *kernel, int block);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Bump allocator over a caller-provided workspace.
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *p) : base(static_cast<char *>(p)) {}
    template <class T>
    T *take(size_t count) {
        off = align_up(off, 256);
        T *p = reinterpret_cast<T *>(base ? base + off : nullptr);
        off += count * sizeof(T);
        return p;
    }
    size_t bytes() const { return align_up(off, 256); }
};

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---------------------------------------------------------------- device side

// Native clang vectors (HIP's float4 is a struct the nontemporal builtins reject).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int lane_id() { return static_cast<int>(threadIdx.x) & (kWave - 1); }

template <class T>
__device__ __forceinline__ T uniform(T v) {
    return __builtin_amdgcn_readfirstlane(v);
}
__device__ __forceinline__ int64_t uniform64(int64_t v) {
    uint64_t u = static_cast<uint64_t>(v);
    uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
    uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// The hardware hands workgroups to the 8 XCDs round-robin (block b runs on
// XCD b % 8).  This renumbering gives each XCD a contiguous range of logical
// blocks, so blocks that share data share that XCD's L2.  It is a bijection
// on [0, gridDim.x).
constexpr unsigned kXcds = 8;
__device__ __forceinline__ unsigned xcd_block() {
    const unsigned b = blockIdx.x, nb = gridDim.x;
    const unsigned x = b % kXcds, k = b / kXcds;
    const unsigned per = nb / kXcds, rem = nb % kXcds;
    return x * per + (x < rem ? x : rem) + k;
}

__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, kWave); }
__device__ __forceinline__ int shfl_xor_i(int v, int m) { return __shfl_xor(v, m, kWave); }

// Inclusive prefix sum over the wave of a 64-bit value.
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v) {
    const int l = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        int64_t o = __shfl_up(v, d, kWave);
        if (l >= d) v += o;
    }
    return v;
}

template <class T>
__device__ __forceinline__ void stg_stream(T *p, T v) {
    __builtin_nontemporal_store(v, p);
}

// Fill kernel (used instead of hipMemsetAsync so that captured graphs stay
// free of memset nodes).
__global__ void fill_u32_kernel(uint32_t *p, uint32_t v, int64_t n);
int fill_u32(void *p, uint32_t v, int64_t n, hipStream_t stream);

}  // namespace tiga
