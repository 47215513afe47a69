// Shared device helpers for the libfw kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "../../include/fw.h"

namespace fw {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Element loads: float32 or bfloat16 storage, widened exactly to float.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __uint_as_float(uint32_t(b) << 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int bytes = 4;
    __device__ __forceinline__ static float load(const float *p, size_t i) { return p[i]; }
};
template <> struct Elem<uint16_t> {
    static constexpr int bytes = 2;
    __device__ __forceinline__ static float load(const uint16_t *p, size_t i) {
        return bf16_bits_to_f32(p[i]);
    }
};

// ---------------------------------------------------------------------------
// Workgroup barrier that orders LDS accesses only (no wait for outstanding
// global loads or stores): for barriers that separate LDS writes from LDS
// reads, where __syncthreads would expose global write latency.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Ordering keys.  ord_key(x) is an unsigned integer that orders like x, with
// -0 and +0 mapped to the same key.  Top-k ranks by (key descending, index
// ascending).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ord_key(float x) {
    uint32_t u = __float_as_uint(x + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_to_float(uint32_t k) {
    uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}
__device__ __forceinline__ uint64_t ord_key64(double x) {
    uint64_t u = (uint64_t)__double_as_longlong(x + 0.0);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Lexicographic order of two equal-size index sets given as bit masks: the
// smallest element of the symmetric difference decides.
__device__ __forceinline__ bool lex_less(uint64_t a, uint64_t b) {
    uint64_t x = a ^ b;
    return x != 0 && (a & (x & (~x + 1))) != 0;
}

// ---------------------------------------------------------------------------
// Workgroup reductions in a fixed order (bitwise repeatable).  `red` must hold
// blockDim.x / 64 elements; every thread must call.
// ---------------------------------------------------------------------------
template <typename T, typename Op>
__device__ T block_reduce(T v, T *red, Op op) {
    // butterfly within each wave (every lane ends with the wave's value,
    // the same bits on each since op is commutative), then the waves'
    // values in wave order; blockDim.x is a multiple of 64
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = op(v, __shfl_xor(v, off));
    if (lane == 0) red[w] = v;
    __syncthreads();
    T r = red[0];
    for (int i = 1; i < nw; ++i) r = op(r, red[i]);
    __syncthreads();
    return r;
}

struct OpMax { template <typename T> __device__ T operator()(T a, T b) const { return a > b ? a : b; } };
struct OpMin { template <typename T> __device__ T operator()(T a, T b) const { return a < b ? a : b; } };
struct OpSum { template <typename T> __device__ T operator()(T a, T b) const { return a + b; } };

// Exclusive scan of one int per thread over the workgroup (Hillis-Steele in
// LDS).  Returns the exclusive prefix; *total receives the sum.
__device__ inline int block_exclusive_scan(int v, int *buf, int *total) {
    const int t = threadIdx.x, nt = blockDim.x;
    buf[t] = v;
    __syncthreads();
    for (int s = 1; s < nt; s <<= 1) {
        int add = (t >= s) ? buf[t - s] : 0;
        __syncthreads();
        buf[t] += add;
        __syncthreads();
    }
    int incl = buf[t];
    int tot = buf[nt - 1];
    __syncthreads();
    if (total) *total = tot;
    return incl - v;
}

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Workgroups are dealt to the eight XCDs round-robin.  Workgroup b of a grid
// of nb takes logical index xcd_order(b, nb): the workgroups of one XCD take
// consecutive logical indices (the tail past a multiple of eight keeps its
// own), so neighbouring logical indices -- rows of one unit reading the same
// keys and values -- share that XCD's L2.
__device__ __forceinline__ int64_t xcd_order(int64_t b, int64_t nb) {
    const int64_t full = nb & ~(int64_t)7;
    if (b >= full) return b;
    return (b & 7) * (full >> 3) + (b >> 3);
}

// Binomial coefficient C(n, r), n <= 64, saturating at 2^62 (exact below).
__host__ __device__ inline uint64_t binom(int n, int r) {
    if (r < 0 || r > n) return 0;
    if (r > n - r) r = n - r;
    uint64_t c = 1;
    for (int i = 1; i <= r; ++i) {
        // c = C(n-r+i-1, i-1); C(n-r+i, i) = c * (n-r+i) / i, exact division
        if (c > (1ull << 62) / 64) return 1ull << 62;
        c = c * (uint64_t)(n - r + i) / (uint64_t)i;
    }
    return c;
}

}  // namespace fw
