// Pieces shared by the fused top-k kernels (k_topk_fused.hip, k_topk_mp.hip):
// vector types, buffer resources, direct-to-LDS loads, wait helpers, the
// kernel argument block and the launches that finish a fused call (rank-order
// sort of the selected keys, exact recomputation of listed rows).
#pragma once

#include "fw_internal.hpp"

namespace fw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));


// An opaque copy: the compiler may not assume it equals its input, so work
// recomputed from it in a later pass is not merged with an earlier pass
// (keeping hundreds of per-logit compare masks alive between passes).
template <typename T>
__device__ __forceinline__ T opaque(T x) {
    asm volatile("" : "+v"(x));
    return x;
}

// Buffer loads: a per-unit descriptor (wave-uniform base and size, reads past
// the size return zero), one 32-bit lane offset and a uniform offset, so the
// unrolled tile loops keep no 64-bit address per tile in vector registers.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ bf16x8 bload8(rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
// Direct-to-LDS loads: lane l's 16 (or 4) bytes land at lds + 16 l (4 l); no
// register is involved, so a wave can keep several tiles in flight.  The
// compiler does not order these writes against later LDS reads: every
// consumer waits explicitly (wait_vm) for the loads it needs.
#define FW_LDS(p) ((__attribute__((address_space(3))) void *)(p))
__device__ __forceinline__ void dma16(rsrc_t r, void *lds, uint32_t voff, uint32_t soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, FW_LDS(lds), 16, voff, soff, 0, 0);
}
__device__ __forceinline__ void dma4(rsrc_t r, void *lds, uint32_t voff, uint32_t soff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, FW_LDS(lds), 4, voff, soff, 0, 0);
}
// wait until at most n vector memory operations of this wave are outstanding
// (loads complete in issue order); n folds to a constant in unrolled loops
#define FW_VM(k) case k: asm volatile("s_waitcnt vmcnt(" #k ")" ::: "memory"); break;
__device__ __forceinline__ void wait_vm(int n) {
    switch (n) {
        FW_VM(0) FW_VM(1) FW_VM(2) FW_VM(3) FW_VM(4) FW_VM(5) FW_VM(6) FW_VM(7)
        FW_VM(8) FW_VM(9) FW_VM(10) FW_VM(11) FW_VM(12) FW_VM(13) FW_VM(14) FW_VM(15)
        FW_VM(16) FW_VM(17) FW_VM(18) FW_VM(19) FW_VM(20) FW_VM(21) FW_VM(22) FW_VM(23)
        FW_VM(24) FW_VM(25) FW_VM(26) FW_VM(27) FW_VM(28) FW_VM(29) FW_VM(30) FW_VM(31)
        FW_VM(32) FW_VM(33) FW_VM(34) FW_VM(35) FW_VM(36) FW_VM(37) FW_VM(38) FW_VM(39)
        FW_VM(40) FW_VM(41) FW_VM(42) FW_VM(43) FW_VM(44) FW_VM(45) FW_VM(46) FW_VM(47)
        FW_VM(48) FW_VM(49) FW_VM(50) FW_VM(51) FW_VM(52) FW_VM(53) FW_VM(54) FW_VM(55)
        FW_VM(56) FW_VM(57) FW_VM(58) FW_VM(59) FW_VM(60) FW_VM(61) FW_VM(62)
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}
#undef FW_VM
__device__ __forceinline__ void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Every barrier of the fused kernel separates LDS writes from LDS reads (the
// direct-to-LDS loads are per wave and waited for by that wave), so it uses
// lds_barrier: a full __syncthreads would also wait for every outstanding
// global store of the wave, exposing write latency at each one.

// Barrier for a ring of direct-to-LDS loads shared by the waves of a
// workgroup: waits for this wave's own LDS reads and writes (lgkmcnt), then
// meets the other waves.  Unlike lds_barrier it carries no memory-model
// fence, whose release would also wait for every direct-to-LDS load still in
// flight; each wave waits for its own ring loads explicitly (wait_vm) before
// it arrives.  The memory clobber keeps the compiler from moving LDS accesses
// across it.
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// the 64-bit value of lane (lane ^ M): quad permutes (DPP) for M = 1, 2,
// swizzles within 32 lanes for M = 4 .. 16, a permute for M = 32
template <int M>
__device__ __forceinline__ unsigned long long xlane64(unsigned long long v) {
    const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
    int a, b;
    if constexpr (M == 1) {
        a = __builtin_amdgcn_mov_dpp(lo, 0xB1, 0xF, 0xF, false);
        b = __builtin_amdgcn_mov_dpp(hi, 0xB1, 0xF, 0xF, false);
    } else if constexpr (M == 2) {
        a = __builtin_amdgcn_mov_dpp(lo, 0x4E, 0xF, 0xF, false);
        b = __builtin_amdgcn_mov_dpp(hi, 0x4E, 0xF, 0xF, false);
    } else if constexpr (M < 32) {
        a = __builtin_amdgcn_ds_swizzle(lo, 0x1F | (M << 10));
        b = __builtin_amdgcn_ds_swizzle(hi, 0x1F | (M << 10));
    } else {
        a = __shfl_xor(lo, 32);
        b = __shfl_xor(hi, 32);
    }
    return ((unsigned long long)(uint32_t)b << 32) | (uint32_t)a;
}
__device__ __forceinline__ unsigned long long xlane64(unsigned long long v, int m) {
    switch (m) {   // m is a constant in the unrolled stages
        case 1: return xlane64<1>(v);
        case 2: return xlane64<2>(v);
        case 4: return xlane64<4>(v);
        case 8: return xlane64<8>(v);
        case 16: return xlane64<16>(v);
        default: return xlane64<32>(v);
    }
}

struct FusedArgs {
    const uint16_t *q, *k, *v;
    const float *scale, *bias;
    int64_t H, G;
    int n;
    KsArg ks;
    float *o, *o_s, *gap, *dropped;
    unsigned long long *sel;  // [R][kmax] selected keys, when indices are requested
    int kmax;
    int32_t *flags, *flag_list, *flag_count;
};

// Launches that complete a fused call: the flag clear before the main kernel,
// and after it the rank-order sort of the selected keys (when topk_idx is
// requested) and the exact recomputation of the rows the main kernel listed.
void launch_fused_clear(int32_t *flag_count, hipStream_t st);
void launch_fused_finish(const FusedArgs &a, int nk, int32_t *topk_idx, hipStream_t st);

}  // namespace fw
