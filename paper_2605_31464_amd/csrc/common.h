// Shared device types and helpers for the gfx950 kernels of libsurrogate.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// bf16 values live in memory as raw 16-bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// float32 -> bf16 bits, round to nearest even (hardware cvt on gfx950).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    __bf16 b = (__bf16)f;
    return (uint32_t)__builtin_bit_cast(uint16_t, b);
}

// Two floats -> packed bf16 pair (lo in bits 0-15), round to nearest even; one
// v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Reductions over the 64 lanes of a wavefront, butterfly order (deterministic).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr float kLog2e = 1.4426950408889634f;

// Column order of the transposed V copy inside each 16-key group: key index bits 2 and 3
// swapped (an involution), so that the 8 keys one lane feeds a PV MFMA are contiguous.
__host__ __device__ __forceinline__ int vt_key_order(int k) {
    return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

// ---- direct-to-LDS loads (shared by the GEMM and attention kernels)

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N <= 63, "vmcnt");
    // s_waitcnt simm16 on gfx9: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt_hi[15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Byte offset of a __shared__ object inside the workgroup's LDS allocation.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
    return (uint32_t)(uintptr_t)(lds_ptr_t)p;
}

// 16 bytes per lane from global memory straight into LDS at lds_addr + 16 * lane
// (lds_addr is wave-uniform and goes through M0).  Written as inline assembly so the
// compiler's wait-count model, which treats LDS DMA conservatively and would force a
// full LDS-read drain before every MFMA group, does not see it: the kernel orders these
// loads itself (explicit vmcnt waits and a barrier before any LDS read of the stage).
__device__ __forceinline__ void dma_load_16B(const void* gptr, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory", "m0");
}

// As dma_load_16B with the address split into a wave-uniform base (SGPRs) and a per-lane
// 32-bit byte offset: global_load_lds_dwordx4 voff, sbase.
__device__ __forceinline__ void dma_load_16B_sbase(const void* sbase, uint32_t voff,
                                                   uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(voff), "s"(sbase), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory", "m0");
}
