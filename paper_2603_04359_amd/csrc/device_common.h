// Device-side types and helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace catk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Load element i of a bf16 (raw bits) or fp32 array as fp32.
template <typename T>
__device__ __forceinline__ float load_as_f32(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_as_f32<float>(const float* p, int64_t i) {
    return p[i];
}
template <>
__device__ __forceinline__ float load_as_f32<uint16_t>(const uint16_t* p, int64_t i) {
    return bf16_bits_to_f32(p[i]);
}

// Reinterpret four dwords as eight bf16 values (MFMA operand).
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
    return __builtin_bit_cast(bf16x8, v);
}

// Unsigned view of a non-negative float: order-preserving for atomicMax.
__device__ __forceinline__ uint32_t abs_bits(float v) {
    return __float_as_uint(v) & 0x7FFFFFFFu;
}

// Packed INT4 (two's complement, element 2m in the low nibble of byte m)
// to int8 values scaled by 16.  From one packed dword (8 codes):
//   lo = bytes (e0, e2, e4, e6) * 16,  hi = bytes (e1, e3, e5, e7) * 16.
// The product of two operands unpacked the same way sums the same index
// pairs (a permutation of the reduction index), scaled by 256.
__device__ __forceinline__ uint32_t unpack_lo16(uint32_t w) {
    return (w << 4) & 0xF0F0F0F0u;
}
__device__ __forceinline__ uint32_t unpack_hi16(uint32_t w) {
    return w & 0xF0F0F0F0u;
}

// s_waitcnt with only the vector-memory counter limited (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier with release/acquire ordering for LDS only: it waits for
// this wave's own LDS operations, while vector-memory loads in flight stay
// in flight (a plain __syncthreads() would also drain them, which defeats a
// multi-stage prefetch).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// LDS byte address of a __shared__ object (the value M0 takes).
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(T* p) {
    return static_cast<uint32_t>(
        reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T*)p));
}

// HBM -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4): lane L
// reads sbase + voff (sbase wave-uniform, voff a per-lane byte offset) and
// its 16 bytes land at LDS byte address lds_base + 16 L (lds_base
// wave-uniform, passed in M0).  Issued through inline asm on purpose: the
// compiler cannot tell which LDS bytes such a copy writes, so with the
// builtin it makes every later LDS read wait for all outstanding global
// loads, which serializes a prefetch ring.  Callers order the copies
// themselves: wait_vmcnt<> for their own copies, then lds_barrier().  M0 is
// saved and restored around the copy, with the one wait state an M0 write
// needs before an LDS DMA.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
    // readfirstlane yields a signed int: go through uint32_t so that the low
    // word is zero-extended, not sign-extended, into the 64-bit address
    const uint64_t b = reinterpret_cast<uint64_t>(sbase);
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
    const uint32_t hi =
        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
    const uint64_t bu = static_cast<uint64_t>(lo) | (static_cast<uint64_t>(hi) << 32);
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, %2\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(voff), "s"(bu), "s"(__builtin_amdgcn_readfirstlane(lds_base))
        : "memory");
}

// As dma16 with 4 bytes per lane (global_load_lds_dword): lane L's dword
// lands at LDS byte address lds_base + 4 L.
__device__ __forceinline__ void dma4(const void* sbase, uint32_t voff, uint32_t lds_base) {
    const uint64_t b = reinterpret_cast<uint64_t>(sbase);
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b)));
    const uint32_t hi =
        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32)));
    const uint64_t bu = static_cast<uint64_t>(lo) | (static_cast<uint64_t>(hi) << 32);
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %3\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dword %1, %2\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "v"(voff), "s"(bu), "s"(__builtin_amdgcn_readfirstlane(lds_base))
        : "memory");
}

}  // namespace catk
