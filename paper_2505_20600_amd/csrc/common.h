// Device-side helpers shared by the maskstep kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ms {

using bf16_t = uint16_t;  // raw bfloat16 storage

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float32 -> bfloat16, round to nearest even, NaN kept (gfx950 v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    __bf16 h = static_cast<__bf16>(f);
    return __builtin_bit_cast(bf16_t, h);
}

// Two floats -> two packed bf16 in one 32-bit word (low = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    bf16x2_t v;
    v.x = static_cast<__bf16>(a);
    v.y = static_cast<__bf16>(b);
    return __builtin_bit_cast(uint32_t, v);
}

// Element-type traits: conversion to/from float and the 16x16 MFMA step.
template <typename T> struct Elt;

template <> struct Elt<float> {
    static constexpr int kKStep = 4;     // K depth of one v_mfma_f32_16x16x4_f32
    static constexpr int kKPerLane = 1;  // K elements each lane feeds per MFMA
    using frag_t = float;
    __device__ __forceinline__ static float to_f32(float v) { return v; }
    __device__ __forceinline__ static float from_f32(float v) { return v; }
    __device__ __forceinline__ static f32x4_t mma(frag_t a, frag_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
};

template <> struct Elt<bf16_t> {
    static constexpr int kKStep = 32;    // K depth of one v_mfma_f32_16x16x32_bf16
    static constexpr int kKPerLane = 8;
    using frag_t = bf16x8_t;
    __device__ __forceinline__ static float to_f32(bf16_t v) { return bf16_to_f32(v); }
    __device__ __forceinline__ static bf16_t from_f32(float v) { return f32_to_bf16(v); }
    __device__ __forceinline__ static f32x4_t mma(frag_t a, frag_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

// 16-byte vector load/store helpers.
struct alignas(16) vec16 { uint32_t w[4]; };

__device__ __forceinline__ vec16 ld16(const void* p) { return *reinterpret_cast<const vec16*>(p); }

// Buffer-resource loads: a wave-uniform base with a byte bound, a per-lane
// byte offset and a scalar byte offset. Reads at or past `bytes` return zeros.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ vec16 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(vec16, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}
__device__ __forceinline__ void st16(void* p, const vec16& v) { *reinterpret_cast<vec16*>(p) = v; }

// Four consecutive elements <-> float4.
template <typename T> __device__ __forceinline__ void load4(const T* p, float out[4]);
template <> __device__ __forceinline__ void load4<float>(const float* p, float out[4]) {
    float4 v = *reinterpret_cast<const float4*>(p);
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
}
template <> __device__ __forceinline__ void load4<bf16_t>(const bf16_t* p, float out[4]) {
    uint2 v = *reinterpret_cast<const uint2*>(p);
    out[0] = __uint_as_float(v.x << 16);
    out[1] = __uint_as_float(v.x & 0xffff0000u);
    out[2] = __uint_as_float(v.y << 16);
    out[3] = __uint_as_float(v.y & 0xffff0000u);
}
template <typename T> __device__ __forceinline__ void store4(T* p, const float v[4]);
template <> __device__ __forceinline__ void store4<float>(float* p, const float v[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
template <> __device__ __forceinline__ void store4<bf16_t>(bf16_t* p, const float v[4]) {
    uint2 o;
    o.x = pack_bf16x2(v[0], v[1]);
    o.y = pack_bf16x2(v[2], v[3]);
    *reinterpret_cast<uint2*>(p) = o;
}

// MI355X dispatches consecutive workgroups of a launch round-robin over its
// 8 XCDs, each with a private L2. Remap the hardware block id so that every
// XCD receives one contiguous range of logical ids: work that shares operands
// (one attention head's K/V, one GEMM weight slice) then shares an L2.
constexpr int kXcds = 8;

__device__ __forceinline__ int xcd_logical_block(int hw, int total) {
    const int x = hw % kXcds, i = hw / kXcds;
    const int per = total / kXcds, rem = total % kXcds;
    return x * per + min(x, rem) + i;
}

// Buffer resource (four SGPRs) over `bytes` bytes from `base`, raw addressing:
// loads at or past `bytes` (per-lane offset plus scalar offset) return zeros.
__device__ __forceinline__ u32x4_t raw_rsrc(const void* base, uint32_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    u32x4_t r;
    r[0] = (uint32_t)b;
    r[1] = (uint32_t)(b >> 32) & 0xffffu;
    r[2] = bytes;
    r[3] = 0x00020000u;
    return r;
}

// One 16-byte-per-lane buffer load into LDS at `lds` + 16 * lane (gfx950
// buffer_load_dwordx4 ... lds), issued as an opaque instruction: the
// compiler does not see the LDS write, so it adds no wait of its own before
// later LDS reads (of other stages); the caller orders them with wait_vmcnt +
// barrier_only. The loads complete in issue order with every other
// vector-memory load, so the compiler's own vmcnt waits stay correct. `soff`
// and `lds` are wave-uniform.
__device__ __forceinline__ void dma_buf16(u32x4_t rsrc, uint32_t voff, uint32_t soff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voff), "s"(rsrc),
                    "s"(__builtin_amdgcn_readfirstlane(soff)) : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void*)(p)));
}

// s_waitcnt with only the vector-memory counter constrained (<= n, n < 64).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x3f70 | (N & 15) | ((N >> 4) << 14));
}

// Workgroup barrier without the memory fence of __syncthreads (callers order
// their own memory operations with explicit waits).
// The empty asm statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void barrier_only() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// 2^x with the hardware v_exp_f32 (no denormal-result fix-up: softmax
// weights below 2^-126 of the running maximum are irrelevant).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Reductions over the four 16-lane rows holding the same column (lanes l,
// l^16, l^32, l^48) with the gfx950 cross-row swaps: given the same register
// twice, each swap returns {own value, partner value} in some order.
__device__ __forceinline__ float rows_max(float x) {
    auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float rows_sum(float x) {
    auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

}  // namespace ms
