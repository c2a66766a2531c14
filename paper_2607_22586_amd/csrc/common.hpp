// Device helpers shared by the gfx950 kernels of libmmshiftkv.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mmskv {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16 bit pattern, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float x) {
    uint32_t b = __float_as_uint(x);
    return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

// Eight consecutive bf16 values (16 bytes) as an MFMA operand.
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
    u32x4 v = *reinterpret_cast<const u32x4*>(p);
    return __builtin_bit_cast(bf16x8, v);
}

// Eight consecutive fp32 values rounded to bf16 as an MFMA operand.
__device__ __forceinline__ bf16x8 load_f32_as_bf16x8(const float* p) {
    float4 a = *reinterpret_cast<const float4*>(p);
    float4 b = *reinterpret_cast<const float4*>(p + 4);
    u32x4 v;
    v[0] = f32_to_bf16_bits(a.x) | (f32_to_bf16_bits(a.y) << 16);
    v[1] = f32_to_bf16_bits(a.z) | (f32_to_bf16_bits(a.w) << 16);
    v[2] = f32_to_bf16_bits(b.x) | (f32_to_bf16_bits(b.y) << 16);
    v[3] = f32_to_bf16_bits(b.z) | (f32_to_bf16_bits(b.w) << 16);
    return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
    u32x4 v = {0u, 0u, 0u, 0u};
    return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
    uint32_t lo = __shfl(static_cast<uint32_t>(v), src, kWave);
    uint32_t hi = __shfl(static_cast<uint32_t>(v >> 32), src, kWave);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m, kWave);
    uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m, kWave);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
    for (int m = 1; m < kWave; m <<= 1) v += shfl_xor_u64(v, m);
    return v;
}

}  // namespace mmskv
