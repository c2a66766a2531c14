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

// Lane moves through DPP (no LDS round trip): x of the source lane for the
// lanes of the rows in ROWS, 0 for the other lanes and for lanes whose
// source falls outside their 16-lane row.  Controls: row_shr:n = 0x110 + n,
// row_bcast:15 = 0x142 (lane 15 of each row to the next row), row_bcast:31
// = 0x143 (lane 31 to rows 2 and 3).
template <int CTRL, int ROWS, typename U>
__device__ __forceinline__ U dpp_take(U x) {
    static_assert(sizeof(U) == 4 || sizeof(U) == 8, "32- or 64-bit lanes");
    auto move = [](uint32_t v) {
        return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, ROWS, 0xF, true));
    };
    if constexpr (sizeof(U) == 4) {
        return static_cast<U>(move(static_cast<uint32_t>(x)));
    } else {
        const uint64_t v = static_cast<uint64_t>(x);
        const uint64_t lo = move(static_cast<uint32_t>(v)), hi = move(static_cast<uint32_t>(v >> 32));
        return static_cast<U>((hi << 32) | lo);
    }
}

// Inclusive prefix sum over the 64 lanes (lane order): shifts of 1, 2, 4
// and 8 within each row, then each row adds the totals of the rows below.
template <typename U>
__device__ __forceinline__ U wave_incl_scan(U x) {
    x += dpp_take<0x111, 0xF>(x);
    x += dpp_take<0x112, 0xF>(x);
    x += dpp_take<0x114, 0xF>(x);
    x += dpp_take<0x118, 0xF>(x);
    x += dpp_take<0x142, 0xA>(x);
    x += dpp_take<0x143, 0xC>(x);
    return x;
}

// Sum over the 64 lanes, the same in every lane.
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
    const uint64_t x = wave_incl_scan(v);
    const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x)), 63));
    const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x >> 32)), 63));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

}  // namespace mmskv
