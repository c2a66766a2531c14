// Counter-based standard normals shared by the proxy kernels: Philox4x32-10
// words (Salmon et al., SC 2011) turned into Box-Muller pairs with ln, sin and
// cos evaluated by fixed series in fp32, every step rounded on its own (no
// fused multiply-add; division and square root correctly rounded), so the
// draws are a fixed function of the counter.  The pairs are widened to fp64
// for the proxy formula.
#pragma once
#pragma clang fp contract(off)

#include "common.hpp"

namespace mmskv {
namespace {

// Philox4x32-10 (Salmon et al., SC 2011): ten rounds of
// (c0,c1,c2,c3) <- (hi(M1 c2)^c1^k0, lo(M1 c2), hi(M0 c0)^c3^k1, lo(M0 c0))
// with the key advanced by the Weyl increments between rounds.
__device__ __forceinline__ void philox4x32_10(uint32_t& c0, uint32_t& c1, uint32_t& c2,
                                              uint32_t& c3, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c0;   // one 32x32->64 multiply each
        const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * c2;
        const uint32_t lo0 = static_cast<uint32_t>(p0), hi0 = static_cast<uint32_t>(p0 >> 32);
        const uint32_t lo1 = static_cast<uint32_t>(p1), hi1 = static_cast<uint32_t>(p1 >> 32);
        // three-input XORs, one v_bitop3_b32 each (truth table 0x96)
        const uint32_t n0 = __builtin_amdgcn_bitop3_b32(hi1, c1, k0, 0x96);
        const uint32_t n2 = __builtin_amdgcn_bitop3_b32(hi0, c3, k1, 0x96);
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
}

// 32-bit word -> (2*(x>>9)+1) * 2^-24, an odd multiple of 2^-24, exact in
// fp32, inside (0,1).
__device__ __forceinline__ float word_to_unit(uint32_t x) {
    return static_cast<float>(2u * (x >> 9) + 1u) * 0x1p-24f;
}

// ln(u), u in (0,1) normal: u = m * 2^e with m in [r, 2r), r = fp32 sqrt(1/2)
// rounded down, taken from the exponent field; ln m = 2 s (1 + s^2/3 + ... +
// s^10/11), s = (m-1)/(m+1), Horner in s^2.
__device__ float ln_unit(float u) {
    const uint32_t bits = __float_as_uint(u);
    int e = static_cast<int>((bits >> 23) & 0xFFu) - 126;
    const float f = __uint_as_float((bits & 0x007FFFFFu) | 0x3F000000u);   // [0.5, 1)
    float m = f;
    if (f < 0x1.6a09e6p-1f) {
        m = f * 2.0f;
        e = e - 1;
    }
    const float s = (m - 1.0f) / (m + 1.0f);
    const float s2 = s * s;
    float h = 1.0f / 11.0f;
#pragma unroll
    for (int k = 4; k >= 0; --k) {
        h = h * s2;
        h = h + 1.0f / static_cast<float>(2 * k + 1);
    }
    float r = 2.0f * s;
    r = r * h;
    const float e_ln2 = static_cast<float>(e) * 0x1.62e430p-1f;
    return e_ln2 + r;
}

// sin / cos of 2*pi*u for u = word_to_unit(x): the nearest quarter turn q of
// 4u = n / 2^22 (n odd, never halfway) comes off in integers, the remainder
// angle (|phi| < pi/4) goes through Taylor series up to phi^11 / phi^10, then
// the quadrant identities.
__device__ void sincos_turn(uint32_t x, float& sn, float& cs) {
    const int n = static_cast<int>(2u * (x >> 9) + 1u);
    const int q = (n + (1 << 21)) >> 22;
    const float f = static_cast<float>(n - q * (1 << 22)) * 0x1p-24f;
    const float phi = f * 0x1.921fb6p+2f;
    const float p2 = phi * phi;
    float as[6], ac[6];
    as[0] = 1.0f;
    ac[0] = 1.0f;
#pragma unroll
    for (int k = 1; k <= 5; ++k) {
        as[k] = -as[k - 1] / static_cast<float>((2 * k) * (2 * k + 1));
        ac[k] = -ac[k - 1] / static_cast<float>((2 * k - 1) * (2 * k));
    }
    float ps = as[5], pc = ac[5];
#pragma unroll
    for (int k = 4; k >= 0; --k) {
        ps = ps * p2;
        ps = ps + as[k];
        pc = pc * p2;
        pc = pc + ac[k];
    }
    const float s0 = phi * ps;
    const float c0 = pc;
    // quadrant q & 3 gives (s0, c0), (c0, -s0), (-s0, -c0), (-c0, s0): an
    // odd q swaps the pair, q & 2 negates the sine and (q + 1) & 2 the
    // cosine (selects and sign flips, no divergent branch)
    const bool swap = (q & 1) != 0;
    const float sv = swap ? c0 : s0, cv = swap ? s0 : c0;
    sn = __uint_as_float(__float_as_uint(sv) ^ ((q & 2) ? 0x80000000u : 0u));
    cs = __uint_as_float(__float_as_uint(cv) ^ (((q + 1) & 2) ? 0x80000000u : 0u));
}

// Four standard normals for dims 4*jq..4*jq+3 of proxy i, query head h,
// batch row b: Philox counter (jq, i, h, (b<<16)|layer), key (k0,k1); words
// (x0,x1) and (x2,x3) each give one Box-Muller pair (r cos, r sin).
__device__ void normal_quad(uint32_t k0, uint32_t k1, int b, int layer, int h, int i, int jq,
                            double z[4]) {
    uint32_t c0 = static_cast<uint32_t>(jq), c1 = static_cast<uint32_t>(i),
             c2 = static_cast<uint32_t>(h),
             c3 = (static_cast<uint32_t>(b) << 16) | (static_cast<uint32_t>(layer) & 0xFFFFu);
    philox4x32_10(c0, c1, c2, c3, k0, k1);
    const uint32_t w[4] = {c0, c1, c2, c3};
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const float r = sqrtf(-2.0f * ln_unit(word_to_unit(w[2 * p])));
        float sn, cs;
        sincos_turn(w[2 * p + 1], sn, cs);
        const float z0 = r * cs;
        const float z1 = r * sn;
        z[2 * p] = static_cast<double>(z0);
        z[2 * p + 1] = static_cast<double>(z1);
    }
}

}  // namespace
}  // namespace mmskv
