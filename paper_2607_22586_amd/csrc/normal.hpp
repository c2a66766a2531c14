// Counter-based standard normals shared by the proxy kernels: Philox4x32-10
// words (Salmon et al., SC 2011) turned into Box-Muller pairs with ln, sin and
// cos evaluated by fixed series in fp64, every step rounded on its own (no
// fused multiply-add), so the draws are a fixed function of the counter.
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
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
}

// 32-bit word -> (2*(x>>9)+1) * 2^-24, exact, inside (0,1).
__device__ __forceinline__ double word_to_unit(uint32_t x) {
    return static_cast<double>(2u * (x >> 9) + 1u) * 0x1p-24;
}

// ln(u), u in (0,1): u = m * 2^e with m in [sqrt(1/2), sqrt(2)) taken from the
// exponent field; ln m = 2 s (1 + s^2/3 + ... + s^22/23), s = (m-1)/(m+1),
// Horner in s^2.
__device__ double ln_unit(double u) {
    const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(u));
    int e = static_cast<int>((bits >> 52) & 0x7FF) - 1022;
    const double f = __longlong_as_double(
        static_cast<long long>((bits & 0x000FFFFFFFFFFFFFull) | 0x3FE0000000000000ull));
    double m = f;
    if (f < 0x1.6a09e667f3bcdp-1) {
        m = f * 2.0;
        e = e - 1;
    }
    const double s = (m - 1.0) / (m + 1.0);
    const double s2 = s * s;
    double h = 1.0 / 23.0;
#pragma unroll
    for (int k = 10; k >= 0; --k) {
        h = h * s2;
        h = h + 1.0 / static_cast<double>(2 * k + 1);
    }
    double r = 2.0 * s;
    r = r * h;
    const double e_ln2 = static_cast<double>(e) * 0x1.62e42fefa39efp-1;
    return e_ln2 + r;
}

// sin / cos of 2*pi*u, u in (0,1): remove the nearest quarter turn exactly,
// Taylor series of the remainder angle (|phi| <= pi/4) up to phi^21 / phi^20,
// then the quadrant identities.
__device__ void sincos_turn(double u, double& sn, double& cs) {
    const int q = static_cast<int>(4.0 * u + 0.5);
    const double f = u - static_cast<double>(q) * 0.25;
    const double phi = f * 0x1.921fb54442d18p+2;
    const double p2 = phi * phi;
    double as[11], ac[11];
    as[0] = 1.0;
    ac[0] = 1.0;
#pragma unroll
    for (int k = 1; k <= 10; ++k) {
        as[k] = -as[k - 1] / static_cast<double>((2 * k) * (2 * k + 1));
        ac[k] = -ac[k - 1] / static_cast<double>((2 * k - 1) * (2 * k));
    }
    double ps = as[10], pc = ac[10];
#pragma unroll
    for (int k = 9; k >= 0; --k) {
        ps = ps * p2;
        ps = ps + as[k];
        pc = pc * p2;
        pc = pc + ac[k];
    }
    const double s0 = phi * ps;
    const double c0 = pc;
    switch (q & 3) {
        case 0: sn = s0; cs = c0; break;
        case 1: sn = c0; cs = -s0; break;
        case 2: sn = -s0; cs = -c0; break;
        default: sn = -c0; cs = s0; break;
    }
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
        const double ua = word_to_unit(w[2 * p]);
        const double ub = word_to_unit(w[2 * p + 1]);
        const double r = sqrt(-2.0 * ln_unit(ua));
        double sn, cs;
        sincos_turn(ub, sn, cs);
        z[2 * p] = r * cs;
        z[2 * p + 1] = r * sn;
    }
}

}  // namespace
}  // namespace mmskv
