// Variance-expanded query proxies (Sec. 3.2.1 Eqs. 4-5; Appendix A.4 Eq. 15)
// and the anchor query of Sec. 3.2.3 Eq. 11, on gfx950.
//
// Every floating-point step here is an fp64 operation rounded on its own
// (no fused multiply-add), so the proxies are a fixed function of the
// inputs: window statistics summed in window order, Philox4x32-10 words,
// Box-Muller with series-evaluated ln / sin / cos, fp64 -> fp32 -> bf16.
#pragma clang fp contract(off)

#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

constexpr int kProxyThreads = 256;
constexpr int kBlockDims = 16;      // dimensions (of every proxy of a head) per workgroup
constexpr int kWinChunk = 64;       // window rows staged in LDS at a time
constexpr int kStatBatch = 16;      // staged rows read per LDS round trip

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

__device__ __forceinline__ double load_q(const ProxyArgs& a, int64_t off) {
    if (a.q_dtype == 0) return static_cast<double>(static_cast<const float*>(a.q)[off]);
    const uint32_t bits = static_cast<uint32_t>(static_cast<const uint16_t*>(a.q)[off]) << 16;
    return static_cast<double>(__uint_as_float(bits));
}

__device__ __forceinline__ uint16_t to_bf16(double x) {
    return static_cast<uint16_t>(f32_to_bf16_bits(static_cast<float>(x)));
}

__global__ void __launch_bounds__(kProxyThreads) build_proxies_kernel(ProxyArgs a) {
    extern __shared__ double smem[];
    const int d = a.d, half = d / 2;
    double* mu = smem;            // [d]  (this block's dims only)
    double* gs = smem + d;        // [d]  gamma * sigma
    float* win = reinterpret_cast<float*>(smem + 2 * d);   // [kWinChunk][kBlockDims] staged window values
    const int h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    const int64_t qbase = static_cast<int64_t>(b) * a.qsb + static_cast<int64_t>(h) * a.qsh;

    // Workgroup x owns quads [x*qpb, (x+1)*qpb) of every proxy of the head
    // (with rotary placement also their partner quads d/8 further on), so it
    // needs the statistics of kBlockDims = 16 dimensions only.
    const bool rope = a.cos_f != nullptr;
    const int qpb = rope ? kBlockDims / 8 : kBlockDims / 4;
    const int q0 = blockIdx.x * qpb;
    auto dim_of = [&](int slot) {
        return rope ? (slot < kBlockDims / 2 ? 4 * q0 + slot : half + 4 * q0 + slot - kBlockDims / 2) : 4 * q0 + slot;
    };
    // stage window rows [w0, w0 + n) of the block's dims in LDS (exact in fp32)
    auto stage = [&](int w0, int n) {
        for (int e = tid; e < n * kBlockDims; e += kProxyThreads) {
            const int w = e / kBlockDims, slot = e % kBlockDims;
            win[e] = static_cast<float>(load_q(a, qbase + static_cast<int64_t>(w0 + w) * a.qst + dim_of(slot)));
        }
    };
    // mean, then (population or sample) variance, summed in window order;
    // thread `slot` < kBlockDims owns one dimension
    const bool owner = tid < kBlockDims;
    double acc = 0.0;
    for (int w0 = 0; w0 < a.W; w0 += kWinChunk) {
        const int n = min(kWinChunk, a.W - w0);
        __syncthreads();
        stage(w0, n);
        __syncthreads();
        if (owner) {
            // LDS reads kStatBatch rows at a time, so one read latency covers a batch
            for (int w0b = 0; w0b < n; w0b += kStatBatch) {
                float v[kStatBatch];
#pragma unroll
                for (int k = 0; k < kStatBatch; ++k) v[k] = w0b + k < n ? win[(w0b + k) * kBlockDims + tid] : 0.f;
#pragma unroll
                for (int k = 0; k < kStatBatch; ++k)
                    if (w0b + k < n) acc = acc + static_cast<double>(v[k]);
            }
        }
    }
    const double m = acc / static_cast<double>(a.W);
    double sq = 0.0;
    const bool one_chunk = a.W <= kWinChunk;
    for (int w0 = 0; w0 < a.W; w0 += kWinChunk) {
        const int n = min(kWinChunk, a.W - w0);
        if (!one_chunk) {
            __syncthreads();
            stage(w0, n);
            __syncthreads();
        }
        if (owner) {
            for (int w0b = 0; w0b < n; w0b += kStatBatch) {
                float v[kStatBatch];
#pragma unroll
                for (int k = 0; k < kStatBatch; ++k) v[k] = w0b + k < n ? win[(w0b + k) * kBlockDims + tid] : 0.f;
#pragma unroll
                for (int k = 0; k < kStatBatch; ++k) {
                    if (w0b + k < n) {
                        const double diff = static_cast<double>(v[k]) - m;
                        const double dd = diff * diff;
                        sq = sq + dd;
                    }
                }
            }
        }
    }
    if (owner) {
        const int j = dim_of(tid);
        const double sg = sqrt(sq / static_cast<double>(a.W - a.ddof));
        mu[j] = m;
        gs[j] = a.gamma * sg;
        if (a.stats != nullptr) {
            double* st = a.stats + (static_cast<int64_t>(b) * a.Hq + h) * 2 * d;
            st[j] = m;
            st[d + j] = sg;
        }
    }
    __syncthreads();

    uint16_t* out_head = a.proxies + (static_cast<int64_t>(b) * a.Hq + h) * a.P * d;
    for (int item = tid; item < a.P * qpb; item += kProxyThreads) {
        const int i = item / qpb;
        const int jq = q0 + item % qpb;
        uint16_t* row = out_head + static_cast<int64_t>(i) * d;
        double z[4];
        normal_quad(a.key0, a.key1, b, a.layer, h, i, jq, z);
        double x[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int j = 4 * jq + e;
            const double t = gs[j] * z[e];
            x[e] = mu[j] + t;
        }
        if (!rope) {
            uint2 pk;
            pk.x = static_cast<uint32_t>(to_bf16(x[0])) | (static_cast<uint32_t>(to_bf16(x[1])) << 16);
            pk.y = static_cast<uint32_t>(to_bf16(x[2])) | (static_cast<uint32_t>(to_bf16(x[3])) << 16);
            *reinterpret_cast<uint2*>(row + 4 * jq) = pk;
        } else {
            // partner dims j + d/2 come from quad jq + d/8
            const int jq2 = jq + d / 8;
            double z2[4], y[4];
            normal_quad(a.key0, a.key1, b, a.layer, h, i, jq2, z2);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int j = 4 * jq2 + e;
                const double t = gs[j] * z2[e];
                y[e] = mu[j] + t;
            }
            uint16_t lo[4], hi[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int j = 4 * jq + e;
                const double c = static_cast<double>(a.cos_f[j]), s = static_cast<double>(a.sin_f[j]);
                const double a0 = x[e] * c, a1 = y[e] * s;
                const double b0 = y[e] * c, b1 = x[e] * s;
                lo[e] = to_bf16(a0 - a1);
                hi[e] = to_bf16(b0 + b1);
            }
            uint2 pl, ph;
            pl.x = lo[0] | (static_cast<uint32_t>(lo[1]) << 16);
            pl.y = lo[2] | (static_cast<uint32_t>(lo[3]) << 16);
            ph.x = hi[0] | (static_cast<uint32_t>(hi[1]) << 16);
            ph.y = hi[2] | (static_cast<uint32_t>(hi[3]) << 16);
            *reinterpret_cast<uint2*>(row + 4 * jq) = pl;
            *reinterpret_cast<uint2*>(row + half + 4 * jq) = ph;
        }
    }

    // anchor query: window row W-1, all dims, by workgroup 0
    if (blockIdx.x == 0) {
        uint16_t* ql = a.q_last + (static_cast<int64_t>(b) * a.Hq + h) * d;
        const int64_t lrow = qbase + static_cast<int64_t>(a.W - 1) * a.qst;
        const bool rope_l = a.cos_l != nullptr;
        for (int j = tid; j < d; j += kProxyThreads) {
            double v = load_q(a, lrow + j);
            if (rope_l) {
                if (j < half) {
                    const double c = static_cast<double>(a.cos_l[j]), s = static_cast<double>(a.sin_l[j]);
                    const double a0 = v * c, a1 = load_q(a, lrow + j + half) * s;
                    v = a0 - a1;
                } else {
                    const int jj = j - half;
                    const double c = static_cast<double>(a.cos_l[jj]), s = static_cast<double>(a.sin_l[jj]);
                    const double b0 = v * c, b1 = load_q(a, lrow + jj) * s;
                    v = b0 + b1;
                }
            }
            ql[j] = to_bf16(v);
        }
    }
}

}  // namespace

hipError_t launch_build_proxies(const ProxyArgs& a, hipStream_t s) {
    dim3 grid(a.d / kBlockDims, a.Hq, a.B);
    const size_t lds = 2 * static_cast<size_t>(a.d) * sizeof(double) +
                       static_cast<size_t>(kWinChunk) * kBlockDims * sizeof(float);
    hipLaunchKernelGGL(build_proxies_kernel, grid, dim3(kProxyThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace mmskv
