// Variance-expanded query proxies (Sec. 3.2.1 Eqs. 4-5; Appendix A.4 Eq. 15)
// and the anchor query of Sec. 3.2.3 Eq. 11, on gfx950.
//
// Every floating-point step here is rounded on its own (no fused
// multiply-add), so the proxies are a fixed function of the inputs: window
// statistics summed in window order (fp64), Philox4x32-10 words, Box-Muller
// with series-evaluated ln / sin / cos (fp32, widened to fp64), the proxy
// formula and the softmax scale log2(e)/sqrt(d) that the queries carry
// (fp64; Sec. 3.2.2 Eq. 7, so the score products are base-2 logits), then
// fp64 -> fp32 -> bf16.  The anchor query is returned unscaled.
#pragma clang fp contract(off)

#include "common.hpp"
#include "kernels.hpp"
#include "normal.hpp"

namespace mmskv {
namespace {

constexpr int kProxyThreads = 256;
constexpr int kBlockDims = 16;      // dimensions (of every proxy of a head) per workgroup
constexpr int kWinChunk = 64;       // window rows staged in LDS at a time
constexpr int kStatBatch = 16;      // staged rows read per LDS round trip

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
    // Draws of this thread's first kPreItems items, made before the
    // statistics are published (they do not depend on them): every wave
    // draws while the statistics lanes run their serial sums.  The draws are
    // fp32 values, so keeping them as fp32 and widening later is exact.
    constexpr int kPreItems = 4;
    const int n_items = a.P * qpb;
    float zp[kPreItems][4], zp2[kPreItems][4];
    if (one_chunk) {
#pragma unroll
        for (int k = 0; k < kPreItems; ++k) {
            const int item = tid + k * kProxyThreads;
            if (item < n_items) {
                const int i = item / qpb, jq = q0 + item % qpb;
                double z[4];
                normal_quad(a.key0, a.key1, b, a.layer, h, i, jq, z);
#pragma unroll
                for (int e = 0; e < 4; ++e) zp[k][e] = static_cast<float>(z[e]);
                if (rope) normal_quad(a.key0, a.key1, b, a.layer, h, i, jq + d / 8, z);
#pragma unroll
                for (int e = 0; e < 4; ++e) zp2[k][e] = rope ? static_cast<float>(z[e]) : 0.f;
            }
        }
    }
    __syncthreads();

    uint16_t* out_head = a.proxies + (static_cast<int64_t>(b) * a.Hq + h) * a.P * d;
    // proxy i, quad jq from its draws z (and z2, the partner quad's, with rotary placement)
    auto emit = [&](int i, int jq, const double (&z)[4], const double (&z2)[4]) {
        uint16_t* row = out_head + static_cast<int64_t>(i) * d;
        double x[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int j = 4 * jq + e;
            const double t = gs[j] * z[e];
            x[e] = mu[j] + t;
        }
        if (!rope) {
            double sx[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) sx[e] = x[e] * a.scale;
            uint2 pk;
            pk.x = static_cast<uint32_t>(to_bf16(sx[0])) | (static_cast<uint32_t>(to_bf16(sx[1])) << 16);
            pk.y = static_cast<uint32_t>(to_bf16(sx[2])) | (static_cast<uint32_t>(to_bf16(sx[3])) << 16);
            *reinterpret_cast<uint2*>(row + 4 * jq) = pk;
        } else {
            // partner dims j + d/2 come from quad jq + d/8
            const int jq2 = jq + d / 8;
            double y[4];
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
                const double rl = a0 - a1, rh = b0 + b1;
                lo[e] = to_bf16(rl * a.scale);
                hi[e] = to_bf16(rh * a.scale);
            }
            uint2 pl, ph;
            pl.x = lo[0] | (static_cast<uint32_t>(lo[1]) << 16);
            pl.y = lo[2] | (static_cast<uint32_t>(lo[3]) << 16);
            ph.x = hi[0] | (static_cast<uint32_t>(hi[1]) << 16);
            ph.y = hi[2] | (static_cast<uint32_t>(hi[3]) << 16);
            *reinterpret_cast<uint2*>(row + 4 * jq) = pl;
            *reinterpret_cast<uint2*>(row + half + 4 * jq) = ph;
        }
    };
    int item = tid;
    if (one_chunk) {
#pragma unroll
        for (int k = 0; k < kPreItems; ++k, item += kProxyThreads) {
            if (item < n_items) {
                double z[4], z2[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    z[e] = static_cast<double>(zp[k][e]);
                    z2[e] = static_cast<double>(zp2[k][e]);
                }
                emit(item / qpb, q0 + item % qpb, z, z2);
            }
        }
    }
    for (; item < n_items; item += kProxyThreads) {
        const int i = item / qpb, jq = q0 + item % qpb;
        double z[4], z2[4] = {0.0, 0.0, 0.0, 0.0};
        normal_quad(a.key0, a.key1, b, a.layer, h, i, jq, z);
        if (rope) normal_quad(a.key0, a.key1, b, a.layer, h, i, jq + d / 8, z2);
        emit(i, jq, z, z2);
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
