// Proxy-induced attention and mass aggregation (Sec. 3.2.2 Eqs. 7-8,
// Sec. 3.2.3 Eq. 11 anchor, Appendix B GQA aggregation) on gfx950.
//
// Layout of the work: a workgroup owns one (batch row b, KV head c, block of
// 256 keys); each of its 4 waves keeps 64 keys resident in registers as
// bf16 MFMA operands for the whole kernel and streams every proxy row of the
// Gh query heads that share KV head c past them in 16-row tiles
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).  No logit ever reaches
// memory.  Because a column mass needs every row's full normaliser, the
// scoring runs twice over the keys:
//   pass 1 (score_lse):  per row, partial (max, sum 2^(s*kappa - max)) over
//                        the workgroup's keys -> part[], merged per row into
//                        a log2-domain log-sum-exp by lse_combine;
//   pass 2 (score_mass): p = 2^(s*kappa - L_row); column sums over the 16*Gh
//                        rows of each proxy group, over all groups (mass) and
//                        over the anchor rows; each key column is owned by
//                        exactly one wave, so there are no atomics and the
//                        result is deterministic.
// kappa = log2(e)/sqrt(d), so 2^(s*kappa) = e^(s/sqrt(d)).
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

constexpr int kThreads = kScoreWaves * kWave;

// Operand fragment of one 16-row tile: lane l holds row (l % 16), columns
// [32*kk + 8*(l/16), +8) for kk < D/32.
template <int D>
struct Frag {
    bf16x8 v[D / 32];
};

template <int D>
__device__ __forceinline__ void load_key_frags(const ScoreArgs& a, int b, int c, int key0,
                                               Frag<D> (&kf)[kScoreSub]) {
    const int lane = lane_id();
    const int col = 8 * (lane >> 4);
#pragma unroll
    for (int s = 0; s < kScoreSub; ++s) {
        const int t = key0 + s * 16 + (lane & 15);
        const bool ok = t < a.T;
        const int64_t off = static_cast<int64_t>(b) * a.ksb + static_cast<int64_t>(c) * a.ksh +
                            static_cast<int64_t>(ok ? t : 0) * a.kst;
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk) {
            if (!ok) {
                kf[s].v[kk] = zero_bf16x8();
            } else if (a.k_dtype == 1) {
                kf[s].v[kk] = load_bf16x8(static_cast<const uint16_t*>(a.k) + off + 32 * kk + col);
            } else {
                kf[s].v[kk] = load_f32_as_bf16x8(static_cast<const float*>(a.k) + off + 32 * kk + col);
            }
        }
    }
}

// Row tile `tile` of KV head c: tiles [0, rows/16) are proxy rows (the Gh
// heads' proxies back to back), the rest are anchor rows (one per head,
// zero-padded to 16).
template <int D>
__device__ __forceinline__ void load_row_frag(const ScoreArgs& a, int b, int c, int tile,
                                              Frag<D>& f) {
    const int lane = lane_id();
    const int col = 8 * (lane >> 4);
    const int r = tile * 16 + (lane & 15);
    const uint16_t* src = nullptr;
    if (r < a.rows) {
        src = a.proxies + (static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh) * a.P * D +
              static_cast<int64_t>(r) * D;
    } else {
        const int hl = r - a.rows;
        if (hl < a.Gh)
            src = a.q_last + (static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh + hl) * D;
    }
#pragma unroll
    for (int kk = 0; kk < D / 32; ++kk)
        f.v[kk] = src ? load_bf16x8(src + 32 * kk + col) : zero_bf16x8();
}

// ---------------------------------------------------------------- pass 1
template <int D>
__global__ void __launch_bounds__(kThreads) score_lse_kernel(ScoreArgs a) {
    __shared__ float2 red[kScoreWaves][kLseChunkTiles * 16];
    const int kb = blockIdx.x, c = blockIdx.y, b = blockIdx.z;
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int key0 = kb * kScoreBlockKeys + wave * (kScoreSub * 16);

    Frag<D> kf[kScoreSub];
    load_key_frags<D>(a, b, c, key0, kf);
    // validity of the keys this lane sees in the K*P^T output layout:
    // key0 + 16*s + 4*(lane/16) + i
    bool kvalid[kScoreSub][4];
#pragma unroll
    for (int s = 0; s < kScoreSub; ++s)
#pragma unroll
        for (int i = 0; i < 4; ++i) kvalid[s][i] = key0 + 16 * s + 4 * (lane >> 4) + i < a.T;

    const int n_tiles = a.rows_pad / 16;
    float2* part = a.part + ((static_cast<int64_t>(b) * a.Hkv + c) * a.n_kb + kb) * a.rows_pad;

    Frag<D> pf, pn;
    load_row_frag<D>(a, b, c, 0, pf);
    for (int chunk = 0; chunk < n_tiles; chunk += kLseChunkTiles) {
        const int chunk_end = min(chunk + kLseChunkTiles, n_tiles);
        for (int tt = chunk; tt < chunk_end; ++tt) {
            if (tt + 1 < n_tiles) load_row_frag<D>(a, b, c, tt + 1, pn);
            floatx4 acc[kScoreSub];
#pragma unroll
            for (int s = 0; s < kScoreSub; ++s) acc[s] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < D / 32; ++kk)
#pragma unroll
                for (int s = 0; s < kScoreSub; ++s) acc[s] = mfma16x16x32(kf[s].v[kk], pf.v[kk], acc[s]);
            // lane holds rows = keys, column = proxy row (lane % 16) of the tile
            float m = -INFINITY;
#pragma unroll
            for (int s = 0; s < kScoreSub; ++s)
#pragma unroll
                for (int i = 0; i < 4; ++i) m = kvalid[s][i] ? fmaxf(m, acc[s][i]) : m;
            m = fmaxf(m, shfl_xor_f(m, 16));
            m = fmaxf(m, shfl_xor_f(m, 32));
            float l = 0.f;
            const float mk = m * a.kappa;
            if (m != -INFINITY) {
#pragma unroll
                for (int s = 0; s < kScoreSub; ++s)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        l += kvalid[s][i] ? fast_exp2(fmaf(acc[s][i], a.kappa, -mk)) : 0.f;
            }
            l += shfl_xor_f(l, 16);
            l += shfl_xor_f(l, 32);
            if (lane < 16) red[wave][(tt - chunk) * 16 + lane] = make_float2(mk, l);
            pf = pn;
        }
        __syncthreads();
        const int n_rows = (chunk_end - chunk) * 16;
        for (int r = threadIdx.x; r < n_rows; r += kThreads) {
            float M = -INFINITY;
#pragma unroll
            for (int w = 0; w < kScoreWaves; ++w) M = fmaxf(M, red[w][r].x);
            float S = 0.f;
            if (M != -INFINITY) {
#pragma unroll
                for (int w = 0; w < kScoreWaves; ++w) S += red[w][r].y * exp2f(red[w][r].x - M);
            }
            part[chunk * 16 + r] = make_float2(M, S);
        }
        __syncthreads();
    }
}

__global__ void __launch_bounds__(256) lse_combine_kernel(ScoreArgs a) {
    const int r = blockIdx.x * 256 + threadIdx.x;
    const int c = blockIdx.y, b = blockIdx.z;
    if (r >= a.rows_pad) return;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const float2* part = a.part + hc * a.n_kb * a.rows_pad + r;
    float M = -INFINITY;
    for (int kb = 0; kb < a.n_kb; ++kb) M = fmaxf(M, part[static_cast<int64_t>(kb) * a.rows_pad].x);
    float S = 0.f;
    for (int kb = 0; kb < a.n_kb; ++kb) {
        const float2 p = part[static_cast<int64_t>(kb) * a.rows_pad];
        S += p.y * exp2f(p.x - M);
    }
    a.lse[hc * a.rows_pad + r] = M + log2f(S);
}

// ---------------------------------------------------------------- pass 2
__device__ __forceinline__ float pick4(const float (&v)[kScoreSub], int q) {
    float r = v[0];
#pragma unroll
    for (int s = 1; s < kScoreSub; ++s) r = (q == s) ? v[s] : r;
    return r;
}

template <int D>
__global__ void __launch_bounds__(kThreads) score_mass_kernel(ScoreArgs a) {
    const int kb = blockIdx.x, c = blockIdx.y, b = blockIdx.z;
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int key0 = kb * kScoreBlockKeys + wave * (kScoreSub * 16);
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;

    Frag<D> kf[kScoreSub];
    load_key_frags<D>(a, b, c, key0, kf);

    const float* L = a.lse + hc * a.rows_pad;
    const int g_rows = a.P / a.G;              // proxies per group (multiple of 16)
    const int gu = g_rows / 16;                // 16-row tiles per (group, head)
    const int tiles_per_group = a.Gh * gu;
    const int n_tiles = a.G * tiles_per_group;
    // this lane writes key column (lane % 16) of sub-tile (lane / 16)
    const int my_key = key0 + 16 * (lane >> 4) + (lane & 15);
    const bool my_ok = my_key < a.T;

    auto tile_row0 = [&](int t) {
        const int g = t / tiles_per_group, rem = t - g * tiles_per_group;
        const int hl = rem / gu, u = rem - hl * gu;
        return hl * a.P + g * g_rows + 16 * u;
    };

    float gacc[kScoreSub], macc[kScoreSub];
#pragma unroll
    for (int s = 0; s < kScoreSub; ++s) { gacc[s] = 0.f; macc[s] = 0.f; }

    Frag<D> pf, pn;
    int r0 = tile_row0(0);
    load_row_frag<D>(a, b, c, r0 / 16, pf);
    float4 lr = *reinterpret_cast<const float4*>(L + r0 + 4 * (lane >> 4));
    for (int t = 0; t < n_tiles; ++t) {
        float4 ln = lr;
        if (t + 1 < n_tiles) {
            const int r1 = tile_row0(t + 1);
            load_row_frag<D>(a, b, c, r1 / 16, pn);
            ln = *reinterpret_cast<const float4*>(L + r1 + 4 * (lane >> 4));
        }
        floatx4 acc[kScoreSub];
#pragma unroll
        for (int s = 0; s < kScoreSub; ++s) acc[s] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk)
#pragma unroll
            for (int s = 0; s < kScoreSub; ++s) acc[s] = mfma16x16x32(pf.v[kk], kf[s].v[kk], acc[s]);
        // lane holds proxy rows 4*(lane/16)+i of the tile, key column lane % 16
#pragma unroll
        for (int s = 0; s < kScoreSub; ++s) {
            gacc[s] += fast_exp2(fmaf(acc[s][0], a.kappa, -lr.x));
            gacc[s] += fast_exp2(fmaf(acc[s][1], a.kappa, -lr.y));
            gacc[s] += fast_exp2(fmaf(acc[s][2], a.kappa, -lr.z));
            gacc[s] += fast_exp2(fmaf(acc[s][3], a.kappa, -lr.w));
        }
        if ((t + 1) % tiles_per_group == 0) {
            const int g = t / tiles_per_group;
#pragma unroll
            for (int s = 0; s < kScoreSub; ++s) {
                gacc[s] += shfl_xor_f(gacc[s], 16);
                gacc[s] += shfl_xor_f(gacc[s], 32);
                macc[s] += gacc[s];
            }
            if (a.group_mass != nullptr && my_ok)
                a.group_mass[(hc * a.G + g) * a.T + my_key] = pick4(gacc, lane >> 4);
#pragma unroll
            for (int s = 0; s < kScoreSub; ++s) gacc[s] = 0.f;
        }
        pf = pn;
        lr = ln;
    }
    if (my_ok) a.mass[hc * a.T + my_key] = pick4(macc, lane >> 4);

    // anchor rows: one per query head of the group, tiles after the proxies
    float aacc[kScoreSub];
#pragma unroll
    for (int s = 0; s < kScoreSub; ++s) aacc[s] = 0.f;
    const int n_anchor_tiles = (a.rows_pad - a.rows) / 16;
    for (int at = 0; at < n_anchor_tiles; ++at) {
        const int rbase = a.rows + 16 * at;
        load_row_frag<D>(a, b, c, rbase / 16, pf);
        const float4 la = *reinterpret_cast<const float4*>(L + rbase + 4 * (lane >> 4));
        floatx4 acc[kScoreSub];
#pragma unroll
        for (int s = 0; s < kScoreSub; ++s) acc[s] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < D / 32; ++kk)
#pragma unroll
            for (int s = 0; s < kScoreSub; ++s) acc[s] = mfma16x16x32(pf.v[kk], kf[s].v[kk], acc[s]);
        const int h0 = 16 * at + 4 * (lane >> 4);
        const float lv[4] = {la.x, la.y, la.z, la.w};
#pragma unroll
        for (int s = 0; s < kScoreSub; ++s)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                aacc[s] += (h0 + i < a.Gh) ? fast_exp2(fmaf(acc[s][i], a.kappa, -lv[i])) : 0.f;
    }
    const float inv_gh = 1.0f / static_cast<float>(a.Gh);
#pragma unroll
    for (int s = 0; s < kScoreSub; ++s) {
        aacc[s] += shfl_xor_f(aacc[s], 16);
        aacc[s] += shfl_xor_f(aacc[s], 32);
        aacc[s] *= inv_gh;
    }
    if (my_ok) a.anchor[hc * a.T + my_key] = pick4(aacc, lane >> 4);
}

template <int D>
hipError_t lse_impl(const ScoreArgs& a, hipStream_t s) {
    dim3 grid(a.n_kb, a.Hkv, a.B);
    hipLaunchKernelGGL(score_lse_kernel<D>, grid, dim3(kThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((a.rows_pad + 255) / 256, a.Hkv, a.B);
    hipLaunchKernelGGL(lse_combine_kernel, g2, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int D>
hipError_t mass_impl(const ScoreArgs& a, hipStream_t s) {
    dim3 grid(a.n_kb, a.Hkv, a.B);
    hipLaunchKernelGGL(score_mass_kernel<D>, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score_lse(const ScoreArgs& a, hipStream_t s) {
    return a.d == 64 ? lse_impl<64>(a, s) : lse_impl<128>(a, s);
}

hipError_t launch_score_mass(const ScoreArgs& a, hipStream_t s) {
    return a.d == 64 ? mass_impl<64>(a, s) : mass_impl<128>(a, s);
}

}  // namespace mmskv
