// Proxy-induced attention and mass aggregation (Sec. 3.2.2 Eqs. 7-8,
// Sec. 3.2.3 Eq. 11 anchor, Appendix B GQA aggregation) on gfx950.
//
// Work decomposition.  A workgroup of WAVES waves owns one (batch row b,
// KV head c) and a block of 64*WAVES prompt keys; each wave keeps its 64 keys
// resident in registers as bf16 MFMA fragments for the whole kernel.  Every
// proxy row of the Gh query heads that share KV head c (then the anchor
// rows) streams past those keys in 32-row tiles: the workgroup stages each
// tile once in LDS (double buffered, XOR-swizzled 16-byte chunks so the
// fragment reads are bank-conflict free) and every wave multiplies it with
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation).  Within a wave the MFMAs of
// tile t are issued alongside the exp/reduction VALU work of tile t-1, which
// keeps both the matrix pipe and the VALU busy.  No logit reaches memory.
//
// An exact column mass needs every row's full normaliser, so the keys are
// scored twice:
//   score_lse:  D = K * P^T (keys as rows).  Per proxy row: max and
//               sum 2^(s*kappa - max) over the wave's keys (in-lane, then one
//               cross-lane step), merged over the waves through LDS into one
//               partial per (row, key block); lse_combine folds the partials
//               into L_row = log2 sum_t 2^(s_t*kappa).
//   score_mass: D = P * K^T (proxies as rows).  p = 2^(s*kappa - L_row);
//               column sums over the 16-row halves of each tile, accumulated
//               over the Gh heads into per-group masses, then over groups
//               into the total mass, and over the anchor rows.  Each key
//               column belongs to one wave, so there are no atomics and the
//               result is deterministic.
// kappa = log2(e)/sqrt(d), so 2^(s*kappa) = e^(s/sqrt(d)).
//
// Workgroups are numbered so that all key blocks of one (b, c) land on the
// same XCD (workgroup i runs on XCD i mod 8), keeping that head's proxies in
// one L2.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kSub = 2;            // 32-key sub-tiles per wave
constexpr int kWaveKeys = 32 * kSub;

__device__ __forceinline__ floatx16 mfma32(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Compile-time buffer parity for the two-stage software pipeline (keeps the
// double-buffered accumulators in registers).
template <int N>
struct Parity {
    static constexpr int value = N;
};

__device__ __forceinline__ floatx16 zero16() {
    floatx16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

// Block -> (head, key block), grouping each head's key blocks on one XCD.
__device__ __forceinline__ void block_work(int n_kb, int& head, int& kb) {
    const int n = static_cast<int>(gridDim.x);
    const int id = static_cast<int>(blockIdx.x);
    const int q = n / 8, r = n % 8, x = id % 8;
    const int logical = x * q + min(x, r) + id / 8;
    head = logical / n_kb;
    kb = logical - head * n_kb;
}

// A 32-row tile of bf16 rows of D elements in LDS: 16-byte chunk c of row r
// is stored at slot r*(D/8) + (c ^ (r & 7)).
template <int D>
struct TileLds {
    static constexpr int kChunks = D / 8;             // 16-byte chunks per row
    static constexpr int kSlots = 32 * kChunks;       // per tile
};

template <int D>
__device__ __forceinline__ bf16x8 lds_frag(const u32x4* stage, int row, int chunk) {
    return __builtin_bit_cast(bf16x8, stage[row * (D / 8) + (chunk ^ (row & 7))]);
}

// Global address of row `r` of the padded row space of head (b, c): rows
// [0, Gh*P) are the proxies of the Gh query heads back to back, the rest the
// anchor (last window) query of each head, zero-padded to a multiple of 32
// (padding rows read head 0's anchor row and are masked out by the users).
template <int D>
__device__ __forceinline__ const uint16_t* row_ptr(const ScoreArgs& a, int b, int c, int r) {
    const int64_t hq0 = static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh;
    if (r < a.rows) return a.proxies + (hq0 * a.P + r) * D;
    int hl = r - a.rows;
    if (hl >= a.Gh) hl = 0;
    return a.q_last + (hq0 + hl) * D;
}

// Per-thread share of staging one tile: thread j moves chunk slots
// j, j + threads, ... (global -> registers now, registers -> LDS later).
template <int D, int WAVES>
struct Stager {
    static constexpr int kThreads = 64 * WAVES;
    static constexpr int kSlots = TileLds<D>::kSlots;
    static constexpr int kPer = (kSlots + kThreads - 1) / kThreads;
    static constexpr bool kExact = (kSlots % kThreads) == 0;
    u32x4 v[kPer];

    __device__ __forceinline__ void load(const ScoreArgs& a, int b, int c, int row0) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int slot = static_cast<int>(threadIdx.x) + k * kThreads;
            if (kExact || slot < kSlots) {
                const int r = slot / TileLds<D>::kChunks;
                const int cs = slot - r * TileLds<D>::kChunks;
                const int cg = cs ^ (r & 7);
                v[k] = *reinterpret_cast<const u32x4*>(row_ptr<D>(a, b, c, row0 + r) + 8 * cg);
            }
        }
    }
    __device__ __forceinline__ void store(u32x4* stage) const {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int slot = static_cast<int>(threadIdx.x) + k * kThreads;
            if (kExact || slot < kSlots) stage[slot] = v[k];
        }
    }
};

// Key fragments of the wave's 64 keys: kf[s][kc] holds key
// key0 + 32*s + (lane % 32), dims [16*kc + 8*(lane/32), +8).
template <int D>
__device__ __forceinline__ void load_keys(const ScoreArgs& a, int b, int c, int key0,
                                          bf16x8 (&kf)[kSub][D / 16]) {
    const int lane = lane_id();
    const int col = 8 * (lane >> 5);
#pragma unroll
    for (int s = 0; s < kSub; ++s) {
        const int t = key0 + 32 * s + (lane & 31);
        const bool ok = t < a.T;
        const int64_t off = static_cast<int64_t>(b) * a.ksb + static_cast<int64_t>(c) * a.ksh +
                            static_cast<int64_t>(ok ? t : 0) * a.kst;
        if (a.k_dtype == 1) {
            const uint16_t* p = static_cast<const uint16_t*>(a.k) + off + col;
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) kf[s][kc] = ok ? load_bf16x8(p + 16 * kc) : zero_bf16x8();
        } else {
            const float* p = static_cast<const float*>(a.k) + off + col;
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) kf[s][kc] = ok ? load_f32_as_bf16x8(p + 16 * kc) : zero_bf16x8();
        }
    }
}

// The MFMAs of one tile.  KEYS_AS_ROWS: D = K * P^T (lane holds one proxy
// column, 16 keys per sub-tile); otherwise D = P * K^T (lane holds one key
// column, 16 proxy rows).
template <int D, bool KEYS_AS_ROWS>
__device__ __forceinline__ void tile_mfma(const u32x4* sp, const bf16x8 (&kf)[kSub][D / 16],
                                          floatx16 (&acc)[kSub], int lane) {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
        const bf16x8 pf = lds_frag<D>(sp, lane & 31, 2 * kc + (lane >> 5));
#pragma unroll
        for (int s = 0; s < kSub; ++s) {
            const floatx16 c0 = (kc == 0) ? zero16() : acc[s];
            acc[s] = KEYS_AS_ROWS ? mfma32(kf[s][kc], pf, c0) : mfma32(pf, kf[s][kc], c0);
        }
    }
}

// ---------------------------------------------------------------- pass 1
// (max*kappa, sum 2^(s*kappa - max*kappa)) of one proxy column over the
// wave's keys; FULL: every key of the block is < T.
template <bool FULL>
__device__ __forceinline__ float2 column_lse(const floatx16 (&acc)[kSub], uint32_t valid, float kappa) {
    float m = -INFINITY;
#pragma unroll
    for (int s = 0; s < kSub; ++s)
#pragma unroll
        for (int i = 0; i < 16; ++i)
            m = (FULL || ((valid >> (16 * s + i)) & 1u)) ? fmaxf(m, acc[s][i]) : m;
    m = fmaxf(m, shfl_xor_f(m, 32));
    const float mk = m * kappa;
    float l = 0.f;
    if (FULL || m != -INFINITY) {
#pragma unroll
        for (int s = 0; s < kSub; ++s)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float e = fast_exp2(fmaf(acc[s][i], kappa, -mk));
                l += (FULL || ((valid >> (16 * s + i)) & 1u)) ? e : 0.f;
            }
    }
    l += shfl_xor_f(l, 32);
    return make_float2(mk, l);
}

template <int D, int WAVES, bool FULL>
__device__ __forceinline__ void lse_body(const ScoreArgs& a, int head, int kb, int b, int c,
                                         u32x4 (&stage)[2][TileLds<D>::kSlots],
                                         float2 (&mrg)[2][WAVES][32]) {
    const int wave = static_cast<int>(threadIdx.x) / kWave, lane = lane_id();
    const int key0 = kb * 64 * WAVES + wave * kWaveKeys;
    const float kappa = a.kappa;

    bf16x8 kf[kSub][D / 16];
    load_keys<D>(a, b, c, key0, kf);
    // keys this lane sees in the K*P^T layout: key0 + 32*s + 8*(i/4) + 4*(lane/32) + i%4
    uint32_t valid = 0;
    if (!FULL) {
#pragma unroll
        for (int s = 0; s < kSub; ++s)
#pragma unroll
            for (int i = 0; i < 16; ++i)
                valid |= (key0 + 32 * s + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3) < a.T) ? (1u << (16 * s + i)) : 0u;
    }

    const int n_tiles = a.rows_pad / 32;
    float2* part = a.part + (static_cast<int64_t>(head) * a.n_kb + kb) * a.rows_pad;
    auto merge = [&](int slot, int tile) {
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) M = fmaxf(M, mrg[slot][w][lane].x);
        float S = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < WAVES; ++w) S += mrg[slot][w][lane].y * exp2f(mrg[slot][w][lane].x - M);
        }
        part[32 * tile + lane] = make_float2(M, S);
    };

    Stager<D, WAVES> st0, st1;
    st0.load(a, b, c, 0);
    st0.store(stage[0]);
    if (n_tiles > 1) st1.load(a, b, c, 32);
    if (n_tiles > 2) st0.load(a, b, c, 64);
    __syncthreads();

    floatx16 acc[2][kSub];
    // tile t: staged in stage[t & 1] during iteration t-1; MFMA in iteration
    // t; column statistics in iteration t+1; merged over waves in t+2
    auto stage_next = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value;
        if (t + 1 < n_tiles) {
            if constexpr (cur == 0) st1.store(stage[1]); else st0.store(stage[0]);
            if (t + 3 < n_tiles) {
                if constexpr (cur == 0) st1.load(a, b, c, 32 * (t + 3)); else st0.load(a, b, c, 32 * (t + 3));
            }
        }
    };
    // iteration 0
    stage_next(Parity<0>{}, 0);
    tile_mfma<D, true>(stage[0], kf, acc[0], lane);
    __syncthreads();
    // steady state: MFMA of tile t next to the statistics of tile t-1
    auto body = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value, prev = cur ^ 1;
        stage_next(parity, t);
        tile_mfma<D, true>(stage[cur], kf, acc[cur], lane);
        const float2 r = column_lse<FULL>(acc[prev], valid, kappa);
        if (lane < 32) mrg[prev][wave][lane] = r;
        if (t >= 2 && wave == (t % WAVES) && lane < 32) merge(cur, t - 2);
        __syncthreads();
    };
    int t = 1;
    for (; t + 1 < n_tiles; t += 2) {
        body(Parity<1>{}, t);
        body(Parity<0>{}, t + 1);
    }
    if (t < n_tiles) {
        body(Parity<1>{}, t);
        ++t;
    }
    // t == n_tiles: statistics of the last tile, merges of the last two
    {
        const int last = n_tiles - 1;
        const int ps = last & 1;
        const float2 r = ps ? column_lse<FULL>(acc[1], valid, kappa) : column_lse<FULL>(acc[0], valid, kappa);
        if (lane < 32) mrg[ps][wave][lane] = r;
        if (n_tiles >= 2 && wave == 0 && lane < 32) merge(ps ^ 1, last - 1);
        __syncthreads();
        if (wave == 1 % WAVES && lane < 32) merge(ps, last);
    }
}

template <int D, int WAVES>
__global__ void __launch_bounds__(64 * WAVES) score_lse_kernel(ScoreArgs a) {
    __shared__ u32x4 stage[2][TileLds<D>::kSlots];
    __shared__ float2 mrg[2][WAVES][32];
    int head, kb;
    block_work(a.n_kb, head, kb);
    const int b = head / a.Hkv, c = head - b * a.Hkv;
    if ((kb + 1) * 64 * WAVES <= a.T)
        lse_body<D, WAVES, true>(a, head, kb, b, c, stage, mrg);
    else
        lse_body<D, WAVES, false>(a, head, kb, b, c, stage, mrg);
}

// L_row = M + log2(sum_kb S_kb * 2^(M_kb - M)), one thread per row.
__global__ void __launch_bounds__(256) lse_combine_kernel(ScoreArgs a) {
    const int r = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
    const int head = static_cast<int>(blockIdx.y);
    if (r >= a.rows_pad) return;
    const float2* p = a.part + static_cast<int64_t>(head) * a.n_kb * a.rows_pad + r;
    float M = -INFINITY, S = 0.f;
    for (int kb = 0; kb < a.n_kb; ++kb) {
        const float2 v = p[static_cast<int64_t>(kb) * a.rows_pad];
        if (v.x > M) {
            S = S * exp2f(M - v.x) + v.y;
            M = v.x;
        } else if (v.x != -INFINITY) {
            S += v.y * exp2f(v.x - M);
        }
    }
    a.lse[static_cast<int64_t>(head) * a.rows_pad + r] = M + log2f(S);
}

// ---------------------------------------------------------------- pass 2
// p = 2^(s*kappa - L) of one tile, summed over this lane's rows 0-15 (hA)
// and rows 16-31 (hB) of the tile; lrow = the tile's 32 L values in LDS.
__device__ __forceinline__ void tile_probs(const floatx16 (&acc)[kSub], const float* lrow, float kappa,
                                           int lane, float (&hA)[kSub], float (&hB)[kSub]) {
    float4 l4[4];
#pragma unroll
    for (int m4 = 0; m4 < 4; ++m4) l4[m4] = *reinterpret_cast<const float4*>(lrow + 8 * m4 + 4 * (lane >> 5));
#pragma unroll
    for (int s = 0; s < kSub; ++s) {
        float sa = 0.f, sb = 0.f;
#pragma unroll
        for (int m4 = 0; m4 < 4; ++m4) {
            const float e0 = fast_exp2(fmaf(acc[s][4 * m4 + 0], kappa, -l4[m4].x));
            const float e1 = fast_exp2(fmaf(acc[s][4 * m4 + 1], kappa, -l4[m4].y));
            const float e2 = fast_exp2(fmaf(acc[s][4 * m4 + 2], kappa, -l4[m4].z));
            const float e3 = fast_exp2(fmaf(acc[s][4 * m4 + 3], kappa, -l4[m4].w));
            if (m4 < 2) sa += (e0 + e1) + (e2 + e3); else sb += (e0 + e1) + (e2 + e3);
        }
        hA[s] = sa;
        hB[s] = sb;
    }
}

template <int D, int WAVES>
__global__ void __launch_bounds__(64 * WAVES) score_mass_kernel(ScoreArgs a) {
    __shared__ u32x4 stage[2][TileLds<D>::kSlots];
    __shared__ __align__(16) float lring[4][32];

    int head, kb;
    block_work(a.n_kb, head, kb);
    const int b = head / a.Hkv, c = head - b * a.Hkv;
    const int wave = static_cast<int>(threadIdx.x) / kWave, lane = lane_id();
    const int key0 = kb * 64 * WAVES + wave * kWaveKeys;
    const float kappa = a.kappa;
    const float* L = a.lse + static_cast<int64_t>(head) * a.rows_pad;

    bf16x8 kf[kSub][D / 16];
    load_keys<D>(a, b, c, key0, kf);

    const int g = a.P / a.G;                 // proxies per group, multiple of 16
    const int n_u = a.P / 32;
    const int n_prox_tiles = n_u * a.Gh;
    const int n_tiles = n_prox_tiles + (a.rows_pad - a.rows) / 32;
    // tile t < n_prox_tiles: proxies 32u.. of head h with u = t / Gh, h = t % Gh;
    // later tiles: anchor rows
    auto tile_row0 = [&](int t) -> int {
        if (t < n_prox_tiles) {
            const int u = t / a.Gh;
            return (t - u * a.Gh) * a.P + 32 * u;
        }
        return a.rows + 32 * (t - n_prox_tiles);
    };

    Stager<D, WAVES> st0, st1;
    float4 lg0 = make_float4(0.f, 0.f, 0.f, 0.f), lg1 = lg0;   // L staging, threads < 8
    const bool lthr = threadIdx.x < 8;
    auto load_l = [&](int t) {
        return *reinterpret_cast<const float4*>(L + tile_row0(t) + 4 * static_cast<int>(threadIdx.x));
    };
    auto store_l = [&](int t, float4 v) {
        *reinterpret_cast<float4*>(&lring[t & 3][4 * threadIdx.x]) = v;
    };
    st0.load(a, b, c, tile_row0(0));
    if (lthr) lg0 = load_l(0);
    st0.store(stage[0]);
    if (lthr) store_l(0, lg0);
    if (n_tiles > 1) {
        st1.load(a, b, c, tile_row0(1));
        if (lthr) lg1 = load_l(1);
    }
    if (n_tiles > 2) {
        st0.load(a, b, c, tile_row0(2));
        if (lthr) lg0 = load_l(2);
    }
    __syncthreads();

    const int64_t gm_base = static_cast<int64_t>(head) * a.G * a.T;
    const int my_key = key0 + lane;          // lanes < 32: sub-tile 0, lanes >= 32: sub-tile 1
    const bool my_ok = my_key < a.T;
    float runA[kSub] = {0.f, 0.f}, runB[kSub] = {0.f, 0.f}, open[kSub] = {0.f, 0.f};
    float macc[kSub] = {0.f, 0.f}, aacc[kSub] = {0.f, 0.f};
    // completes group `gi` for this wave's 64 key columns: sum the two
    // half-waves, add to the total mass, store, reset
    auto flush_group = [&](float (&o)[kSub], int gi) {
#pragma unroll
        for (int s = 0; s < kSub; ++s) {
            o[s] += shfl_xor_f(o[s], 32);
            macc[s] += o[s];
        }
        if (a.group_mass != nullptr && my_ok)
            a.group_mass[gm_base + static_cast<int64_t>(gi) * a.T + my_key] = (lane < 32) ? o[0] : o[1];
#pragma unroll
        for (int s = 0; s < kSub; ++s) o[s] = 0.f;
    };
    // rows 0-15 of tile (u, h) belong to proxy group (32u)/g, rows 16-31 to
    // (32u+16)/g; runA / runB sum each half over the Gh heads and `open`
    // carries a group that spans several tiles
    auto group_step = [&](int tp, const float (&hA)[kSub], const float (&hB)[kSub]) {
#pragma unroll
        for (int s = 0; s < kSub; ++s) {
            runA[s] += hA[s];
            runB[s] += hB[s];
        }
        const int u = tp / a.Gh;
        if (tp - u * a.Gh == a.Gh - 1) {
#pragma unroll
            for (int s = 0; s < kSub; ++s) {
                open[s] += runA[s];
                runA[s] = 0.f;
            }
            if (((32 * u + 16) % g) == 0) flush_group(open, (32 * u) / g);
#pragma unroll
            for (int s = 0; s < kSub; ++s) {
                open[s] += runB[s];
                runB[s] = 0.f;
            }
            if (((32 * u + 32) % g) == 0) flush_group(open, (32 * u + 16) / g);
        }
    };
    auto anchor_step = [&](int tp, const floatx16 (&ac)[kSub]) {
        // anchor rows of tile tp: query head 32*(tp - n_prox_tiles) + row
        const float* lrow = lring[tp & 3];
        const int h0 = 32 * (tp - n_prox_tiles) + 4 * (lane >> 5);
#pragma unroll
        for (int m4 = 0; m4 < 4; ++m4) {
            const float4 l4 = *reinterpret_cast<const float4*>(lrow + 8 * m4 + 4 * (lane >> 5));
            const float lj[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
            for (int s = 0; s < kSub; ++s)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float e = fast_exp2(fmaf(ac[s][4 * m4 + j], kappa, -lj[j]));
                    aacc[s] += (h0 + 8 * m4 + j < a.Gh) ? e : 0.f;
                }
        }
    };

    floatx16 acc[2][kSub];
    // tile t: staged during iteration t-1 (proxy rows in stage[t & 1], L
    // values in lring[t & 3]); MFMA in iteration t; probabilities in t+1
    auto stage_next = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value;
        if (t + 1 < n_tiles) {
            if constexpr (cur == 0) {
                st1.store(stage[1]);
                if (lthr) store_l(t + 1, lg1);
            } else {
                st0.store(stage[0]);
                if (lthr) store_l(t + 1, lg0);
            }
            if (t + 3 < n_tiles) {
                if constexpr (cur == 0) {
                    st1.load(a, b, c, tile_row0(t + 3));
                    if (lthr) lg1 = load_l(t + 3);
                } else {
                    st0.load(a, b, c, tile_row0(t + 3));
                    if (lthr) lg0 = load_l(t + 3);
                }
            }
        }
    };
    stage_next(Parity<0>{}, 0);
    tile_mfma<D, false>(stage[0], kf, acc[0], lane);
    __syncthreads();
    // steady state over proxy tiles: MFMA of tile t next to the
    // probabilities of tile t-1 (the last of these MFMAs may be an anchor tile)
    auto body = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value, prev = cur ^ 1;
        stage_next(parity, t);
        tile_mfma<D, false>(stage[cur], kf, acc[cur], lane);
        float hA[kSub], hB[kSub];
        tile_probs(acc[prev], lring[(t - 1) & 3], kappa, lane, hA, hB);
        group_step(t - 1, hA, hB);
        __syncthreads();
    };
    int t = 1;
    for (; t + 1 <= n_prox_tiles; t += 2) {
        body(Parity<1>{}, t);
        body(Parity<0>{}, t + 1);
    }
    if (t <= n_prox_tiles) {
        body(Parity<1>{}, t);
        ++t;
    }
    // anchor tiles (t - 1 >= n_prox_tiles)
    auto anchor_body = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value, prev = cur ^ 1;
        if (t < n_tiles) {
            stage_next(parity, t);
            tile_mfma<D, false>(stage[cur], kf, acc[cur], lane);
        }
        anchor_step(t - 1, acc[prev]);
        __syncthreads();
    };
    for (; t <= n_tiles; ++t) {
        if (t & 1) anchor_body(Parity<1>{}, t); else anchor_body(Parity<0>{}, t);
    }
    const float inv_gh = 1.0f / static_cast<float>(a.Gh);
#pragma unroll
    for (int s = 0; s < kSub; ++s) aacc[s] = (aacc[s] + shfl_xor_f(aacc[s], 32)) * inv_gh;
    if (my_ok) {
        const int64_t o = static_cast<int64_t>(head) * a.T + my_key;
        a.mass[o] = (lane < 32) ? macc[0] : macc[1];
        a.anchor[o] = (lane < 32) ? aacc[0] : aacc[1];
    }
}

template <int D, int WAVES>
hipError_t lse_impl(const ScoreArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((score_lse_kernel<D, WAVES>), dim3(a.B * a.Hkv * a.n_kb), dim3(64 * WAVES), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((a.rows_pad + 255) / 256, a.B * a.Hkv);
    hipLaunchKernelGGL(lse_combine_kernel, g2, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int D, int WAVES>
hipError_t mass_impl(const ScoreArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((score_mass_kernel<D, WAVES>), dim3(a.B * a.Hkv * a.n_kb), dim3(64 * WAVES), 0, s, a);
    return hipGetLastError();
}

}  // namespace

int score_block_waves(int B, int Hkv, int T) {
    // 8-wave blocks (512 keys) when that still gives every CU two blocks of
    // work, else 4-wave blocks (256 keys)
    const long blocks8 = static_cast<long>(B) * Hkv * ((T + 511) / 512);
    return blocks8 >= 512 ? 8 : 4;
}

hipError_t launch_score_lse(const ScoreArgs& a, hipStream_t s) {
    const int w = a.block_keys / 64;
    if (a.d == 64) return w == 8 ? lse_impl<64, 8>(a, s) : lse_impl<64, 4>(a, s);
    return w == 8 ? lse_impl<128, 8>(a, s) : lse_impl<128, 4>(a, s);
}

hipError_t launch_score_mass(const ScoreArgs& a, hipStream_t s) {
    const int w = a.block_keys / 64;
    if (a.d == 64) return w == 8 ? mass_impl<64, 8>(a, s) : mass_impl<64, 4>(a, s);
    return w == 8 ? mass_impl<128, 8>(a, s) : mass_impl<128, 4>(a, s);
}

}  // namespace mmskv
