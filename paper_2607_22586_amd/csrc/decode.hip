// Decode-time check on gfx950: the attention-mass coverage of Fig. 1b (the
// share of a decoding query's softmax mass over all prompt keys that falls
// on the keys kept after prefilling) and decode attention over the fixed
// compacted cache (Sec. 3.1's prefill-only protocol).
//
// Coverage: one workgroup of 4 waves per (b, c, block of 256 keys), each wave
// holding 64 keys in registers.  The Gh * n_dec decode queries of KV head c,
// scaled once like the anchor query (log2(e)/sqrt(d) in fp64, then fp32,
// then bf16), are staged in LDS and streamed past the keys in 32-row tiles
// with v_mfma_f32_32x32x16_bf16 in the K * Q^T layout (lane = query row, its
// 32 values = its keys), so a row's block statistics are in-lane sums.  Per
// (row, block) the kernel writes (m, sum of 2^(s - m) over all keys, the same
// over the kept keys).  The keys are read once: the pass is bound by HBM
// reads of K and by the exps.
//
// Compacted attention, bf16 cache: one workgroup of 4 waves per (b, c, 32
// decode rows) on the matrix cores (S = K' Q^T, then O = P V' with P split
// into two bf16 parts), which also merges the coverage partials of its rows.
// fp32 cache: a merge kernel, then one wave per decode query with fp32
// products on the VALU (a few hundred keys).
#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kDecWaves = 4;
constexpr int kDecSub = 1;                 // 64-key sub-blocks per wave, loaded together
constexpr int kDecKeys = 64 * kDecWaves * kDecSub;   // keys per workgroup
constexpr int kDecMaxRows = 256;           // Gh * n_dec, padded to 32
constexpr int kDecMaxCompact = 2048;       // rows of the compacted cache (c_max)

__device__ __forceinline__ floatx16 mfma_32x32x16(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx16 zero16() {
    floatx16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

__device__ __forceinline__ float pair_max2(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// the value of lane l ^ 32 (the swap leaves lane l < 32's own value in the
// first result and its partner's in the second, and the reverse for l >= 32)
__device__ __forceinline__ float pair_other(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(lane_id() < 32 ? r[1] : r[0]);
}

__device__ __forceinline__ float pair_sum2(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// bf16 bits of v * scale (fp64 product, rounded to fp32, then to bf16)
__device__ __forceinline__ uint32_t scaled_bf16(uint32_t bits16, double scale) {
    const double v = static_cast<double>(__uint_as_float(bits16 << 16)) * scale;
    return f32_to_bf16_bits(static_cast<float>(v));
}

// the decode queries of each KV head scaled once, in the coverage kernel's
// row order (row r = head c*Gh + r / n_dec, query r % n_dec; rows past
// Gh * n_dec zero): qsc [B*Hkv, rows_pad, d] bf16; one 16-byte chunk per thread
__global__ void __launch_bounds__(256) decode_scale_kernel(DecodeArgs a) {
    const int chunks = a.d / 8;
    const int i = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
    const int bc = blockIdx.y;
    if (i >= a.rows_pad * chunks) return;
    const int r = i / chunks, ch = i - r * chunks;
    const int b = bc / a.Hkv, c = bc - b * a.Hkv;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < a.rows) {
        const int h = c * a.Gh + r / a.n_dec, j = r - (r / a.n_dec) * a.n_dec;
        const u32x4 raw = *reinterpret_cast<const u32x4*>(
            a.q_dec + ((static_cast<int64_t>(b) * a.Hq + h) * a.n_dec + j) * a.d + 8 * ch);
#pragma unroll
        for (int w = 0; w < 4; ++w)
            v[w] = scaled_bf16(raw[w] & 0xFFFFu, a.scale) | (scaled_bf16(raw[w] >> 16, a.scale) << 16);
    }
    *reinterpret_cast<u32x4*>(a.qsc + (static_cast<int64_t>(bc) * a.rows_pad + r) * a.d + 8 * ch) = v;
}

// One key block of the coverage pass; FULL: every key of the block is < T.
template <int D, bool FULL>
__device__ __forceinline__ void cover_block(const DecodeArgs& a, int kb, int bc, u32x4* qs,
                                            const uint32_t* kept, float4 (*part)[kDecMaxRows],
                                            bf16x8 (&kfs)[kDecSub][2][D / 16]) {
    constexpr int KC = D / 16;                 // 16-element k steps
    constexpr int kRow = D / 8 + 1;            // LDS row in 16-byte chunks (one pad chunk)
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int key_base = kb * kDecKeys;
#pragma unroll
    for (int sb = 0; sb < kDecSub; ++sb) {
        const int key0 = key_base + 256 * sb + 64 * wave;
        const bf16x8 (&kf)[2][KC] = kfs[sb];
        // value i of sub-tile s of this lane is key key0 + 32 s + 8 (i / 4) + 4 (lane / 32) + i % 4;
        // bit 16 s + i of valid / keep: that key is below T / kept
        uint32_t valid = 0xFFFFFFFFu, keep = 0u;
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int t = key0 + 32 * s + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
                const int tl = t - key_base;
                const bool ok = FULL || t < a.T;
                if (!FULL && !ok) valid &= ~(1u << (16 * s + i));
                if (ok && ((kept[tl >> 5] >> (tl & 31)) & 1u)) keep |= 1u << (16 * s + i);
            }
        // (key0 is the same in every lane: the MFMAs and lane swaps below run in
        // whole waves)
        if (!FULL && key0 >= a.T) continue;
        // most 32-key sub-tiles hold no kept key: their kept sums are skipped
        const bool kept0 = __ballot((keep & 0xFFFFu) != 0u) != 0, kept1 = __ballot((keep >> 16) != 0u) != 0;
        // the kept sum as one fused multiply-add per value with a 0 / 1 factor
        auto kmul = [&](int j) { return static_cast<float>((keep >> j) & 1u); };
        for (int r0 = 0; r0 < a.rows_pad; r0 += 32) {
            // opaque per row tile, so that the 0 / 1 factors are formed where
            // they are used instead of being kept in 32 registers
            asm volatile("" : "+v"(keep));
            floatx16 acc[2];
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const bf16x8 q = __builtin_bit_cast(bf16x8, qs[(r0 + (lane & 31)) * kRow + 2 * kc + (lane >> 5)]);
#pragma unroll
                for (int s = 0; s < 2; ++s) acc[s] = mfma_32x32x16(kf[s][kc], q, kc == 0 ? zero16() : acc[s]);
            }
            // sums of 2^s relative to 0 while every lane's sum is in
            // [2^-60, lane_sum_limit(T, 32)) (as in the row log-sum-exp pass),
            // else relative to the exact per-column maximum
            float mx = 0.f, la = -0.f, lk = -0.f;
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float e = (FULL || ((valid >> (16 * s + i)) & 1u)) ? fast_exp2(acc[s][i]) : 0.f;
                    acc[s][i] = e;
                    la += e;
                }
            if (kept0) {
#pragma unroll
                for (int i = 0; i < 16; ++i) lk = fmaf(acc[0][i], kmul(i), lk);
            }
            if (kept1) {
#pragma unroll
                for (int i = 0; i < 16; ++i) lk = fmaf(acc[1][i], kmul(16 + i), lk);
            }
            const bool in_range = (la >= 0x1p-60f || (!FULL && valid == 0u)) && la < a.lane_sum_hi;
            if (__ballot(!in_range) != 0) {
                // the logits again (the exps above replaced them) for the exact form
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) {
                    const bf16x8 q = __builtin_bit_cast(bf16x8, qs[(r0 + (lane & 31)) * kRow + 2 * kc + (lane >> 5)]);
#pragma unroll
                    for (int s = 0; s < 2; ++s) acc[s] = mfma_32x32x16(kf[s][kc], q, kc == 0 ? zero16() : acc[s]);
                }
                mx = -INFINITY;
#pragma unroll
                for (int s = 0; s < 2; ++s)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (FULL || ((valid >> (16 * s + i)) & 1u)) mx = fmaxf(mx, acc[s][i]);
                mx = pair_max2(mx);
                la = 0.f;
                lk = 0.f;
                if (mx != -INFINITY) {
#pragma unroll
                    for (int s = 0; s < 2; ++s)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const float e = (FULL || ((valid >> (16 * s + i)) & 1u)) ? fast_exp2(acc[s][i] - mx) : 0.f;
                            la += e;
                            lk = fmaf(e, kmul(16 * s + i), lk);
                        }
                }
            }
            la = pair_sum2(la);
            lk = pair_sum2(lk);
            if (lane < 32 && la > 0.f) {
                const float4 o = part[wave][r0 + lane];
                const float M = fmaxf(o.x, mx);
                const float fo = o.x == -INFINITY ? 0.f : fast_exp2(o.x - M), fn = fast_exp2(mx - M);
                part[wave][r0 + lane] = make_float4(M, o.y * fo + la * fn, o.z * fo + lk * fn, 0.f);
            }
        }
    }
}

template <int D>
__global__ void __launch_bounds__(64 * kDecWaves, 2) decode_cover_kernel(DecodeArgs a) {
    constexpr int KC = D / 16;                 // 16-element k steps
    constexpr int kRow = D / 8 + 1;            // LDS row in 16-byte chunks (one pad chunk)
    extern __shared__ u32x4 qs[];              // [rows_pad * kRow]
    __shared__ uint32_t kept[kDecKeys / 32];
    __shared__ float4 part[kDecWaves][kDecMaxRows];

    const int kb = blockIdx.x, bc = blockIdx.y;
    const int b = bc / a.Hkv, c = bc - b * a.Hkv;
    const int tid = threadIdx.x, wave = tid / kWave, lane = lane_id();
    const int key_base = kb * kDecKeys;
    constexpr int kThreads = 64 * kDecWaves;

    // Every global load of the prologue is issued before the first wait: the
    // head's scaled queries (decode_scale_kernel; L2-resident), the kept
    // indices, then the block's keys (HBM).  Indices are clamped instead of
    // branched on, so nothing serialises the loads.
    // (query chunks in rounds of kQPer per thread: one round up to 128 rows at d = 128)
    constexpr int kQPer = 8;
    const int nq = a.rows_pad * (D / 8);
    const u32x4* qsrc = reinterpret_cast<const u32x4*>(a.qsc + static_cast<int64_t>(bc) * a.rows_pad * D);
    u32x4 qv[kQPer];
#pragma unroll
    for (int j = 0; j < kQPer; ++j) qv[j] = qsrc[min(tid + kThreads * j, nq - 1)];
    constexpr int kIdxPer = kDecMaxCompact / kThreads;
    const int n_kept = min(max(a.counts[bc], 0), a.c_max);
    const int32_t* ids = a.idx + static_cast<int64_t>(bc) * a.c_max;
    int32_t iv[kIdxPer];
#pragma unroll
    for (int j = 0; j < kIdxPer; ++j) iv[j] = ids[min(tid + kThreads * j, a.c_max - 1)];

    // the wave's sub-block sb holds keys key_base + 256 sb + 64 wave + [0, 64):
    // kf[s][kc] = key key0 + 32 s + lane % 32, dims 16 kc + 8 (lane / 32) ..
    // A key past T reads key T - 1 instead (unconditional loads, issued
    // together); its values are masked out of every sum.
    bf16x8 kfs[kDecSub][2][KC];
    auto load_keys = [&](bf16x8 (&kf)[2][KC], int key0) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int t = min(key0 + 32 * s + (lane & 31), a.T - 1);
            const int64_t off = static_cast<int64_t>(b) * a.ksb + static_cast<int64_t>(c) * a.ksh +
                                static_cast<int64_t>(t) * a.kst + 8 * (lane >> 5);
            if (a.k_dtype == 1) {
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) kf[s][kc] = load_bf16x8(static_cast<const uint16_t*>(a.k) + off + 16 * kc);
            } else {
#pragma unroll
                for (int kc = 0; kc < KC; ++kc) kf[s][kc] = load_f32_as_bf16x8(static_cast<const float*>(a.k) + off + 16 * kc);
            }
        }
    };
#pragma unroll
    for (int sb = 0; sb < kDecSub; ++sb) load_keys(kfs[sb], key_base + 256 * sb + 64 * wave);

    // queries to LDS, kept flags cleared, per (wave, row) running (m, sum
    // all, sum kept) reset; then the kept flags of this block's keys (idx is
    // any list of in-range indices)
    for (int i0 = 0; i0 < nq; i0 += kThreads * kQPer) {
        if (i0 > 0) {
#pragma unroll
            for (int j = 0; j < kQPer; ++j) qv[j] = qsrc[min(i0 + tid + kThreads * j, nq - 1)];
        }
#pragma unroll
        for (int j = 0; j < kQPer; ++j) {
            const int i = i0 + tid + kThreads * j;
            if (i < nq) {
                const int r = i / (D / 8), ch = i - r * (D / 8);
                qs[r * kRow + ch] = qv[j];
            }
        }
    }
    if (tid < kDecKeys / 32) kept[tid] = 0u;
    for (int r = lane; r < a.rows_pad; r += kWave) part[wave][r] = make_float4(-INFINITY, 0.f, 0.f, 0.f);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kIdxPer; ++j) {
        const int t = iv[j] - key_base;
        if (tid + kThreads * j < n_kept && t >= 0 && t < kDecKeys && t + key_base < a.T)
            atomicOr(&kept[t >> 5], 1u << (t & 31));
    }
    __syncthreads();
    if (key_base + kDecKeys <= a.T)
        cover_block<D, true>(a, kb, bc, qs, kept, part, kfs);
    else
        cover_block<D, false>(a, kb, bc, qs, kept, part, kfs);
    __syncthreads();
    // merge the 4 waves: one thread per row
    for (int r = tid; r < a.rows_pad; r += 64 * kDecWaves) {
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, part[w][r].x);
        float sa = 0.f, sk = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kDecWaves; ++w) {
                const float f = fast_exp2(part[w][r].x - M);
                sa += part[w][r].y * f;
                sk += part[w][r].z * f;
            }
        }
        a.part[(static_cast<int64_t>(bc) * a.n_kb + kb) * a.rows_pad + r] = make_float4(M, sa, sk, 0.f);
    }
}

// coverage = (sum over blocks of the kept sums) / (sum of all sums), both
// rescaled to the row's largest block maximum; one wave per row, lanes over
// the key blocks
__global__ void __launch_bounds__(256) decode_cover_combine_kernel(DecodeArgs a) {
    const int lane = lane_id();
    const int r = static_cast<int>(blockIdx.x) * 4 + static_cast<int>(threadIdx.x) / kWave;
    const int bc = blockIdx.y;
    if (r >= a.rows) return;                                           // wave-uniform
    const float4* p = a.part + static_cast<int64_t>(bc) * a.n_kb * a.rows_pad + r;
    float M = -INFINITY;
    for (int kb = lane; kb < a.n_kb; kb += kWave) M = fmaxf(M, p[static_cast<int64_t>(kb) * a.rows_pad].x);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    float sa = 0.f, sk = 0.f;
    for (int kb = lane; kb < a.n_kb; kb += kWave) {
        const float4 v = p[static_cast<int64_t>(kb) * a.rows_pad];
        if (v.x != -INFINITY) {
            const float f = exp2f(v.x - M);
            sa += v.y * f;
            sk += v.z * f;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        sa += __shfl_xor(sa, o);
        sk += __shfl_xor(sk, o);
    }
    if (lane == 0) {
        const int b = bc / a.Hkv, c = bc - b * a.Hkv;
        const int h = c * a.Gh + r / a.n_dec, j = r - (r / a.n_dec) * a.n_dec;
        a.coverage[(static_cast<int64_t>(b) * a.Hq + h) * a.n_dec + j] = sk / sa;
    }
}

// bf16 bits of two fp32 values, round to nearest even, packed (lo, hi)
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// decode attention over a bf16 compacted cache on the matrix cores: one
// workgroup of 4 waves per (b, c, 32 decode rows of KV head c), walking the
// counts[b, c] cached keys in chunks of 256, 64 per wave.  Per chunk, wave w:
//   S = K'_w Q^T (keys as MFMA rows, so lane l % 32 is decode row l % 32 and
//   its 32 values are the wave's keys); the chunk's row maxima merged over
//   the waves through LDS into the running maximum M; p = 2^(s - M), the
//   earlier partial output and sum rescaled by 2^(M_old - M);
//   O_w += P V'_w, with P as the MFMA's A operand straight from the S
//   registers (value i of 16-key step kk holds key 16 kk + 8 (j / 4) +
//   4 (l / 32) + j % 4, j = i - 8 kk, and V' is read in the same key order)
//   split into two bf16 parts p = hi + lo so that the weights keep ~16 bits,
//   V' staged in LDS (one 16-byte-padded row per key) and read as 2-byte
//   columns.
// At the end the waves' partial outputs and sums are added through LDS and
// divided.  fp32 accumulation throughout; the scaled queries are
// decode_scale_kernel's.
template <int D>
__global__ void __launch_bounds__(64 * kDecWaves) decode_attend_mfma_kernel(DecodeArgs a) {
    constexpr int KC = D / 16;                     // 16-dim k steps of S
    constexpr int NT = D / 32;                     // 32-dim output tiles
    constexpr int kVRow = D + 8;                   // staged V' row, bf16 elements (16-byte pad)
    constexpr int kWaveV = 64 * kVRow;             // a wave's staged rows (bf16 elements)
    static_assert(32 * D * 4 <= kWaveV * 2, "a wave's partial output fits its staging area");
    __shared__ u32x4 vstage[kDecWaves * kWaveV / 8];
    __shared__ float mx_w[kDecWaves][32];
    __shared__ float l_w[kDecWaves][32];
    __shared__ __align__(16) float fac_s[32];
    __shared__ float4 cov_w[kDecWaves][32];
    const int tile = blockIdx.x, bc = blockIdx.y;
    const int b = bc / a.Hkv, c = bc - b * a.Hkv;
    const int tid = threadIdx.x, wave = tid / kWave, lane = lane_id();
    const int h = lane >> 5, l32 = lane & 31;
    const int n = min(max(a.counts[bc], 0), a.c_max);
    const uint16_t* kc_base = static_cast<const uint16_t*>(a.k_out) + static_cast<int64_t>(bc) * a.c_max * D;
    const uint16_t* vc_base = static_cast<const uint16_t*>(a.v_out) + static_cast<int64_t>(bc) * a.c_max * D;
    uint16_t* vw = reinterpret_cast<uint16_t*>(vstage) + wave * kWaveV;

    // coverage of the tile's rows, the merge of the coverage kernel's per-key-
    // block partials (m, sum all, sum kept): thread t takes row t % 32 and key
    // blocks t / 32 + 8 j; its first 8 partials are fetched here, with the
    // other loads, and merged at the end
    constexpr int kCovPer = 8;
    const int cr = tid & 31, cg = tid >> 5;
    const float4* pp = a.part + static_cast<int64_t>(bc) * a.n_kb * a.rows_pad + 32 * tile + cr;
    float4 pv[kCovPer];
#pragma unroll
    for (int j = 0; j < kCovPer; ++j) pv[j] = pp[static_cast<int64_t>(min(cg + 8 * j, a.n_kb - 1)) * a.rows_pad];
    // query fragments: decode row 32 tile + l32, dims 16 kc + 8 h ..
    bf16x8 qf[KC];
    {
        const uint16_t* qrow = a.qsc + (static_cast<int64_t>(bc) * a.rows_pad + 32 * tile + l32) * D + 8 * h;
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) qf[kc] = load_bf16x8(qrow + 16 * kc);
    }
    floatx16 o[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) o[t] = zero16();
    float M = -INFINITY, lsum = 0.f;               // running maximum and partial sum of row l32

    for (int k0 = 0; k0 < n; k0 += 64 * kDecWaves) {
        const int kw = k0 + 64 * wave;             // the wave's first key (same in every lane)
        // the wave's K' fragments (keys kw + 32 s + l32 as rows, dims 16 kc +
        // 8 h) and V' rows (16-byte chunk q of its 64 x D/8), all loads issued
        // together; a key at or past n reads row n - 1 instead (its weight is 0)
        bf16x8 kf[2][KC];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            const uint16_t* kr = kc_base + static_cast<int64_t>(min(kw + 32 * s2 + l32, n - 1)) * D + 8 * h;
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) kf[s2][kc] = load_bf16x8(kr + 16 * kc);
        }
        u32x4 vst[D / 8];
#pragma unroll
        for (int j = 0; j < D / 8; ++j) {
            const int q = lane + kWave * j, r = q / (D / 8), ch = q - r * (D / 8);
            vst[j] = *reinterpret_cast<const u32x4*>(vc_base + static_cast<int64_t>(min(kw + r, n - 1)) * D + 8 * ch);
        }
        floatx16 sv[2];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) sv[s2] = mfma_32x32x16(kf[s2][kc], qf[kc], kc == 0 ? zero16() : sv[s2]);
#pragma unroll
        for (int j = 0; j < D / 8; ++j) {
            const int q = lane + kWave * j, r = q / (D / 8), ch = q - r * (D / 8);
            *reinterpret_cast<u32x4*>(vw + r * kVRow + 8 * ch) = vst[j];
        }
        // keys past n drop out; the wave's row maxima
        float mloc = -INFINITY;
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = kw + 32 * s2 + 8 * (i >> 2) + 4 * h + (i & 3);
                if (key >= n) sv[s2][i] = -INFINITY;
                mloc = fmaxf(mloc, sv[s2][i]);
            }
        mloc = pair_max2(mloc);
        if (lane < 32) mx_w[wave][lane] = mloc;
        __syncthreads();
        float mc = mx_w[0][l32];
#pragma unroll
        for (int w = 1; w < kDecWaves; ++w) mc = fmaxf(mc, mx_w[w][l32]);
        const float Mn = fmaxf(M, mc);             // finite: key k0 < n is in this chunk
        const float fac = M == -INFINITY ? 0.f : fast_exp2(M - Mn);
        M = Mn;
        if (wave == 0 && lane < 32) fac_s[lane] = fac;
        float ps = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = fast_exp2(sv[s2][i] - Mn);
                sv[s2][i] = p;
                ps += p;
            }
        lsum = lsum * fac + ps;
        __syncthreads();
        if (k0 > 0) {
            // rows 8 m4 + 4 h + j of the output values
#pragma unroll
            for (int m4 = 0; m4 < 4; ++m4) {
                const float4 f = *reinterpret_cast<const float4*>(fac_s + 8 * m4 + 4 * h);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    o[t][4 * m4 + 0] *= f.x;
                    o[t][4 * m4 + 1] *= f.y;
                    o[t][4 * m4 + 2] *= f.z;
                    o[t][4 * m4 + 3] *= f.w;
                }
            }
        }
        // O += P V': 16-key steps (s2, kk)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                u32x4 hi, lo;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const float p0 = sv[s2][8 * kk + 2 * w], p1 = sv[s2][8 * kk + 2 * w + 1];
                    const uint32_t hb = pack_bf16(p0, p1);
                    hi[w] = hb;
                    lo[w] = pack_bf16(p0 - __uint_as_float(hb << 16), p1 - __uint_as_float(hb & 0xFFFF0000u));
                }
                const bf16x8 ph = __builtin_bit_cast(bf16x8, hi), pl = __builtin_bit_cast(bf16x8, lo);
                // this lane's 8 keys of the step, in the A operand's order
                const int rbase = 32 * s2 + 16 * kk + 4 * h;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const uint16_t* col = vw + 32 * t + l32;
                    u32x4 vv;
#pragma unroll
                    for (int w = 0; w < 4; ++w) {
                        const int j0 = 2 * w, j1 = 2 * w + 1;
                        const int r0 = rbase + 8 * (j0 >> 2) + (j0 & 3), r1 = rbase + 8 * (j1 >> 2) + (j1 & 3);
                        vv[w] = static_cast<uint32_t>(col[r0 * kVRow]) | (static_cast<uint32_t>(col[r1 * kVRow]) << 16);
                    }
                    const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
                    o[t] = mfma_32x32x16(ph, vf, o[t]);
                    o[t] = mfma_32x32x16(pl, vf, o[t]);
                }
            }
    }
    // the waves' partial outputs and sums, added through LDS
    const float L = pair_sum2(lsum);
    __syncthreads();                               // every wave is done with its staged rows
    float* ob = reinterpret_cast<float*>(vw);      // [32 rows][D] of this wave
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) ob[(8 * (i >> 2) + 4 * h + (i & 3)) * D + 32 * t + l32] = o[t][i];
    if (lane < 32) l_w[wave][lane] = L;
    __syncthreads();
    // thread tid: row tid / 8, dims [D/8 * (tid % 8), +D/8)
    constexpr int kDims = D / 8;
    const int r = tid >> 3, d0 = kDims * (tid & 7);
    const int row = 32 * tile + r;
    if (row < a.rows) {
        float tot = 0.f;
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) tot += l_w[w][r];
        const float inv = tot > 0.f ? 1.f / tot : 0.f;
        const int hq = c * a.Gh + row / a.n_dec, jq = row - (row / a.n_dec) * a.n_dec;
        float* dst = a.out + ((static_cast<int64_t>(b) * a.Hq + hq) * a.n_dec + jq) * D + d0;
#pragma unroll
        for (int e = 0; e < kDims; e += 4) {
            float4 acc4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int w = 0; w < kDecWaves; ++w) {
                const float4 v = *reinterpret_cast<const float4*>(
                    reinterpret_cast<const float*>(vstage) + w * (kWaveV / 2) + r * D + d0 + e);
                acc4.x += v.x; acc4.y += v.y; acc4.z += v.z; acc4.w += v.w;
            }
            *reinterpret_cast<float4*>(dst + e) = make_float4(acc4.x * inv, acc4.y * inv, acc4.z * inv, acc4.w * inv);
        }
    }
    // coverage = (kept sums) / (all sums), both rescaled to the row's largest
    // block maximum: merged in the thread, over the lane pair l, l ^ 32, then
    // over the waves through LDS
    {
        float m = -INFINITY, sa = 0.f, sk = 0.f;
        auto merge = [&](float vm, float va, float vk) {
            if (vm == -INFINITY) return;
            const float mn = fmaxf(m, vm);
            const float fo = m == -INFINITY ? 0.f : exp2f(m - mn), fv = exp2f(vm - mn);
            sa = sa * fo + va * fv;
            sk = sk * fo + vk * fv;
            m = mn;
        };
        for (int kb0 = 0; kb0 < a.n_kb; kb0 += 8 * kCovPer) {
            if (kb0 > 0) {
#pragma unroll
                for (int j = 0; j < kCovPer; ++j)
                    pv[j] = pp[static_cast<int64_t>(min(kb0 + cg + 8 * j, a.n_kb - 1)) * a.rows_pad];
            }
#pragma unroll
            for (int j = 0; j < kCovPer; ++j)
                if (kb0 + cg + 8 * j < a.n_kb) merge(pv[j].x, pv[j].y, pv[j].z);
        }
        {
            const float om = pair_other(m), oa = pair_other(sa), ok = pair_other(sk);
            merge(om, oa, ok);
        }
        if (lane < 32) cov_w[wave][lane] = make_float4(m, sa, sk, 0.f);
        __syncthreads();
        if (tid < 32) {
            m = -INFINITY;
            sa = 0.f;
            sk = 0.f;
#pragma unroll
            for (int w = 0; w < kDecWaves; ++w) merge(cov_w[w][tid].x, cov_w[w][tid].y, cov_w[w][tid].z);
            const int row = 32 * tile + tid;
            if (row < a.rows) {
                const int hq = c * a.Gh + row / a.n_dec, jq = row - (row / a.n_dec) * a.n_dec;
                a.coverage[(static_cast<int64_t>(b) * a.Hq + hq) * a.n_dec + jq] = sk / sa;
            }
        }
    }
}

// decode attention over an fp32 compacted cache: one wave per decode query.
// Logits: lane i takes keys i, i + 64, ..., with the whole scaled query in
// registers and the key row in 16-byte loads.  Output: lane 16 g + u adds
// keys g, g + 4, ... on dims [8u, 8u + 8) (16-byte loads of v'), then the
// four key groups are summed across lanes.
template <int D>
__global__ void __launch_bounds__(256) decode_attend_kernel(DecodeArgs a) {
    constexpr int kChunks = D / 8;                 // 16-byte bf16 chunks of a row
    constexpr int kGroups = kWave / kChunks;       // keys in flight in the output loop
    __shared__ float wsh[4][kDecMaxCompact];
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wave;   // (b, h, j)
    const int64_t n_rows = static_cast<int64_t>(a.B) * a.Hq * a.n_dec;
    if (row >= n_rows) return;                                          // wave-uniform
    const int h = static_cast<int>((row / a.n_dec) % a.Hq);
    const int b = static_cast<int>(row / (static_cast<int64_t>(a.Hq) * a.n_dec));
    const int64_t bc = static_cast<int64_t>(b) * a.Hkv + h / a.Gh;
    const int n = min(max(a.counts[bc], 0), a.c_max);
    // the scaled query (decode_scale_kernel's row (h % Gh) * n_dec + j of KV
    // head bc), fp32 values of its bf16 bits, in every lane
    const int jq = static_cast<int>(row % a.n_dec);
    const uint16_t* qrow = a.qsc + (bc * a.rows_pad + (h % a.Gh) * a.n_dec + jq) * D;
    float q[D];
#pragma unroll
    for (int c8 = 0; c8 < kChunks; ++c8) {
        const u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 8 * c8);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            q[8 * c8 + 2 * w] = __uint_as_float(raw[w] << 16);
            q[8 * c8 + 2 * w + 1] = __uint_as_float(raw[w] & 0xFFFF0000u);
        }
    }
    float mx = -INFINITY;
    for (int i = lane; i < n; i += kWave) {
        const int64_t kr = (bc * a.c_max + i) * D;
        float dot = 0.f;
#pragma unroll
        for (int c8 = 0; c8 < kChunks; ++c8) {
            const bf16x8 kv = a.k_dtype == 1 ? load_bf16x8(static_cast<const uint16_t*>(a.k_out) + kr + 8 * c8)
                                             : load_f32_as_bf16x8(static_cast<const float*>(a.k_out) + kr + 8 * c8);
            const u32x4 kb = __builtin_bit_cast(u32x4, kv);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                dot = fmaf(q[8 * c8 + 2 * w], __uint_as_float(kb[w] << 16), dot);
                dot = fmaf(q[8 * c8 + 2 * w + 1], __uint_as_float(kb[w] & 0xFFFF0000u), dot);
            }
        }
        wsh[wave][i] = dot;
        mx = fmaxf(mx, dot);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    float sum = 0.f;
    for (int i = lane; i < n; i += kWave) {
        const float e = fast_exp2(wsh[wave][i] - mx);
        wsh[wave][i] = e;
        sum += e;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
    __builtin_amdgcn_wave_barrier();
    const int g = lane / kChunks, u = lane - g * kChunks;
    float o8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o8[e] = 0.f;
    // kUnroll keys per lane group in flight
    constexpr int kUnroll = 8;
    for (int i0 = g; i0 < n; i0 += kGroups * kUnroll) {
        if (a.k_dtype == 1) {
            u32x4 v[kUnroll];
#pragma unroll
            for (int m = 0; m < kUnroll; ++m) {
                const int i = i0 + kGroups * m;
                v[m] = i < n ? *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v_out) +
                                                                (bc * a.c_max + i) * D + 8 * u)
                             : u32x4{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int m = 0; m < kUnroll; ++m) {
                const int i = i0 + kGroups * m;
                const float w = i < n ? wsh[wave][i] : 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    o8[2 * e] = fmaf(w, __uint_as_float(v[m][e] << 16), o8[2 * e]);
                    o8[2 * e + 1] = fmaf(w, __uint_as_float(v[m][e] & 0xFFFF0000u), o8[2 * e + 1]);
                }
            }
        } else {
            float4 v[kUnroll][2];
#pragma unroll
            for (int m = 0; m < kUnroll; ++m) {
                const int i = i0 + kGroups * m;
                const float* vp = static_cast<const float*>(a.v_out) + (bc * a.c_max + (i < n ? i : 0)) * D + 8 * u;
                v[m][0] = *reinterpret_cast<const float4*>(vp);
                v[m][1] = *reinterpret_cast<const float4*>(vp + 4);
            }
#pragma unroll
            for (int m = 0; m < kUnroll; ++m) {
                const int i = i0 + kGroups * m;
                const float w = i < n ? wsh[wave][i] : 0.f;
                o8[0] = fmaf(w, v[m][0].x, o8[0]); o8[1] = fmaf(w, v[m][0].y, o8[1]);
                o8[2] = fmaf(w, v[m][0].z, o8[2]); o8[3] = fmaf(w, v[m][0].w, o8[3]);
                o8[4] = fmaf(w, v[m][1].x, o8[4]); o8[5] = fmaf(w, v[m][1].y, o8[5]);
                o8[6] = fmaf(w, v[m][1].z, o8[6]); o8[7] = fmaf(w, v[m][1].w, o8[7]);
            }
        }
    }
    // sum the key groups: lanes u, u + kChunks, ... hold the same dims
#pragma unroll
    for (int o = kChunks; o < kWave; o <<= 1)
#pragma unroll
        for (int e = 0; e < 8; ++e) o8[e] += __shfl_xor(o8[e], o);
    if (g == 0) {
        const float inv = n > 0 ? 1.f / sum : 0.f;
        float* dst = a.out + row * D + 8 * u;
        *reinterpret_cast<float4*>(dst) = make_float4(o8[0] * inv, o8[1] * inv, o8[2] * inv, o8[3] * inv);
        *reinterpret_cast<float4*>(dst + 4) = make_float4(o8[4] * inv, o8[5] * inv, o8[6] * inv, o8[7] * inv);
    }
}

}  // namespace

int decode_rows_pad(int Gh, int n_dec) { return (Gh * n_dec + 31) / 32 * 32; }
int decode_max_rows() { return kDecMaxRows; }
int decode_max_compact() { return kDecMaxCompact; }
int decode_key_blocks(int T) { return (T + kDecKeys - 1) / kDecKeys; }

hipError_t launch_decode_check(const DecodeArgs& a, hipStream_t s) {
    dim3 g0((a.rows_pad * (a.d / 8) + 255) / 256, a.B * a.Hkv);
    hipLaunchKernelGGL(decode_scale_kernel, g0, dim3(256), 0, s, a);
    dim3 g1(a.n_kb, a.B * a.Hkv);
    // staged queries: up to 256 rows of 17 chunks (69.6 KB at d = 128)
    const size_t lds = static_cast<size_t>(a.rows_pad) * (a.d / 8 + 1) * 16;
    hipError_t e;
    if (a.d == 64) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_cover_kernel<64>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(decode_cover_kernel<64>, g1, dim3(64 * kDecWaves), lds, s, a);
    } else {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_cover_kernel<128>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(decode_cover_kernel<128>, g1, dim3(64 * kDecWaves), lds, s, a);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.k_dtype == 1) {
        // bf16 cache: the matrix-core kernel, one workgroup per 32 decode rows
        // of a KV head (it also merges the coverage partials of its rows)
        dim3 g3(a.rows_pad / 32, a.B * a.Hkv);
        if (a.d == 64)
            hipLaunchKernelGGL(decode_attend_mfma_kernel<64>, g3, dim3(64 * kDecWaves), 0, s, a);
        else
            hipLaunchKernelGGL(decode_attend_mfma_kernel<128>, g3, dim3(64 * kDecWaves), 0, s, a);
        return hipGetLastError();
    }
    // fp32 cache: the coverage merge, then fp32 products on the VALU, one
    // wave per decode query
    dim3 g2((a.rows + 3) / 4, a.B * a.Hkv);
    hipLaunchKernelGGL(decode_cover_combine_kernel, g2, dim3(256), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t n_rows = static_cast<int64_t>(a.B) * a.Hq * a.n_dec;
    dim3 g3(static_cast<unsigned>((n_rows + 3) / 4));
    if (a.d == 64)
        hipLaunchKernelGGL(decode_attend_kernel<64>, g3, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(decode_attend_kernel<128>, g3, dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace mmskv
