// Decode-time check on gfx950: the attention-mass coverage of Fig. 1b (the
// share of a decoding query's softmax mass over all prompt keys that falls
// on the keys kept after prefilling) and decode attention over the fixed
// compacted cache (Sec. 3.1's prefill-only protocol).
//
// Coverage: one workgroup of 4 waves per (b, c, block of 512 keys).  The
// Gh * n_dec decode queries of KV head c, scaled once like the anchor query
// (log2(e)/sqrt(d) in fp64, then fp32, then bf16), are staged in LDS and
// streamed past the block's keys in 32-row tiles with v_mfma_f32_32x32x16_bf16
// in the K * Q^T layout (lane = query row, its 32 values = its keys), so a
// row's block statistics are in-lane sums.  Per (row, block) the kernel
// writes (m, sum of 2^(s - m) over all keys, the same over the kept keys);
// a second kernel merges the blocks and divides.  The keys are read once:
// the pass is HBM-bound on K.
//
// Compacted attention: one wave per decode query over the counts[b, c] rows
// of the compacted cache, fp32 on the VALU (a few hundred keys).
#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kDecWaves = 4;
constexpr int kDecSub = 2;                 // 64-key sub-blocks per wave, loaded together
constexpr int kDecKeys = 64 * kDecWaves * kDecSub;   // keys per workgroup
constexpr int kDecMaxRows = 256;           // Gh * n_dec, padded to 32
constexpr int kDecMaxCompact = 2048;       // rows of the compacted cache (c_max)

__device__ __forceinline__ floatx16 mfma_32x32x16(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float pair_max2(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
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

template <int D>
__global__ void __launch_bounds__(64 * kDecWaves) decode_cover_kernel(DecodeArgs a) {
    constexpr int KC = D / 16;                 // 16-element k steps
    constexpr int kRow = D / 8 + 1;            // LDS row in 16-byte chunks (one pad chunk)
    extern __shared__ u32x4 qs[];              // [rows_pad * kRow]
    __shared__ uint32_t kept[kDecKeys / 32];
    __shared__ float4 part[kDecWaves][kDecMaxRows];

    const int kb = blockIdx.x, bc = blockIdx.y;
    const int b = bc / a.Hkv, c = bc - b * a.Hkv;
    const int tid = threadIdx.x, wave = tid / kWave, lane = lane_id();
    const int key_base = kb * kDecKeys;

    // kept flags of this block's keys (idx is any list of in-range indices)
    if (tid < kDecKeys / 32) kept[tid] = 0u;
    __syncthreads();
    const int n_kept = min(max(a.counts[bc], 0), a.c_max);
    for (int i = tid; i < n_kept; i += 64 * kDecWaves) {
        const int t = a.idx[static_cast<int64_t>(bc) * a.c_max + i] - key_base;
        if (t >= 0 && t < kDecKeys && t + key_base < a.T) atomicOr(&kept[t >> 5], 1u << (t & 31));
    }

    // the wave's sub-block sb holds keys key_base + 256 sb + 64 wave + [0, 64):
    // kf[s][kc] = key key0 + 32 s + lane % 32, dims 16 kc + 8 (lane / 32) ..
    bf16x8 kfs[kDecSub][2][KC];
    auto load_keys = [&](bf16x8 (&kf)[2][KC], int key0) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int t = key0 + 32 * s + (lane & 31);
            const bool ok = t < a.T;
            const int64_t off = static_cast<int64_t>(b) * a.ksb + static_cast<int64_t>(c) * a.ksh +
                                static_cast<int64_t>(ok ? t : 0) * a.kst + 8 * (lane >> 5);
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                if (a.k_dtype == 1)
                    kf[s][kc] = ok ? load_bf16x8(static_cast<const uint16_t*>(a.k) + off + 16 * kc) : zero_bf16x8();
                else
                    kf[s][kc] = ok ? load_f32_as_bf16x8(static_cast<const float*>(a.k) + off + 16 * kc)
                                   : zero_bf16x8();
            }
        }
    };
#pragma unroll
    for (int sb = 0; sb < kDecSub; ++sb) load_keys(kfs[sb], key_base + 256 * sb + 64 * wave);
    // the head's scaled queries (decode_scale_kernel), copied to LDS while the keys arrive
    const u32x4* qsrc = reinterpret_cast<const u32x4*>(a.qsc + static_cast<int64_t>(bc) * a.rows_pad * D);
    for (int i = tid; i < a.rows_pad * (D / 8); i += 64 * kDecWaves) {
        const int r = i / (D / 8), ch = i - r * (D / 8);
        qs[r * kRow + ch] = qsrc[i];
    }
    // per (wave, row) running (m, sum all, sum kept), merged over the sub-blocks
    for (int r = lane; r < a.rows_pad; r += kWave) part[wave][r] = make_float4(-INFINITY, 0.f, 0.f, 0.f);
    __syncthreads();
#pragma unroll
    for (int sb = 0; sb < kDecSub; ++sb) {
        const int key0 = key_base + 256 * sb + 64 * wave;
        const bf16x8 (&kf)[2][KC] = kfs[sb];
        // value i of sub-tile s of this lane is key key0 + 32 s + 8 (i / 4) + 4 (lane / 32) + i % 4
        uint32_t valid = 0u, keep = 0u;
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int t = key0 + 32 * s + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
                const int tl = t - key_base;
                if (t < a.T) valid |= 1u << (16 * s + i);
                if (t < a.T && ((kept[tl >> 5] >> (tl & 31)) & 1u)) keep |= 1u << (16 * s + i);
            }
        // (key0 is the same in every lane: the MFMAs and lane swaps below run in
        // whole waves)
        for (int r0 = 0; r0 < a.rows_pad && key0 < a.T; r0 += 32) {
            floatx16 acc[2];
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[s][i] = 0.f;
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                const bf16x8 q = __builtin_bit_cast(bf16x8, qs[(r0 + (lane & 31)) * kRow + 2 * kc + (lane >> 5)]);
#pragma unroll
                for (int s = 0; s < 2; ++s) acc[s] = mfma_32x32x16(kf[s][kc], q, acc[s]);
            }
            // sums of 2^s relative to 0 while every lane's sum is in
            // [2^-60, lane_sum_limit(T, 32)) (as in the row log-sum-exp pass),
            // else relative to the exact per-column maximum
            float mx = 0.f, la = 0.f, lk = 0.f;
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float e = ((valid >> (16 * s + i)) & 1u) ? fast_exp2(acc[s][i]) : 0.f;
                    la += e;
                    lk += ((keep >> (16 * s + i)) & 1u) ? e : 0.f;
                }
            const bool in_range = (la >= 0x1p-60f || valid == 0u) && la < a.lane_sum_hi;
            if (__ballot(!in_range) != 0) {
                mx = -INFINITY;
#pragma unroll
                for (int s = 0; s < 2; ++s)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if ((valid >> (16 * s + i)) & 1u) mx = fmaxf(mx, acc[s][i]);
                mx = pair_max2(mx);
                la = 0.f;
                lk = 0.f;
                if (mx != -INFINITY) {
#pragma unroll
                    for (int s = 0; s < 2; ++s)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            const float e = ((valid >> (16 * s + i)) & 1u) ? fast_exp2(acc[s][i] - mx) : 0.f;
                            la += e;
                            lk += ((keep >> (16 * s + i)) & 1u) ? e : 0.f;
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

// decode attention over the compacted cache: one wave per decode query.
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
