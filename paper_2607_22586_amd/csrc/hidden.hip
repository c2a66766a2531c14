// Hidden-state form of the proxies (Sec. 3.2.1 Eqs. 4-6 as written, and
// Algorithm 1): statistics of a layer's prefill hidden states, variance-
// expanded samples of them, and their projection by every head's query
// weights, on gfx950.
//
// hidden_stats   per (batch row, feature): S = sum h and SS = sum h^2 over
//                chunks of tokens (token order inside a chunk, one thread
//                per 8 features, fp64), then the chunk sums in chunk order;
//                mean = S/T, std = sqrt((SS - S*mean)/(T - ddof)).
// hidden_proxies x = mu + (gamma*sigma) z per (batch row, sample, feature),
//                z from the counter-based generator with the head field set
//                to 0xFFFFFFFF (one set of samples per layer, shared by all
//                heads), fp64 -> fp32 -> bf16.
// project        q[b, h, i, :] = W_Q^(h) H~[b, i, :]: a bf16 GEMM of the
//                (B*P) x D samples against the (Hq*d) x D weights (both with
//                the reduction dimension contiguous) with fp32 accumulation.
//                Without rotary tables, on full 128 x 224 tiles: four waves
//                of 64 x 112 on v_mfma_f32_16x16x32_bf16.  Otherwise 128x128
//                tiles of four 64x64 waves on v_mfma_f32_32x32x16_bf16, the
//                epilogue through LDS so that the rotary pairs (e, e + d/2)
//                of a head meet in one thread.  Both multiply by the query
//                scale log2(e)/sqrt(d) in fp64 and round to bf16.
#pragma clang fp contract(off)

#include <math.h>

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "normal.hpp"

namespace mmskv {
namespace {

constexpr int kStatThreads = 64;           // one wave per workgroup (no shared state)

// fp32 value times the query scale, in fp64, rounded back to fp32.
__device__ __forceinline__ float scaled(float v, double scale) {
    const double y = static_cast<double>(v) * scale;
    return static_cast<float>(y);
}
constexpr int kStatVec = 8;                 // features per thread (one 16-byte bf16 load)
constexpr int kStatFlight = 8;              // tokens per group of loads in flight

// Running sums of one token's kStatVec features.  The square of a bf16 or fp32
// value is exact in fp64, so the fused multiply-add rounds exactly like a
// separate product and sum.
__device__ __forceinline__ void accum_token(const double (&v)[kStatVec], double (&s)[kStatVec],
                                       double (&ss)[kStatVec]) {
#pragma unroll
    for (int e = 0; e < kStatVec; ++e) {
        s[e] = s[e] + v[e];
        ss[e] = fma(v[e], v[e], ss[e]);
    }
}

__device__ __forceinline__ void unpack_bf16x8(const u32x4& r, double (&v)[kStatVec]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[2 * q] = static_cast<double>(__uint_as_float(r[q] << 16));
        v[2 * q + 1] = static_cast<double>(__uint_as_float(r[q] & 0xFFFF0000u));
    }
}

// 8 consecutive fp32 features of one token as fp64.
__device__ __forceinline__ void load8_f32(const HiddenArgs& a, int64_t off, double (&v)[kStatVec]) {
    const float4 x = *reinterpret_cast<const float4*>(static_cast<const float*>(a.hidden) + off);
    const float4 y = *reinterpret_cast<const float4*>(static_cast<const float*>(a.hidden) + off + 4);
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
}

// Chunk sums: grid (n_chunks, ceil(D / (8*64)), B); thread j owns features
// [8j, 8j+8) of the block and sums them over the chunk's tokens in token
// order.  bf16 rows: the raw 16-byte loads of the next kStatFlight tokens
// are issued before the current ones are summed (two register sets used in
// turn), so up to two groups of loads are in flight per thread.
__global__ void __launch_bounds__(kStatThreads) hidden_stats_partial_kernel(HiddenArgs a) {
    const int c = blockIdx.x, b = blockIdx.z;
    const int j0 = (static_cast<int>(blockIdx.y) * kStatThreads + static_cast<int>(threadIdx.x)) * kStatVec;
    if (j0 >= a.D) return;
    const int t0 = c * a.chunk, t1 = min(t0 + a.chunk, a.T);
    double s[kStatVec], ss[kStatVec];
#pragma unroll
    for (int e = 0; e < kStatVec; ++e) { s[e] = 0.0; ss[e] = 0.0; }
    const int64_t base = static_cast<int64_t>(b) * a.sb + j0;
    if (a.dtype == 1) {
        const uint16_t* h = static_cast<const uint16_t*>(a.hidden) + base;
        auto fetch = [&](int t, u32x4 (&r)[kStatFlight]) {
#pragma unroll
            for (int u = 0; u < kStatFlight; ++u)
                if (t + u < t1) r[u] = *reinterpret_cast<const u32x4*>(h + static_cast<int64_t>(t + u) * a.st);
        };
        auto sum = [&](int t, const u32x4 (&r)[kStatFlight]) {
#pragma unroll
            for (int u = 0; u < kStatFlight; ++u) {
                if (t + u < t1) {
                    double v[kStatVec];
                    unpack_bf16x8(r[u], v);
                    accum_token(v, s, ss);
                }
            }
        };
        // two register sets, A for tokens [t, t+F), B for [t+F, t+2F)
        u32x4 ra[kStatFlight], rb[kStatFlight];
        fetch(t0, ra);
        for (int t = t0; t < t1; t += 2 * kStatFlight) {
            if (t + kStatFlight < t1) fetch(t + kStatFlight, rb);
            sum(t, ra);
            if (t + 2 * kStatFlight < t1) fetch(t + 2 * kStatFlight, ra);
            if (t + kStatFlight < t1) sum(t + kStatFlight, rb);
        }
    } else {
        for (int t = t0; t < t1; ++t) {
            double v[kStatVec];
            load8_f32(a, base + static_cast<int64_t>(t) * a.st, v);
            accum_token(v, s, ss);
        }
    }
    double2* out = a.partial + (static_cast<int64_t>(b) * a.n_chunks + c) * a.D + j0;
#pragma unroll
    for (int e = 0; e < kStatVec; ++e) out[e] = make_double2(s[e], ss[e]);
}

// Chunk sums in chunk order -> mean, std: grid (ceil(D/256), B).
__global__ void __launch_bounds__(256) hidden_stats_final_kernel(HiddenArgs a) {
    const int j = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x), b = blockIdx.y;
    if (j >= a.D) return;
    const double2* p = a.partial + static_cast<int64_t>(b) * a.n_chunks * a.D + j;
    double S = 0.0, SS = 0.0;
    // kFinalBatch chunk partials fetched at once (their latencies overlap),
    // then added in chunk order
    constexpr int kFinalBatch = 16;
    for (int c0 = 0; c0 < a.n_chunks; c0 += kFinalBatch) {
        double2 v[kFinalBatch];
#pragma unroll
        for (int u = 0; u < kFinalBatch; ++u)
            if (c0 + u < a.n_chunks) v[u] = p[static_cast<int64_t>(c0 + u) * a.D];
#pragma unroll
        for (int u = 0; u < kFinalBatch; ++u) {
            if (c0 + u < a.n_chunks) {
                S = S + v[u].x;
                SS = SS + v[u].y;
            }
        }
    }
    const double mean = S / static_cast<double>(a.T);
    const double sm = S * mean;
    double var = (SS - sm) / static_cast<double>(a.T - a.ddof);
    if (var < 0.0) var = 0.0;
    a.stats[(static_cast<int64_t>(b) * 2) * a.D + j] = mean;
    a.stats[(static_cast<int64_t>(b) * 2 + 1) * a.D + j] = sqrt(var);
}

// Samples: one thread per (sample i, feature quad jq); grid (ceil(P*D/4 / 256), B).
__global__ void __launch_bounds__(256) hidden_proxies_kernel(HiddenArgs a) {
    const int b = blockIdx.y;
    const int quads = a.D / 4;
    const int64_t item = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (item >= static_cast<int64_t>(a.P) * quads) return;
    const int i = static_cast<int>(item / quads), jq = static_cast<int>(item % quads);
    const double* mu = a.stats + (static_cast<int64_t>(b) * 2) * a.D;
    const double* sg = a.stats + (static_cast<int64_t>(b) * 2 + 1) * a.D;
    double z[4];
    normal_quad(a.key0, a.key1, b, a.layer, -1, i, jq, z);
    uint16_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int j = 4 * jq + e;
        const double gs = a.gamma * sg[j];
        const double t = gs * z[e];
        const double x = mu[j] + t;
        o[e] = static_cast<uint16_t>(f32_to_bf16_bits(static_cast<float>(x)));
    }
    uint2 pk;
    pk.x = o[0] | (static_cast<uint32_t>(o[1]) << 16);
    pk.y = o[2] | (static_cast<uint32_t>(o[3]) << 16);
    *reinterpret_cast<uint2*>(a.hp + (static_cast<int64_t>(b) * a.P + i) * a.D + 4 * jq) = pk;
}

// ------------------------------------------------------------ projection GEMM
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kGemmThreads = 256;
constexpr int kRowChunks = kBK / 8;            // 16-byte chunks per tile row
constexpr int kRowSlots = kRowChunks + 1;      // padded row (one spare chunk)
constexpr int kTileSlots = kBM * kRowSlots;    // per operand tile
constexpr int kLoads = kBM * kRowChunks / kGemmThreads;   // chunks per thread per operand

__device__ __forceinline__ floatx16 mfma32(bf16x8 a, bf16x8 b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Rows r of A (M x K) and of W (N x K) in 16-byte chunks; rows past the
// matrix and k past D read as zero.
struct GemmStage {
    u32x4 a[kLoads], w[kLoads];
};

__device__ __forceinline__ void gemm_fetch(const ProjectArgs& p, int m0, int n0, int k0, GemmStage& st) {
#pragma unroll
    for (int q = 0; q < kLoads; ++q) {
        const int c = static_cast<int>(threadIdx.x) + q * kGemmThreads;
        const int r = c / kRowChunks, kc = c % kRowChunks;
        const int k = k0 + 8 * kc;
        const u32x4 zero = {0u, 0u, 0u, 0u};
        st.a[q] = (m0 + r < p.M && k < p.K)
                      ? *reinterpret_cast<const u32x4*>(p.a + static_cast<int64_t>(m0 + r) * p.K + k) : zero;
        st.w[q] = (n0 + r < p.N && k < p.K)
                      ? *reinterpret_cast<const u32x4*>(p.w + static_cast<int64_t>(n0 + r) * p.K + k) : zero;
    }
}

__device__ __forceinline__ void gemm_store(const GemmStage& st, u32x4* la, u32x4* lw) {
#pragma unroll
    for (int q = 0; q < kLoads; ++q) {
        const int c = static_cast<int>(threadIdx.x) + q * kGemmThreads;
        const int r = c / kRowChunks, kc = c % kRowChunks;
        la[r * kRowSlots + kc] = st.a[q];
        lw[r * kRowSlots + kc] = st.w[q];
    }
}

// Epilogue of a 128 x 128 output tile: the fp32 accumulators (wave (wm, wn)
// holds rows wm*64.., columns wn*64..) through LDS, then the rotary pairs,
// the softmax scale and the bf16 rounding, to the proxies' layout.
__device__ __forceinline__ void project_epilogue(const ProjectArgs& p, const floatx16 (&acc)[2][2], u32x4* lds,
                                                 int m0, int n0, int wm, int wn, int lane) {
    constexpr int kLd = kBN + 4;
    float* tile = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = wm * 64 + 32 * x + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
                const int cc = wn * 64 + 32 * y + (lane & 31);
                tile[r * kLd + cc] = acc[x][y][i];
            }
    __syncthreads();
    const int d = p.d, half = d / 2;
    const bool rope = p.cos != nullptr;
    // each thread: one row, 8 consecutive output columns (one head's
    // lower half when rotary pairs are formed)
    const int groups = rope ? kBN / 16 : kBN / 8;     // 8-column groups per row
    for (int g = static_cast<int>(threadIdx.x); g < kBM * groups; g += kGemmThreads) {
        const int r = g / groups, cg = g % groups;
        const int m = m0 + r;
        if (m >= p.M) continue;
        const int bb = m / p.P, i = m % p.P;
        int col;
        if (rope) {
            const int c8 = cg * 8;                     // lower-half column index inside the tile's heads
            col = (c8 / half) * d + (c8 % half);
        } else {
            col = cg * 8;
        }
        const int n = n0 + col;
        if (n >= p.N) continue;
        const int h = n / d, e = n % d;
        uint16_t* out = p.out + ((static_cast<int64_t>(bb) * p.Hq + h) * p.P + i) * d;
        u32x4 lo, hi;
        if (!rope) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                lo[q] = f32_to_bf16_bits(scaled(tile[r * kLd + col + 2 * q], p.scale)) |
                        (f32_to_bf16_bits(scaled(tile[r * kLd + col + 2 * q + 1], p.scale)) << 16);
            *reinterpret_cast<u32x4*>(out + e) = lo;
        } else {
            uint32_t l16[8], h16[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const float x0 = tile[r * kLd + col + q], x1 = tile[r * kLd + col + half + q];
                const float c = p.cos[e + q], s = p.sin[e + q];
                const float a0 = x0 * c, a1 = x1 * s, b0 = x1 * c, b1 = x0 * s;
                l16[q] = f32_to_bf16_bits(scaled(a0 - a1, p.scale));
                h16[q] = f32_to_bf16_bits(scaled(b0 + b1, p.scale));
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                lo[q] = l16[2 * q] | (l16[2 * q + 1] << 16);
                hi[q] = h16[2 * q] | (h16[2 * q + 1] << 16);
            }
            *reinterpret_cast<u32x4*>(out + e) = lo;
            *reinterpret_cast<u32x4*>(out + e + half) = hi;
        }
    }
}

// Any shape (ragged tiles): register-staged loads, two LDS stages.
__global__ void __launch_bounds__(kGemmThreads) project_kernel(ProjectArgs p) {
    // two stages of (A tile, W tile); the fp32 output tile reuses the space
    __shared__ u32x4 lds[2 * 2 * kTileSlots];
    const int m0 = static_cast<int>(blockIdx.x) * kBM, n0 = static_cast<int>(blockIdx.y) * kBN;
    const int wave = static_cast<int>(threadIdx.x) / kWave, lane = lane_id();
    const int wm = wave >> 1, wn = wave & 1;           // 64 x 64 quadrant of the wave
    const int n_k = (p.K + kBK - 1) / kBK;

    floatx16 acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;

    // k steps: LDS holds steps ks (being multiplied) and ks+1 (written during
    // step ks); two register stages hold the global loads of steps ks+1 and
    // ks+2, so every load has two steps of MFMA work to arrive in
    GemmStage s0, s1;
    gemm_fetch(p, m0, n0, 0, s0);
    gemm_store(s0, lds, lds + kTileSlots);
    if (1 < n_k) gemm_fetch(p, m0, n0, kBK, s1);
    if (2 < n_k) gemm_fetch(p, m0, n0, 2 * kBK, s0);
    __syncthreads();
    // step ks; `nx` holds the loads of step ks+1 and is refilled with ks+3
    auto step = [&](int ks, GemmStage& nx) {
        const int cur = ks & 1;
        const u32x4* la = lds + cur * 2 * kTileSlots;
        const u32x4* lw = la + kTileSlots;
#pragma unroll
        for (int kc = 0; kc < kBK / 16; ++kc) {
            bf16x8 fa[2], fw[2];
            const int chunk = 2 * kc + (lane >> 5);
#pragma unroll
            for (int x = 0; x < 2; ++x) {
                fa[x] = __builtin_bit_cast(bf16x8, la[(wm * 64 + 32 * x + (lane & 31)) * kRowSlots + chunk]);
                fw[x] = __builtin_bit_cast(bf16x8, lw[(wn * 64 + 32 * x + (lane & 31)) * kRowSlots + chunk]);
            }
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) acc[x][y] = mfma32(fa[x], fw[y], acc[x][y]);
        }
        if (ks + 1 < n_k) {
            u32x4* na = lds + (cur ^ 1) * 2 * kTileSlots;
            gemm_store(nx, na, na + kTileSlots);
            if (ks + 3 < n_k) gemm_fetch(p, m0, n0, (ks + 3) * kBK, nx);
        }
        __syncthreads();
    };
    int ks = 0;
    for (; ks < n_k; ks += 2) {
        step(ks, s1);
        if (ks + 1 < n_k) step(ks + 1, s0);
    }

    project_epilogue(p, acc, lds, m0, n0, wm, wn, lane);
}

// Full tiles with direct-to-LDS loads (global_load_lds_dwordx4): the tiles
// of k step ks land in LDS stage ks % NS without passing through registers,
// issued NS - 1 steps ahead; one barrier per step.  The waits are written out
// (each wave waits for its own share of stage ks, the barrier then covers
// every wave's share and every wave's reads of step ks - 1, whose stage the
// step's new loads overwrite).  A row of a stage is DK / 8 chunks of 16
// bytes, chunk c of row r at slot c ^ f(r), f chosen so that the 8 rows read
// in one 128-byte LDS phase (one chunk each) fall in 8 different bank groups.
template <int DK>
struct DmaTile {
    static constexpr int kChunks = DK / 8;                 // 16-byte chunks per row
    static constexpr int kRow = DK * 2;                    // bytes per row
    static constexpr int kTile = kBM * kRow;               // bytes per operand tile
    static constexpr int kStage = 2 * kTile;               // A tile, then W tile
    static constexpr int kRowsPerOp = 1024 / kRow;         // rows per 1 KB instruction
    static constexpr int kOps = 32 / kRowsPerOp;           // instructions per operand per wave
    static constexpr int kPerStage = 2 * kOps;             // loads per wave per stage
    static __device__ __forceinline__ int slot(int r, int c) {
        return kChunks == 4 ? c ^ ((r >> 1) & 3) : c ^ (r & 7);
    }
};

// wave w issues rows 32 w .. 32 w + 31 of both tiles of one step
template <int DK>
__device__ __forceinline__ void dma_step(const ProjectArgs& p, int m0, int n0, int k0, char* stage, int wave, int lane) {
    using T = DmaTile<DK>;
#pragma unroll
    for (int op = 0; op < 2; ++op) {
        const uint16_t* src = op == 0 ? p.a + static_cast<int64_t>(m0) * p.K : p.w + static_cast<int64_t>(n0) * p.K;
#pragma unroll
        for (int j = 0; j < T::kOps; ++j) {
            const int r0 = 32 * wave + T::kRowsPerOp * j, r = r0 + lane / T::kChunks;
            const int c = T::slot(r, lane % T::kChunks);
            __builtin_amdgcn_global_load_lds(src + static_cast<int64_t>(r) * p.K + k0 + 8 * c,
                                             (__attribute__((address_space(3))) void*)(stage + op * T::kTile + r0 * T::kRow),
                                             16, 0, 0);
        }
    }
}

// s_waitcnt with vmcnt = N and the other counters not waited on
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N < 64, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

template <int DK, int NS>
__global__ void __launch_bounds__(kGemmThreads) project_dma_kernel(ProjectArgs p) {
    using T = DmaTile<DK>;
    static_assert(kBM == kBN && kBM == 128, "four waves of 32 rows per operand");
    // the stages, or the epilogue's fp32 tile if that is larger
    constexpr int kBytes = NS * T::kStage > kBM * (kBN + 4) * 4 ? NS * T::kStage : kBM * (kBN + 4) * 4;
    __shared__ u32x4 lds[kBytes / 16];
    char* base = reinterpret_cast<char*>(lds);
    const int m0 = static_cast<int>(blockIdx.x) * kBM, n0 = static_cast<int>(blockIdx.y) * kBN;
    const int wave = static_cast<int>(threadIdx.x) / kWave, lane = lane_id();
    const int wm = wave >> 1, wn = wave & 1;
    const int n_k = p.K / DK;
    floatx16 acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[x][y][i] = 0.f;
#pragma unroll
    for (int st = 0; st < NS - 1; ++st)
        if (st < n_k) dma_step<DK>(p, m0, n0, st * DK, base + st * T::kStage, wave, lane);
    for (int ks = 0; ks < n_k; ++ks) {
        // this wave's loads of stage ks are the oldest outstanding; later
        // stages in flight: min(NS - 2, n_k - 1 - ks)
        const int later = min(NS - 2, n_k - 1 - ks);
        if (later >= 3) wait_vm<3 * T::kPerStage>();
        else if (later == 2) wait_vm<2 * T::kPerStage>();
        else if (later == 1) wait_vm<T::kPerStage>();
        else wait_vm<0>();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (ks + NS - 1 < n_k)
            dma_step<DK>(p, m0, n0, (ks + NS - 1) * DK, base + ((ks + NS - 1) % NS) * T::kStage, wave, lane);
        const char* sa = base + (ks % NS) * T::kStage;
        const char* sw = sa + T::kTile;
        // fragments of k chunk kc + 1 are read while the MFMAs of kc run
        bf16x8 fa[2][2], fw[2][2];
        auto read_frags = [&](int kc, int buf) {
            const int c = 2 * kc + (lane >> 5);
#pragma unroll
            for (int x = 0; x < 2; ++x) {
                const int ra = wm * 64 + 32 * x + (lane & 31), rw = wn * 64 + 32 * x + (lane & 31);
                fa[buf][x] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sa + ra * T::kRow + 16 * T::slot(ra, c)));
                fw[buf][x] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sw + rw * T::kRow + 16 * T::slot(rw, c)));
            }
        };
        read_frags(0, 0);
#pragma unroll
        for (int kc = 0; kc < DK / 16; ++kc) {
            if (kc + 1 < DK / 16) read_frags(kc + 1, (kc + 1) & 1);
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y) acc[x][y] = mfma32(fa[kc & 1][x], fw[kc & 1][y], acc[x][y]);
        }
    }
    // every wave's reads done before the tile reuses the stages
    asm volatile("" ::: "memory");
    __syncthreads();
    project_epilogue(p, acc, lds, m0, n0, wm, wn, lane);
}

// Full tiles without rotary tables: 128 x 224 output tiles (the benchmark
// shape has 16 x 16 of them, one per CU), four waves of 64 x 112 on
// v_mfma_f32_16x16x32_bf16 (4 x 7 accumulator blocks per wave).  A k step is
// 64 wide and lands in one of two LDS stages by direct loads: each wave issues
// 11 of the step's 44 loads of 8 rows x 128 bytes, from a uniform base
// advanced per step plus loop-invariant 32-bit lane offsets (chunk c of row r
// at slot c ^ (r & 7)).  A step runs its two 32-wide halves back to back: the
// A fragments of the next half are read before a half's 28 MFMAs, and each W
// fragment is refilled right after the four MFMAs that last read it.  The
// barrier sits between the halves: by then every wave has its own loads of
// the next stage and its reads of the current one complete, so after it the
// next stage can be read and the loads two steps ahead overwrite the current
// stage.
constexpr int kWM = 128, kWN = 224, kWK = 64;
constexpr int kWRow = kWK * 2;                      // bytes per staged row
constexpr int kWTileA = kWM * kWRow;                // the A rows of a stage
constexpr int kWStage = (kWM + kWN) * kWRow;        // 45,056 bytes
constexpr int kWLoads = (kWM + kWN) / 8 / 4;        // loads per wave and stage
constexpr int kWLd = kWN + 4;                       // epilogue row pitch (floats)
constexpr int kWLds = 2 * kWStage > kWM * kWLd * 4 ? 2 * kWStage : kWM * kWLd * 4;
// the four waves issue the 8-row groups of a stage in turn: the A tile's 16
// groups are loads j < 4 of every wave, the W tile's 28 the rest
static_assert((kWM + kWN) % 32 == 0 && kWM / 8 == 4 * 4 && kGemmThreads == 4 * kWave, "load split");
static_assert(kWN == 2 * 112 && kWM == 2 * 64, "four waves of 64 x 112");
typedef float floatx4 __attribute__((ext_vector_type(4)));

// s_waitcnt vmcnt(0) lgkmcnt(0)
__device__ __forceinline__ void wait_vm_lgkm0() { __builtin_amdgcn_s_waitcnt(0x0070); }

__global__ void __launch_bounds__(kGemmThreads) project_wide_kernel(ProjectArgs p) {
    __shared__ u32x4 lds[kWLds / 16];
    char* base = reinterpret_cast<char*>(lds);
    const int nN = p.N / kWN;
    const int m0 = static_cast<int>(blockIdx.x) / nN * kWM, n0 = static_cast<int>(blockIdx.x) % nN * kWN;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave), lane = lane_id();
    const int wm = wave >> 1, wn = wave & 1;
    const int n_k = p.K / kWK;                      // at least 2 (checked by the host)
    floatx4 acc[4][7];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 7; ++y) acc[x][y] = floatx4{0.f, 0.f, 0.f, 0.f};

    // load j of a stage: rows 8 (wave + 4 j) .. + 7 of the A tile (j < 4) or
    // of the W tile (j >= 4, less 16 groups); lane -> row + (lane >> 3), slot lane & 7
    uint32_t voff[kWLoads];
#pragma unroll
    for (int j = 0; j < kWLoads; ++j) {
        const int g = wave + 4 * j - (j < 4 ? 0 : kWM / 8);
        const int r = 8 * g + (lane >> 3);
        voff[j] = static_cast<uint32_t>(((j < 4 ? m0 : n0) + r) * p.K * 2 + 16 * ((lane & 7) ^ (r & 7)));
    }
    auto loads = [&](int k0, char* stage) {
        const char* ab = reinterpret_cast<const char*>(p.a) + 2 * k0;
        const char* wb = reinterpret_cast<const char*>(p.w) + 2 * k0;
#pragma unroll
        for (int j = 0; j < kWLoads; ++j) {
            const int g = wave + 4 * j - (j < 4 ? 0 : kWM / 8);
            char* dst = stage + (j < 4 ? 0 : kWTileA) + 8 * g * kWRow;
            __builtin_amdgcn_global_load_lds((j < 4 ? ab : wb) + voff[j],
                                             (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
        }
    };
    // fragment rows wm*64 + 16x + (lane & 15) and wn*112 + 16y + (lane & 15)
    // (both = lane & 7 mod 8), 16-byte chunk 4 h + (lane >> 4) of half h
    const int rA = wm * 64 + (lane & 15), rW = wn * 112 + (lane & 15);
    const int oA0 = rA * kWRow + 16 * ((lane >> 4) ^ (lane & 7));
    const int oA1 = rA * kWRow + 16 * ((4 + (lane >> 4)) ^ (lane & 7));
    const int oW0 = kWTileA + rW * kWRow + 16 * ((lane >> 4) ^ (lane & 7));
    const int oW1 = kWTileA + rW * kWRow + 16 * ((4 + (lane >> 4)) ^ (lane & 7));
    auto rd = [&](const char* q) { return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(q)); };
    bf16x8 fa0[4], fa1[4], fw[7];

    loads(0, base);
    loads(kWK, base + kWStage);
    wait_vm<kWLoads>();
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
#pragma unroll
    for (int x = 0; x < 4; ++x) fa0[x] = rd(base + oA0 + x * 16 * kWRow);
#pragma unroll
    for (int y = 0; y < 7; ++y) fw[y] = rd(base + oW0 + y * 16 * kWRow);

    // step ks on stage st (half 0's fragments already in fa0 / fw); nst is
    // the next stage; the loads of step ks + 2 go to st
    auto step = [&](int ks, char* st, const char* nst, auto last_tag) {
        constexpr bool kLast = decltype(last_tag)::value;
#pragma unroll
        for (int x = 0; x < 4; ++x) fa1[x] = rd(st + oA1 + x * 16 * kWRow);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int y = 0; y < 7; ++y) {
#pragma unroll
            for (int x = 0; x < 4; ++x) acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa0[x], fw[y], acc[x][y], 0, 0, 0);
            fw[y] = rd(st + oW1 + y * 16 * kWRow);
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (!kLast) {
            wait_vm_lgkm0();
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            if (ks + 2 < n_k) loads((ks + 2) * kWK, st);
#pragma unroll
            for (int x = 0; x < 4; ++x) fa0[x] = rd(nst + oA0 + x * 16 * kWRow);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int y = 0; y < 7; ++y) {
#pragma unroll
            for (int x = 0; x < 4; ++x) acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa1[x], fw[y], acc[x][y], 0, 0, 0);
            if constexpr (!kLast) fw[y] = rd(nst + oW0 + y * 16 * kWRow);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    int ks = 0;
    for (; ks + 2 < n_k; ks += 2) {
        step(ks, base, base + kWStage, std::false_type{});
        step(ks + 1, base + kWStage, base, std::false_type{});
    }
    if (ks + 1 < n_k) {
        step(ks, base, base + kWStage, std::false_type{});
        ++ks;
    }
    step(ks, base + (ks & 1) * kWStage, nullptr, std::true_type{});

    // epilogue: the fp32 tile through LDS (every wave's stage reads are done),
    // then 8 consecutive columns of one row per thread and group: the query
    // scale in fp64, bf16, one 16-byte store into the proxies' layout
    asm volatile("" ::: "memory");
    __syncthreads();
    float* tile = reinterpret_cast<float*>(lds);
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 7; ++y)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                tile[(wm * 64 + 16 * x + 4 * (lane >> 4) + i) * kWLd + wn * 112 + 16 * y + (lane & 15)] = acc[x][y][i];
    __syncthreads();
    constexpr int kGroups = kWN / 8;
    for (int g = static_cast<int>(threadIdx.x); g < kWM * kGroups; g += kGemmThreads) {
        const int r = g / kGroups, c = 8 * (g % kGroups);
        const int m = m0 + r, n = n0 + c;
        const int bb = m / p.P, i = m % p.P, h = n / p.d, e = n % p.d;
        const float* src = tile + r * kWLd + c;
        u32x4 v;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            v[q] = f32_to_bf16_bits(scaled(src[2 * q], p.scale)) | (f32_to_bf16_bits(scaled(src[2 * q + 1], p.scale)) << 16);
        *reinterpret_cast<u32x4*>(p.out + ((static_cast<int64_t>(bb) * p.Hq + h) * p.P + i) * p.d + e) = v;
    }
}

}  // namespace

hipError_t launch_hidden_stats(const HiddenArgs& a, hipStream_t s) {
    dim3 g1(a.n_chunks, (a.D + kStatThreads * kStatVec - 1) / (kStatThreads * kStatVec), a.B);
    hipLaunchKernelGGL(hidden_stats_partial_kernel, g1, dim3(kStatThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((a.D + 255) / 256, a.B);
    hipLaunchKernelGGL(hidden_stats_final_kernel, g2, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_hidden_proxies(const HiddenArgs& a, hipStream_t s) {
    const int64_t items = static_cast<int64_t>(a.P) * (a.D / 4);
    dim3 g(static_cast<unsigned>((items + 255) / 256), a.B);
    hipLaunchKernelGGL(hidden_proxies_kernel, g, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_project(const ProjectArgs& p, hipStream_t s) {
    // without rotary tables, on full 128 x 224 tiles whose lane offsets fit
    // in 31 bits: one 128 x 224 tile per workgroup
    if (p.cos == nullptr && p.M % kWM == 0 && p.N % kWN == 0 && p.K % kWK == 0 && p.K >= 2 * kWK &&
        static_cast<int64_t>(p.M > p.N ? p.M : p.N) * p.K * 2 < (static_cast<int64_t>(1) << 31)) {
        hipLaunchKernelGGL(project_wide_kernel, dim3((p.M / kWM) * (p.N / kWN)), dim3(kGemmThreads), 0, s, p);
        return hipGetLastError();
    }
    dim3 g((p.M + kBM - 1) / kBM, (p.N + kBN - 1) / kBN);
    // full tiles: 64-wide k steps in two LDS stages loaded directly (two
    // workgroups per CU; deeper rings of 32- or 64-wide steps leave one per
    // CU, or more barriers per MFMA, and measured slower)
    if (p.M % kBM == 0 && p.N % kBN == 0 && p.K % 64 == 0)
        hipLaunchKernelGGL((project_dma_kernel<64, 2>), g, dim3(kGemmThreads), 0, s, p);
    else
        hipLaunchKernelGGL(project_kernel, g, dim3(kGemmThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace mmskv
