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

// A 32-row tile of bf16 rows of D elements in LDS, each row padded by one
// 16-byte chunk: chunk c of row r sits at slot r*(D/8 + 1) + c.  The padding
// shifts consecutive rows by 4 banks, so the 16 rows read by 16 consecutive
// lanes (same chunk) hit 16 different bank groups, and a lane's fragment
// reads differ only by an immediate offset.
template <int D>
struct TileLds {
    static constexpr int kChunks = D / 8;             // 16-byte chunks per row
    static constexpr int kRow = kChunks + 1;          // padded row, in chunks
    static constexpr int kSlots = 32 * kRow;          // per tile
};

template <int D>
__device__ __forceinline__ bf16x8 lds_frag(const u32x4* stage, int row, int chunk) {
    return __builtin_bit_cast(bf16x8, stage[row * TileLds<D>::kRow + chunk]);
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

// Per-thread share of staging one tile: thread j moves 16-byte chunks
// j, j + threads, ... of the tile's 32 x D/8 chunks (global -> registers now,
// registers -> LDS later).  For a tile of proxy rows the source is one
// contiguous 32-row block, so the per-thread offsets are fixed and only the
// tile's base pointer changes.
template <int D, int WAVES>
struct Stager {
    static constexpr int kThreads = 64 * WAVES;
    static constexpr int kChunks = 32 * TileLds<D>::kChunks;
    static constexpr int kPer = (kChunks + kThreads - 1) / kThreads;
    static constexpr bool kExact = (kChunks % kThreads) == 0;
    u32x4 v[kPer];

    static __device__ __forceinline__ int chunk_of(int k) { return static_cast<int>(threadIdx.x) + k * kThreads; }
    static __device__ __forceinline__ bool active(int k) { return kExact || chunk_of(k) < kChunks; }
    // element offset of the chunk within a contiguous 32-row block
    static __device__ __forceinline__ int src_off(int k) { return 8 * chunk_of(k); }
    // LDS slot of the chunk
    static __device__ __forceinline__ int dst_slot(int k) {
        const int q = chunk_of(k);
        const int r = q / TileLds<D>::kChunks;
        return r * TileLds<D>::kRow + (q - r * TileLds<D>::kChunks);
    }
    // 32 consecutive proxy rows starting at `base`
    __device__ __forceinline__ void load_block(const uint16_t* base, const int (&off)[kPer]) {
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            if (active(k)) v[k] = *reinterpret_cast<const u32x4*>(base + off[k]);
    }
    // any tile of the padded row space (anchor rows)
    __device__ __forceinline__ void load_rows(const ScoreArgs& a, int b, int c, int row0) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            if (active(k)) {
                const int q = chunk_of(k);
                const int r = q / TileLds<D>::kChunks;
                const int cs = q - r * TileLds<D>::kChunks;
                v[k] = *reinterpret_cast<const u32x4*>(row_ptr<D>(a, b, c, row0 + r) + 8 * cs);
            }
        }
    }
    __device__ __forceinline__ void store(u32x4* stage) const {
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            if (active(k)) stage[dst_slot(k)] = v[k];
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

// Fragments of one 32-row tile for this lane: row (lane % 32), 16-byte
// chunks 2*kc + lane/32.
template <int D>
__device__ __forceinline__ void read_frags(const u32x4* sp, bf16x8 (&A)[D / 16], int lane) {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) A[kc] = lds_frag<D>(sp, lane & 31, 2 * kc + (lane >> 5));
}

// The MFMAs of one tile from the fragments in A; as soon as chunk kc has been
// issued, A[kc] is refilled from the next tile's LDS slot, so the LDS latency
// hides behind the remaining MFMAs.  KEYS_AS_ROWS: D = K * P^T (lane holds one
// proxy column, 16 keys per sub-tile); otherwise D = P * K^T (lane holds one
// key column, 16 proxy rows).
template <int D, bool KEYS_AS_ROWS>
__device__ __forceinline__ void tile_mfma(bf16x8 (&A)[D / 16], const u32x4* next,
                                          const bf16x8 (&kf)[kSub][D / 16], floatx16 (&acc)[kSub],
                                          int lane, const floatx16& init) {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
#pragma unroll
        for (int s = 0; s < kSub; ++s) {
            const floatx16 c0 = (kc == 0) ? init : acc[s];
            acc[s] = KEYS_AS_ROWS ? mfma32(kf[s][kc], A[kc], c0) : mfma32(A[kc], kf[s][kc], c0);
        }
        A[kc] = lds_frag<D>(next, lane & 31, 2 * kc + (lane >> 5));
    }
}

// Accumulator start for a P * K^T tile whose rows begin at `rowv`: each
// lane's 16 rows (8*m + 4*(lane/32) + j) get -L_row/kappa, so the MFMA result
// is s - L/kappa and the probability is 2^(kappa * acc).
__device__ __forceinline__ floatx16 row_offsets(const float* rowv, int lane) {
    floatx16 c;
#pragma unroll
    for (int m4 = 0; m4 < 4; ++m4) {
        const float4 v = *reinterpret_cast<const float4*>(rowv + 8 * m4 + 4 * (lane >> 5));
        c[4 * m4 + 0] = v.x;
        c[4 * m4 + 1] = v.y;
        c[4 * m4 + 2] = v.z;
        c[4 * m4 + 3] = v.w;
    }
    return c;
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

constexpr int kMergeTiles = 16;   // pass-1 tiles whose cross-wave merge is batched

template <int D, int WAVES, bool FULL>
__device__ __forceinline__ void lse_body(const ScoreArgs& a, int head, int kb, int b, int c,
                                         u32x4 (&stage)[3][TileLds<D>::kSlots],
                                         float2 (&mrg)[2][kMergeTiles][WAVES][32]) {
    using St = Stager<D, WAVES>;
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
    const int n_prox = a.rows / 32;
    const uint16_t* pbase =
        a.proxies + (static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh) * a.P * D;
    int off[St::kPer];
#pragma unroll
    for (int k = 0; k < St::kPer; ++k) off[k] = St::src_off(k);
    // tile t = rows [32t, 32t+32) of the padded row space
    auto load_tile = [&](St& st, int t) {
        if (t < n_prox) st.load_block(pbase + static_cast<int64_t>(32 * t) * D, off);
        else st.load_rows(a, b, c, 32 * t);
    };

    float2* part = a.part + (static_cast<int64_t>(head) * a.n_kb + kb) * a.rows_pad;
    // merged (max, sum) over the waves of tiles [16k, 16k+16), all threads
    auto merge_chunk = [&](int k) {
        const int n_in = min(kMergeTiles, n_tiles - kMergeTiles * k);
        for (int i = static_cast<int>(threadIdx.x); i < n_in * 32; i += 64 * WAVES) {
            const int tl = i >> 5, r = i & 31;
            float M = -INFINITY;
#pragma unroll
            for (int w = 0; w < WAVES; ++w) M = fmaxf(M, mrg[k & 1][tl][w][r].x);
            float S = 0.f;
            if (M != -INFINITY) {
#pragma unroll
                for (int w = 0; w < WAVES; ++w)
                    S += mrg[k & 1][tl][w][r].y * fast_exp2(mrg[k & 1][tl][w][r].x - M);
            }
            part[32 * (kMergeTiles * k + tl) + r] = make_float2(M, S);
        }
    };

    // Pipeline (LDS slots t % 3): in iteration t the proxy rows of tile t+2
    // go registers -> LDS, tile t+3 is fetched into registers, the MFMAs of
    // tile t run from A while A is refilled with tile t+1, and the column
    // statistics of tile t-1 are computed.
    St st;
    bf16x8 A[D / 16];
    load_tile(st, 0);
    st.store(stage[0]);
    if (n_tiles > 1) {
        load_tile(st, 1);
        st.store(stage[1]);
    }
    if (n_tiles > 2) load_tile(st, 2);
    __syncthreads();
    read_frags<D>(stage[0], A, lane);

    floatx16 acc[2][kSub];
    auto stage_next = [&](int t) {
        if (t + 2 < n_tiles) {
            st.store(stage[(t + 2) % 3]);
            if (t + 3 < n_tiles) load_tile(st, t + 3);
        }
    };
    auto stats_of = [&](const floatx16 (&ac)[kSub], int tile) {
        const float2 r = column_lse<FULL>(ac, valid, kappa);
        if (lane < 32) mrg[(tile / kMergeTiles) & 1][tile % kMergeTiles][wave][lane] = r;
    };
    // iteration 0
    stage_next(0);
    tile_mfma<D, true>(A, stage[1 % 3], kf, acc[0], lane, zero16());
    __syncthreads();
    // steady state; the merge of chunk k once its last tile's statistics are
    // in LDS
    auto body = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value, prev = cur ^ 1;
        stage_next(t);
        tile_mfma<D, true>(A, stage[(t + 1) % 3], kf, acc[cur], lane, zero16());
        stats_of(acc[prev], t - 1);
        if (t >= kMergeTiles + 1 && ((t - kMergeTiles - 1) % kMergeTiles) == 0)
            merge_chunk((t - kMergeTiles - 1) / kMergeTiles);
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
    // t == n_tiles: statistics of the last tile, then the unmerged chunks
    if ((n_tiles - 1) & 1) stats_of(acc[1], n_tiles - 1); else stats_of(acc[0], n_tiles - 1);
    __syncthreads();
    // the loop merged chunk k at t = 16k + 17 for every such t <= n_tiles - 1
    const int merged = n_tiles >= kMergeTiles + 2 ? (n_tiles - kMergeTiles - 2) / kMergeTiles + 1 : 0;
    for (int k = merged; k * kMergeTiles < n_tiles; ++k) merge_chunk(k);
}

template <int D, int WAVES>
__global__ void __launch_bounds__(64 * WAVES) score_lse_kernel(ScoreArgs a) {
    __shared__ u32x4 stage[3][TileLds<D>::kSlots];
    __shared__ float2 mrg[2][kMergeTiles][WAVES][32];
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
// p = 2^(kappa * acc) of one tile (acc already holds s - L/kappa), summed
// over this lane's rows 0-15 (hA) and rows 16-31 (hB) of the tile.
__device__ __forceinline__ void tile_probs(const floatx16 (&acc)[kSub], float kappa, float (&hA)[kSub],
                                           float (&hB)[kSub]) {
#pragma unroll
    for (int s = 0; s < kSub; ++s) {
        float sa = 0.f, sb = 0.f;
#pragma unroll
        for (int m4 = 0; m4 < 4; ++m4) {
            const float e0 = fast_exp2(acc[s][4 * m4 + 0] * kappa);
            const float e1 = fast_exp2(acc[s][4 * m4 + 1] * kappa);
            const float e2 = fast_exp2(acc[s][4 * m4 + 2] * kappa);
            const float e3 = fast_exp2(acc[s][4 * m4 + 3] * kappa);
            if (m4 < 2) sa += (e0 + e1) + (e2 + e3); else sb += (e0 + e1) + (e2 + e3);
        }
        hA[s] = sa;
        hB[s] = sb;
    }
}

// Position of a pass-2 tile: proxy block u (rows 32u.. of each head) and
// head h, visited u-major; advance() steps to the next tile.
struct TileCursor {
    int t, u, h;
    __device__ __forceinline__ void advance(int Gh) {
        ++t;
        if (++h == Gh) {
            h = 0;
            ++u;
        }
    }
};

template <int D, int WAVES>
__global__ void __launch_bounds__(64 * WAVES) score_mass_kernel(ScoreArgs a) {
    using St = Stager<D, WAVES>;
    __shared__ u32x4 stage[3][TileLds<D>::kSlots];
    extern __shared__ float4 dyn_lds[];
    float* Llds = reinterpret_cast<float*>(dyn_lds);     // [rows_pad]

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
    const int n_prox_tiles = (a.P / 32) * a.Gh;
    const int n_tiles = n_prox_tiles + (a.rows_pad - a.rows) / 32;
    const uint16_t* pbase =
        a.proxies + (static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh) * a.P * D;
    int off[St::kPer];
#pragma unroll
    for (int k = 0; k < St::kPer; ++k) off[k] = St::src_off(k);

    // this head's row offsets -L/kappa, all rows, stay in LDS for the whole kernel
    const float inv_kappa = 1.0f / kappa;
    for (int i = static_cast<int>(threadIdx.x); i < a.rows_pad; i += 64 * WAVES) Llds[i] = -L[i] * inv_kappa;

    // tiles t < n_prox_tiles: proxies 32u.. of head h; later: anchor rows
    auto load_tile = [&](St& st, const TileCursor& q) {
        if (q.t < n_prox_tiles)
            st.load_block(pbase + static_cast<int64_t>(q.h * a.P + 32 * q.u) * D, off);
        else
            st.load_rows(a, b, c, a.rows + 32 * (q.t - n_prox_tiles));
    };

    // Pipeline (LDS slots t % 3): in iteration t the rows of tile t+2 go
    // registers -> LDS, tile t+3 is fetched into registers, the MFMAs of tile
    // t run from A while A is refilled with tile t+1, and the probabilities
    // of tile t-1 are formed.
    St st;
    bf16x8 A[D / 16];
    TileCursor q3{0, 0, 0};                  // next tile to fetch
    load_tile(st, q3);
    st.store(stage[0]);
    q3.advance(a.Gh);
    if (n_tiles > 1) {
        load_tile(st, q3);
        st.store(stage[1]);
    }
    q3.advance(a.Gh);
    if (n_tiles > 2) load_tile(st, q3);
    q3.advance(a.Gh);
    __syncthreads();
    read_frags<D>(stage[0], A, lane);

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
    TileCursor q1{0, 0, 0};                  // tile whose probabilities come next
    auto group_step = [&](const float (&hA)[kSub], const float (&hB)[kSub]) {
#pragma unroll
        for (int s = 0; s < kSub; ++s) {
            runA[s] += hA[s];
            runB[s] += hB[s];
        }
        if (q1.h == a.Gh - 1) {
            const int u = q1.u;
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
        q1.advance(a.Gh);
    };
    auto anchor_step = [&](int tp, const floatx16 (&ac)[kSub]) {
        // anchor rows of tile tp: query head 32*(tp - n_prox_tiles) + row
        const int h0 = 32 * (tp - n_prox_tiles) + 4 * (lane >> 5);
#pragma unroll
        for (int m4 = 0; m4 < 4; ++m4)
#pragma unroll
            for (int s = 0; s < kSub; ++s)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float e = fast_exp2(ac[s][4 * m4 + j] * kappa);
                    aacc[s] += (h0 + 8 * m4 + j < a.Gh) ? e : 0.f;
                }
    };

    floatx16 acc[2][kSub];
    auto stage_next = [&](int t) {
        if (t + 2 < n_tiles) {
            st.store(stage[(t + 2) % 3]);
            if (t + 3 < n_tiles) load_tile(st, q3);
        }
        q3.advance(a.Gh);
    };
    TileCursor q0{0, 0, 0};                  // tile whose MFMAs come next
    auto tile_row = [&](const TileCursor& q) {
        return q.t < n_prox_tiles ? q.h * a.P + 32 * q.u : a.rows + 32 * (q.t - n_prox_tiles);
    };
    stage_next(0);
    tile_mfma<D, false>(A, stage[1 % 3], kf, acc[0], lane, row_offsets(Llds + tile_row(q0), lane));
    q0.advance(a.Gh);
    __syncthreads();
    // steady state over proxy tiles: MFMA of tile t next to the
    // probabilities of tile t-1 (the last of these MFMAs may be an anchor tile)
    auto body = [&](auto parity, int t) {
        constexpr int cur = decltype(parity)::value, prev = cur ^ 1;
        stage_next(t);
        tile_mfma<D, false>(A, stage[(t + 1) % 3], kf, acc[cur], lane, row_offsets(Llds + tile_row(q0), lane));
        q0.advance(a.Gh);
        float hA[kSub], hB[kSub];
        tile_probs(acc[prev], kappa, hA, hB);
        group_step(hA, hB);
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
            stage_next(t);
            tile_mfma<D, false>(A, stage[(t + 1) % 3], kf, acc[cur], lane, row_offsets(Llds + tile_row(q0), lane));
            q0.advance(a.Gh);
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
    hipLaunchKernelGGL((score_mass_kernel<D, WAVES>), dim3(a.B * a.Hkv * a.n_kb), dim3(64 * WAVES),
                       static_cast<size_t>(a.rows_pad) * sizeof(float), s, a);
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
