// Proxy-induced attention and mass aggregation (Sec. 3.2.2 Eqs. 7-8,
// Sec. 3.2.3 Eq. 11 anchor, Appendix B GQA aggregation) on gfx950.
//
// Work decomposition.  A workgroup of WAVES waves owns one (batch row b,
// KV head c) and a block of prompt keys; each wave keeps its keys (32*NS in
// pass 1, 64 in pass 2) resident in registers as bf16 MFMA fragments for
// the whole kernel.  Every proxy row of the Gh query heads that share KV
// head c (then the anchor rows) streams past those keys in 32-row tiles:
// the workgroup stages each tile once in a 4-slot LDS ring (rows padded by
// one 16-byte chunk so the fragment reads are bank-conflict free) and every
// wave multiplies it with v_mfma_f32_32x32x16_bf16 (fp32 accumulation).
// Within a wave the MFMAs of one tile (or chain) are issued alongside the
// exp/reduction VALU work of the previous one, so the matrix pipe and the
// VALU work side by side.  No logit reaches memory.
//
// An exact column mass needs every row's full normaliser, so the keys are
// scored twice:
//   score_lse:  D = K * P^T (keys as rows).  Per proxy row: the sum of 2^s
//               over the wave's keys, relative to zero while it stays in a
//               safe range and relative to the exact maximum otherwise,
//               merged over the waves through LDS into one (max, sum)
//               partial per (row, key block); lse_combine folds the partials
//               into L_row = log2 sum_t 2^(s_t).
//   score_mass: D = P * K^T (proxies as rows).  p = 2^(s - L_row);
//               column sums over the 16-row halves of each tile, accumulated
//               over the Gh heads into per-group masses, then over groups
//               into the total mass, and over the anchor rows.  Each key
//               column belongs to one wave, so there are no atomics and the
//               result is deterministic.
// The query rows carry the softmax scale log2(e)/sqrt(d) (the proxies from
// their construction, the anchor rows from their staging here, both in fp64
// before the bf16 rounding), so s = q~ . k is a base-2 logit and
// 2^s = e^(q.k/sqrt(d)).
//
// Workgroups are numbered so that all key blocks of one (b, c) land on the
// same XCD (workgroup i runs on XCD i mod 8), keeping that head's proxies in
// one L2.
//
// Early phase.  Every workgroup needs its whole key block before the
// pipeline can start, and all of them fetch their keys at once at the start
// of a pass.  Where the blocks allow it (full blocks of bf16 keys; pass 1
// with four sub-tiles per wave, pass 2 with 8-wave blocks at d = 128 and
// the paper's 16 proxies per group), the first 8 proxy tiles are staged in
// LDS slots of their own before any key load is issued, and their chains run
// sub-tile by sub-tile while the rest of the keys arrive, each round
// fetching the next sub-tile's keys.  Per tile the sums are formed in the
// pipeline's order, so the results are the same bits either way.
#include <math.h>

#include <utility>

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

// bf16 bits of the anchor value v (bf16 bits) times log2(e)/sqrt(d): the
// product in fp64, rounded fp64 -> fp32 -> bf16 like the proxies.
__device__ __forceinline__ uint32_t scaled_anchor(uint32_t v, double scale) {
    return f32_to_bf16_bits(static_cast<float>(static_cast<double>(__uint_as_float(v << 16)) * scale));
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
    // anchor tile ta of KV head (b, c), formed from the last window queries:
    // row r is query head c*Gh + 32 ta + r scaled (zero past Gh); hq0 is the
    // index of query head (b, c*Gh)
    __device__ __forceinline__ void load_anchor(const ScoreArgs& a, int64_t hq0, int ta) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            if (!active(k)) continue;
            const int q = chunk_of(k), r = q / TileLds<D>::kChunks, ch = q - r * TileLds<D>::kChunks;
            const int h = 32 * ta + r;
            u32x4 x = {0u, 0u, 0u, 0u};
            if (h < a.Gh) {
                const u32x4 raw = *reinterpret_cast<const u32x4*>(a.q_last + (hq0 + h) * D + 8 * ch);
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    x[w] = scaled_anchor(raw[w] & 0xFFFFu, a.anchor_scale) |
                           (scaled_anchor(raw[w] >> 16, a.anchor_scale) << 16);
            }
            v[k] = x;
        }
    }
    __device__ __forceinline__ void store(u32x4* stage) const {
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            if (active(k)) stage[dst_slot(k)] = v[k];
    }
};

// Key fragments of the wave's 32*NS keys: kf[s][kc] holds key
// key0 + 32*s + (lane % 32), dims [16*kc + 8*(lane/32), +8).
// (BF16_FULL: the caller has checked that the keys are bf16 and that every
// key of the sub-tile is < T, so the loads are unconditional and carry no
// branch, which keeps the compiler's count of outstanding loads exact)
template <int D, bool BF16_FULL = false>
__device__ __forceinline__ void load_key_sub(const ScoreArgs& a, int b, int c, int key0, int s,
                                             bf16x8 (&ks)[D / 16]) {
    const int lane = lane_id();
    const int col = 8 * (lane >> 5);
    const int t = key0 + 32 * s + (lane & 31);
    const bool ok = BF16_FULL || t < a.T;
    const int64_t off = static_cast<int64_t>(b) * a.ksb + static_cast<int64_t>(c) * a.ksh +
                        static_cast<int64_t>(ok ? t : 0) * a.kst;
    if (BF16_FULL || a.k_dtype == 1) {
        const uint16_t* p = static_cast<const uint16_t*>(a.k) + off + col;
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc) ks[kc] = ok ? load_bf16x8(p + 16 * kc) : zero_bf16x8();
    } else {
        const float* p = static_cast<const float*>(a.k) + off + col;
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc) ks[kc] = ok ? load_f32_as_bf16x8(p + 16 * kc) : zero_bf16x8();
    }
}

template <int D, int NS = kSub>
__device__ __forceinline__ void load_keys(const ScoreArgs& a, int b, int c, int key0,
                                          bf16x8 (&kf)[NS][D / 16]) {
#pragma unroll
    for (int s = 0; s < NS; ++s) load_key_sub<D>(a, b, c, key0, s, kf[s]);
}

// Fragments of one 32-row tile for this lane: row (lane % 32), 16-byte
// chunks 2*kc + lane/32.
template <int D>
__device__ __forceinline__ void read_frags(const u32x4* sp, bf16x8 (&A)[D / 16], int lane) {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) A[kc] = lds_frag<D>(sp, lane & 31, 2 * kc + (lane >> 5));
}

// Accumulator start for a P * K^T tile whose rows begin at `rowv`: each
// lane's 16 rows (8*m + 4*(lane/32) + j) get -L_row, so the MFMA result is
// s - L and the probability is 2^acc.
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

// Column totals over both half-waves for the wave's 64 keys: lane l < 32
// returns x0(l) + x0(l + 32) (sub-tile 0, key l), lane l >= 32 returns
// x1(l - 32) + x1(l) (sub-tile 1, key l), so lane l ends with key key0 + l.
__device__ __forceinline__ float pair_sum(float x0, float x1) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x0), __float_as_uint(x1), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Both half-waves' sum in every lane.
__device__ __forceinline__ float pair_total(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

constexpr int kRing = 4;   // LDS tile slots of the pipelined passes

template <int N>
struct Tag {
    static constexpr int value = N;
};

// f(Tag<0>{}), ..., f(Tag<N-1>{}), unrolled at compile time.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(Tag<I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ---------------------------------------------------------------- pass 1
constexpr int kMergeTiles = 16;   // pass-1 tiles whose cross-wave merge is batched
constexpr int kEarlyTiles = 8;    // pass-1 tiles taken sub-tile by sub-tile while the keys arrive
constexpr int kEarlySubs = 4;     // sub-tiles per wave of that schedule

// Pass 1 in the K * P^T layout.  Each wave holds NS sub-tiles of 32 keys; for
// every 32-row tile of the row space it runs one chain of D/16 dependent
// MFMAs per sub-tile (keys as rows, the tile's proxy rows as columns), so
// lane l holds column l % 32 (row 32t + l % 32) and keys key0 + 32*s +
// 8*(i/4) + 4*(l/32) + i%4 of sub-tile s (value i).  The 16 values of a
// chain are turned into 2^s and summed while the next chain's MFMAs run;
// two accumulator sets alternate between the chains.  The accumulators start
// at zero, so the MFMA leaves the base-2 logit itself and every logit costs
// one exp and one add (in a block with keys past T, a chain's accumulator
// starts at -inf on their rows instead).  A lane's running sum over the
// tile's chains is kept relative to zero while it lies in [2^-60, H) with
// H = lane_sum_hi, the bound under which no partial of a row's total can
// overflow; at 2^-60 or more the terms that underflow (each below 2^-126)
// are negligible against the sum.  A chain that would take it out of that
// range is taken again by the whole wave relative to each lane's exact
// maximum while its values are still in registers, and the lane's
// (max, sum) pair is merged by the max-and-rescale rule.  Per tile, the two half-waves' sums of each
// column are combined and the waves' pairs are merged every kMergeTiles tiles
// into one partial per (row, key block).  FULL: every key of the block is < T.
template <int D, int WAVES, int NS, bool FULL, bool EARLY, int SLOTS>
__device__ __forceinline__ void lse_body(const ScoreArgs& a, int head, int kb, int b, int c,
                                         u32x4 (&stage)[SLOTS][TileLds<D>::kSlots],
                                         float2 (&mrg)[2][kMergeTiles][WAVES][32]) {
    using St = Stager<D, WAVES>;
    constexpr int KC = D / 16;                 // MFMAs per chain
    static_assert(NS % 2 == 0, "chains alternate between two accumulator sets");
    static_assert(!EARLY || (FULL && NS == kEarlySubs && SLOTS >= kEarlyTiles && kEarlyTiles >= kRing),
                  "the early tiles are full blocks of four sub-tiles in their own LDS slots");
    const int wave = static_cast<int>(threadIdx.x) / kWave, lane = lane_id();
    const int key0 = kb * (32 * NS * WAVES) + wave * (32 * NS);

    bf16x8 kf[NS][KC];
    if constexpr (!EARLY) load_keys<D, NS>(a, b, c, key0, kf);
    // keys of sub-tile s held by this lane that are < T: value i is key
    // key0 + 32 s + 8 (i / 4) + 4 (lane / 32) + i % 4, valid while
    // 8 (i / 4) + i % 4 < n_keys(s)
    auto n_keys = [&](int s2) { return a.T - key0 - 32 * s2 - 4 * (lane >> 5); };

    const int n_tiles = a.rows_pad / 32;
    const int n_prox = a.rows / 32;
    const int64_t hq0 = static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh;
    const uint16_t* pbase = a.proxies + hq0 * a.P * D;
    int off[St::kPer];
#pragma unroll
    for (int k = 0; k < St::kPer; ++k) off[k] = St::src_off(k);
    St st;
    // tile t = rows [32t, 32t+32) of the padded row space
    auto load_tile = [&](int t) {
        if (t < n_prox) st.load_block(pbase + static_cast<int64_t>(32 * t) * D, off);
        else st.load_anchor(a, hq0, t - n_prox);
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

    // fragments of tile t in set t % 2; the other set is refilled with tile
    // t+1 while tile t's chains run, one 16-byte read per NS/2 MFMAs
    bf16x8 A[2][KC];
    floatx16 acc[2];
    if constexpr (!EARLY) {
        // Prologue: tiles 0-2 to LDS slots 0-2, tile 3 in the staging registers.
        for (int k = 0; k < 3; ++k) {
            if (k < n_tiles) {
                load_tile(k);
                st.store(stage[k]);
            }
        }
        if (3 < n_tiles) load_tile(3);
        __syncthreads();
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) A[0][kc] = lds_frag<D>(stage[0], lane & 31, 2 * kc + (lane >> 5));
    }
    // per-lane pair of the tile being summed: fast part relative to zero
    // (the running sum over the tile's chains so far), exact part (max, sum)
    // from chains that left the fast range; me and se are back at -inf and 0
    // whenever exact_tile is false
    float sf = 0.f, me = -INFINITY, se = 0.f;
    int exact_tile = 0;                        // wave-uniform flag

    // finish chain (values in acc[SETP], sub-tile SP) after its exps; nsf is
    // the running sum with this chain's values added: range check and, if
    // needed, the exact form
    auto finish_chain = [&](auto setp, auto sp, float nsf) {
        constexpr int SETP = decltype(setp)::value, SP = decltype(sp)::value;
        // a lane whose keys are all past T has nothing to sum
        const bool in_range = (nsf >= 0x1p-60f || (!FULL && n_keys(SP) <= 0)) && nsf < a.lane_sum_hi;
        if (__ballot(!in_range) == 0) {
            sf = nsf;
        } else {
            // the tile's first chain starts the running sum
            if (SP == 0) sf = 0.f;
            // (keys past T hold -inf and drop out of both)
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, acc[SETP][i]);
            if (mx != -INFINITY) {
                float ls = 0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) ls += fast_exp2(acc[SETP][i] - mx);
                const float mm = fmaxf(me, mx);
                se = (me == -INFINITY ? 0.f : se * fast_exp2(me - mm)) + ls * fast_exp2(mx - mm);
                me = mm;
            }
            // set here, inside the branch that the whole wave takes or
            // skips (as a select on the ballot it would cost two VALU ops
            // on the fast path)
            exact_tile = 1;
            asm volatile("" : "+s"(exact_tile));
        }
    };
    // column (max, sum) of a tile from both half-waves: fast part sfv
    // (relative to zero) and, when `exact` (wave-uniform), the exact part
    // (mev, sev)
    auto tile_pair = [&](float sfv, float mev, float sev, bool exact) {
        float mrow = 0.f, l;
        if (!exact) {
            // every chain was in range, so in a full block l >= 2^-60
            l = pair_total(sfv);
            if (!FULL && !(l > 0.f)) mrow = -INFINITY;
        } else {
            // lane pair: fast part (max 0) and exact part
            float M = sfv > 0.f ? fmaxf(0.f, mev) : mev;
            float S = 0.f;
            if (M != -INFINITY) S = (sfv > 0.f ? sfv * fast_exp2(-M) : 0.f) + (mev == -INFINITY ? 0.f : sev * fast_exp2(mev - M));
            const auto rm = __builtin_amdgcn_permlane32_swap(__float_as_uint(M), __float_as_uint(M), false, false);
            const auto rs = __builtin_amdgcn_permlane32_swap(__float_as_uint(S), __float_as_uint(S), false, false);
            const float m0 = __uint_as_float(rm[0]), m1 = __uint_as_float(rm[1]);
            const float s0 = __uint_as_float(rs[0]), s1 = __uint_as_float(rs[1]);
            mrow = fmaxf(m0, m1);
            l = 0.f;
            if (mrow != -INFINITY)
                l = (m0 == -INFINITY ? 0.f : s0 * fast_exp2(m0 - mrow)) + (m1 == -INFINITY ? 0.f : s1 * fast_exp2(m1 - mrow));
            // an empty sum (no valid key) carries no maximum, so it cannot
            // outweigh the pairs it is merged with
            if (!(l > 0.f)) mrow = -INFINITY;
        }
        return make_float2(mrow, l);
    };
    // column (max, sum) of tile tp from both half-waves, to LDS
    auto finish_tile = [&](int tp, bool merge_now) {
        const float2 pr = tile_pair(sf, me, se, exact_tile != 0);
        if (exact_tile) {
            me = -INFINITY;
            se = 0.f;
            exact_tile = 0;
        }
        if (lane < 32) mrg[(tp / kMergeTiles) & 1][tp % kMergeTiles][wave][lane] = pr;
        if (merge_now) merge_chunk((tp - kMergeTiles) / kMergeTiles);
    };

    // One pipeline iteration over tile t (LDS slot t % 4): chain s of tile t
    // runs its MFMAs while the exps of the chain before it (the last chain of
    // tile t-1 for s = 0) are formed; the last chain refills the fragments
    // with tile t+1; then tile t+3 is staged (registers -> LDS) and tile t+4
    // fetched; one barrier after every even iteration.  PREV: tile t-1
    // exists.  MF: tile t exists.  FAST: tile t+3 is staged and tile t+4 is
    // a proxy tile.
    auto iter = [&](auto t4, auto prev, auto mf, auto fast, int t) {
        constexpr int T4 = decltype(t4)::value;
        constexpr bool PREV = decltype(prev)::value != 0, MF = decltype(mf)::value != 0,
                       FAST = decltype(fast)::value != 0;
        const u32x4* next = stage[(T4 + 1) % kRing];
        auto chain = [&](auto si) {
            constexpr int S = decltype(si)::value;
            constexpr int CUR = S & 1, PRV = CUR ^ 1, SP = (S + NS - 1) % NS;
            constexpr bool HAVE_PREV = S > 0 ? MF : PREV;
            constexpr int AS = T4 & 1, AN = AS ^ 1;    // fragment sets of tiles t and t+1
            // the previous chain's values are added to the running sum (a
            // tile's first chain, SP == 0, starts it from -0, the additive
            // identity, so that first add is no instruction)
            float l0 = SP == 0 ? -0.f : sf, l1 = -0.f;
            if (!FULL && MF) {
                // keys past T start at -inf, so their 2^s is 0 (the mask is
                // opaque here so that the start values are not kept live
                // across the loop)
                int nk = n_keys(S);
                asm volatile("" : "+v"(nk));
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[CUR][i] = (8 * (i >> 2) + (i & 3) < nk) ? 0.f : -INFINITY;
            }
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                if (MF) acc[CUR] = mfma32(kf[S][kc], A[AS][kc], kc == 0 ? (FULL ? zero16() : acc[CUR]) : acc[CUR]);
                __builtin_amdgcn_sched_barrier(0);
                // the previous chain's values go to slots 1 .. KC-1, so none of
                // them is read before its last MFMA has had a slot to finish
                if (HAVE_PREV && kc > 0) {
                    constexpr int kSlots = KC - 1;
#pragma unroll
                    for (int i = 16 * (kc - 1) / kSlots; i < 16 * kc / kSlots; ++i) {
                        const float e = fast_exp2(acc[PRV][i]);
                        if (i & 1) l1 += e; else l0 += e;
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
                // MFMA slot j = S * KC + kc of the tile refills fragment j / NS
                // of tile t+1 after every NS-th slot
                if (MF && ((S * KC + kc) % NS) == NS - 1) {
                    const int f = (S * KC + kc) / NS;
                    A[AN][f] = lds_frag<D>(next, lane & 31, 2 * f + (lane >> 5));
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            if (HAVE_PREV) {
                finish_chain(Tag<PRV>{}, Tag<SP>{}, l0 + l1);
                if (S == 0) {
                    const int tp = t - 1;
                    finish_tile(tp, T4 == 1 && tp >= kMergeTiles && (tp - kMergeTiles) % kMergeTiles == 0);
                }
            }
        };
        // tile t+3 to LDS and tile t+4 into the staging registers, between
        // the chains so that their latency is covered by MFMAs
        auto staging = [&]() {
            if (FAST) {
                st.store(stage[(T4 + 3) % kRing]);
                st.load_block(pbase + static_cast<int64_t>(32 * (t + 4)) * D, off);
            } else if (t + 3 < n_tiles) {
                st.store(stage[(T4 + 3) % kRing]);
                if (t + 4 < n_tiles) load_tile(t + 4);
            }
        };
        chain(Tag<0>{});
        if constexpr (MF) {
            chain(Tag<1>{});
            staging();
            if constexpr (NS > 2) {
                chain(Tag<2>{});
                chain(Tag<3>{});
            }
        } else {
            staging();
        }
        if ((T4 & 1) == 0) __syncthreads();
    };
    int t0 = 0;
    if constexpr (EARLY) {
        // Early tiles: the first kEarlyTiles proxy tiles are staged in their
        // own LDS slots before any key load is issued, and their chains run
        // sub-tile by sub-tile (sub-tile 0 of every early tile, then
        // sub-tile 1, ...).  Only sub-tile 0's keys are fetched up front;
        // round s issues the loads of sub-tile s+1, so a quarter of the key
        // block is in flight at a time and each round waits for its own
        // quarter only (with every key load issued at once, the memory system
        // serves them in its own order, and since a wave's loads complete in
        // issue order the first quarter would be complete only near the end
        // of the whole burst).  Per tile, the chains are summed in the same
        // order as in the pipeline below, so the partials are the same
        // numbers.
        {
            St pre[kEarlyTiles];
#pragma unroll
            for (int k = 0; k < kEarlyTiles; ++k) pre[k].load_block(pbase + static_cast<int64_t>(32 * k) * D, off);
            load_key_sub<D, true>(a, b, c, key0, 0, kf[0]);
#pragma unroll
            for (int k = 0; k < kEarlyTiles; ++k) pre[k].store(stage[k]);
        }
        __syncthreads();
        float sp[kEarlyTiles];                 // running fast sum of each early tile
#pragma unroll
        for (int k = 0; k < kEarlyTiles; ++k) sp[k] = 0.f;
        int exact_mask = 0;                    // wave-uniform: early tiles with exact partials
        // exact partials (max, sum) per (early tile, lane) of this wave, in
        // the second merge buffer, which the pipeline first writes for tile
        // kMergeTiles (after the barriers below)
        float2* xs = &mrg[1][0][0][0] + wave * (kEarlyTiles * 64);
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) A[0][kc] = lds_frag<D>(stage[0], lane & 31, 2 * kc + (lane >> 5));
        // chain (sub-tile PS, tile PT) summed: running sum nsf, values in acc[PRV]
        auto early_finish = [&](auto prv, auto ps, auto pt, float nsf) {
            constexpr int PRV = decltype(prv)::value, PS = decltype(ps)::value, PT = decltype(pt)::value;
            const bool in_range = nsf >= 0x1p-60f && nsf < a.lane_sum_hi;
            if (__ballot(!in_range) == 0) {
                sp[PT] = nsf;
            } else {
                if (PS == 0) sp[PT] = 0.f;
                float mx = -INFINITY;
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, acc[PRV][i]);
                float2 ex = ((exact_mask >> PT) & 1) ? xs[PT * 64 + lane] : make_float2(-INFINITY, 0.f);
                if (mx != -INFINITY) {
                    float ls = 0.f;
#pragma unroll
                    for (int i = 0; i < 16; ++i) ls += fast_exp2(acc[PRV][i] - mx);
                    const float mm = fmaxf(ex.x, mx);
                    ex.y = (ex.x == -INFINITY ? 0.f : ex.y * fast_exp2(ex.x - mm)) + ls * fast_exp2(mx - mm);
                    ex.x = mm;
                }
                xs[PT * 64 + lane] = ex;
                exact_mask |= 1 << PT;
                asm volatile("" : "+s"(exact_mask));
            }
        };
        static_for<kEarlySubs * kEarlyTiles>([&](auto ci) {
            constexpr int C = decltype(ci)::value;
            constexpr int S = C / kEarlyTiles, TT = C % kEarlyTiles;
            constexpr int CUR = C & 1, PRV = CUR ^ 1;
            constexpr int PC = C > 0 ? C - 1 : 0, PS = PC / kEarlyTiles, PT = PC % kEarlyTiles;
            constexpr int NT = (TT + 1) % kEarlyTiles;     // the next chain's tile
            if constexpr (TT == 0 && S + 1 < kEarlySubs) load_key_sub<D, true>(a, b, c, key0, S + 1, kf[S + 1]);
            float l0 = (C > 0 && PS != 0) ? sp[PT] : -0.f, l1 = -0.f;
#pragma unroll
            for (int kc = 0; kc < KC; ++kc) {
                acc[CUR] = mfma32(kf[S][kc], A[C & 1][kc], kc == 0 ? zero16() : acc[CUR]);
                __builtin_amdgcn_sched_barrier(0);
                if (C > 0 && kc > 0) {
                    constexpr int kSlots = KC - 1;
#pragma unroll
                    for (int i = 16 * (kc - 1) / kSlots; i < 16 * kc / kSlots; ++i) {
                        const float e = fast_exp2(acc[PRV][i]);
                        if (i & 1) l1 += e; else l0 += e;
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
                if (C + 1 < kEarlySubs * kEarlyTiles)
                    A[(C + 1) & 1][kc] = lds_frag<D>(stage[NT], lane & 31, 2 * kc + (lane >> 5));
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (C > 0) early_finish(Tag<PRV>{}, Tag<PS>{}, Tag<PT>{}, l0 + l1);
        });
        // the pipeline's start: tiles kEarlyTiles .. +2 to ring slots 0-2,
        // the next in the staging registers (fetched before the last chain
        // is summed, stored once every wave is done with the early slots)
        constexpr int kLast = kEarlySubs * kEarlyTiles - 1;
        {
            St pre[3];
#pragma unroll
            for (int k = 0; k < 3; ++k) pre[k].load_block(pbase + static_cast<int64_t>(32 * (kEarlyTiles + k)) * D, off);
            load_tile(kEarlyTiles + 3);
            {
                float l0 = sp[kEarlyTiles - 1], l1 = -0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float e = fast_exp2(acc[kLast & 1][i]);
                    if (i & 1) l1 += e; else l0 += e;
                }
                early_finish(Tag<kLast & 1>{}, Tag<kEarlySubs - 1>{}, Tag<kEarlyTiles - 1>{}, l0 + l1);
            }
#pragma unroll
            for (int k = 0; k < kEarlyTiles; ++k) {
                const bool ex = ((exact_mask >> k) & 1) != 0;
                const float2 xe = ex ? xs[k * 64 + lane] : make_float2(-INFINITY, 0.f);
                const float2 pr = tile_pair(sp[k], xe.x, xe.y, ex);
                if (lane < 32) mrg[0][k][wave][lane] = pr;
            }
            __syncthreads();
#pragma unroll
            for (int k = 0; k < 3; ++k) pre[k].store(stage[k]);
        }
        __syncthreads();
#pragma unroll
        for (int kc = 0; kc < KC; ++kc) A[0][kc] = lds_frag<D>(stage[0], lane & 31, 2 * kc + (lane >> 5));
        t0 = kEarlyTiles;
    }
    using Off = Tag<0>;
    using On = Tag<1>;
    iter(Tag<0>{}, Off{}, On{}, Off{}, t0);
    int t = t0 + 1;
    __builtin_amdgcn_s_waitcnt(0);
    for (; t + 3 + 4 < n_prox; t += 4) {
        iter(Tag<1>{}, On{}, On{}, On{}, t);
        iter(Tag<2>{}, On{}, On{}, On{}, t + 1);
        iter(Tag<3>{}, On{}, On{}, On{}, t + 2);
        iter(Tag<0>{}, On{}, On{}, On{}, t + 3);
    }
    for (; t < n_tiles; t += 4) {
        iter(Tag<1>{}, On{}, On{}, Off{}, t);
        if (t + 1 < n_tiles) iter(Tag<2>{}, On{}, On{}, Off{}, t + 1);
        if (t + 2 < n_tiles) iter(Tag<3>{}, On{}, On{}, Off{}, t + 2);
        if (t + 3 < n_tiles) iter(Tag<0>{}, On{}, On{}, Off{}, t + 3);
    }
    // drain: the exps of the last tile's last chain (t == n_tiles here)
    switch (n_tiles & 3) {
        case 0: iter(Tag<0>{}, On{}, Off{}, Off{}, n_tiles); break;
        case 1: iter(Tag<1>{}, On{}, Off{}, Off{}, n_tiles); break;
        case 2: iter(Tag<2>{}, On{}, Off{}, Off{}, n_tiles); break;
        default: iter(Tag<3>{}, On{}, Off{}, Off{}, n_tiles); break;
    }
    __syncthreads();
    // chunk k was merged in iteration 16k+17 when that iteration ran (t <= n_tiles)
    const int merged = n_tiles >= kMergeTiles + 1 ? (n_tiles - kMergeTiles - 1) / kMergeTiles + 1 : 0;
    for (int k = merged; k * kMergeTiles < n_tiles; ++k) merge_chunk(k);
}

template <int D, int WAVES, int NS>
__global__ void __launch_bounds__(64 * WAVES) score_lse_kernel(ScoreArgs a) {
    constexpr bool kEarly = NS == kEarlySubs;
    constexpr int kSlotsAll = kEarly ? kEarlyTiles : kRing;
    __shared__ u32x4 stage[kSlotsAll][TileLds<D>::kSlots];
    __shared__ float2 mrg[2][kMergeTiles][WAVES][32];
    int head, kb;
    block_work(a.n_kb, head, kb);
    const int b = head / a.Hkv, c = head - b * a.Hkv;
    if ((kb + 1) * (32 * NS * WAVES) <= a.T) {
        // the early schedule needs every tile it stages ahead to be a proxy
        // tile, and bf16 keys (loaded without conversion)
        if constexpr (kEarly) {
            if (a.rows / 32 >= 2 * kMergeTiles && a.k_dtype == 1) {
                lse_body<D, WAVES, NS, true, true>(a, head, kb, b, c, stage, mrg);
                return;
            }
        }
        lse_body<D, WAVES, NS, true, false>(a, head, kb, b, c, stage, mrg);
    } else {
        lse_body<D, WAVES, NS, false, false>(a, head, kb, b, c, stage, mrg);
    }
}

// L_row = M + log2(sum_kb S_kb * 2^(M_kb - M)), one thread per row; the
// partials are fetched kCombineBatch at a time so their latencies overlap.
constexpr int kCombineBatch = 16;
__global__ void __launch_bounds__(256) lse_combine_kernel(ScoreArgs a) {
    const int r = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
    const int head = static_cast<int>(blockIdx.y);
    if (r >= a.rows_pad) return;
    const float2* p = a.part + static_cast<int64_t>(head) * a.n_kb * a.rows_pad + r;
    float M = -INFINITY, S = 0.f;
    for (int kb0 = 0; kb0 < a.n_kb; kb0 += kCombineBatch) {
        float2 v[kCombineBatch];
#pragma unroll
        for (int j = 0; j < kCombineBatch; ++j)
            v[j] = kb0 + j < a.n_kb ? p[static_cast<int64_t>(kb0 + j) * a.rows_pad] : make_float2(-INFINITY, 0.f);
        float bm = -INFINITY;
#pragma unroll
        for (int j = 0; j < kCombineBatch; ++j) bm = fmaxf(bm, v[j].x);
        if (bm > M) {
            S = (M == -INFINITY) ? 0.f : S * exp2f(M - bm);
            M = bm;
        }
        if (M != -INFINITY) {
#pragma unroll
            for (int j = 0; j < kCombineBatch; ++j)
                if (v[j].x != -INFINITY) S += v[j].y * exp2f(v[j].x - M);
        }
    }
    a.lse[static_cast<int64_t>(head) * a.rows_pad + r] = M + log2f(S);
}

// ---------------------------------------------------------------- pass 2
// Position of a pass-2 tile: proxy block u (rows 32u.. of each head) and
// head h, visited u-major, then the anchor tiles.
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

// EARLY: a full block of bf16 keys, 16 proxies per group (each 16-row half
// of a tile is one group) and 5 to 8 query heads per KV head (tiles 0-7 then
// close exactly one proxy block); see the early phase below.
template <int D, int WAVES, bool EARLY, int SLOTS>
__device__ __forceinline__ void mass_body(const ScoreArgs& a, int head, int kb,
                                          u32x4 (&stage)[SLOTS][TileLds<D>::kSlots], float* Llds) {
    using St = Stager<D, WAVES>;
    static_assert(!EARLY || SLOTS >= kEarlyTiles, "the early tiles have their own LDS slots");
    const int b = head / a.Hkv, c = head - b * a.Hkv;
    // the wave index in a scalar register, so that the priority branch below
    // is a scalar branch that each wave takes or skips
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave), lane = lane_id();
    const int key0 = kb * 64 * WAVES + wave * kWaveKeys;
    const float* L = a.lse + static_cast<int64_t>(head) * a.rows_pad;

    bf16x8 kf[kSub][D / 16];
    if constexpr (!EARLY) load_keys<D>(a, b, c, key0, kf);

    const int g16 = a.P / a.G / 16;          // 16-row halves per proxy group
    const int n_prox = (a.P / 32) * a.Gh;
    const int n_anc = (a.rows_pad - a.rows) / 32;
    const int64_t hq0 = static_cast<int64_t>(b) * a.Hq + static_cast<int64_t>(c) * a.Gh;
    const uint16_t* pbase = a.proxies + hq0 * a.P * D;
    int off[St::kPer];
#pragma unroll
    for (int k = 0; k < St::kPer; ++k) off[k] = St::src_off(k);

    // proxy tile (u, h): rows 32u.. of head h, first row h*P + 32u
    auto tile_row = [&](const TileCursor& q) { return q.h * a.P + 32 * q.u; };
    auto load_tile = [&](St& st, const TileCursor& q) {
        st.load_block(pbase + static_cast<int64_t>(tile_row(q)) * D, off);
    };

    // Pipeline over the proxy tiles t (LDS slot t % 4).  Iteration t issues
    // the MFMAs of tile t (fragments in A, accumulator start in Cn) while
    // refilling A with tile t+1, forms the probabilities of tile t-1 from the
    // other accumulator set, writes tile t+3 from registers to LDS, fetches
    // tile t+5 into registers and reads the accumulator start of tile t+1.
    // A slot is written two iterations before it is read and rewritten two
    // iterations after its last read, so one barrier after every even
    // iteration orders all LDS traffic.
    // Prologue: every load (keys above, the row offsets, tiles 0-4) is in
    // flight before the first store waits on any of them.  Tiles 0-2 go to
    // LDS slots 0-2; tiles 3 and 4 wait in the two staging register sets
    // (tile k in set k % 2), so each tile is fetched two iterations before
    // it is stored.
    St pre[3], st[2];
    TileCursor ld{0, 0, 0};                  // next tile to fetch
    constexpr int kLBatch = 8;               // row offsets fetched per thread at once
    auto l_batch = [&](int i0, auto&& between) {
        float lv[kLBatch];
#pragma unroll
        for (int j = 0; j < kLBatch; ++j) {
            const int i = i0 + j * 64 * WAVES;
            lv[j] = i < a.rows_pad ? L[i] : 0.f;
        }
        between();
#pragma unroll
        for (int j = 0; j < kLBatch; ++j) {
            const int i = i0 + j * 64 * WAVES;
            if (i < a.rows_pad) Llds[i] = -lv[j];
        }
    };
    TileCursor mm{0, 0, 0};                  // tile whose accumulator start is read next
    // accumulator starts of tiles t (set t % 2) and t + 1: read one tile ahead
    // into the other set, so none is copied
    floatx16 Cn[2];
    bf16x8 A[D / 16];
    if constexpr (!EARLY) {
        l_batch(static_cast<int>(threadIdx.x), [&]() {
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                if (ld.t < n_prox) load_tile(pre[k], ld);
                ld.advance(a.Gh);
            }
#pragma unroll
            for (int k = 3; k < 5; ++k) {
                if (ld.t < n_prox) load_tile(st[k & 1], ld);
                ld.advance(a.Gh);
            }
        });
        for (int i0 = static_cast<int>(threadIdx.x) + kLBatch * 64 * WAVES; i0 < a.rows_pad; i0 += kLBatch * 64 * WAVES)
            l_batch(i0, []() {});
#pragma unroll
        for (int k = 0; k < 3; ++k)
            if (k < n_prox) pre[k].store(stage[k]);
        __syncthreads();
        read_frags<D>(stage[0], A, lane);
        Cn[0] = row_offsets(Llds + tile_row(mm), lane);
        mm.advance(a.Gh);
    }

    const int64_t gm_base = static_cast<int64_t>(head) * a.G * a.T;
    const int my_key = key0 + lane;
    const bool my_ok = my_key < a.T;
    float runA[kSub][2] = {}, runB[kSub][2] = {}, open[kSub] = {0.f, 0.f};
    float macc = 0.f;
    int g_half = 0, g_idx = 0;               // halves in the open group, its index
    auto close_half = [&](float (&run)[kSub][2]) {
#pragma unroll
        for (int s = 0; s < kSub; ++s) {
            open[s] += run[s][0] + run[s][1];
            run[s][0] = run[s][1] = 0.f;
        }
        if (++g_half == g16) {
            const float tot = pair_sum(open[0], open[1]);
            macc += tot;
            if (a.group_mass != nullptr && my_ok) a.group_mass[gm_base + static_cast<int64_t>(g_idx) * a.T + my_key] = tot;
#pragma unroll
            for (int s = 0; s < kSub; ++s) open[s] = 0.f;
            g_half = 0;
            ++g_idx;
        }
    };
    // rows 0-15 of proxy tile (u, h) are half 2u of head h, rows 16-31 half
    // 2u+1; runA / runB sum each half over the Gh heads, and after the last
    // head both halves are closed
    int gs_h = 0;                            // head of the tile whose probabilities come next
    auto group_step = [&]() {
        if (++gs_h == a.Gh) {
            gs_h = 0;
            close_half(runA);
            close_half(runB);
        }
    };

    floatx16 acc[2][kSub];
    // One pipeline iteration; PROBS: tile t-1 exists (t > 0).  FAST: tile t
    // exists, tile t+3 is staged and tile t+5 fetched, so nothing branches.
    // The issue order is fixed by hand: after MFMA slot j of tile t come the
    // sums of value group j-1 and the exps of group j of tile t-1 (kPer32 of
    // its 32 accumulator values per group; the accumulator already holds the
    // base-2 exponent s - L), so no VALU step waits on the one before it and
    // the matrix pipe and the VALU work side by side; the fragment refill
    // follows the second MFMA of each k-chunk, the accumulator start of tile
    // t+1 is read halfway and the staging sits at the end.
    constexpr int kMfmas = kSub * (D / 16);
    constexpr int kPer32 = 32 / kMfmas;
    auto iter = [&](auto t4, auto probs, auto fast, int t) {
        constexpr int T4 = decltype(t4)::value;
        constexpr bool PROBS = decltype(probs)::value != 0, FAST = decltype(fast)::value != 0;
        constexpr int cur = T4 & 1, prev = cur ^ 1;
        const u32x4* next = stage[(T4 + 1) % kRing];
        const bool mfma_on = FAST || t < n_prox;
        // Issue priority: on every other tile the younger wave of each SIMD
        // (w >= WAVES/2) runs at the higher priority, so that the older one,
        // which otherwise wins every arbitration, does not run ahead and wait
        // at the barrier; on the other tiles both are equal.
        if ((T4 & 1) != 0 || wave >= WAVES / 2)
            __builtin_amdgcn_s_setprio(1);
        else
            __builtin_amdgcn_s_setprio(0);
        float ev[kPer32];
        auto add_group = [&](int g) {
#pragma unroll
            for (int v = 0; v < kPer32; ++v) {
                const int idx = g * kPer32 + v, s2 = idx / 16, i = idx % 16;
                if (i < 8) runA[s2][v & 1] += ev[v]; else runB[s2][v & 1] += ev[v];
            }
        };
        auto exp_group = [&](int g) {
#pragma unroll
            for (int v = 0; v < kPer32; ++v) {
                const int idx = g * kPer32 + v;
                ev[v] = fast_exp2(acc[prev][idx / 16][idx % 16]);
            }
        };
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc) {
#pragma unroll
            for (int s = 0; s < kSub; ++s) {
                const int slot = kSub * kc + s;
                if (mfma_on) acc[cur][s] = mfma32(A[kc], kf[s][kc], kc == 0 ? Cn[cur] : acc[cur][s]);
                if (PROBS) {
                    if (slot >= 1) add_group(slot - 1);
                    exp_group(slot);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            if (mfma_on) A[kc] = lds_frag<D>(next, lane & 31, 2 * kc + (lane >> 5));
            if (kc == D / 32) {
                // accumulator start of tile t+1 (a valid row block even past the end)
                Cn[prev] = row_offsets(Llds + ((FAST || mm.t < n_prox) ? tile_row(mm) : 0), lane);
                mm.advance(a.Gh);
            }
            if (kc == D / 32 - 1) {
                // tile t+3 (set (t+3) % 2) to LDS, then tile t+5 into the same
                // set, halfway through the MFMAs so their latency is covered
                constexpr int set = (T4 + 1) & 1;
                if (FAST) {
                    st[set].store(stage[(T4 + 3) % kRing]);
                    load_tile(st[set], ld);
                } else if (t + 3 < n_prox) {
                    st[set].store(stage[(T4 + 3) % kRing]);
                    if (ld.t < n_prox) load_tile(st[set], ld);
                }
                ld.advance(a.Gh);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (PROBS) {
            add_group(kMfmas - 1);
#pragma unroll
            for (int s = 0; s < kSub; ++s)
#pragma unroll
                for (int q = 0; q < 2; ++q) asm volatile("" : "+v"(runA[s][q]), "+v"(runB[s][q]));
        }
        if (PROBS) group_step();
        if ((T4 & 1) == 0) __syncthreads();
    };
    int t0 = 0;
    if constexpr (EARLY) {
        // Early phase (as in the log-sum-exp pass): tiles 0-7 are staged in
        // their own LDS slots before any key load, only sub-tile 0's keys are
        // fetched up front, and the tiles' 16 chains (8 MFMAs each) run
        // sub-tile by sub-tile, the first round fetching sub-tile 1's keys, so
        // each round waits only for its own half of the keys.  Each sub-tile
        // sums into its own runA / runB, in the same order as in the
        // pipeline; the proxy block that tiles 0 .. Gh-1 close is folded per
        // sub-tile when its last head passes and its two group masses are
        // formed once both sub-tiles are in.
        {
            St pre8[kEarlyTiles];
            l_batch(static_cast<int>(threadIdx.x), [&]() {
#pragma unroll
                for (int k = 0; k < kEarlyTiles; ++k) load_tile(pre8[k], TileCursor{k, k / a.Gh, k % a.Gh});
                load_key_sub<D, true>(a, b, c, key0, 0, kf[0]);
            });
            for (int i0 = static_cast<int>(threadIdx.x) + kLBatch * 64 * WAVES; i0 < a.rows_pad;
                 i0 += kLBatch * 64 * WAVES)
                l_batch(i0, []() {});
#pragma unroll
            for (int k = 0; k < kEarlyTiles; ++k) pre8[k].store(stage[k]);
        }
        __syncthreads();
        bf16x8 Ae[2][D / 16];
        floatx16 ce[2];                      // accumulators of the current and the previous chain
        float fold[2][kSub];                 // [half A / B][sub-tile]: the first proxy block's sums
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc) Ae[0][kc] = lds_frag<D>(stage[0], lane & 31, 2 * kc + (lane >> 5));
        Cn[0] = row_offsets(Llds + tile_row(TileCursor{0, 0, 0}), lane);
        // the sums of chain (sub-tile PS, tile PT), values in ce[PRV]; when
        // tile PT is the last head of proxy block 0, that block's sums of
        // sub-tile PS are set aside
        auto early_sum = [&](auto prv, auto ps, int pt, int i0, int i1) {
            constexpr int PRV = decltype(prv)::value, PS = decltype(ps)::value;
            (void)pt;
#pragma unroll
            for (int i = i0; i < i1; ++i) {
                const float e = fast_exp2(ce[PRV][i]);
                if (i < 8) runA[PS][i & 1] += e; else runB[PS][i & 1] += e;
            }
        };
        auto early_close = [&](auto ps, int pt) {
            constexpr int PS = decltype(ps)::value;
            if (pt == a.Gh - 1) {
                fold[0][PS] = runA[PS][0] + runA[PS][1];
                fold[1][PS] = runB[PS][0] + runB[PS][1];
                runA[PS][0] = runA[PS][1] = runB[PS][0] = runB[PS][1] = 0.f;
            }
        };
        static_for<kSub * kEarlyTiles>([&](auto ci) {
            constexpr int C = decltype(ci)::value;
            constexpr int S = C / kEarlyTiles, TT = C % kEarlyTiles;
            constexpr int CUR = C & 1, PRV = CUR ^ 1;
            constexpr int PC = C > 0 ? C - 1 : 0, PS = PC / kEarlyTiles, PT = PC % kEarlyTiles;
            constexpr int NT = (TT + 1) % kEarlyTiles;
            if constexpr (TT == 0 && S + 1 < kSub) load_key_sub<D, true>(a, b, c, key0, S + 1, kf[S + 1]);
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) {
                ce[CUR] = mfma32(Ae[C & 1][kc], kf[S][kc], kc == 0 ? Cn[C & 1] : ce[CUR]);
                __builtin_amdgcn_sched_barrier(0);
                // the previous chain's 16 values in slots 1-7 (none read
                // before its last MFMA has had a slot to finish)
                if (C > 0 && kc > 0) early_sum(Tag<PRV>{}, Tag<PS>{}, PT, 16 * (kc - 1) / 7, 16 * kc / 7);
                __builtin_amdgcn_sched_barrier(0);
                if (C + 1 < kSub * kEarlyTiles)
                    Ae[(C + 1) & 1][kc] = lds_frag<D>(stage[NT], lane & 31, 2 * kc + (lane >> 5));
                if (kc == D / 32 && C + 1 < kSub * kEarlyTiles)
                    Cn[(C + 1) & 1] = row_offsets(Llds + tile_row(TileCursor{NT, NT / a.Gh, NT % a.Gh}), lane);
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (C > 0) early_close(Tag<PS>{}, PT);
        });
        // the pipeline's start: tiles 8-10 to ring slots 0-2, tiles 11 and 12
        // in the staging registers (tile k in set k % 2), fetched before the
        // last chain is summed and stored once every wave is done with the
        // early slots
        constexpr int kLast = kSub * kEarlyTiles - 1;
        ld = TileCursor{kEarlyTiles, kEarlyTiles / a.Gh, kEarlyTiles % a.Gh};
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            load_tile(pre[k], ld);
            ld.advance(a.Gh);
        }
#pragma unroll
        for (int k = 3; k < 5; ++k) {
            load_tile(st[(kEarlyTiles + k) & 1], ld);
            ld.advance(a.Gh);
        }
        early_sum(Tag<kLast & 1>{}, Tag<kSub - 1>{}, kEarlyTiles - 1, 0, 16);
        early_close(Tag<kSub - 1>{}, kEarlyTiles - 1);
        // proxy block 0's two groups (halves A and B), as the pipeline forms
        // them: the sub-tile sums, then the pair of sub-tiles per key
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
            const float tot = pair_sum(fold[h2][0], fold[h2][1]);
            macc += tot;
            if (a.group_mass != nullptr) a.group_mass[gm_base + static_cast<int64_t>(h2) * a.T + my_key] = tot;
        }
        g_idx = 2;
        gs_h = kEarlyTiles % a.Gh;           // heads of proxy block 1 already summed
        // the anchor tile (Gh <= 8 rows: one tile) goes to early slot 4,
        // which nothing writes again, so the pipeline's end reads it there
        // without a barrier of its own
        St anc;
        anc.load_anchor(a, hq0, 0);
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 3; ++k) pre[k].store(stage[k]);
        anc.store(stage[kRing]);
        __syncthreads();
        read_frags<D>(stage[0], A, lane);
        mm = TileCursor{kEarlyTiles, kEarlyTiles / a.Gh, kEarlyTiles % a.Gh};
        Cn[0] = row_offsets(Llds + tile_row(mm), lane);
        mm.advance(a.Gh);
        t0 = kEarlyTiles;
    }
    using Off = Tag<0>;
    using On = Tag<1>;
    iter(Tag<0>{}, Off{}, Off{}, t0);
    int t = t0 + 1;
    // drain the key and staging loads of the prologue here, once, so that no
    // wait for them lands inside the loop
    __builtin_amdgcn_s_waitcnt(0);
    // steady state: t + 5 < n_prox
    for (; t + 3 + 5 < n_prox; t += 4) {
        iter(Tag<1>{}, On{}, On{}, t);
        iter(Tag<2>{}, On{}, On{}, t + 1);
        iter(Tag<3>{}, On{}, On{}, t + 2);
        iter(Tag<0>{}, On{}, On{}, t + 3);
    }
    // the rest, up to the probabilities of the last proxy tile (t = 1 mod 4 here)
    for (; t <= n_prox; t += 4) {
        iter(Tag<1>{}, On{}, Off{}, t);
        if (t + 1 <= n_prox) iter(Tag<2>{}, On{}, Off{}, t + 1);
        if (t + 2 <= n_prox) iter(Tag<3>{}, On{}, Off{}, t + 2);
        if (t + 3 <= n_prox) iter(Tag<0>{}, On{}, Off{}, t + 3);
    }

    // anchor tiles (the last window query of each of the Gh heads), outside
    // the pipeline: query head 32*ta + row of anchor tile ta
    float aacc[kSub] = {0.f, 0.f};
    for (int ta = 0; ta < n_anc; ++ta) {
        if constexpr (EARLY) {
            // staged after the early phase (n_anc == 1)
            read_frags<D>(stage[kRing], A, lane);
        } else {
            __syncthreads();
            st[0].load_anchor(a, hq0, ta);
            st[0].store(stage[0]);
            __syncthreads();
            read_frags<D>(stage[0], A, lane);
        }
        floatx16 ac[kSub];
        const floatx16 c0 = row_offsets(Llds + a.rows + 32 * ta, lane);
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc)
#pragma unroll
            for (int s = 0; s < kSub; ++s) ac[s] = mfma32(A[kc], kf[s][kc], kc == 0 ? c0 : ac[s]);
        const int h0 = 32 * ta + 4 * (lane >> 5);
#pragma unroll
        for (int m4 = 0; m4 < 4; ++m4)
#pragma unroll
            for (int s = 0; s < kSub; ++s)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float e = fast_exp2(ac[s][4 * m4 + j]);
                    aacc[s] += (h0 + 8 * m4 + j < a.Gh) ? e : 0.f;
                }
    }
    const float anc = pair_sum(aacc[0], aacc[1]) * (1.0f / static_cast<float>(a.Gh));
    if (my_ok) {
        const int64_t o = static_cast<int64_t>(head) * a.T + my_key;
        a.mass[o] = macc;
        a.anchor[o] = anc;
    }
}

template <int D, int WAVES>
__global__ void __launch_bounds__(64 * WAVES) score_mass_kernel(ScoreArgs a) {
    constexpr bool kEarly = WAVES == 8 && D == 128;
    __shared__ u32x4 stage[kEarly ? kEarlyTiles : kRing][TileLds<D>::kSlots];
    extern __shared__ float4 dyn_lds[];
    float* Llds = reinterpret_cast<float*>(dyn_lds);     // [rows_pad]
    int head, kb;
    block_work(a.mass_n_kb, head, kb);
    if constexpr (kEarly) {
        // (the early phase and the pipeline's start load tiles 0 .. 12 as
        // proxy tiles, so a head must have at least 16 of them)
        if ((kb + 1) * 64 * WAVES <= a.T && a.k_dtype == 1 && a.P == 16 * a.G && a.Gh >= 5 &&
            a.Gh <= kEarlyTiles && (a.P / 32) * a.Gh >= 2 * kEarlyTiles) {
            mass_body<D, WAVES, true>(a, head, kb, stage, Llds);
            return;
        }
    }
    mass_body<D, WAVES, false>(a, head, kb, stage, Llds);
}

template <int D, int WAVES, int NS>
hipError_t lse_impl(const ScoreArgs& a, int stages, hipStream_t s) {
    if (stages & kLseBlocks) {
        hipLaunchKernelGGL((score_lse_kernel<D, WAVES, NS>), dim3(a.B * a.Hkv * a.n_kb), dim3(64 * WAVES), 0, s, a);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (stages & kLseMerge) {
        dim3 g2((a.rows_pad + 255) / 256, a.B * a.Hkv);
        hipLaunchKernelGGL(lse_combine_kernel, g2, dim3(256), 0, s, a);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <int D, int WAVES>
hipError_t mass_impl(const ScoreArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((score_mass_kernel<D, WAVES>), dim3(a.B * a.Hkv * a.mass_n_kb), dim3(64 * WAVES),
                       static_cast<size_t>(a.rows_pad) * sizeof(float), s, a);
    return hipGetLastError();
}

}  // namespace

float lane_sum_limit(int T, int keys_per_sum) {
    const long n = (static_cast<long>(T) + keys_per_sum - 1) / keys_per_sum;   // lane sums per row
    int bits = 0;
    while ((1L << bits) < n) ++bits;                   // ceil(log2 n)
    const int e = 127 - bits < 120 ? 127 - bits : 120;
    return ldexpf(1.0f, e);
}

ScorePlan score_plan(int B, int Hkv, int T) {
    // the largest key blocks that still give every CU one block of work:
    // pass 1 with 8 waves of 128 keys, else 8 waves of 64, else 4 waves of
    // 64; pass 2 with 8-wave blocks (512 keys) when that gives every CU two
    // blocks, else 4-wave blocks (256 keys)
    const long heads = static_cast<long>(B) * Hkv;
    ScorePlan p;
    if (heads * ((T + 1023) / 1024) >= 256) {
        p.lse_waves = 8;
        p.lse_sub = 4;
    } else if (heads * ((T + 511) / 512) >= 256) {
        p.lse_waves = 8;
        p.lse_sub = 2;
    } else {
        p.lse_waves = 4;
        p.lse_sub = 2;
    }
    p.mass_waves = heads * ((T + 511) / 512) >= 512 ? 8 : 4;
    return p;
}

hipError_t launch_score_lse(const ScoreArgs& a, int stages, hipStream_t s) {
    const int w = a.lse_waves, ns = a.lse_sub;
    if (a.d == 64) {
        if (w == 8) return ns == 4 ? lse_impl<64, 8, 4>(a, stages, s) : lse_impl<64, 8, 2>(a, stages, s);
        return lse_impl<64, 4, 2>(a, stages, s);
    }
    if (w == 8) return ns == 4 ? lse_impl<128, 8, 4>(a, stages, s) : lse_impl<128, 8, 2>(a, stages, s);
    return lse_impl<128, 4, 2>(a, stages, s);
}

hipError_t launch_score_mass(const ScoreArgs& a, hipStream_t s) {
    const int w = a.block_keys / 64;
    if (a.d == 64) return w == 8 ? mass_impl<64, 8>(a, s) : mass_impl<64, 4>(a, s);
    return w == 8 ? mass_impl<128, 8>(a, s) : mass_impl<128, 4>(a, s);
}

}  // namespace mmskv
