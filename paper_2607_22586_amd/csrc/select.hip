// tau-sets, votes, anchor score and budgeted selection (Sec. 3.2.2 Eqs. 9-10,
// Sec. 3.2.3 Eq. 11, Algorithm 1) on gfx950.
//
// tau_cut   one workgroup per (b, c, group): a mass-weighted radix select on
//           the fp32 bit patterns of the group masses (non-negative floats
//           order like their bits; 11/11/9-bit digits below the sign bit)
//           finds the cut mass theta and, among keys whose mass equals theta,
//           the last admitted index, such that
//           {mass > theta} u {mass == theta, index <= tcut} is the shortest
//           (mass desc, index asc) prefix whose mass reaches tau * total.
//           Masses are summed as integers in units of 2^-S (converted from
//           the float bits exactly), so every decision is independent of
//           summation order.  The register-resident variant (T <= 32768)
//           stops its passes early once the crossing bucket holds one key;
//           the sweep variant always runs all three.  Both end by writing
//           the group's membership plane: one bit per key, 32 keys a word.
// vote      one wave per two membership words at a time: vote = #groups
//           whose set holds the key, counted with one ballot per bit position;
//           score = vote + lambda*anchor (fp64), or the total mass.
// topk      one workgroup per (b, c): radix select (11-bit digits, stopping
//           early once a bucket is taken whole) of the (C-1)-th largest score
//           key over [0, T-1) (or the C-th over [0, T)), then an
//           index-ordered compaction writes the kept tokens in ascending
//           order and appends token T-1.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kTauThreads = 512;                 // register-resident tau cut

// floor(m * 2^S) for the finite, non-negative float with bit pattern `bits`,
// computed exactly from the significand and exponent (the product m * 2^S
// stays below 2^63 for every mass the score pass can produce).
__device__ __forceinline__ uint64_t fixed_of(uint32_t bits, int S) {
    const uint32_t e = (bits >> 23) & 0xFFu;
    const uint64_t man = static_cast<uint64_t>((bits & 0x7FFFFFu) | (e != 0 ? 0x800000u : 0u));
    // value = man * 2^(e - 150) (normal) or man * 2^-149 (subnormal)
    const int sh = (e != 0 ? static_cast<int>(e) : 1) - 150 + S;
    if (sh >= 0) return man << sh;
    if (sh <= -24) return 0ull;
    return man >> (-sh);
}

// The fixed-point value floor(m * 2^S) of a non-negative float m = man *
// 2^(e' - 150) (e' = max(e, 1), man with the implicit bit when e > 0) is
// man << sh for sh = e' - 150 + S >= 0 and man >> -sh otherwise.  Every key
// in one bucket of the tau-cut passes has the same exponent (the first digit
// holds the exponent bits, the later passes keep them in the prefix), so a
// bucket can sum mant_part(bits) = man >> max(-sh, 0) (under 2^24) and take
// the common factor 2^max(sh, 0) once: bucket_fixed(sum, e) is then exactly
// the sum of fixed_of over the bucket.
__device__ __forceinline__ int fixed_shift(uint32_t e, int S) {
    return (e != 0 ? static_cast<int>(e) : 1) - 150 + S;
}
__device__ __forceinline__ uint32_t mant_part(uint32_t bits, int S) {
    const uint32_t e = bits >> 23;           // sign bit is 0
    const uint32_t man = (bits & 0x7FFFFFu) | (e != 0 ? 0x800000u : 0u);
    const int rs = -fixed_shift(e, S);
    return rs <= 0 ? man : (rs >= 24 ? 0u : man >> rs);
}
__device__ __forceinline__ uint64_t bucket_fixed(uint64_t sum, uint32_t e, int S) {
    const int sh = fixed_shift(e, S);
    return sh > 0 ? sum << min(sh, 63) : sum;   // sh stays below 40 for any non-empty bucket
}

// Adds (count 1, value f) of every active lane to bucket `digit`, combining
// lanes of the wave that share a digit (skewed digit distributions would
// otherwise serialise on one LDS address).
__device__ __forceinline__ void hist_add(bool active, uint32_t digit, uint64_t f, uint32_t* cnt,
                                         unsigned long long* sum) {
    const int lane = lane_id();
    uint64_t pending = __ballot(active);
    for (int peel = 0; pending != 0; ++peel) {
        if (peel == 4) {
            if (active) {
                atomicAdd(&cnt[digit], 1u);
                if (sum) atomicAdd(&sum[digit], static_cast<unsigned long long>(f));
            }
            break;
        }
        const int leader = __ffsll(static_cast<unsigned long long>(pending)) - 1;
        const uint32_t d0 = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(digit), leader));
        const bool mine = active && digit == d0;
        const uint64_t m = __ballot(mine);
        if (sum) {
            const uint64_t v = wave_sum_u64(mine ? f : 0ull);
            if (lane == leader) atomicAdd(&sum[d0], static_cast<unsigned long long>(v));
        }
        if (lane == leader) atomicAdd(&cnt[d0], static_cast<uint32_t>(__popcll(m)));
        if (mine) active = false;
        pending &= ~m;
    }
}

// Block-wide exclusive prefix count of `flag` over the NT threads in thread
// order; returns the prefix and writes the block total.
template <int NT = kSelThreads>
__device__ __forceinline__ uint32_t block_excl_count(bool flag, uint32_t* wtot, uint32_t& total) {
    constexpr int kW = NT / kWave;
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const uint64_t m = __ballot(flag);
    const uint32_t below = static_cast<uint32_t>(__popcll(m & ((1ull << lane) - 1ull)));
    if (lane == 0) wtot[wave] = static_cast<uint32_t>(__popcll(m));
    __syncthreads();
    uint32_t before = 0, tot = 0;
    for (int w = 0; w < kW; ++w) {
        const uint32_t x = wtot[w];
        before += (w < wave) ? x : 0u;
        tot += x;
    }
    __syncthreads();
    total = tot;
    return before + below;
}

// Block-wide exclusive prefix sum of `v` over the NT threads in thread
// order; also returns the block total.
template <typename U, int NT = kSelThreads, bool kFence = true>
__device__ __forceinline__ U block_excl_scan(U v, U* wtot, U& total) {
    constexpr int kW = NT / kWave;
    const int lane = lane_id(), wave = static_cast<int>(threadIdx.x) / kWave;
    const U x = wave_incl_scan(v);
    if (lane == kWave - 1) wtot[wave] = x;
    __syncthreads();
    U before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kW; ++w) {
        const U t = wtot[w];
        before += (w < wave) ? t : U(0);
        tot += t;
    }
    // without kFence the caller puts a barrier before wtot is written again
    if (kFence) __syncthreads();
    total = tot;
    return before + x - v;
}

// Digits [0, 2048) visited in descending order, thread i of NT covering the
// 2048/NT digits below 2048 - (2048/NT)*i, bucket d holding val_of(d): finds
// the digit whose bucket takes the running total (from the top) to need =
// need_of(total of all buckets) (1 <= need <= total; no digit when need is
// 0).  Returns the total; writes, through shared memory, the digit, `need`
// minus the total of higher buckets, and the bucket's count (when `cnt` is
// given).
template <typename U, int NT, typename ValOf, typename NeedOf>
__device__ __forceinline__ U crossing_of(ValOf val_of, const uint32_t* cnt, NeedOf need_of, U* wtot,
                                         uint32_t* s_digit, U* s_rem, uint32_t* s_cnt) {
    constexpr int kPer = 2048 / NT;
    const int top = 2047 - kPer * static_cast<int>(threadIdx.x);
    U v[kPer];
    U mine = 0;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        v[k] = val_of(top - k);
        mine += v[k];
    }
    U total;
    U excl = block_excl_scan<U, NT, false>(mine, wtot, total);   // the barrier below guards wtot
    const U need = need_of(total);
    if (excl < need && need <= excl + mine) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            if (excl < need && need <= excl + v[k]) {
                *s_digit = top - k;
                *s_rem = need - excl;
                if (cnt != nullptr) *s_cnt = cnt[top - k];
            }
            excl += v[k];
        }
    }
    __syncthreads();
    return total;
}

template <typename U, int NT = kSelThreads>
__device__ __forceinline__ void descending_crossing(const U* val, const uint32_t* cnt, U need, U* wtot,
                                                    uint32_t* s_digit, U* s_rem, uint32_t* s_cnt) {
    crossing_of<U, NT>([val](int d) { return val[d]; }, cnt, [need](U) { return need; }, wtot, s_digit, s_rem,
                       s_cnt);
}

template <int NT = kSelThreads>
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, unsigned long long* scratch) {
    constexpr int kW = NT / kWave;
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    v = wave_sum_u64(v);
    if (lane == 0) scratch[wave] = v;
    __syncthreads();
    uint64_t t = 0;
    for (int w = 0; w < kW; ++w) t += scratch[w];
    __syncthreads();
    return t;
}

// tau-cut digits: bits 30..20, 19..9, 8..0 of the (sign-free) mass bits.
__device__ __forceinline__ int tau_shift(int pass) { return pass == 0 ? 20 : pass == 1 ? 9 : 0; }
__device__ __forceinline__ uint32_t tau_mask(int pass) { return pass == 0 ? 0u : pass == 1 ? 0xFFF00000u : 0xFFFFFE00u; }
__device__ __forceinline__ uint32_t tau_digit(uint32_t bits, int pass) {
    return (bits >> tau_shift(pass)) & (pass == 2 ? 0x1FFu : 0x7FFu);
}
// bits fixed once pass `pass` has chosen its digit
__device__ __forceinline__ uint32_t tau_fixed(int pass) {
    return pass == 0 ? 0xFFF00000u : pass == 1 ? 0xFFFFFE00u : 0xFFFFFFFFu;
}

// tau-set membership of key t for cut (theta, tcut): mass above the cut, or
// equal to it at an index up to tcut
__device__ __forceinline__ bool in_tau_set(uint32_t bits, int t, uint32_t theta, int32_t tcut) {
    return bits > theta || (bits == theta && t <= tcut);
}

// Position of score key t of a head in `keys`: thread-major for the
// register-resident top-k (thread i owns keys i*kpt .. i*kpt + kpt - 1 and
// reads its j-th at j*1024 + i, so the reads are contiguous), else t.
__device__ __forceinline__ int key_pos(const SelectArgs& a, int t) {
    return a.kpt > 0 ? (t % a.kpt) * 1024 + t / a.kpt : t;
}

// Group g's share of clearing the first-digit histogram of head hc (the
// vote kernel fills it).
__device__ __forceinline__ void clear_hist0_share(const SelectArgs& a, int64_t hc, int g) {
    const int lo = static_cast<int>((2048L * g) / a.G), hi = static_cast<int>((2048L * (g + 1)) / a.G);
    for (int i = lo + static_cast<int>(threadIdx.x); i < hi; i += static_cast<int>(blockDim.x)) a.hist0[hc * 2048 + i] = 0u;
}

// Word w of group g's membership plane of head hc.
__device__ __forceinline__ uint32_t* plane_word(const SelectArgs& a, int64_t hc, int g, int w) {
    const int nw = (a.T + 31) / 32;
    return a.planes + (hc * a.G + g) * nw + w;
}

// ---------------------------------------------------------------- tau cut
__global__ void __launch_bounds__(kSelThreads) tau_cut_kernel(SelectArgs a) {
    __shared__ uint32_t cnt[2048];
    __shared__ unsigned long long sum[2048];
    __shared__ unsigned long long wtot64[kSelWaves];
    __shared__ uint32_t wtot[kSelWaves];
    __shared__ uint32_t s_digit, s_cnt;
    __shared__ unsigned long long s_rem;
    __shared__ int32_t s_tcut;

    const int g = blockIdx.x, c = blockIdx.y, b = blockIdx.z;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const int64_t hcg = hc * a.G + g;
    const uint32_t* m = reinterpret_cast<const uint32_t*>(a.group_mass) + hcg * a.T;
    const int tid = threadIdx.x;
    const int S = a.fix_shift;
    clear_hist0_share(a, hc, g);

    uint64_t local = 0;
    for (int t = tid; t < a.T; t += kSelThreads) local += fixed_of(m[t], S);
    const uint64_t total = block_sum_u64(local, wtot64);
    // every mass below the fixed-point resolution: empty set
    uint32_t theta = 0xFFFFFFFFu;
    int32_t tcut = -1;
    if (total != 0) {
        unsigned long long need = static_cast<unsigned long long>(ceil(a.tau * static_cast<double>(total)));
        if (need < 1) need = 1;
        if (need > total) need = total;

        uint32_t prefix = 0;
        for (int pass = 0; pass < 3; ++pass) {
            const uint32_t mask = tau_mask(pass);
            for (int i = tid; i < 2048; i += kSelThreads) { cnt[i] = 0; sum[i] = 0; }
            __syncthreads();
            // uniform trip count: hist_add needs every lane of the wave
            for (int base = 0; base < a.T; base += kSelThreads) {
                const int t = base + tid;
                const uint32_t bits = t < a.T ? m[t] : 0u;
                const bool in = t < a.T && (bits & mask) == prefix;
                hist_add(in, tau_digit(bits, pass), in ? fixed_of(bits, S) : 0ull, cnt, sum);
            }
            __syncthreads();
            descending_crossing<unsigned long long>(sum, cnt, need, wtot64, &s_digit, &s_rem, &s_cnt);
            prefix |= s_digit << tau_shift(pass);
            need = s_rem;
        }
        // keys with mass == theta each carry f_theta; the first k_eq by index
        // enter the set (all of them when k_eq covers the bucket)
        theta = prefix;
        const uint64_t f_theta = fixed_of(prefix, S);
        const uint64_t k_eq = f_theta == 0 ? 1 : (need + f_theta - 1) / f_theta;
        if (k_eq >= s_cnt) {
            tcut = a.T;
        } else {
            if (tid == 0) s_tcut = a.T - 1;
            __syncthreads();
            uint64_t seen = 0;
            for (int base = 0; base < a.T; base += kSelThreads) {
                const int t = base + tid;
                const bool eq = t < a.T && m[t] == prefix;
                uint32_t tot;
                const uint32_t before = block_excl_count(eq, wtot, tot);
                if (eq && seen + before + 1 == k_eq) s_tcut = t;
                seen += tot;
                if (seen >= k_eq) break;
            }
            __syncthreads();
            tcut = s_tcut;
        }
    }
    if (tid == 0) {
        a.theta[hcg] = theta;
        a.tcut[hcg] = tcut;
    }
    // membership plane: each wave's 64 keys of a sweep step are two words
    const int lane = lane_id();
    for (int base = 0; base < a.T; base += kSelThreads) {
        const int t = base + tid;
        const uint64_t mb = __ballot(t < a.T && in_tau_set(m[t], t, theta, tcut));
        const int w = (base + (tid & ~(kWave - 1))) / 32 + lane;
        if (lane < 2 && 32 * w < a.T) *plane_word(a, hc, g, w) = static_cast<uint32_t>(mb >> (32 * lane));
    }
}

// ---------------------------------------------------------------- vote + score
// One workgroup per 32 membership words (128-byte lines of every group's
// plane) of one head, each wave two words at a time: in each half-wave,
// lane l reads the word of group l (32 groups at a time), and one ballot per
// bit position j counts, for both words at once, the groups whose set holds
// key j; lane j of each half keeps its own key's count.
constexpr int kVoteThreads = 256;
constexpr int kVoteWords = 32;                          // words per workgroup
constexpr int kVoteSteps = kVoteWords * kWave / (2 * kVoteThreads);

__global__ void __launch_bounds__(kVoteThreads) vote_score_kernel(SelectArgs a) {
    __shared__ uint32_t lh[2048];            // this workgroup's first-digit counts
    const int c = blockIdx.y, b = blockIdx.z;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const int lane = lane_id(), half = lane >> 5, j0 = lane & 31;
    const int nw = (a.T + 31) / 32;
    const int pool = a.keep_last ? a.T - 1 : a.T;
    const int wbase = static_cast<int>(blockIdx.x) * kVoteWords + 2 * kVoteSteps * (static_cast<int>(threadIdx.x) / kWave);
    for (int i = threadIdx.x; i < 2048; i += kVoteThreads) lh[i] = 0u;
    __syncthreads();
#pragma unroll
    for (int step = 0; step < kVoteSteps; ++step) {
        const int w = wbase + 2 * step + half;
        const int t = 32 * w + j0;
        double score = 0.0;
        if (a.mode == 0) {
            uint32_t vote = 0;
            for (int g0 = 0; g0 < a.G; g0 += 32) {
                const int g = g0 + j0;
                const uint32_t word = (w < nw && g < a.G) ? *plane_word(a, hc, g, w) : 0u;
#pragma unroll
                for (int j = 0; j < 32; ++j) {
                    const uint64_t m = __ballot((word >> j) & 1u);
                    const uint32_t n0 = static_cast<uint32_t>(__popcll(m & 0xFFFFFFFFull));
                    const uint32_t n1 = static_cast<uint32_t>(__popcll(m >> 32));
                    if (j0 == j) vote += half ? n1 : n0;
                }
            }
            if (t < a.T) {
                score = static_cast<double>(vote) + a.lambda * static_cast<double>(a.anchor[hc * a.T + t]);
                if (a.votes != nullptr) a.votes[hc * a.T + t] = static_cast<uint8_t>(vote);
            }
        } else if (t < a.T) {
            score = static_cast<double>(a.mass[hc * a.T + t]);
        }
        if (t < a.T) {
            const uint64_t key = static_cast<uint64_t>(__double_as_longlong(score));
            a.keys[hc * a.key_stride + key_pos(a, t)] = key;
            if (t < pool) atomicAdd(&lh[static_cast<uint32_t>(key >> 53) & 2047u], 1u);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 2048; i += kVoteThreads)
        if (lh[i] != 0u) atomicAdd(&a.hist0[hc * 2048 + i], lh[i]);
}

// Clears the first-digit histograms where no tau cut runs before the vote
// kernel (MASS mode).
__global__ void __launch_bounds__(256) clear_hist0_kernel(SelectArgs a) {
    const int64_t n = static_cast<int64_t>(a.B) * a.Hkv * 2048;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256)
        a.hist0[i] = 0u;
}

// ---------------------------------------------------------------- top-k
// Radix search for the selection threshold over the 64-bit score keys of
// the pool: 11-bit digits from the top (bits 63..53, ..., 9..0), stopping
// once the crossing bucket is taken whole.  `each(f)` calls f(key, ok) with
// the same trip count on every thread, ok marking the pool keys this thread
// owns.  On return, the selected keys are {key > theta} plus the first k_eq
// keys (by index) with key == theta.  Requires 1 <= want < pool size.  The
// first pass takes its counts from h0 (all pool keys by bits 63..53).
struct TopkShared {
    uint32_t cnt[2][2048];       // pass p counts into cnt[p % 2]
    uint32_t wtot[kSelWaves];
    uint32_t s_digit, s_cnt, s_rem;
};

template <typename Each>
__device__ __forceinline__ void topk_threshold(uint32_t want, Each each, const uint32_t* h0, TopkShared& sh,
                                               uint64_t& theta, uint32_t& k_eq) {
    const int tid = threadIdx.x;
    uint64_t prefix = 0, mask = 0;
    uint32_t need = want;
    // the first digit's counts, made by the vote kernel; the other buffer
    // cleared for the second pass
    for (int i = tid; i < 2048; i += kSelThreads) {
        sh.cnt[0][i] = h0[i];
        sh.cnt[1][i] = 0;
    }
    __syncthreads();
    for (int pass = 0; pass < 6; ++pass) {
        const int shift = pass == 5 ? 0 : 53 - 11 * pass;
        uint32_t* cnt = sh.cnt[pass & 1];
        if (pass > 0) {
            // plain LDS atomics over the keys left in the crossing bucket
            each([&](uint64_t kv, bool ok) {
                if (ok && (kv & mask) == prefix) atomicAdd(&cnt[static_cast<uint32_t>(kv >> shift) & 2047u], 1u);
            });
            __syncthreads();
        }
        descending_crossing<uint32_t>(cnt, cnt, need, sh.wtot, &sh.s_digit, &sh.s_rem, &sh.s_cnt);
        // every read of this buffer is done (the crossing ends with a
        // barrier): clear it for pass + 2, two barriers away
        for (int i = tid; i < 2048; i += kSelThreads) cnt[i] = 0;
        prefix |= static_cast<uint64_t>(sh.s_digit) << shift;
        mask |= (shift == 0 ? 0x1FFull : 0x7FFull) << shift;
        need = sh.s_rem;
        if (sh.s_cnt == need) {
            // the whole bucket is taken: every key >= its lower bound (> 0,
            // since the pool holds more keys than are wanted)
            theta = prefix - 1;
            k_eq = 0;
            return;
        }
    }
    theta = prefix;
    k_eq = need;
}

__global__ void __launch_bounds__(kSelThreads) topk_kernel(SelectArgs a) {
    __shared__ TopkShared sh;

    const int c = blockIdx.x, b = blockIdx.y;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const int tid = threadIdx.x;
    int32_t* out = a.idx + hc * a.c_max;
    int budget = a.budget;
    if (a.budgets != nullptr) budget = min(max(a.budgets[hc], 1), a.c_max);

    if (a.T <= budget) {
        for (int j = tid; j < a.c_max; j += kSelThreads) out[j] = (j < a.T) ? j : -1;
        if (tid == 0) a.counts[hc] = a.T;
        return;
    }
    const int pool = a.keep_last ? a.T - 1 : a.T;
    const uint32_t want = static_cast<uint32_t>(a.keep_last ? budget - 1 : budget);
    const uint64_t* key = a.keys + hc * a.key_stride;

    uint64_t theta = 0;
    uint32_t k_eq = 0;
    if (want > 0) {
        topk_threshold(want, [&](auto&& f) {
            for (int base = 0; base < pool; base += kSelThreads) {
                const int t = base + tid;
                f(t < pool ? key[t] : 0ull, t < pool);
            }
        }, a.hist0 + hc * 2048, sh, theta, k_eq);
    }
    uint32_t eq_seen = 0, written = 0;
    for (int base = 0; base < pool; base += kSelThreads) {
        const int t = base + tid;
        const bool in = t < pool;
        const uint64_t kv = in ? key[t] : 0ull;
        const bool gt = in && want > 0 && kv > theta;
        const bool eq = in && want > 0 && k_eq > 0 && kv == theta;
        uint32_t eq_tot;
        const uint32_t eq_before = block_excl_count(eq, sh.wtot, eq_tot);
        const bool sel = gt || (eq && eq_seen + eq_before < k_eq);
        uint32_t sel_tot;
        const uint32_t pos = block_excl_count(sel, sh.wtot, sel_tot);
        if (sel && written + pos < want) out[written + pos] = t;
        eq_seen += eq_tot;
        written = min(written + sel_tot, want);
    }
    if (a.keep_last) {
        if (tid == 0) out[written] = a.T - 1;
        written += 1;
    }
    for (int j = static_cast<int>(written) + tid; j < a.c_max; j += kSelThreads) out[j] = -1;
    if (tid == 0) a.counts[hc] = static_cast<int32_t>(written);
}

// ------------------------------------------- register-resident variants
// For T <= 1024 * KPT the whole row of one workgroup fits in registers:
// thread j holds elements [KPT*j, KPT*j + KPT) (index order), so the data
// is read from memory once and every index-ordered step (ties, compaction)
// needs one block scan instead of a sweep.

// tau cut of one (b, c, group); same result as tau_cut_kernel.  NT threads
// (512 up to T = 16384, so two workgroups share a CU and a launch of 512
// workgroups is resident at once; 1024 up to T = 32768) of at most 128
// VGPRs.  Thread i holds keys
// 2048 q + 4 i + e (q < KPT / 4, e < 4), so every load is one contiguous
// 16-byte piece per lane; the index-ordered steps (ties, the plane) go
// through the 2048-key chunks q in order.
template <int KPT, int NT>
__global__ void __launch_bounds__(NT) tau_cut_reg_kernel(SelectArgs a) {
    static_assert(KPT % 4 == 0, "whole 4-key pieces per thread");
    constexpr int kQ = KPT / 4;
    constexpr int kChunk = 4 * NT;
    constexpr int kW = NT / kWave;
    __shared__ uint32_t cnt[2048];
    __shared__ unsigned long long sum[2048];
    __shared__ unsigned long long wtot64[kW];
    __shared__ uint32_t wtot[kW];
    __shared__ uint32_t s_digit, s_cnt;
    __shared__ unsigned long long s_rem;
    __shared__ int32_t s_tcut;
    __shared__ uint32_t s_theta;

    const int g = blockIdx.x, c = blockIdx.y, b = blockIdx.z;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const int64_t hcg = hc * a.G + g;
    const uint32_t* m = reinterpret_cast<const uint32_t*>(a.group_mass) + hcg * a.T;
    const int tid = threadIdx.x, lane = lane_id();
    const int S = a.fix_shift;
    clear_hist0_share(a, hc, g);
    auto key_of = [&](int q, int e) { return kChunk * q + 4 * tid + e; };

    // masses (bits), held for all passes (their fixed-point values are
    // recomputed where needed); keys past T read as mass 0
    uint32_t mb[KPT];
    if ((a.T & 3) == 0 && (reinterpret_cast<uintptr_t>(m) & 15u) == 0) {
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            u32x4 x = {0u, 0u, 0u, 0u};
            if (key_of(q, 0) < a.T) x = *reinterpret_cast<const u32x4*>(m + key_of(q, 0));
            mb[4 * q] = x[0]; mb[4 * q + 1] = x[1]; mb[4 * q + 2] = x[2]; mb[4 * q + 3] = x[3];
        }
    } else {
#pragma unroll
        for (int q = 0; q < kQ; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) mb[4 * q + e] = key_of(q, e) < a.T ? m[key_of(q, e)] : 0u;
    }
    // every mass below the fixed-point resolution: empty set
    uint32_t theta = 0xFFFFFFFFu;
    int32_t tcut = -1;
    unsigned long long need = 0;
    uint32_t prefix = 0;
    bool found = true;
    {
#pragma nounroll
        for (int pass = 0; pass < 3; ++pass) {
            const uint32_t mask = tau_mask(pass);
            for (int i = tid; i < 2048; i += NT) { cnt[i] = 0; sum[i] = 0; }
            __syncthreads();
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                // opaque inside the pass loop, so the per-key values are not
                // hoisted out of it and kept live
                asm volatile("" : "+v"(mb[j]));
                if (key_of(j / 4, j % 4) < a.T && (mb[j] & mask) == prefix) {
                    const uint32_t dg = tau_digit(mb[j], pass);
                    atomicAdd(&cnt[dg], 1u);
                    atomicAdd(&sum[dg], static_cast<unsigned long long>(mant_part(mb[j], S)));
                }
            }
            __syncthreads();
            // bucket d's exponent: the digit's top 8 bits in the first pass,
            // the prefix's in the later ones
            const uint32_t e_pre = prefix >> 23;
            const unsigned long long total = crossing_of<unsigned long long, NT>(
                [&](int d) {
                    return static_cast<unsigned long long>(
                        bucket_fixed(sum[d], pass == 0 ? static_cast<uint32_t>(d) >> 3 : e_pre, S));
                },
                cnt,
                [&](unsigned long long tot) {
                    if (pass == 0) {
                        // the shortest prefix reaching tau * total (at least one key)
                        need = static_cast<unsigned long long>(ceil(a.tau * static_cast<double>(tot)));
                        if (need < 1) need = 1;
                        if (need > tot) need = tot;
                    }
                    return need;
                },
                wtot64, &s_digit, &s_rem, &s_cnt);
            if (pass == 0 && total == 0) {
                found = false;
                break;
            }
            prefix |= s_digit << tau_shift(pass);
            need = s_rem;
            if (pass < 2 && s_cnt == 1u) {
                // one key left in the crossing bucket: its mass is theta, and the
                // remaining passes would only spell out its low bits
#pragma unroll
                for (int j = 0; j < KPT; ++j)
                    if (key_of(j / 4, j % 4) < a.T && (mb[j] & tau_fixed(pass)) == prefix) s_theta = mb[j];
                __syncthreads();
                prefix = s_theta;
                break;
            }
        }
    }
    if (found) {
        theta = prefix;
        const uint64_t f_theta = fixed_of(prefix, S);
        const uint64_t k_eq = f_theta == 0 ? 1 : (need + f_theta - 1) / f_theta;
        if (k_eq >= s_cnt) {
            tcut = a.T;
        } else {
            // the k_eq-th key (by index) whose mass equals theta, chunk by chunk
            if (tid == 0) s_tcut = a.T - 1;
            uint64_t seen = 0;
#pragma nounroll
            for (int q = 0; q < kQ; ++q) {
                uint32_t n_eq = 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) n_eq += (key_of(q, e) < a.T && mb[4 * q + e] == prefix) ? 1u : 0u;
                uint32_t tot;
                const uint32_t before = block_excl_scan<uint32_t, NT>(n_eq, wtot, tot);
                if (seen + before < k_eq && k_eq <= seen + before + n_eq) {
                    uint64_t at = seen + before;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (key_of(q, e) < a.T && mb[4 * q + e] == prefix && ++at == k_eq) s_tcut = key_of(q, e);
                }
                seen += tot;
                if (seen >= k_eq) break;
            }
            __syncthreads();
            tcut = s_tcut;
        }
    }
    if (tid == 0) {
        a.theta[hcg] = theta;
        a.tcut[hcg] = tcut;
    }
    // membership plane: each lane's 4 bits, merged over the 8 lanes of a word
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
        uint32_t word = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = key_of(q, e);
            word |= (t < a.T && in_tau_set(mb[4 * q + e], t, theta, tcut)) ? 1u << (4 * (lane & 7) + e) : 0u;
        }
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) word |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(word), o, kWave));
        if ((lane & 7) == 0 && key_of(q, 0) < a.T) *plane_word(a, hc, g, key_of(q, 0) / 32) = word;
    }
}

// Budgeted selection of one (b, c); same result as topk_kernel.
template <int KPT>
__global__ void __launch_bounds__(kSelThreads) topk_reg_kernel(SelectArgs a) {
    __shared__ TopkShared sh;

    const int c = blockIdx.x, b = blockIdx.y;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const int tid = threadIdx.x;
    int32_t* out = a.idx + hc * a.c_max;
    int budget = a.budget;
    if (a.budgets != nullptr) budget = min(max(a.budgets[hc], 1), a.c_max);

    if (a.T <= budget) {
        for (int j = tid; j < a.c_max; j += kSelThreads) out[j] = (j < a.T) ? j : -1;
        if (tid == 0) a.counts[hc] = a.T;
        return;
    }
    const int pool = a.keep_last ? a.T - 1 : a.T;
    const uint32_t want = static_cast<uint32_t>(a.keep_last ? budget - 1 : budget);
    const uint64_t* key = a.keys + hc * a.key_stride;
    const int t0 = tid * KPT;
    uint64_t kv[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) kv[j] = (t0 + j < pool) ? key[j * kSelThreads + tid] : 0ull;

    uint64_t theta = 0;
    uint32_t k_eq = 0;
    if (want > 0) {
        topk_threshold(want, [&](auto&& f) {
#pragma unroll
            for (int j = 0; j < KPT; ++j) f(kv[j], t0 + j < pool);
        }, a.hist0 + hc * 2048, sh, theta, k_eq);
    }
    // index-ordered compaction: keys > theta, then the first k_eq equal keys
    uint32_t n_eq = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) n_eq += (want > 0 && k_eq > 0 && t0 + j < pool && kv[j] == theta) ? 1u : 0u;
    uint32_t eq_total = 0, eq_seen = 0;
    if (want > 0 && k_eq > 0) eq_seen = block_excl_scan<uint32_t>(n_eq, sh.wtot, eq_total);
    uint32_t sel_mask = 0, n_sel = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        const bool in = want > 0 && t0 + j < pool;
        const bool gt = in && kv[j] > theta;
        bool eq = in && k_eq > 0 && kv[j] == theta;
        if (eq) eq = eq_seen++ < k_eq;
        if (gt || eq) {
            sel_mask |= 1u << j;
            ++n_sel;
        }
    }
    uint32_t sel_total;
    uint32_t pos = block_excl_scan<uint32_t>(n_sel, sh.wtot, sel_total);
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        if ((sel_mask >> j) & 1u) {
            if (pos < want) out[pos] = t0 + j;
            ++pos;
        }
    }
    uint32_t written = min(sel_total, want);
    if (a.keep_last) {
        if (tid == 0) out[written] = a.T - 1;
        written += 1;
    }
    for (int j = static_cast<int>(written) + tid; j < a.c_max; j += kSelThreads) out[j] = -1;
    if (tid == 0) a.counts[hc] = static_cast<int32_t>(written);
}

}  // namespace

int select_kpt(int T) {
    // register-resident top-k while a row fits in 32 keys per thread of 1024
    const int per = (T + kSelThreads - 1) / kSelThreads;
    return per <= 4 ? 4 : per <= 8 ? 8 : per <= 16 ? 16 : per <= 32 ? 32 : 0;
}

hipError_t launch_select(const SelectArgs& a, int stages, hipStream_t s) {
    if (a.kpt != select_kpt(a.T) || a.key_stride != select_key_stride(a.T)) return hipErrorInvalidValue;
    hipError_t e = hipSuccess;
    if (stages & kSelectTau) {
        if (a.mode == 0) {
            // register-resident tau cut while a row fits in 32 masses per
            // thread of 512, then of 1024; the sweep kernel beyond
            dim3 g1(a.G, a.Hkv, a.B);
            const int tper = (a.T + kTauThreads - 1) / kTauThreads;
            const int tkpt = tper <= 8 ? 8 : tper <= 16 ? 16 : tper <= 32 ? 32 : tper <= 64 ? 64 : 0;
            switch (tkpt) {
                case 8: hipLaunchKernelGGL((tau_cut_reg_kernel<8, kTauThreads>), g1, dim3(kTauThreads), 0, s, a); break;
                case 16: hipLaunchKernelGGL((tau_cut_reg_kernel<16, kTauThreads>), g1, dim3(kTauThreads), 0, s, a); break;
                case 32: hipLaunchKernelGGL((tau_cut_reg_kernel<32, kTauThreads>), g1, dim3(kTauThreads), 0, s, a); break;
                case 64: hipLaunchKernelGGL((tau_cut_reg_kernel<32, kSelThreads>), g1, dim3(kSelThreads), 0, s, a); break;
                default: hipLaunchKernelGGL(tau_cut_kernel, g1, dim3(kSelThreads), 0, s, a); break;
            }
        } else {
            const int64_t n = static_cast<int64_t>(a.B) * a.Hkv * 2048;
            const int64_t blocks = (n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024;
            hipLaunchKernelGGL(clear_hist0_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, a);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (stages & kSelectVote) {
        const int nw = (a.T + 31) / 32;
        dim3 g2((nw + kVoteWords - 1) / kVoteWords, a.Hkv, a.B);
        hipLaunchKernelGGL(vote_score_kernel, g2, dim3(kVoteThreads), 0, s, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (stages & kSelectPick) {
        dim3 g3(a.Hkv, a.B);
        switch (a.kpt) {
            case 4: hipLaunchKernelGGL(topk_reg_kernel<4>, g3, dim3(kSelThreads), 0, s, a); break;
            case 8: hipLaunchKernelGGL(topk_reg_kernel<8>, g3, dim3(kSelThreads), 0, s, a); break;
            case 16: hipLaunchKernelGGL(topk_reg_kernel<16>, g3, dim3(kSelThreads), 0, s, a); break;
            case 32: hipLaunchKernelGGL(topk_reg_kernel<32>, g3, dim3(kSelThreads), 0, s, a); break;
            default: hipLaunchKernelGGL(topk_kernel, g3, dim3(kSelThreads), 0, s, a); break;
        }
        e = hipGetLastError();
    }
    return e;
}

}  // namespace mmskv
