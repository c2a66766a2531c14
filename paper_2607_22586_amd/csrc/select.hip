// tau-sets, votes, anchor score and budgeted selection (Sec. 3.2.2 Eqs. 9-10,
// Sec. 3.2.3 Eq. 11, Algorithm 1) on gfx950.
//
// tau_cut   one workgroup per (b, c, group): a mass-weighted radix select on
//           the fp32 bit patterns of the group masses (non-negative floats
//           order like their bits; 11/11/10-bit digits) finds the cut mass
//           theta and, among keys whose mass equals theta, the last admitted
//           index, such that {mass > theta} u {mass == theta, index <= tcut}
//           is the shortest (mass desc, index asc) prefix whose mass reaches
//           tau * total.  Masses are summed as 2^S fixed-point integers, so
//           every decision is independent of summation order.
// vote      one thread per key: vote = #groups whose set holds the key;
//           score = vote + lambda*anchor (fp64) or the total mass.
// topk      one workgroup per (b, c): radix select (11-bit digits, stopping
//           early once a bucket is taken whole) of the (C-1)-th largest score
//           key over [0, T-1) (or the C-th over [0, T)), then an index-ordered
//           compaction writes the kept tokens in ascending order and appends
//           token T-1.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace mmskv {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

__device__ __forceinline__ uint64_t to_fixed(float m, double scale) {
    return static_cast<uint64_t>(static_cast<double>(m) * scale);
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
        const uint32_t d0 = __shfl(digit, leader, kWave);
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

// Block-wide exclusive prefix count of `flag` over the 1024 threads in
// thread order; returns the prefix and writes the block total.
__device__ __forceinline__ uint32_t block_excl_count(bool flag, uint32_t* wtot, uint32_t& total) {
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    const uint64_t m = __ballot(flag);
    const uint32_t below = static_cast<uint32_t>(__popcll(m & ((1ull << lane) - 1ull)));
    if (lane == 0) wtot[wave] = static_cast<uint32_t>(__popcll(m));
    __syncthreads();
    uint32_t before = 0, tot = 0;
    for (int w = 0; w < kSelWaves; ++w) {
        const uint32_t x = wtot[w];
        before += (w < wave) ? x : 0u;
        tot += x;
    }
    __syncthreads();
    total = tot;
    return before + below;
}

// Block-wide exclusive prefix sum of `v` over the 1024 threads in thread
// order; also returns the block total.
template <typename U>
__device__ __forceinline__ U block_excl_scan(U v, U* wtot, U& total) {
    const int lane = lane_id(), wave = static_cast<int>(threadIdx.x) / kWave;
    U x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        U y;
        if constexpr (sizeof(U) == 8)
            y = shfl_u64(x, lane >= o ? lane - o : lane);
        else
            y = __shfl(x, lane >= o ? lane - o : lane, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) wtot[wave] = x;
    __syncthreads();
    U before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        const U t = wtot[w];
        before += (w < wave) ? t : U(0);
        tot += t;
    }
    __syncthreads();
    total = tot;
    return before + x - v;
}

// Digits [0, 2048) visited in descending order, thread i covering digits
// 2047-2i and 2046-2i: finds the digit whose bucket takes the running total
// (from the top) to `need` (need >= 1, need <= total).  Returns, through
// shared memory, the digit, `need` minus the total of higher buckets, and the
// bucket's count.
template <typename U>
__device__ __forceinline__ void descending_crossing(const U* val, const uint32_t* cnt, U need, U* wtot,
                                                    uint32_t* s_digit, U* s_rem, uint32_t* s_cnt) {
    const int i = static_cast<int>(threadIdx.x);
    const int d_hi = 2047 - 2 * i, d_lo = 2046 - 2 * i;
    const U v_hi = val[d_hi], v_lo = val[d_lo];
    U total;
    const U excl = block_excl_scan<U>(v_hi + v_lo, wtot, total);
    if (excl < need && need <= excl + v_hi + v_lo) {
        if (excl + v_hi >= need) {
            *s_digit = d_hi;
            *s_rem = need - excl;
            *s_cnt = cnt[d_hi];
        } else {
            *s_digit = d_lo;
            *s_rem = need - excl - v_hi;
            *s_cnt = cnt[d_lo];
        }
    }
    __syncthreads();
}

__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, unsigned long long* scratch) {
    const int lane = lane_id(), wave = threadIdx.x / kWave;
    v = wave_sum_u64(v);
    if (lane == 0) scratch[wave] = v;
    __syncthreads();
    uint64_t t = 0;
    for (int w = 0; w < kSelWaves; ++w) t += scratch[w];
    __syncthreads();
    return t;
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
    const int64_t hcg = (static_cast<int64_t>(b) * a.Hkv + c) * a.G + g;
    const float* m = a.group_mass + hcg * a.T;
    const int tid = threadIdx.x;

    uint64_t local = 0;
    for (int t = tid; t < a.T; t += kSelThreads) local += to_fixed(m[t], a.fix_scale);
    const uint64_t total = block_sum_u64(local, wtot64);
    if (total == 0) {
        // every mass is below the fixed-point resolution: empty set
        if (tid == 0) { a.theta[hcg] = 0xFFFFFFFFu; a.tcut[hcg] = -1; }
        return;
    }
    unsigned long long need = static_cast<unsigned long long>(ceil(a.tau * static_cast<double>(total)));
    if (need < 1) need = 1;
    if (need > total) need = total;

    // digits: bits 31..21, 20..10, 9..0 (the sign bit is 0)
    const int shifts[3] = {21, 10, 0};
    const uint32_t masks[3] = {0u, 0xFFE00000u, 0xFFFFFC00u};
    uint32_t prefix = 0;
    for (int pass = 0; pass < 3; ++pass) {
        const int shift = shifts[pass];
        const uint32_t mask = masks[pass];
        for (int i = tid; i < 2048; i += kSelThreads) { cnt[i] = 0; sum[i] = 0; }
        __syncthreads();
        for (int t = tid; t < a.T; t += kSelThreads) {
            const float mv = m[t];
            const uint32_t bits = __float_as_uint(mv);
            if ((bits & mask) == prefix) {
                const uint32_t dg = (bits >> shift) & 2047u;
                atomicAdd(&cnt[dg], 1u);
                atomicAdd(&sum[dg], static_cast<unsigned long long>(to_fixed(mv, a.fix_scale)));
            }
        }
        __syncthreads();
        descending_crossing<unsigned long long>(sum, cnt, need, wtot64, &s_digit, &s_rem, &s_cnt);
        prefix |= s_digit << shift;
        need = s_rem;
    }
    // keys with mass == theta each carry f_theta; the first k_eq by index
    // enter the set (all of them when k_eq covers the bucket)
    const uint64_t f_theta = to_fixed(__uint_as_float(prefix), a.fix_scale);
    const uint64_t k_eq = f_theta == 0 ? 1 : (need + f_theta - 1) / f_theta;
    if (k_eq >= s_cnt) {
        if (tid == 0) { a.theta[hcg] = prefix; a.tcut[hcg] = a.T; }
        return;
    }
    if (tid == 0) s_tcut = a.T - 1;
    __syncthreads();
    uint64_t seen = 0;
    for (int base = 0; base < a.T; base += kSelThreads) {
        const int t = base + tid;
        const bool eq = t < a.T && __float_as_uint(m[t]) == prefix;
        uint32_t tot;
        const uint32_t before = block_excl_count(eq, wtot, tot);
        if (eq && seen + before + 1 == k_eq) s_tcut = t;
        seen += tot;
        if (seen >= k_eq) break;
    }
    __syncthreads();
    if (tid == 0) {
        a.theta[hcg] = prefix;
        a.tcut[hcg] = s_tcut;
    }
}

// ---------------------------------------------------------------- vote + score
__global__ void __launch_bounds__(256) vote_score_kernel(SelectArgs a) {
    __shared__ uint32_t th[256];
    __shared__ int32_t tc[256];
    const int c = blockIdx.y, b = blockIdx.z;
    const int64_t hc = static_cast<int64_t>(b) * a.Hkv + c;
    const bool vote_mode = a.mode == 0;
    if (vote_mode) {
        for (int i = threadIdx.x; i < a.G; i += 256) {
            th[i] = a.theta[hc * a.G + i];
            tc[i] = a.tcut[hc * a.G + i];
        }
    }
    __syncthreads();
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= a.T) return;
    double score;
    if (vote_mode) {
        int vote = 0;
        const float* gm = a.group_mass + hc * a.G * static_cast<int64_t>(a.T) + t;
        for (int g = 0; g < a.G; ++g) {
            const uint32_t bits = __float_as_uint(gm[static_cast<int64_t>(g) * a.T]);
            vote += (bits > th[g] || (bits == th[g] && t <= tc[g])) ? 1 : 0;
        }
        score = static_cast<double>(vote) + a.lambda * static_cast<double>(a.anchor[hc * a.T + t]);
        if (a.votes != nullptr) a.votes[hc * a.T + t] = static_cast<uint8_t>(vote);
    } else {
        score = static_cast<double>(a.mass[hc * a.T + t]);
    }
    a.keys[hc * a.T + t] = static_cast<uint64_t>(__double_as_longlong(score));
}

// ---------------------------------------------------------------- top-k
__global__ void __launch_bounds__(kSelThreads) topk_kernel(SelectArgs a) {
    __shared__ uint32_t cnt[2048];
    __shared__ uint32_t wtot[kSelWaves];
    __shared__ uint32_t s_digit, s_cnt, s_rem;

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
    const uint64_t* key = a.keys + hc * a.T;

    // selected: key > theta, or key == theta among the first k_eq by index
    uint64_t theta = 0;
    uint32_t k_eq = 0;
    if (want > 0) {
        const int shifts[6] = {53, 42, 31, 20, 9, 0};
        uint64_t prefix = 0, mask = 0;
        uint32_t need = want;
        bool settled = false;
        for (int pass = 0; pass < 6 && !settled; ++pass) {
            const int shift = shifts[pass];
            for (int i = tid; i < 2048; i += kSelThreads) cnt[i] = 0;
            __syncthreads();
            for (int base = 0; base < pool; base += kSelThreads) {
                const int t = base + tid;
                const bool in = t < pool;
                const uint64_t kv = in ? key[t] : 0ull;
                const bool cand = in && (kv & mask) == prefix;
                hist_add(cand, static_cast<uint32_t>(kv >> shift) & 2047u, 0ull, cnt, nullptr);
            }
            __syncthreads();
            descending_crossing<uint32_t>(cnt, cnt, need, wtot, &s_digit, &s_rem, &s_cnt);
            prefix |= static_cast<uint64_t>(s_digit) << shift;
            mask |= (shift == 0 ? 0x1FFull : 0x7FFull) << shift;
            need = s_rem;
            if (s_cnt == need) {
                // the whole bucket is taken: every key >= its lower bound
                // (> 0, since the pool holds more keys than are wanted)
                theta = prefix - 1;
                k_eq = 0;
                settled = true;
            }
        }
        if (!settled) {
            theta = prefix;
            k_eq = need;
        }
    }
    uint32_t eq_seen = 0, written = 0;
    for (int base = 0; base < pool; base += kSelThreads) {
        const int t = base + tid;
        const bool in = t < pool;
        const uint64_t kv = in ? key[t] : 0ull;
        const bool gt = in && want > 0 && kv > theta;
        const bool eq = in && want > 0 && k_eq > 0 && kv == theta;
        uint32_t eq_tot;
        const uint32_t eq_before = block_excl_count(eq, wtot, eq_tot);
        const bool sel = gt || (eq && eq_seen + eq_before < k_eq);
        uint32_t sel_tot;
        const uint32_t pos = block_excl_count(sel, wtot, sel_tot);
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

// tau cut of one (b, c, group); same result as tau_cut_kernel.
template <int KPT>
__global__ void __launch_bounds__(kSelThreads) tau_cut_reg_kernel(SelectArgs a) {
    __shared__ uint32_t cnt[2048];
    __shared__ unsigned long long sum[2048];
    __shared__ unsigned long long wtot64[kSelWaves];
    __shared__ uint32_t wtot[kSelWaves];
    __shared__ uint32_t s_digit, s_cnt;
    __shared__ unsigned long long s_rem;
    __shared__ int32_t s_tcut;

    const int g = blockIdx.x, c = blockIdx.y, b = blockIdx.z;
    const int64_t hcg = (static_cast<int64_t>(b) * a.Hkv + c) * a.G + g;
    const float* m = a.group_mass + hcg * a.T;
    const int tid = threadIdx.x;
    const int t0 = tid * KPT;

    float mv[KPT];
    uint64_t local = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        mv[j] = (t0 + j < a.T) ? m[t0 + j] : 0.f;
        local += to_fixed(mv[j], a.fix_scale);
    }
    const uint64_t total = block_sum_u64(local, wtot64);
    if (total == 0) {
        if (tid == 0) { a.theta[hcg] = 0xFFFFFFFFu; a.tcut[hcg] = -1; }
        return;
    }
    unsigned long long need = static_cast<unsigned long long>(ceil(a.tau * static_cast<double>(total)));
    if (need < 1) need = 1;
    if (need > total) need = total;

    const int shifts[3] = {21, 10, 0};
    const uint32_t masks[3] = {0u, 0xFFE00000u, 0xFFFFFC00u};
    uint32_t prefix = 0;
    for (int pass = 0; pass < 3; ++pass) {
        const int shift = shifts[pass];
        const uint32_t mask = masks[pass];
        for (int i = tid; i < 2048; i += kSelThreads) { cnt[i] = 0; sum[i] = 0; }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const uint32_t bits = __float_as_uint(mv[j]);
            if (t0 + j < a.T && (bits & mask) == prefix) {
                const uint32_t dg = (bits >> shift) & 2047u;
                atomicAdd(&cnt[dg], 1u);
                atomicAdd(&sum[dg], static_cast<unsigned long long>(to_fixed(mv[j], a.fix_scale)));
            }
        }
        __syncthreads();
        descending_crossing<unsigned long long>(sum, cnt, need, wtot64, &s_digit, &s_rem, &s_cnt);
        prefix |= s_digit << shift;
        need = s_rem;
    }
    const uint64_t f_theta = to_fixed(__uint_as_float(prefix), a.fix_scale);
    const uint64_t k_eq = f_theta == 0 ? 1 : (need + f_theta - 1) / f_theta;
    if (k_eq >= s_cnt) {
        if (tid == 0) { a.theta[hcg] = prefix; a.tcut[hcg] = a.T; }
        return;
    }
    // the k_eq-th key (by index) whose mass equals theta
    uint32_t n_eq = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) n_eq += (t0 + j < a.T && __float_as_uint(mv[j]) == prefix) ? 1u : 0u;
    uint32_t eq_total;
    const uint32_t eq_before = block_excl_scan<uint32_t>(n_eq, wtot, eq_total);
    if (eq_before < k_eq && k_eq <= eq_before + n_eq) {
        uint32_t seen = eq_before;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            if (t0 + j < a.T && __float_as_uint(mv[j]) == prefix) {
                if (++seen == k_eq) s_tcut = t0 + j;
            }
        }
    }
    __syncthreads();
    if (tid == 0) {
        a.theta[hcg] = prefix;
        a.tcut[hcg] = s_tcut;
    }
}

// Budgeted selection of one (b, c); same result as topk_kernel.
template <int KPT>
__global__ void __launch_bounds__(kSelThreads) topk_reg_kernel(SelectArgs a) {
    __shared__ uint32_t cnt[2048];
    __shared__ uint32_t wtot[kSelWaves];
    __shared__ uint32_t s_digit, s_cnt, s_rem;

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
    const uint64_t* key = a.keys + hc * a.T;
    const int t0 = tid * KPT;
    uint64_t kv[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) kv[j] = (t0 + j < pool) ? key[t0 + j] : 0ull;

    uint64_t theta = 0;
    uint32_t k_eq = 0;
    if (want > 0) {
        const int shifts[6] = {53, 42, 31, 20, 9, 0};
        uint64_t prefix = 0, mask = 0;
        uint32_t need = want;
        bool settled = false;
        for (int pass = 0; pass < 6 && !settled; ++pass) {
            const int shift = shifts[pass];
            for (int i = tid; i < 2048; i += kSelThreads) cnt[i] = 0;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                const bool cand = t0 + j < pool && (kv[j] & mask) == prefix;
                hist_add(cand, static_cast<uint32_t>(kv[j] >> shift) & 2047u, 0ull, cnt, nullptr);
            }
            __syncthreads();
            descending_crossing<uint32_t>(cnt, cnt, need, wtot, &s_digit, &s_rem, &s_cnt);
            prefix |= static_cast<uint64_t>(s_digit) << shift;
            mask |= (shift == 0 ? 0x1FFull : 0x7FFull) << shift;
            need = s_rem;
            if (s_cnt == need) {
                theta = prefix - 1;
                k_eq = 0;
                settled = true;
            }
        }
        if (!settled) {
            theta = prefix;
            k_eq = need;
        }
    }
    // index-ordered compaction: keys > theta, then the first k_eq equal keys
    uint32_t n_eq = 0;
#pragma unroll
    for (int j = 0; j < KPT; ++j) n_eq += (want > 0 && k_eq > 0 && t0 + j < pool && kv[j] == theta) ? 1u : 0u;
    uint32_t eq_total;
    uint32_t eq_seen = block_excl_scan<uint32_t>(n_eq, wtot, eq_total);
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
    uint32_t pos = block_excl_scan<uint32_t>(n_sel, wtot, sel_total);
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

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    // register-resident kernels while a row fits in 16 (tau cut) or 32
    // (top-k) elements per thread
    const int per = (a.T + kSelThreads - 1) / kSelThreads;
    const int kpt = per <= 4 ? 4 : per <= 8 ? 8 : per <= 16 ? 16 : per <= 32 ? 32 : 0;
    if (a.mode == 0) {
        dim3 g1(a.G, a.Hkv, a.B);
        switch (kpt) {
            case 4: hipLaunchKernelGGL(tau_cut_reg_kernel<4>, g1, dim3(kSelThreads), 0, s, a); break;
            case 8: hipLaunchKernelGGL(tau_cut_reg_kernel<8>, g1, dim3(kSelThreads), 0, s, a); break;
            case 16: hipLaunchKernelGGL(tau_cut_reg_kernel<16>, g1, dim3(kSelThreads), 0, s, a); break;
            default: hipLaunchKernelGGL(tau_cut_kernel, g1, dim3(kSelThreads), 0, s, a); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    dim3 g2((a.T + 255) / 256, a.Hkv, a.B);
    hipLaunchKernelGGL(vote_score_kernel, g2, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g3(a.Hkv, a.B);
    switch (kpt) {
        case 4: hipLaunchKernelGGL(topk_reg_kernel<4>, g3, dim3(kSelThreads), 0, s, a); break;
        case 8: hipLaunchKernelGGL(topk_reg_kernel<8>, g3, dim3(kSelThreads), 0, s, a); break;
        case 16: hipLaunchKernelGGL(topk_reg_kernel<16>, g3, dim3(kSelThreads), 0, s, a); break;
        case 32: hipLaunchKernelGGL(topk_reg_kernel<32>, g3, dim3(kSelThreads), 0, s, a); break;
        default: hipLaunchKernelGGL(topk_kernel, g3, dim3(kSelThreads), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace mmskv
