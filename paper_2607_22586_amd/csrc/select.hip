// tau-sets, votes, anchor score and budgeted selection (Sec. 3.2.2 Eqs. 9-10,
// Sec. 3.2.3 Eq. 11, Algorithm 1) on gfx950.
//
// tau_cut   one workgroup per (b, c, group): a mass-weighted radix select on
//           the fp32 bit patterns of the group masses (non-negative floats
//           order like their bits) finds the cut mass theta and, among keys
//           whose mass equals theta, the last admitted index, such that the
//           set {mass > theta} u {mass == theta, index <= tcut} is the shortest
//           (mass desc, index asc) prefix whose mass reaches tau * total.
//           Masses are summed as 2^S fixed-point integers, so every decision
//           is independent of summation order.
// vote      one thread per key: vote = #groups whose set holds the key;
//           score = vote + lambda*anchor (fp64) or the total mass.
// topk      one workgroup per (b, c): radix select of the (C-1)-th largest
//           score key over [0, T-1) (or the C-th over [0, T)), then an
//           index-ordered compaction writes the kept tokens in ascending
//           order and appends token T-1.
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
    __shared__ uint32_t cnt[256];
    __shared__ unsigned long long sum[256];
    __shared__ unsigned long long scratch[kSelWaves];
    __shared__ uint32_t wtot[kSelWaves];
    __shared__ uint32_t s_digit;
    __shared__ unsigned long long s_need;
    __shared__ int32_t s_tcut;

    const int g = blockIdx.x, c = blockIdx.y, b = blockIdx.z;
    const int64_t hcg = (static_cast<int64_t>(b) * a.Hkv + c) * a.G + g;
    const float* m = a.group_mass + hcg * a.T;
    const int tid = threadIdx.x;

    uint64_t local = 0;
    for (int t = tid; t < a.T; t += kSelThreads) local += to_fixed(m[t], a.fix_scale);
    const uint64_t total = block_sum_u64(local, scratch);
    uint64_t need = static_cast<uint64_t>(ceil(a.tau * static_cast<double>(total)));
    if (need < 1) need = 1;
    if (need > total) need = total;
    if (total == 0) {
        // every mass is below the fixed-point resolution: empty set
        if (tid == 0) { a.theta[hcg] = 0xFFFFFFFFu; a.tcut[hcg] = -1; }
        return;
    }

    uint32_t prefix = 0, mask = 0;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int i = tid; i < 256; i += kSelThreads) { cnt[i] = 0; sum[i] = 0; }
        if (tid == 0) { s_digit = 0; s_need = need; }
        __syncthreads();
        for (int base = 0; base < a.T; base += kSelThreads) {
            const int t = base + tid;
            const bool in = t < a.T;
            const float mv = in ? m[t] : 0.f;
            const uint32_t bits = __float_as_uint(mv);
            const bool cand = in && (bits & mask) == prefix;
            hist_add(cand, (bits >> shift) & 255u, to_fixed(mv, a.fix_scale), cnt, sum);
        }
        __syncthreads();
        if (tid < kWave) {
            // lane l covers digits 255-4l .. 252-4l (descending)
            const int lane = tid;
            uint64_t s4[4];
            uint64_t mine = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) { s4[j] = sum[255 - 4 * lane - j]; mine += s4[j]; }
            uint64_t incl = mine;
            for (int o = 1; o < kWave; o <<= 1) {
                const uint64_t y = shfl_u64(incl, lane >= o ? lane - o : lane);
                if (lane >= o) incl += y;
            }
            const uint64_t excl = incl - mine;
            const bool hit = excl < need && need <= incl;
            if (hit) {
                uint64_t acc = excl;
                int j = 0;
                for (; j < 3; ++j) {
                    if (acc + s4[j] >= need) break;
                    acc += s4[j];
                }
                s_digit = 255 - 4 * lane - j;
                s_need = need - acc;
            }
        }
        __syncthreads();
        prefix |= s_digit << shift;
        mask |= 255u << shift;
        need = s_need;
        __syncthreads();
    }
    // keys with mass == theta each carry f_theta; take the first k_eq by index
    const uint64_t f_theta = to_fixed(__uint_as_float(prefix), a.fix_scale);
    const uint64_t k_eq = f_theta == 0 ? 1 : (need + f_theta - 1) / f_theta;
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
    __shared__ uint32_t cnt[256];
    __shared__ uint32_t wtot[kSelWaves];
    __shared__ uint32_t s_digit, s_need;

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

    uint64_t prefix = 0, mask = 0;
    uint32_t need = want;
    if (want > 0) {
        for (int pass = 0; pass < 8; ++pass) {
            const int shift = 56 - 8 * pass;
            for (int i = tid; i < 256; i += kSelThreads) cnt[i] = 0;
            if (tid == 0) { s_digit = 0; s_need = need; }
            __syncthreads();
            for (int base = 0; base < pool; base += kSelThreads) {
                const int t = base + tid;
                const bool in = t < pool;
                const uint64_t kv = in ? key[t] : 0ull;
                const bool cand = in && (kv & mask) == prefix;
                hist_add(cand, static_cast<uint32_t>(kv >> shift) & 255u, 0ull, cnt, nullptr);
            }
            __syncthreads();
            if (tid < kWave) {
                const int lane = tid;
                uint32_t c4[4], mine = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) { c4[j] = cnt[255 - 4 * lane - j]; mine += c4[j]; }
                uint32_t incl = mine;
                for (int o = 1; o < kWave; o <<= 1) {
                    const uint32_t y = __shfl(incl, lane >= o ? lane - o : lane, kWave);
                    if (lane >= o) incl += y;
                }
                const uint32_t excl = incl - mine;
                if (excl < need && need <= incl) {
                    uint32_t acc = excl;
                    int j = 0;
                    for (; j < 3; ++j) {
                        if (acc + c4[j] >= need) break;
                        acc += c4[j];
                    }
                    s_digit = 255 - 4 * lane - j;
                    s_need = need - acc;
                }
            }
            __syncthreads();
            prefix |= static_cast<uint64_t>(s_digit) << shift;
            mask |= 255ull << shift;
            need = s_need;
            __syncthreads();
        }
    }
    // selected: key > theta, or key == theta among the first `need` by index
    const uint64_t theta = prefix;
    const uint32_t k_eq = (want > 0) ? need : 0u;
    uint32_t eq_seen = 0, written = 0;
    for (int base = 0; base < pool; base += kSelThreads) {
        const int t = base + tid;
        const bool in = t < pool;
        const uint64_t kv = in ? key[t] : 0ull;
        const bool gt = in && want > 0 && kv > theta;
        const bool eq = in && want > 0 && kv == theta;
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

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    if (a.mode == 0) {
        dim3 g1(a.G, a.Hkv, a.B);
        hipLaunchKernelGGL(tau_cut_kernel, g1, dim3(kSelThreads), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    dim3 g2((a.T + 255) / 256, a.Hkv, a.B);
    hipLaunchKernelGGL(vote_score_kernel, g2, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g3(a.Hkv, a.B);
    hipLaunchKernelGGL(topk_kernel, g3, dim3(kSelThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace mmskv
