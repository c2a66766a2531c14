// Internal launch interface between the C-ABI layer (api.cpp) and the
// gfx950 kernels.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mmskv {

// Workgroup shapes of the two score passes for a problem size: pass 1 runs
// lse_waves waves of 32 * lse_sub keys each, pass 2 mass_waves waves of 64.
struct ScorePlan {
    int lse_waves, lse_sub, mass_waves;
};
ScorePlan score_plan(int B, int Hkv, int T);

struct ProxyArgs {
    const void* q;        // [B, Hq, W, d]
    int q_dtype;          // 0 fp32, 1 bf16
    int64_t qsb, qsh, qst;
    const float* cos_f; const float* sin_f;   // [d/2] or null
    const float* cos_l; const float* sin_l;   // [d/2] or null
    uint16_t* proxies;    // [B, Hq, P, d]
    uint16_t* q_last;     // [B, Hq, d]
    double* stats;        // [B, Hq, 2, d] or null
    int B, Hq, W, d, P, ddof, layer;
    double gamma;
    double scale;         // log2(e) / sqrt(d), applied before the rounding
    uint32_t key0, key1;
};

struct ScoreArgs {
    const uint16_t* proxies;   // [B, Hq, P, d]
    const uint16_t* q_last;    // [B, Hq, d]
    const void* k;             // [B, Hkv, T, d]
    int k_dtype;
    int64_t ksb, ksh, kst;
    int B, Hq, Hkv, T, d, P, G, Gh;
    int lse_waves, lse_sub;    // pass 1: waves per workgroup, 32-key sub-tiles per wave
    int n_kb;                  // pass-1 key blocks (32 * lse_sub * lse_waves keys each)
    int block_keys;            // pass 2: keys per workgroup (64 * waves)
    int mass_n_kb;             // pass-2 key blocks
    int rows;                  // Gh * P proxy rows per KV head
    int rows_pad;              // rows + 32 * ceil(Gh / 32) (anchor rows, padded)
    double anchor_scale;       // log2(e) / sqrt(d), applied to the anchor rows as they are staged
    float lane_sum_hi;         // pass 1 sums from zero while every lane sum is below this
    float2* part;              // [B, Hkv, n_kb, rows_pad]  (max, sum), base 2
    float* lse;                // [B, Hkv, rows_pad]        log2-domain
    float* group_mass;         // [B, Hkv, G, T] or null
    float* mass;               // [B, Hkv, T]
    float* anchor;             // [B, Hkv, T]
};

struct SelectArgs {
    const float* group_mass;   // [B, Hkv, G, T]
    const float* mass;         // [B, Hkv, T]
    const float* anchor;       // [B, Hkv, T]
    const int32_t* budgets;    // [B, Hkv] or null
    int B, Hkv, T, G, mode, keep_last, budget, c_max;
    double tau, lambda;
    int fix_shift;             // S: tau sums count masses in units of 2^-S
    uint32_t* theta;           // [B, Hkv, G] cut mass (fp32 bits)
    int32_t* tcut;             // [B, Hkv, G] last admitted index among equals
    uint64_t* keys;            // [B, Hkv, T] score bits (fp64, non-negative)
    uint32_t* planes;          // [B, Hkv, G, ceil(T/32)] tau-set membership, bit j of word (g, w): key 32w+j in S_g
    uint32_t* hist0;           // [B, Hkv, 2048] pool keys per top digit (bits 63..53) of the score key
    int kpt;                   // keys per top-k thread (register path), 0 for the sweep path
    int key_stride;            // per-head stride of `keys`: kpt * 1024 (key t at (t % kpt) * 1024 + t / kpt), else T
    int32_t* idx;              // [B, Hkv, c_max]
    int32_t* counts;           // [B, Hkv]
    uint8_t* votes;            // [B, Hkv, T] or null
};

struct GatherArgs {
    const void* k; const void* v;
    int64_t ksb, ksh, kst, vsb, vsh, vst;   // element strides
    int elem_bytes, row_bytes;
    const int32_t* idx; const int32_t* counts;
    int B, Hkv, T, c_max;
    void* k_out; void* v_out;
};

struct HiddenArgs {
    const void* hidden;   // [B, T, D], D contiguous
    int dtype;            // 0 fp32, 1 bf16
    int64_t sb, st;       // element strides of batch row and token
    int B, T, D, chunk, n_chunks, ddof;
    double2* partial;     // [B, n_chunks, D] per-chunk (sum, sum of squares)
    double* stats;        // [B, 2, D] mean then std
    uint16_t* hp;         // [B, P, D] hidden-space samples (bf16)
    int P, layer;
    double gamma;
    uint32_t key0, key1;
};

struct ProjectArgs {
    const uint16_t* a;    // [M, K] hidden-space samples, M = B * P
    const uint16_t* w;    // [N, K] query weights, N = Hq * d
    const float* cos; const float* sin;   // [d/2] or null
    uint16_t* out;        // [B, Hq, P, d]
    double scale;         // log2(e) / sqrt(d), applied before the rounding
    int M, N, K, P, Hq, d;
};

struct DecodeArgs {
    const uint16_t* q_dec;     // [B, Hq, n_dec, d] bf16, unscaled
    const void* k;             // [B, Hkv, T, d] full prompt cache
    int k_dtype;               // dtype of k, k_out and v_out
    int64_t ksb, ksh, kst;
    const int32_t* idx;        // [B, Hkv, c_max]
    const int32_t* counts;     // [B, Hkv]
    const void* k_out;         // [B, Hkv, c_max, d] compacted cache
    const void* v_out;
    int B, Hq, Hkv, T, d, Gh, n_dec, c_max;
    int rows;                  // Gh * n_dec decode queries per KV head
    int rows_pad;              // rows rounded up to 32
    int n_kb;                  // key blocks
    double scale;              // log2(e) / sqrt(d), applied to the queries
    float lane_sum_hi;         // block sums from zero while every lane sum is below this
    float4* part;              // [B, Hkv, n_kb, rows_pad] (max, sum all, sum kept), base 2
    uint16_t* qsc;             // [B, Hkv, rows_pad, d] scaled decode queries (bf16)
    float* coverage;           // [B, Hq, n_dec]
    float* out;                // [B, Hq, n_dec, d]
};

struct WindowArgs {
    const void* q;             // [B, Hq, W, d] window queries
    int q_dtype;
    int64_t qsb, qsh, qst;
    int B, Hq, W, d, n;
    double scale;              // log2(e) / sqrt(d)
    uint16_t* rows;            // [B, Hq, n, d] bf16
    uint16_t* q_last;          // [B, Hq, d] bf16
};

struct ShapeArgs {
    const float* mass;         // [B, Hkv, T] (unused by StreamingLLM)
    float* score;              // [B, Hkv, T]
    int B, Hkv, T, kind, window, pool, sinks;
};

// Upper end of the lane sums (keys_per_sum terms of 2^s each) that the score
// and decode kernels add relative to zero.  A row's total over T keys is
// made of at most n = ceil(T / keys_per_sum) such sums, so with every one
// below 2^(127 - ceil(log2 n)) the total stays below 2^127 and no partial or
// merged sum can overflow fp32; capped at 2^120.
float lane_sum_limit(int T, int keys_per_sum);

int decode_rows_pad(int Gh, int n_dec);
int decode_key_blocks(int T);
int decode_max_rows();
int decode_max_compact();

hipError_t launch_build_proxies(const ProxyArgs& a, hipStream_t s);
// Pass-1 stages: the per-(row, key block) partials, then their merge into L.
constexpr int kLseBlocks = 1, kLseMerge = 2;
hipError_t launch_score_lse(const ScoreArgs& a, int stages, hipStream_t s);
hipError_t launch_score_mass(const ScoreArgs& a, hipStream_t s);
// Selection stages: tau cuts and membership planes (VOTE) or clearing the
// first-digit counts (MASS); votes, scores and first-digit counts; top-k.
constexpr int kSelectTau = 1, kSelectVote = 2, kSelectPick = 4;
hipError_t launch_select(const SelectArgs& a, int stages, hipStream_t s);
// Keys per thread of the register-resident top-k for T keys (0: the sweep
// kernel), and the per-head stride of the score keys it implies.
int select_kpt(int T);
inline int select_key_stride(int T) {
    const int k = select_kpt(T);
    return k > 0 ? k * 1024 : T;
}
hipError_t launch_gather(const GatherArgs& a, hipStream_t s);
hipError_t launch_hidden_stats(const HiddenArgs& a, hipStream_t s);
hipError_t launch_hidden_proxies(const HiddenArgs& a, hipStream_t s);
hipError_t launch_project(const ProjectArgs& p, hipStream_t s);
hipError_t launch_decode_check(const DecodeArgs& a, hipStream_t s);
hipError_t launch_window_rows(const WindowArgs& a, hipStream_t s);
hipError_t launch_shape_scores(const ShapeArgs& a, hipStream_t s);

}  // namespace mmskv
