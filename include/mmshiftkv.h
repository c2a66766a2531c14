/*
 * mmshiftkv.h -- C ABI of the MI355X (gfx950) library for MM-ShiftKV
 * prefill-stage KV scoring and selection (arxiv 2607.22586).
 *
 * Per layer, for every (batch row, KV head), the library
 *   1. builds variance-expanded query proxies from the observation-window
 *      queries                                (Sec. 3.2.1 Eqs. 4-5),
 *   2. computes each proxy's softmax over all prompt keys and sums the
 *      attention mass per proxy group across the query heads of the GQA
 *      group, plus the last-query anchor       (Sec. 3.2.2 Eqs. 7-8,
 *                                               Sec. 3.2.3 Eq. 11, Appendix B),
 *   3. forms the tau-sets and votes, ranks keys by vote + lambda*anchor and
 *      keeps the most recent key plus the top C-1 (Sec. 3.2.2 Eqs. 9-10,
 *                                               Sec. 3.2.3, Algorithm 1),
 *   4. gathers the retained K/V rows, in temporal order, into a compacted
 *      cache                                   (Appendix B).
 *
 * Conventions (all entry points):
 *   - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *     library never allocates, frees or synchronises; scratch memory comes
 *     from the caller, sized by the *_workspace() queries.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls only enqueue
 *     work on it and return; results are valid once the stream reaches them.
 *   - Arguments are validated on the host before anything is launched; an
 *     invalid call returns a negative mmskv_status and enqueues nothing.
 *     MMSKV_EHIP reports a launch error from the HIP runtime.
 *   - bf16 tensors are passed as uint16_t bit patterns.
 *   - Inputs containing NaN or Inf give unspecified (but memory-safe) results.
 *   - Calls are thread-safe.  The only global state is the per-GPU scratch
 *     array of mmshiftkv_score_noalloc (see there).
 */
#ifndef MMSHIFTKV_H
#define MMSHIFTKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MMSKV_OK = 0,
    MMSKV_EINVAL = -1,       /* invalid argument: shape, pointer, parameter */
    MMSKV_EUNSUPPORTED = -2, /* valid per the paper but not built: see each call */
    MMSKV_EWORKSPACE = -3,   /* workspace pointer NULL or smaller than required */
    MMSKV_EHIP = -4,         /* the HIP runtime reported a launch error */
    MMSKV_ESCRATCH = -5      /* mmshiftkv_score_noalloc: the problem needs more
                                than MMSKV_NOALLOC_SCRATCH_BYTES of scratch */
} mmskv_status;

typedef enum { MMSKV_F32 = 0, MMSKV_BF16 = 1 } mmskv_dtype;

typedef enum {
    MMSKV_VOTE = 0, /* the paper's rule: tau-set votes + lambda * anchor */
    MMSKV_MASS = 1  /* total proxy mass (votes and anchor not used) */
} mmskv_mode;

/* Problem sizes of one layer.  Each call reads the fields its comment names
 * (the proxy, score, decode and window calls read all of them; the others
 * ignore the rest, which may then hold any value).
 *   B    batch rows (<= 65535)        Hq   query heads
 *   Hkv  KV heads (Hq % Hkv == 0; the Gh = Hq/Hkv query heads h with
 *        h / Gh == c share KV head c)
 *   T    prompt keys per KV head (>= 1)
 *   W    window queries per query head (>= 1)
 *   d    head dimension: 64 or 128 (others -> MMSKV_EUNSUPPORTED) */
typedef struct {
    int32_t B, Hq, Hkv, T, W, d;
} mmskv_shape;

/* Element strides of a 4-D tensor [batch, head, token, d]; d is contiguous
 * and every row must start on a 16-byte boundary. */
typedef struct {
    int64_t sb, sh, st;
} mmskv_strides;

/* Method parameters (paper defaults: P=512, G=32, gamma=10, tau=0.95,
 * lambda=1; Sec. 4.1 and Appendix B).
 *   P         proxies per query head (the paper's N); P % G == 0 and the
 *             group size P/G must be a multiple of 16
 *   G         proxy groups, 1..255 (groups are contiguous proxy blocks)
 *   gamma     >= 0; multiplies the window std (x = mu + gamma*sigma*z)
 *   tau       in (0, 1]: tau-set mass fraction
 *   lambda    >= 0: anchor weight
 *   std_ddof  0 (population std) or 1; W - std_ddof >= 1
 *   layer     0..65535 and seed: fields of the Philox4x32-10 counter / key
 *   mode      mmskv_mode
 *   keep_last 1: token T-1 is always kept and the rest of the budget is
 *             filled from [0, T-1); 0: plain top-C over [0, T) */
typedef struct {
    int32_t P, G;
    double gamma, tau, lambda;
    int32_t std_ddof, layer;
    uint64_t seed;
    int32_t mode, keep_last;
} mmskv_params;

/* Step 1 -- query proxies (Sec. 3.2.1 Eqs. 4-5; Appendix A.4 Eq. 15).
 * Per (b, query head h) and dimension j: mu, sigma over the W window queries
 * (fp64, summed in window order, divisor W - std_ddof).  Proxy i of head h:
 *   x_j = mu_j + (gamma * sigma_j) * z_j,
 * z from Philox4x32-10 (counter (j/4, i, h, (b<<16)|layer), key = seed) and
 * Box-Muller on series-evaluated ln/sin/cos in fp32 (each product and sum
 * rounded separately, division and square root correctly rounded), widened
 * to fp64; optional rotate-half rotary embedding (pairs j, j+d/2)
 * from the caller's cos/sin tables; then multiplied by the softmax scale
 * c = log2(e)/sqrt(d) (fp64; the proxies carry Eq. 7's 1/sqrt(d), so their
 * products with the keys are base-2 logits) and rounded fp64 -> fp32 ->
 * bf16, both round to nearest even.  q_last[b,h] is window query W-1
 * (rotated by the *_l tables when given), rounded the same way but NOT
 * scaled; it is the anchor query of Eq. 11.
 *   q_win     [B, Hq, W, d] q_dtype, strides q_strides (elements)
 *   rope_*_f  [d/2] fp32 cos/sin at the proxies' future position, or both NULL
 *   rope_*_l  [d/2] fp32 cos/sin at the last query's position, or both NULL
 *   proxies   [B, Hq, P, d] bf16 out, contiguous (scaled by c)
 *   q_last    [B, Hq, d] bf16 out, contiguous (not scaled)
 *   stats     [B, Hq, 2, d] fp64 out (mu then sigma) or NULL */
int mmshiftkv_build_proxies(const mmskv_shape *shape, const mmskv_params *params,
                            const void *q_win, int32_t q_dtype, const mmskv_strides *q_strides,
                            const float *rope_cos_f, const float *rope_sin_f,
                            const float *rope_cos_l, const float *rope_sin_l,
                            uint16_t *proxies, uint16_t *q_last, double *stats, void *stream);

/* Step 2 -- proxy attention and masses (Sec. 3.2.2 Eqs. 7-8; Sec. 3.2.3
 * Eq. 11; Appendix B GQA aggregation).  For KV head c of batch row b, every
 * proxy row of the Gh query heads that share c gets its softmax over all T
 * keys: the proxies arrive scaled by c = log2(e)/sqrt(d) (as the proxy calls
 * make them), so p_t = 2^(s_t - L) with s_t = q~ . k_t and
 * L = log2 sum_t 2^(s_t) (bf16 operands, fp32 accumulation; fp32 keys are
 * rounded to bf16 for scoring).  The anchor queries q_last arrive unscaled
 * and are scaled the same way here (fp64 product with c, then fp32, then
 * bf16).  Outputs, fp32, contiguous:
 *   group_mass [B, Hkv, G, T]  sum over the group's proxies and heads
 *                              (may be NULL in MMSKV_MASS mode)
 *   mass       [B, Hkv, T]     sum over all groups
 *   anchor     [B, Hkv, T]     mean over the Gh heads of softmax(q_last)
 * The logit matrix never reaches memory: the call runs a row log-sum-exp
 * pass and a mass pass over the keys.  Workspace: mmshiftkv_score_workspace
 * bytes (256-byte aligned pointer). */
size_t mmshiftkv_score_workspace(const mmskv_shape *shape, const mmskv_params *params);
int mmshiftkv_score(const mmskv_shape *shape, const mmskv_params *params,
                    const uint16_t *proxies, const uint16_t *q_last,
                    const void *k, int32_t k_dtype, const mmskv_strides *k_strides,
                    float *group_mass, float *mass, float *anchor,
                    void *workspace, size_t workspace_bytes, void *stream);

/* mmshiftkv_score without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): same arguments, results and kernels as
 * mmshiftkv_score, with the scratch memory taken from a library-owned array
 * of MMSKV_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU instead of the workspace.
 * The call itself allocates nothing and never frees; the array of a GPU is
 * set up on the first call with that GPU current and held until the process
 * ends.  It runs on the CURRENT device (hipGetDevice), so `stream` must
 * belong to that device.  Every call on one GPU shares that GPU's array:
 * calls that overlap in time on one GPU (different streams, or threads
 * without ordering) race and give undefined results; calls ordered on one
 * stream are safe.  Nothing in the array needs clearing between calls (each
 * call writes every byte it reads first).  A problem whose workspace
 * (mmshiftkv_score_workspace) exceeds the array returns MMSKV_ESCRATCH with
 * nothing enqueued; the benchmark workloads need at most ~17 MiB. */
#define MMSKV_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int mmshiftkv_score_noalloc(const mmskv_shape *shape, const mmskv_params *params,
                            const uint16_t *proxies, const uint16_t *q_last,
                            const void *k, int32_t k_dtype, const mmskv_strides *k_strides,
                            float *group_mass, float *mass, float *anchor, void *stream);

/* The two passes of mmshiftkv_score as separate calls (same arguments and
 * workspace), for callers that schedule or time them separately:
 * mmshiftkv_score_lse writes each row's log-sum-exp into the workspace;
 * mmshiftkv_score_mass then reads it and writes the outputs. */
int mmshiftkv_score_lse(const mmskv_shape *shape, const mmskv_params *params,
                        const uint16_t *proxies, const uint16_t *q_last,
                        const void *k, int32_t k_dtype, const mmskv_strides *k_strides,
                        void *workspace, size_t workspace_bytes, void *stream);
int mmshiftkv_score_mass(const mmskv_shape *shape, const mmskv_params *params,
                         const uint16_t *proxies, const uint16_t *q_last,
                         const void *k, int32_t k_dtype, const mmskv_strides *k_strides,
                         float *group_mass, float *mass, float *anchor,
                         void *workspace, size_t workspace_bytes, void *stream);

/* The two halves of mmshiftkv_score_lse (the row normaliser of Sec. 3.2.2
 * Eq. 7), same arguments and workspace, for callers that schedule or time
 * them separately; in this order they are mmshiftkv_score_lse, and nothing
 * else may write the workspace between them:
 * mmshiftkv_score_lse_blocks: for every proxy and anchor row and every block
 * of keys, the block's (max, sum of 2^(s - max)) pair (base 2), into the
 * workspace; mmshiftkv_score_lse_merge: each row's log-sum-exp over all T
 * keys from those pairs (the largest maximum as reference, every sum
 * rescaled to it), into the workspace.  Errors as mmshiftkv_score_lse. */
int mmshiftkv_score_lse_blocks(const mmskv_shape *shape, const mmskv_params *params,
                               const uint16_t *proxies, const uint16_t *q_last,
                               const void *k, int32_t k_dtype, const mmskv_strides *k_strides,
                               void *workspace, size_t workspace_bytes, void *stream);
int mmshiftkv_score_lse_merge(const mmskv_shape *shape, const mmskv_params *params,
                              const uint16_t *proxies, const uint16_t *q_last,
                              const void *k, int32_t k_dtype, const mmskv_strides *k_strides,
                              void *workspace, size_t workspace_bytes, void *stream);

/* Step 3 -- tau-sets, votes and budgeted selection (Sec. 3.2.2 Eqs. 9-10;
 * Sec. 3.2.3 Eq. 11; Algorithm 1).
 * VOTE: for each group, S_g = keys taken in (mass desc, index asc) order up to
 * the first prefix whose mass reaches tau * the group total (masses summed in
 * 2^-k fixed point, so the cut is deterministic); vote(t) = #groups with t in
 * S_g; score = vote + lambda * anchor in fp64.  MASS: score = mass.
 * Selection per (b, c) with budget C (budgets[b*Hkv+c] when `budgets` is a
 * device array, else `budget`): if T <= C all keys; else token T-1 plus the
 * C-1 best of [0, T-1) by (score desc, index asc) (keep_last = 1), or the C
 * best of [0, T) (keep_last = 0).
 *   idx    [B, Hkv, c_max] int32 out: ascending token indices, -1 padded
 *   counts [B, Hkv] int32 out: min(C, T)
 *   votes  [B, Hkv, T] uint8 out or NULL (VOTE mode only)
 * Requires c_max >= min(C, T) for every head (checked on the host for the
 * scalar budget; per-head budgets above c_max are clamped to c_max).
 * Reads shape->B, Hq, Hkv, T (W and d are ignored) and params->P, G, tau,
 * lambda, mode, keep_last.  Workspace: mmshiftkv_select_workspace bytes. */
size_t mmshiftkv_select_workspace(const mmskv_shape *shape, const mmskv_params *params);
int mmshiftkv_select_topk(const mmskv_shape *shape, const mmskv_params *params,
                          const float *group_mass, const float *mass, const float *anchor,
                          const int32_t *budgets, int32_t budget, int32_t c_max,
                          int32_t *idx, int32_t *counts, uint8_t *votes,
                          void *workspace, size_t workspace_bytes, void *stream);

/* The three stages of mmshiftkv_select_topk as separate calls (same
 * arguments, same workspace), for callers that schedule or time them
 * separately; called in this order on one stream they are
 * mmshiftkv_select_topk.  Each keeps its state in the workspace for the
 * next, so nothing else may write the workspace between them.
 * mmshiftkv_select_tau: VOTE mode, the tau cut of every group (reads
 * group_mass); MASS mode, only clears the workspace's digit counts.
 * mmshiftkv_select_vote: votes (VOTE; `votes` out or NULL) and the score of
 * every key (reads anchor in VOTE mode, mass in MASS mode).
 * mmshiftkv_select_pick: the budgeted top-k into idx and counts.
 * Each checks the arguments it reads as mmshiftkv_select_topk does. */
int mmshiftkv_select_tau(const mmskv_shape *shape, const mmskv_params *params, const float *group_mass,
                         void *workspace, size_t workspace_bytes, void *stream);
int mmshiftkv_select_vote(const mmskv_shape *shape, const mmskv_params *params, const float *mass,
                          const float *anchor, uint8_t *votes, void *workspace, size_t workspace_bytes,
                          void *stream);
int mmshiftkv_select_pick(const mmskv_shape *shape, const mmskv_params *params, const int32_t *budgets,
                          int32_t budget, int32_t c_max, int32_t *idx, int32_t *counts,
                          void *workspace, size_t workspace_bytes, void *stream);

/* Step 4 -- compacted cache (Appendix B: retained tokens in temporal order,
 * inserted through the standard cache update).  For j < counts[b,c]:
 *   k_out[b,c,j,:] = k[b,c,idx[b,c,j],:], v_out likewise (byte copies);
 * rows j >= counts[b,c] are zero-filled.  Reads shape->B, Hkv, T and d
 * (Hq and W are ignored); a row of d elements must be a whole number of
 * 16-byte vectors (d * element size % 16 == 0, d <= 65536).
 *   k, v          [B, Hkv, T, d] dtype, strides k_strides / v_strides
 *   k_out, v_out  [B, Hkv, c_max, d] dtype, contiguous
 * idx entries outside [0, T) are not read (their row is zero-filled). */
int mmshiftkv_gather_kv(const mmskv_shape *shape, const void *k, const void *v, int32_t dtype,
                        const mmskv_strides *k_strides, const mmskv_strides *v_strides,
                        const int32_t *idx, const int32_t *counts, int32_t c_max,
                        void *k_out, void *v_out, void *stream);

/* ---- Hidden-state form of the proxies (Sec. 3.2.1 Eqs. 4-6 as written;
 * Algorithm 1).  The statistics are taken over a layer's prefill hidden
 * states (the input of the query projection), the samples are drawn in
 * hidden space, and every query head's proxies are its projection W_Q^(h) of
 * the same samples, rotated to the future position.  The three calls replace
 * mmshiftkv_build_proxies; their output feeds mmshiftkv_score unchanged, with
 * q_last taken from the model's own last query.
 *
 * Sizes of one layer's hidden states: B batch rows (<= 65535), T prompt
 * tokens (>= 1), D hidden features (a multiple of 8). */
typedef struct {
    int32_t B, T, D;
} mmskv_hshape;

/* Eq. 4 over hidden [B, T, D] (dtype, element strides sb / st; features
 * contiguous, rows on 16-byte boundaries): per (b, feature) fp64 mean and
 * std with divisor T - std_ddof (std_ddof 0 or 1, T - std_ddof >= 1).  Sums
 * of values and of squares are taken per chunk of 256 tokens in token order,
 * then added in chunk order; var = (SS - S*mean) / (T - std_ddof), negative
 * values clamped to 0.
 *   stats [B, 2, D] fp64 out (mean row, then std row), contiguous
 * Workspace: mmshiftkv_hidden_stats_workspace bytes (256-byte aligned). */
size_t mmshiftkv_hidden_stats_workspace(const mmskv_hshape *shape);
int mmshiftkv_hidden_stats(const mmskv_hshape *shape, int32_t std_ddof,
                           const void *hidden, int32_t dtype, int64_t sb, int64_t st,
                           double *stats, void *workspace, size_t workspace_bytes, void *stream);

/* Eq. 5 in hidden space: sample i of batch row b, feature j,
 *   x = mu_j + (gamma * sigma_j) * z,
 * z from the generator of mmshiftkv_build_proxies with the head field of the
 * counter set to 0xFFFFFFFF (one sample set per layer, shared by all heads);
 * fp64 -> fp32 -> bf16.  Uses params->P, gamma, seed and layer only.
 *   stats [B, 2, D] fp64 from mmshiftkv_hidden_stats
 *   hp    [B, P, D] bf16 out, contiguous, 8-byte aligned */
int mmshiftkv_hidden_proxies(const mmskv_hshape *shape, const mmskv_params *params,
                             const double *stats, uint16_t *hp, void *stream);

/* Eq. 6: proxies[b, h, i, :] = W_Q^(h) hp[b, i, :] (bf16 operands, fp32
 * accumulation on the matrix cores), then, when rope_cos / rope_sin are
 * given, the rotate-half rotary embedding at the future position (pairs
 * e, e + d/2, fp32), then the softmax scale log2(e)/sqrt(d) (fp64 product,
 * rounded to fp32), rounded to bf16.
 *   hp        [B, P, D] bf16, contiguous
 *   wq        [Hq * d, D] bf16, contiguous (row h*d + e is output feature e
 *             of head h; no bias)
 *   rope_*    [d/2] fp32 or both NULL
 *   proxies   [B, Hq, P, d] bf16 out, contiguous
 * d is 64 or 128; hp, wq and proxies start on 16-byte boundaries. */
int mmshiftkv_project_proxies(const mmskv_hshape *shape, int32_t P, int32_t Hq, int32_t d,
                              const uint16_t *hp, const uint16_t *wq,
                              const float *rope_cos, const float *rope_sin,
                              uint16_t *proxies, void *stream);

/* ---- Decode-time check (not part of the selection; it measures it).  The
 * attention-mass coverage of Fig. 1b -- the share of a decoding query's
 * softmax mass over all T prompt keys that falls on the keys kept after
 * prefilling -- and decode attention over the compacted cache, which stays
 * fixed while decoding under the prefill-only protocol (Sec. 3.1,
 * Sec. 3.2.3).  For decode query j of query head h (KV head c = h / Gh) of
 * batch row b, with q~ = bf16(fp32(q * log2(e)/sqrt(d))) (fp64 product, as
 * for the anchor query) and base-2 logits s_t = q~ . k_t (bf16 operands,
 * fp32 accumulation; fp32 keys rounded to bf16):
 *   coverage[b,h,j] = sum over kept t of 2^(s_t - L),  L = log2 sum_t 2^(s_t),
 * with kept = idx[b,c,0..counts[b,c]) (entries outside [0, T) ignored), and
 *   out[b,h,j,:]    = sum_{i < counts[b,c]} 2^(s'_i - L') v'_i,
 * s'_i = q~ . k'_i over the compacted rows, L' = log2 sum_i 2^(s'_i) (fp32);
 * out is zero when counts[b,c] is 0.  counts are clamped to [0, c_max].
 *   q_dec        [B, Hq, n_dec, d] bf16, contiguous, not scaled
 *   k            [B, Hkv, T, d] dtype, strides k_strides (the prompt cache)
 *   idx, counts  as returned by mmshiftkv_select_topk (c_max columns)
 *   k_out, v_out [B, Hkv, c_max, d] dtype, contiguous (mmshiftkv_gather_kv)
 *   coverage     [B, Hq, n_dec] fp32 out;  out [B, Hq, n_dec, d] fp32 out
 * (Hq/Hkv) * n_dec <= 256 and c_max <= 2048 (else MMSKV_EUNSUPPORTED).
 * Workspace: mmshiftkv_decode_workspace bytes (0 for an invalid shape). */
size_t mmshiftkv_decode_workspace(const mmskv_shape *shape, int32_t n_dec);
int mmshiftkv_decode_check(const mmskv_shape *shape, int32_t n_dec, const uint16_t *q_dec,
                           const void *k, int32_t dtype, const mmskv_strides *k_strides,
                           const int32_t *idx, const int32_t *counts, int32_t c_max,
                           const void *k_out, const void *v_out, float *coverage, float *out,
                           void *workspace, size_t workspace_bytes, void *stream);

/* ---- Baseline selectors on the same kernels: the comparison methods of
 * Sec. 4.1 with the settings of the paper's appendix on the baselines.  Each
 * one is a per-key score for mmshiftkv_select_topk in MMSKV_MASS mode with
 * keep_last = 0 (score = mass; a kept key scores 2^100, above any mass):
 *   SnapKV        rows of mmshiftkv_window_rows (window 32) scored by
 *                 mmshiftkv_score (P = 32, G = 1, MASS), then
 *                 MMSKV_SHAPE_SNAPKV (pooling 5);
 *   StreamingLLM  MMSKV_SHAPE_STREAMING (4 sinks, recency), no scoring;
 *   ExpectedAttn  proxies with gamma = 1 (512 samples, no variance
 *                 expansion) scored in MASS mode, then MMSKV_SHAPE_SINKS (4);
 *   LastAttn      the method itself with tau = 1 (Table 5's first row).
 *
 * The last n window queries of each head in the form of proxies: window
 * query w = W-n+i as a bf16 value (fp32 inputs rounded to nearest even),
 * times log2(e)/sqrt(d) in fp64, rounded to fp32 then bf16, and q_last[b,h]
 * = window query W-1 as a bf16 value (not scaled), as mmshiftkv_build_proxies
 * gives it.  1 <= n <= W.
 *   q_win  [B, Hq, W, d] q_dtype, strides q_strides (elements)
 *   rows   [B, Hq, n, d] bf16 out, contiguous;  q_last [B, Hq, d] bf16 out */
int mmshiftkv_window_rows(const mmskv_shape *shape, int32_t n, const void *q_win, int32_t q_dtype,
                          const mmskv_strides *q_strides, uint16_t *rows, uint16_t *q_last, void *stream);

typedef enum {
    MMSKV_SHAPE_SNAPKV = 0,    /* keys t < T-window: average of mass[u] over
                                  |u-t| <= pool/2, u < T-window, divided by
                                  pool (zeros outside); t >= T-window kept */
    MMSKV_SHAPE_STREAMING = 1, /* t < sinks kept, else score t (recency) */
    MMSKV_SHAPE_SINKS = 2      /* t < sinks kept, else mass[t] */
} mmskv_shape_kind;

/* Per-key baseline score from a mass (fp32 sums in ascending u); reads
 * shape->B, Hkv and T only:
 *   mass   [B, Hkv, T] fp32 (may be NULL for MMSKV_SHAPE_STREAMING)
 *   score  [B, Hkv, T] fp32 out
 * 0 <= window <= T, sinks >= 0, pool odd >= 1, T <= 2^24. */
int mmshiftkv_shape_scores(const mmskv_shape *shape, int32_t kind, int32_t window, int32_t pool, int32_t sinks,
                           const float *mass, float *score, void *stream);

/* Human-readable text for an mmskv_status value (static storage). */
const char *mmshiftkv_status_string(int status);

/* Library version: major*10000 + minor*100 + patch. */
int mmshiftkv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MMSHIFTKV_H */
