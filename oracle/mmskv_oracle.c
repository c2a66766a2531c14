/*
 * mmskv_oracle.c -- plain, slow fp64 CPU oracle for MM-ShiftKV prefill-stage
 * KV scoring and selection.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant generator
 * with the HIP library: every step is written out here from the paper
 * (MM-ShiftKV, arxiv 2607.22586) and from the published definitions of the
 * counter-based generator, in plain loops, double precision, one row at a
 * time, with no blocking, fusion or reordering beyond what the definitions
 * state.
 *
 * Readings of the paper that this file adopts (each is a choice where the
 * paper is silent or ambiguous):
 *   - Statistics are taken in query space over the W given window queries of
 *     each (batch, query head), per feature dimension (Sec. 3.2.1 Eq. 4 takes
 *     element-wise mean/std; Appendix A.4 Eq. 15 states the proxy law in
 *     query space).  std uses divisor (W - ddof), ddof = 0 by default.
 *   - Sampling uses a diagonal Gaussian, x = mu + (gamma*sigma)*z, i.e. gamma
 *     multiplies the standard deviation (Sec. 3.2.1 Eq. 5, diag((gamma sigma)^2)).
 *   - Noise z is independent per (batch, layer, query head, proxy, dim).
 *   - Optional rotary embedding uses caller tables (rotate-half pairing j,
 *     j+d/2) for one synthetic future position (Sec. 3.2.1, last paragraph).
 *   - The softmax scale of Sec. 3.2.2 Eq. 7, 1/sqrt(head_dim), is carried by
 *     the queries: proxies are multiplied by c = log2(e)/sqrt(head_dim) in
 *     fp64 and then rounded fp64 -> fp32 -> bf16 (round to nearest even);
 *     the anchor query, a bf16 input, is scaled the same way (fp64 product
 *     of its bf16 value and c, then fp32, then bf16), so it is rounded twice.
 *     The paper fixes no rounding point for its mixed-precision inference
 *     (Sec. 4.1; the FlashAttention kernel it names applies the scale to the
 *     fp32 scores instead).  This point is a convention, chosen because it
 *     saves the GPU kernel one multiply per logit; the other choice, bf16
 *     queries with the scale on the logit, moves individual probabilities
 *     by about 1% at gamma = 10, so the two are not interchangeable at the
 *     parity bar.  Scoring keys are rounded fp32 -> bf16 the same way.  The
 *     logits q~ . k are then computed in fp64 on those bf16 values and are
 *     base-2 logits: the softmax is 2^(s - L) with L = log2 sum_t 2^(s_t),
 *     which equals exp(q.k/sqrt(d) - lse) up to the bf16 rounding of the
 *     scaled queries.
 *   - Softmax over all T prompt keys (Sec. 3.2.2 Eq. 7).
 *   - Groups are contiguous proxy blocks I_g = {g*P/G .. (g+1)*P/G - 1}
 *     (Sec. 3.2.2 Eq. 8 leaves the partition open).
 *   - GQA: the masses of the query heads that share a KV head are summed
 *     inside each group before the tau-set is formed (Appendix B; Sec. 4.1).
 *   - tau-set: keys ordered by (group mass desc, index asc); the shortest
 *     prefix whose running sum is >= tau * (sum of all keys in that same
 *     order) (Sec. 3.2.2 Eq. 9 uses >=).
 *   - Anchor: the mean over the GQA group of the softmax of each query head's
 *     last window query (Sec. 3.2.3 Eq. 11), so the anchor never exceeds one
 *     vote step.  Score = vote + lambda*anchor in fp64.
 *   - Selection: if T <= C keep all; else keep token T-1 plus the top C-1 of
 *     [0, T-1) by (score desc, index asc); output in ascending index order
 *     (Sec. 3.2.3; Appendix B; Algorithm 1).
 *   - Hidden-state form (Sec. 3.2.1 as written, Algorithm 1): statistics of
 *     the layer's prefill hidden states (the query projection's input) per
 *     batch row and feature over all T prompt tokens; one set of N samples
 *     per (batch row, layer) shared by every head, projected by each head's
 *     query weights W_Q (no bias term, as in Eq. 6); the same rotary
 *     placement and roundings as the query-space form.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (see build.py).
 * The -ffp-contract=off flag keeps every a*b+c as two rounded operations,
 * which the counter-based normal generator below relies on.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Counter-based generator: Philox4x32-10 (Salmon, Moraes, Dror, Shaw,       */
/* "Parallel random numbers: as easy as 1, 2, 3", SC 2011).                  */
/* One round maps counter (c0,c1,c2,c3) with key (k0,k1) to                  */
/*   (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0)),       */
/* M0 = 0xD2511F53, M1 = 0xCD9E8D57; the key is bumped by the Weyl constants */
/* (0x9E3779B9, 0xBB67AE85) between rounds; ten rounds.                      */
/* ------------------------------------------------------------------------ */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        uint64_t prod0 = (uint64_t)0xD2511F53u * (uint64_t)c0;
        uint64_t prod1 = (uint64_t)0xCD9E8D57u * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
        uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* A 32-bit word x -> uniform (2*(x>>9) + 1) * 2^-24: an odd multiple of
 * 2^-24, exact in fp32, strictly inside (0, 1). */
float oracle_uniform(uint32_t x)
{
    return (float)(2u * (x >> 9) + 1u) * (1.0f / 16777216.0f);
}

/* Natural logarithm for u in (0,1), in fp32, written from the series
 *   ln m = 2 * sum_{k=0..5} s^(2k+1) / (2k+1),  s = (m-1)/(m+1),
 * after splitting u = m * 2^e with m in [r, 2r), r the fp32 value of
 * sqrt(1/2) rounded down; |s| <= 0.1716, so the first omitted term is below
 * 1e-10 of the result.  Horner form, plain fp32 mul/add; the coefficients
 * are 1.0f/(2k+1). */
float oracle_ln(float u)
{
    int e;
    float f = frexpf(u, &e);               /* u = f * 2^e, f in [0.5, 1) */
    float m = f;
    if (f < 0x1.6a09e6p-1f) {
        m = 2.0f * f;
        e = e - 1;
    }
    float s = (m - 1.0f) / (m + 1.0f);
    float s2 = s * s;
    float poly = 1.0f / 11.0f;
    for (int k = 4; k >= 0; --k) {
        poly = poly * s2;
        poly = poly + 1.0f / (float)(2 * k + 1);
    }
    float ln_m = 2.0f * s;
    ln_m = ln_m * poly;
    float ln2 = 0x1.62e430p-1f;            /* nearest fp32 to ln 2 */
    float eln2 = (float)e * ln2;
    return eln2 + ln_m;
}

/* sin and cos of 2*pi*u, in fp32, for the uniform u = n * 2^-24 of word x
 * (n = 2*(x>>9) + 1, odd): the quarter turn q nearest to 4u = n / 2^22 is
 * removed in integer arithmetic (n is odd, so 4u is never halfway), which
 * leaves f = u - q/4 = (n - q 2^22) 2^-24 with |f| < 1/8, exact in fp32;
 * phi = f * 2pi (2pi rounded to fp32); Taylor series of sin to phi^11 and
 * of cos to phi^10 (|phi| < pi/4, first omitted terms below 1e-10),
 * coefficients by repeated fp32 division, Horner form; the quarter turns
 * are then restored by the quadrant identities. */
void oracle_sincos_2pi(uint32_t x, float *sin_out, float *cos_out)
{
    int32_t n = (int32_t)(2u * (x >> 9) + 1u);
    int32_t q = (n + (1 << 21)) >> 22;
    int32_t rem = n - q * (1 << 22);
    float f = (float)rem * (1.0f / 16777216.0f);
    float two_pi = 0x1.921fb6p+2f;         /* nearest fp32 to 2 pi */
    float phi = f * two_pi;
    float p2 = phi * phi;

    float cs[6], cc[6];
    cs[0] = 1.0f;
    cc[0] = 1.0f;
    for (int k = 1; k <= 5; ++k) {
        cs[k] = -cs[k - 1] / (float)((2 * k) * (2 * k + 1));
        cc[k] = -cc[k - 1] / (float)((2 * k - 1) * (2 * k));
    }
    float ps = cs[5], pc = cc[5];
    for (int k = 4; k >= 0; --k) {
        ps = ps * p2;
        ps = ps + cs[k];
        pc = pc * p2;
        pc = pc + cc[k];
    }
    float sp = phi * ps;
    float cp = pc;
    switch (q & 3) {
    case 0: *sin_out = sp;  *cos_out = cp;  break;
    case 1: *sin_out = cp;  *cos_out = -sp; break;
    case 2: *sin_out = -sp; *cos_out = -cp; break;
    default: *sin_out = -cp; *cos_out = sp; break;
    }
}

/* Standard normals for dims 4*jq .. 4*jq+3 of proxy i of query head h,
 * batch b, layer l: Philox counter (jq, i, h, (b<<16)|l), key = seed split in
 * two 32-bit halves; words (x0,x1) and (x2,x3) each give one Box-Muller
 * pair (Box & Muller 1958): r = sqrt(-2 ln u_a), z = (r cos 2pi u_b,
 * r sin 2pi u_b), in fp32 (correctly rounded division and square root),
 * then widened to fp64 for the proxy formula. */
void oracle_normal4(uint64_t seed, int b, int layer, int h, int i, int jq, double z[4])
{
    uint32_t ctr[4] = {(uint32_t)jq, (uint32_t)i, (uint32_t)h,
                       ((uint32_t)b << 16) | ((uint32_t)layer & 0xFFFFu)};
    uint32_t key[2] = {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)};
    uint32_t x[4];
    oracle_philox4x32_10(ctr, key, x);
    for (int pair = 0; pair < 2; ++pair) {
        float ua = oracle_uniform(x[2 * pair]);
        float r = sqrtf(-2.0f * oracle_ln(ua));
        float sn, cs;
        oracle_sincos_2pi(x[2 * pair + 1], &sn, &cs);
        float z0 = r * cs;
        float z1 = r * sn;
        z[2 * pair] = (double)z0;
        z[2 * pair + 1] = (double)z1;
    }
}

/* ------------------------------------------------------------------------ */
/* bf16 helpers (round to nearest even; NaN is not expected in inputs).      */
/* ------------------------------------------------------------------------ */
uint16_t oracle_f32_to_bf16(float x)
{
    uint32_t bits;
    memcpy(&bits, &x, 4);
    uint32_t lsb = (bits >> 16) & 1u;
    bits = bits + 0x7FFFu + lsb;
    return (uint16_t)(bits >> 16);
}

double oracle_bf16_to_f64(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

/* dtype codes: 0 = fp32, 1 = bf16 (raw 16-bit patterns). */
static double load_elem(const void *base, int dtype, int64_t off)
{
    if (dtype == 0)
        return (double)((const float *)base)[off];
    return oracle_bf16_to_f64(((const uint16_t *)base)[off]);
}

/* Scoring value of a key element: fp32 keys are first rounded to bf16. */
static double load_key_bf16(const void *base, int dtype, int64_t off)
{
    if (dtype == 0)
        return oracle_bf16_to_f64(oracle_f32_to_bf16(((const float *)base)[off]));
    return oracle_bf16_to_f64(((const uint16_t *)base)[off]);
}

/* Softmax scale carried by the queries: log2(e) / sqrt(d), fp64. */
double oracle_query_scale(int d)
{
    return 1.4426950408889634074 / sqrt((double)d);
}

/* ------------------------------------------------------------------------ */
/* Step 1 -- proxies (Sec. 3.2.1 Eqs. 4-5, Appendix A.4 Eq. 15).             */
/* ------------------------------------------------------------------------ */
/*
 * q_win      [B, Hq, W, d] contiguous, dtype 0/1
 * rope_cos_f / rope_sin_f: [d/2] fp32 tables for the proxies' future
 *            position, or NULL (no rotary embedding)
 * rope_cos_l / rope_sin_l: [d/2] fp32 tables for the last query's position
 *            (used for the anchor query), or NULL
 * proxies    [B, Hq, P, d] bf16 out (x times log2(e)/sqrt(d), rounded)
 * q_last     [B, Hq, d] bf16 out (the last window query, not scaled)
 * stats      [B, Hq, 2, d] fp64 out (mu, sigma), may be NULL
 * returns 0, or -1 on invalid arguments
 */
/* b0 / h0: global batch row and query head of the first row/head of q_win,
 * so that a slice of a larger problem draws the same noise (the generator
 * counter uses the global indices). */
int oracle_build_proxies_at(int B, int Hq, int W, int d, int P, double gamma, int ddof,
                            uint64_t seed, int layer, int b0, int h0, const void *q_win, int dtype,
                            const float *rope_cos_f, const float *rope_sin_f,
                            const float *rope_cos_l, const float *rope_sin_l,
                            uint16_t *proxies, uint16_t *q_last, double *stats)
{
    if (B < 1 || Hq < 1 || W < 1 || d < 4 || (d % 4) != 0 || P < 1 || W - ddof < 1 ||
        ddof < 0 || layer < 0 || layer > 0xFFFF || b0 < 0 || h0 < 0 || B + b0 > 0xFFFF)
        return -1;
    int use_rope = (rope_cos_f != NULL && rope_sin_f != NULL);
    int use_rope_last = (rope_cos_l != NULL && rope_sin_l != NULL);
    int half = d / 2;
    double qs = oracle_query_scale(d);

#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < Hq; ++h) {
            double *mu = (double *)malloc(sizeof(double) * (size_t)d);
            double *sg = (double *)malloc(sizeof(double) * (size_t)d);
            double *x = (double *)malloc(sizeof(double) * (size_t)d);
            int64_t qbase = ((int64_t)b * Hq + h) * (int64_t)W * d;
            /* mean and std over the window, per dimension, summed in order */
            for (int j = 0; j < d; ++j) {
                double acc = 0.0;
                for (int w = 0; w < W; ++w)
                    acc = acc + load_elem(q_win, dtype, qbase + (int64_t)w * d + j);
                double m = acc / (double)W;
                double sq = 0.0;
                for (int w = 0; w < W; ++w) {
                    double diff = load_elem(q_win, dtype, qbase + (int64_t)w * d + j) - m;
                    double dd = diff * diff;
                    sq = sq + dd;
                }
                double var = sq / (double)(W - ddof);
                mu[j] = m;
                sg[j] = sqrt(var);
            }
            if (stats) {
                double *st = stats + ((int64_t)b * Hq + h) * 2 * d;
                for (int j = 0; j < d; ++j) {
                    st[j] = mu[j];
                    st[d + j] = sg[j];
                }
            }
            /* proxies */
            for (int i = 0; i < P; ++i) {
                for (int jq = 0; jq < d / 4; ++jq) {
                    double z[4];
                    oracle_normal4(seed, b0 + b, layer, h0 + h, i, jq, z);
                    for (int e = 0; e < 4; ++e) {
                        int j = 4 * jq + e;
                        double gs = gamma * sg[j];
                        double t = gs * z[e];
                        x[j] = mu[j] + t;
                    }
                }
                uint16_t *out = proxies + (((int64_t)b * Hq + h) * P + i) * d;
                if (use_rope) {
                    for (int j = 0; j < half; ++j) {
                        double c = (double)rope_cos_f[j], s = (double)rope_sin_f[j];
                        double a0 = x[j] * c, a1 = x[j + half] * s;
                        double b0 = x[j + half] * c, b1 = x[j] * s;
                        double lo = a0 - a1, hi = b0 + b1;
                        double slo = lo * qs, shi = hi * qs;
                        out[j] = oracle_f32_to_bf16((float)slo);
                        out[j + half] = oracle_f32_to_bf16((float)shi);
                    }
                } else {
                    for (int j = 0; j < d; ++j) {
                        double sx = x[j] * qs;
                        out[j] = oracle_f32_to_bf16((float)sx);
                    }
                }
            }
            /* anchor query: the last window query of this head */
            {
                for (int j = 0; j < d; ++j)
                    x[j] = load_elem(q_win, dtype, qbase + (int64_t)(W - 1) * d + j);
                uint16_t *out = q_last + ((int64_t)b * Hq + h) * d;
                if (use_rope_last) {
                    for (int j = 0; j < half; ++j) {
                        double c = (double)rope_cos_l[j], s = (double)rope_sin_l[j];
                        double a0 = x[j] * c, a1 = x[j + half] * s;
                        double b0 = x[j + half] * c, b1 = x[j] * s;
                        double lo = a0 - a1, hi = b0 + b1;
                        out[j] = oracle_f32_to_bf16((float)lo);
                        out[j + half] = oracle_f32_to_bf16((float)hi);
                    }
                } else {
                    for (int j = 0; j < d; ++j)
                        out[j] = oracle_f32_to_bf16((float)x[j]);
                }
            }
            free(mu);
            free(sg);
            free(x);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Step 1, hidden-state form (Sec. 3.2.1 Eqs. 4-6, Algorithm 1): statistics  */
/* of the prefill hidden states of one layer, variance-expanded samples of  */
/* them, and their projection by the query weights of every head.          */
/* ------------------------------------------------------------------------ */
/*
 * Per (batch row, feature dimension): mean and standard deviation over the
 * T prompt tokens (Eq. 4), by their definitions, in two passes:
 *   mean = (sum_t h_t) / T,
 *   var  = (sum_t (h_t - mean)^2) / (T - ddof),  std = sqrt(var),
 * each sum taken sequentially in token order.
 * hidden [B, T, D] (row stride D), dtype 0 fp32 / 1 bf16; stats [B, 2, D].
 */
int oracle_hidden_stats(int B, int T, int D, int ddof, const void *hidden, int dtype, double *stats)
{
    if (B < 1 || T < 1 || D < 1 || ddof < 0 || T - ddof < 1)
        return -1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int j = 0; j < D; ++j) {
            double s = 0.0;
            for (int t = 0; t < T; ++t)
                s = s + load_elem(hidden, dtype, ((int64_t)b * T + t) * D + j);
            double mean = s / (double)T;
            double ss = 0.0;
            for (int t = 0; t < T; ++t) {
                double dv = load_elem(hidden, dtype, ((int64_t)b * T + t) * D + j) - mean;
                double sq = dv * dv;
                ss = ss + sq;
            }
            stats[((int64_t)b * 2) * D + j] = mean;
            stats[((int64_t)b * 2 + 1) * D + j] = sqrt(ss / (double)(T - ddof));
        }
    }
    return 0;
}

/*
 * N proxy hidden states per batch row (Eq. 5): x = mu + (gamma*sigma)*z,
 * z from the same counter-based generator with the head field of the
 * counter set to 0xFFFFFFFF (hidden space, shared by all heads of the
 * layer), fp64 -> fp32 -> bf16.  stats [B, 2, D]; hp [B, P, D] bf16.
 * b0: global batch row of the first row.
 */
int oracle_hidden_proxies(int B, int D, int P, double gamma, uint64_t seed, int layer, int b0,
                          const double *stats, uint16_t *hp)
{
    if (B < 1 || D < 4 || (D % 4) != 0 || P < 1 || layer < 0 || layer > 0xFFFF || b0 < 0 ||
        B + b0 > 0xFFFF)
        return -1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int i = 0; i < P; ++i) {
            const double *mu = stats + ((int64_t)b * 2) * D;
            const double *sg = stats + ((int64_t)b * 2 + 1) * D;
            uint16_t *out = hp + ((int64_t)b * P + i) * D;
            for (int jq = 0; jq < D / 4; ++jq) {
                double z[4];
                oracle_normal4(seed, b0 + b, layer, -1, i, jq, z);
                for (int e = 0; e < 4; ++e) {
                    int j = 4 * jq + e;
                    double gs = gamma * sg[j];
                    double t = gs * z[e];
                    double x = mu[j] + t;
                    out[j] = oracle_f32_to_bf16((float)x);
                }
            }
        }
    }
    return 0;
}

/*
 * Query proxies (Eq. 6): q[b, h, i, e] = sum_k H~[b, i, k] * W_Q[h*d + e, k]
 * over the bf16 values, summed in k order in fp64, then the optional rotary
 * placement (rotate-half pairs e, e + d/2, caller tables for one future
 * position), times the query scale log2(e)/sqrt(d) in fp64, then
 * fp64 -> fp32 -> bf16.  hp [B, P, D]; wq [Hq*d, D] bf16;
 * proxies [B, Hq, P, d] bf16; pre [B, Hq, P, d] fp64 values before the
 * rounding (scaled), or NULL.
 */
int oracle_project_proxies(int B, int P, int D, int Hq, int d, const uint16_t *hp, const uint16_t *wq,
                           const float *rope_cos, const float *rope_sin, uint16_t *proxies, double *pre)
{
    if (B < 1 || P < 1 || D < 1 || Hq < 1 || d < 2 || (d % 2) != 0)
        return -1;
    int use_rope = (rope_cos != NULL && rope_sin != NULL);
    int half = d / 2;
    double qs = oracle_query_scale(d);
#pragma omp parallel for collapse(3) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < Hq; ++h) {
            for (int i = 0; i < P; ++i) {
                double *x = (double *)malloc(sizeof(double) * (size_t)d);
                const uint16_t *hv = hp + ((int64_t)b * P + i) * D;
                for (int e = 0; e < d; ++e) {
                    const uint16_t *wr = wq + ((int64_t)h * d + e) * D;
                    double acc = 0.0;
                    for (int k = 0; k < D; ++k) {
                        double pr = oracle_bf16_to_f64(hv[k]) * oracle_bf16_to_f64(wr[k]);
                        acc = acc + pr;
                    }
                    x[e] = acc;
                }
                int64_t o = (((int64_t)b * Hq + h) * P + i) * d;
                for (int e = 0; e < (use_rope ? half : d); ++e) {
                    if (use_rope) {
                        double c = (double)rope_cos[e], s = (double)rope_sin[e];
                        double a0 = x[e] * c, a1 = x[e + half] * s;
                        double b0 = x[e + half] * c, b1 = x[e] * s;
                        double lo = a0 - a1, hi = b0 + b1;
                        double slo = lo * qs, shi = hi * qs;
                        proxies[o + e] = oracle_f32_to_bf16((float)slo);
                        proxies[o + e + half] = oracle_f32_to_bf16((float)shi);
                        if (pre) {
                            pre[o + e] = slo;
                            pre[o + e + half] = shi;
                        }
                    } else {
                        double sx = x[e] * qs;
                        proxies[o + e] = oracle_f32_to_bf16((float)sx);
                        if (pre)
                            pre[o + e] = sx;
                    }
                }
                free(x);
            }
        }
    }
    return 0;
}

int oracle_build_proxies(int B, int Hq, int W, int d, int P, double gamma, int ddof,
                         uint64_t seed, int layer, const void *q_win, int dtype,
                         const float *rope_cos_f, const float *rope_sin_f,
                         const float *rope_cos_l, const float *rope_sin_l,
                         uint16_t *proxies, uint16_t *q_last, double *stats)
{
    return oracle_build_proxies_at(B, Hq, W, d, P, gamma, ddof, seed, layer, 0, 0, q_win, dtype,
                                   rope_cos_f, rope_sin_f, rope_cos_l, rope_sin_l, proxies, q_last,
                                   stats);
}

/* ------------------------------------------------------------------------ */
/* Step 2 -- proxy attention and masses (Sec. 3.2.2 Eqs. 7-8; Sec. 3.2.3     */
/* Eq. 11 for the anchor; Appendix B for the GQA aggregation).               */
/* ------------------------------------------------------------------------ */

/* softmax over t for one scaled bf16 query row q~: base-2 logits
 * s_t = q~ . k_t (fp64 on the bf16 values), p_t = 2^(s_t - L) with
 * L = log2 sum_t 2^(s_t); writes p[T]. */
static void softmax_row(const uint16_t *q, const void *k, int kdtype, int64_t kbase, int T,
                        int d, double *logit, double *p)
{
    double mx = -INFINITY;
    for (int t = 0; t < T; ++t) {
        double dot = 0.0;
        for (int j = 0; j < d; ++j) {
            double prod = oracle_bf16_to_f64(q[j]) * load_key_bf16(k, kdtype, kbase + (int64_t)t * d + j);
            dot = dot + prod;
        }
        logit[t] = dot;
        if (logit[t] > mx)
            mx = logit[t];
    }
    double sum = 0.0;
    for (int t = 0; t < T; ++t)
        sum = sum + exp2(logit[t] - mx);
    double lse2 = mx + log2(sum);
    for (int t = 0; t < T; ++t)
        p[t] = exp2(logit[t] - lse2);
}

/* The anchor query scaled like the proxies: fp64 product of its bf16 value
 * and log2(e)/sqrt(d), then fp32, then bf16. */
static void scale_query(const uint16_t *q, int d, uint16_t *out)
{
    double qs = oracle_query_scale(d);
    for (int j = 0; j < d; ++j) {
        double v = oracle_bf16_to_f64(q[j]) * qs;
        out[j] = oracle_f32_to_bf16((float)v);
    }
}

/*
 * proxies  [B, Hq, P, d] bf16, scaled by log2(e)/sqrt(d) (as step 1 makes them)
 * q_last   [B, Hq, d] bf16, not scaled (the anchor queries)
 * k        [B, Hkv, T, d] contiguous, dtype 0 (fp32, rounded to bf16) / 1
 * group_mass [B, Hkv, G, T] fp64 out (may be NULL)
 * mass       [B, Hkv, T] fp64 out;  anchor [B, Hkv, T] fp64 out
 */
int oracle_score(int B, int Hq, int Hkv, int T, int d, int P, int G,
                 const uint16_t *proxies, const uint16_t *q_last, const void *k, int kdtype,
                 double *group_mass, double *mass, double *anchor)
{
    if (B < 1 || Hq < 1 || Hkv < 1 || (Hq % Hkv) != 0 || T < 1 || d < 1 || P < 1 || G < 1 ||
        (P % G) != 0)
        return -1;
    int Gh = Hq / Hkv;
    int g = P / G;
    double *gm = group_mass;
    double *gm_own = NULL;
    if (!gm) {
        gm_own = (double *)malloc(sizeof(double) * (size_t)B * Hkv * G * T);
        gm = gm_own;
    }

    /* one task per (b, kv head, group): the group's rows are summed in a
     * fixed order (head, then proxy), independent of the thread count */
#pragma omp parallel for collapse(3) schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        for (int c = 0; c < Hkv; ++c) {
            for (int gi = 0; gi < G; ++gi) {
                double *logit = (double *)malloc(sizeof(double) * (size_t)T);
                double *p = (double *)malloc(sizeof(double) * (size_t)T);
                double *acc = gm + (((int64_t)b * Hkv + c) * G + gi) * T;
                for (int t = 0; t < T; ++t)
                    acc[t] = 0.0;
                int64_t kbase = ((int64_t)b * Hkv + c) * (int64_t)T * d;
                for (int hl = 0; hl < Gh; ++hl) {
                    int h = c * Gh + hl;
                    for (int i = gi * g; i < (gi + 1) * g; ++i) {
                        const uint16_t *q = proxies + (((int64_t)b * Hq + h) * P + i) * d;
                        softmax_row(q, k, kdtype, kbase, T, d, logit, p);
                        for (int t = 0; t < T; ++t)
                            acc[t] = acc[t] + p[t];
                    }
                }
                free(logit);
                free(p);
            }
        }
    }

#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int c = 0; c < Hkv; ++c) {
            double *logit = (double *)malloc(sizeof(double) * (size_t)T);
            double *p = (double *)malloc(sizeof(double) * (size_t)T);
            uint16_t *qa = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)d);
            int64_t kbase = ((int64_t)b * Hkv + c) * (int64_t)T * d;
            double *ms = mass + ((int64_t)b * Hkv + c) * T;
            double *an = anchor + ((int64_t)b * Hkv + c) * T;
            for (int t = 0; t < T; ++t) {
                double s = 0.0;
                for (int gi = 0; gi < G; ++gi)
                    s = s + gm[(((int64_t)b * Hkv + c) * G + gi) * T + t];
                ms[t] = s;
                an[t] = 0.0;
            }
            for (int hl = 0; hl < Gh; ++hl) {
                int h = c * Gh + hl;
                scale_query(q_last + ((int64_t)b * Hq + h) * d, d, qa);
                softmax_row(qa, k, kdtype, kbase, T, d, logit, p);
                for (int t = 0; t < T; ++t)
                    an[t] = an[t] + p[t];
            }
            for (int t = 0; t < T; ++t)
                an[t] = an[t] / (double)Gh;
            free(logit);
            free(p);
            free(qa);
        }
    }
    free(gm_own);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Step 3 -- tau-sets, votes, anchor score, budgeted top-k, temporal order   */
/* (Sec. 3.2.2 Eqs. 9-10; Sec. 3.2.3 Eq. 11; Appendix B; Algorithm 1).       */
/* ------------------------------------------------------------------------ */
typedef struct {
    double v;
    int t;
} keyed;

/* order: value descending, then index ascending */
static int cmp_desc(const void *a, const void *b)
{
    const keyed *x = (const keyed *)a, *y = (const keyed *)b;
    if (x->v > y->v) return -1;
    if (x->v < y->v) return 1;
    return (x->t > y->t) - (x->t < y->t);
}

static int cmp_int(const void *a, const void *b)
{
    int x = *(const int *)a, y = *(const int *)b;
    return (x > y) - (x < y);
}

/*
 * mode 0 = VOTE (paper): score = vote + lambda * anchor
 * mode 1 = MASS: score = total mass
 * group_mass [B, Hkv, G, T] (needed for VOTE), mass/anchor [B, Hkv, T] fp64
 * idx [B, Hkv, c_max] int32 out (ascending, -1 padded), counts [B, Hkv] out
 * votes [B, Hkv, T] int32 out or NULL; score [B, Hkv, T] fp64 out or NULL
 * cut_mass [B, Hkv, G] fp64 out or NULL: the mass of the last key that enters
 *   each tau-set; cut_size [B, Hkv, G] int32 out or NULL: the tau-set sizes
 */
int oracle_select(int B, int Hkv, int T, int G, int mode, double tau, double lambda,
                  int keep_last, int budget, int c_max, const double *group_mass,
                  const double *mass, const double *anchor, int32_t *idx, int32_t *counts,
                  int32_t *votes, double *score, double *cut_mass, int32_t *cut_size)
{
    if (B < 1 || Hkv < 1 || T < 1 || G < 1 || budget < 1 || c_max < budget ||
        !(tau > 0.0 && tau <= 1.0) || !(lambda >= 0.0) || (mode != 0 && mode != 1))
        return -1;

#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int b = 0; b < B; ++b) {
        for (int c = 0; c < Hkv; ++c) {
            int64_t hc = (int64_t)b * Hkv + c;
            keyed *kv = (keyed *)malloc(sizeof(keyed) * (size_t)T);
            int *vote = (int *)malloc(sizeof(int) * (size_t)T);
            double *S = (double *)malloc(sizeof(double) * (size_t)T);
            int *sel = (int *)malloc(sizeof(int) * (size_t)(T + 1));
            for (int t = 0; t < T; ++t)
                vote[t] = 0;
            if (mode == 0) {
                for (int gi = 0; gi < G; ++gi) {
                    const double *a = group_mass + (hc * G + gi) * T;
                    for (int t = 0; t < T; ++t) {
                        kv[t].v = a[t];
                        kv[t].t = t;
                    }
                    qsort(kv, (size_t)T, sizeof(keyed), cmp_desc);
                    double total = 0.0;
                    for (int r = 0; r < T; ++r)
                        total = total + kv[r].v;
                    double target = tau * total;
                    double run = 0.0;
                    int n = 0;
                    while (n < T) {
                        run = run + kv[n].v;
                        n = n + 1;
                        if (run >= target)
                            break;
                    }
                    for (int r = 0; r < n; ++r)
                        vote[kv[r].t] += 1;
                    if (cut_mass) cut_mass[hc * G + gi] = kv[n - 1].v;
                    if (cut_size) cut_size[hc * G + gi] = n;
                }
                for (int t = 0; t < T; ++t)
                    S[t] = (double)vote[t] + lambda * anchor[hc * T + t];
            } else {
                for (int t = 0; t < T; ++t)
                    S[t] = mass[hc * T + t];
            }
            if (votes)
                for (int t = 0; t < T; ++t)
                    votes[hc * T + t] = vote[t];
            if (score)
                for (int t = 0; t < T; ++t)
                    score[hc * T + t] = S[t];

            int nsel = 0;
            if (T <= budget) {
                for (int t = 0; t < T; ++t)
                    sel[nsel++] = t;
            } else {
                int pool = keep_last ? T - 1 : T;
                int want = keep_last ? budget - 1 : budget;
                for (int t = 0; t < pool; ++t) {
                    kv[t].v = S[t];
                    kv[t].t = t;
                }
                qsort(kv, (size_t)pool, sizeof(keyed), cmp_desc);
                for (int r = 0; r < want; ++r)
                    sel[nsel++] = kv[r].t;
                if (keep_last)
                    sel[nsel++] = T - 1;
                qsort(sel, (size_t)nsel, sizeof(int), cmp_int);
            }
            for (int j = 0; j < c_max; ++j)
                idx[hc * c_max + j] = (j < nsel) ? sel[j] : -1;
            counts[hc] = nsel;
            free(kv);
            free(vote);
            free(S);
            free(sel);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Step 4 -- gather the retained rows into the compacted cache (Appendix B:  */
/* restore temporal order, insert through the standard cache update).        */
/* src [B, H, T, row_bytes], idx [B, H, c_max], counts [B, H];               */
/* dst [B, H, c_max, row_bytes]; padding rows are zero-filled.               */
/* ------------------------------------------------------------------------ */
int oracle_gather(int B, int H, int T, int64_t row_bytes, int c_max, const void *src,
                  const int32_t *idx, const int32_t *counts, void *dst)
{
    if (B < 1 || H < 1 || T < 1 || row_bytes < 1 || c_max < 1)
        return -1;
    for (int64_t bh = 0; bh < (int64_t)B * H; ++bh) {
        for (int j = 0; j < c_max; ++j) {
            unsigned char *o = (unsigned char *)dst + (bh * c_max + j) * row_bytes;
            if (j < counts[bh]) {
                int t = idx[bh * c_max + j];
                if (t < 0 || t >= T)
                    return -1;
                memcpy(o, (const unsigned char *)src + (bh * T + t) * row_bytes, (size_t)row_bytes);
            } else {
                memset(o, 0, (size_t)row_bytes);
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Decode-time check: the attention-mass coverage of Fig. 1b (the fraction  */
/* of a decoding query's attention mass that falls on the prompt keys kept  */
/* after prefilling) and decode attention over the compacted cache, which   */
/* stays fixed while decoding under the prefill-only protocol (Sec. 3.1,    */
/* Sec. 3.2.3).  For decode query j of query head h (KV head c = h / Gh) of */
/* batch row b, with q~ the query scaled like the anchor query above and    */
/* p its softmax over all T prompt keys (Eq. 7, base-2 logits):             */
/*   coverage[b,h,j] = sum of p_t over the kept keys t (index order);       */
/*   out[b,h,j,:]    = sum_i p'_i v'_i, p' the softmax of q~ over the       */
/*                     counts[b,c] rows k'_i of the compacted cache.        */
/* q_dec [B, Hq, n_dec, d] bf16, not scaled; k [B, Hkv, T, d] contiguous,   */
/* kdtype; idx [B, Hkv, c_max] (ascending, -1 padded), counts [B, Hkv];     */
/* k_out, v_out [B, Hkv, c_max, d] kvdtype; coverage [B, Hq, n_dec] fp64    */
/* out; out [B, Hq, n_dec, d] fp64 out.                                     */
/* ------------------------------------------------------------------------ */
int oracle_decode_check(int B, int Hq, int Hkv, int T, int d, int n_dec,
                        const uint16_t *q_dec, const void *k, int kdtype,
                        const int32_t *idx, const int32_t *counts, int c_max,
                        const void *k_out, const void *v_out, int kvdtype,
                        double *coverage, double *out)
{
    if (B < 1 || Hq < 1 || Hkv < 1 || (Hq % Hkv) != 0 || T < 1 || d < 1 || n_dec < 1 || c_max < 1)
        return -1;
    for (int64_t bc = 0; bc < (int64_t)B * Hkv; ++bc) {
        if (counts[bc] < 0 || counts[bc] > c_max)
            return -1;
        for (int i = 0; i < counts[bc]; ++i) {
            int t = idx[bc * c_max + i];
            if (t < 0 || t >= T)
                return -1;
        }
    }
    const int Gh = Hq / Hkv;
    const int64_t rows = (int64_t)B * Hq * n_dec;
    int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
    for (int64_t r = 0; r < rows; ++r) {
        const int b = (int)(r / ((int64_t)Hq * n_dec));
        const int h = (int)((r / n_dec) % Hq);
        const int64_t bc = (int64_t)b * Hkv + h / Gh;
        uint16_t *qs = malloc(sizeof(uint16_t) * (size_t)d);
        double *logit = malloc(sizeof(double) * (size_t)T);
        double *p = malloc(sizeof(double) * (size_t)T);
        const int n = counts[bc];
        double *lc = malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
        if (!qs || !logit || !p || !lc) {
            bad = 1;
        } else {
            scale_query(q_dec + r * d, d, qs);
            softmax_row(qs, k, kdtype, bc * T * d, T, d, logit, p);
            double cov = 0.0;
            for (int i = 0; i < n; ++i)
                cov = cov + p[idx[bc * c_max + i]];
            coverage[r] = cov;
            /* softmax over the compacted rows, then the weighted sum of V' */
            double mx = -INFINITY;
            for (int i = 0; i < n; ++i) {
                double dot = 0.0;
                for (int j = 0; j < d; ++j) {
                    double prod = oracle_bf16_to_f64(qs[j]) * load_key_bf16(k_out, kvdtype, (bc * c_max + i) * d + j);
                    dot = dot + prod;
                }
                lc[i] = dot;
                if (dot > mx)
                    mx = dot;
            }
            double sum = 0.0;
            for (int i = 0; i < n; ++i)
                sum = sum + exp2(lc[i] - mx);
            const double lse2 = mx + log2(sum);
            for (int j = 0; j < d; ++j)
                out[r * d + j] = 0.0;
            for (int i = 0; i < n; ++i) {
                const double w = exp2(lc[i] - lse2);
                for (int j = 0; j < d; ++j)
                    out[r * d + j] = out[r * d + j] + w * load_elem(v_out, kvdtype, (bc * c_max + i) * d + j);
            }
        }
        free(qs);
        free(logit);
        free(p);
        free(lc);
    }
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Baseline selectors on the same scoring and selection (the comparison     */
/* methods of Sec. 4.1 as the paper configures them in its appendix on the  */
/* baselines).  Each one becomes a per-key score that the MASS-mode top-C   */
/* of oracle_select (keep_last = 0) turns into the kept set:                */
/*   SnapKV: the attention of the last `window` prompt queries (rows from   */
/*     oracle_window_rows, scored by oracle_score), summed over the GQA     */
/*     group, average-pooled over the prompt keys before the window         */
/*     (kernel `pool`, zero padding counted); the window itself is kept;    */
/*   StreamingLLM: the first `sinks` keys and then the most recent ones;    */
/*   ExpectedAttn: the proxy mass of N samples drawn without variance       */
/*     expansion (gamma = 1), the first `sinks` keys kept.                  */
/* A kept key gets score KEEP = 2^100, above any mass.                      */
/* ------------------------------------------------------------------------ */

/* the last n window queries of each head, scaled like the proxies
 * (times log2(e)/sqrt(d) in fp64, then fp32, then bf16):
 * q_win [B, Hq, W, d] dtype 0/1; rows [B, Hq, n, d] bf16 out */
int oracle_window_rows(int B, int Hq, int W, int d, int n, const void *q_win, int dtype, uint16_t *rows)
{
    if (B < 1 || Hq < 1 || W < 1 || d < 1 || n < 1 || n > W)
        return -1;
    const double qs = oracle_query_scale(d);
    for (int64_t bh = 0; bh < (int64_t)B * Hq; ++bh)
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < d; ++j) {
                /* window queries enter as bf16 values (fp32 inputs rounded first) */
                double x = oracle_bf16_to_f64(oracle_f32_to_bf16((float)load_elem(q_win, dtype, (bh * W + (W - n + i)) * d + j)));
                rows[(bh * n + i) * d + j] = oracle_f32_to_bf16((float)(x * qs));
            }
    return 0;
}

enum { ORACLE_SHAPE_SNAPKV = 0, ORACLE_SHAPE_STREAMING = 1, ORACLE_SHAPE_SINKS = 2 };

/* mass [B, Hkv, T] fp64 in; score [B, Hkv, T] fp64 out */
int oracle_shape_scores(int B, int Hkv, int T, int kind, int window, int pool, int sinks,
                        const double *mass, double *score)
{
    const double keep = ldexp(1.0, 100);
    if (B < 1 || Hkv < 1 || T < 1 || window < 0 || sinks < 0 || pool < 1 || (pool % 2) == 0)
        return -1;
    for (int64_t bc = 0; bc < (int64_t)B * Hkv; ++bc) {
        const double *m = mass + bc * T;
        double *o = score + bc * T;
        for (int t = 0; t < T; ++t) {
            if (kind == ORACLE_SHAPE_SNAPKV) {
                const int prefix = T - window;
                if (t >= prefix) {
                    o[t] = keep;
                } else {
                    double s = 0.0;
                    for (int u = t - pool / 2; u <= t + pool / 2; ++u)
                        if (u >= 0 && u < prefix)
                            s = s + m[u];
                    o[t] = s / pool;
                }
            } else if (kind == ORACLE_SHAPE_STREAMING) {
                o[t] = t < sinks ? keep : (double)t;
            } else if (kind == ORACLE_SHAPE_SINKS) {
                o[t] = t < sinks ? keep : m[t];
            } else {
                return -1;
            }
        }
    }
    return 0;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
