/* Memory- and UB-check driver for the C oracle (test infrastructure, CPU only).
 *
 * Built together with mmskv_oracle.c under -fsanitize=address,undefined by
 * tests/test_oracle_sanitize.py and run once: every exported oracle routine
 * is called on small inputs held in heap buffers of exactly the documented
 * sizes (so that a read or write past any of them is reported), in both
 * input dtypes and with the optional outputs present and absent, plus the
 * argument checks that must refuse.  Inputs come from a plain xorshift
 * stream of this file; no result is compared here (the pins and parity tests
 * do that), only the return codes.  Exit status 0 when every call returned
 * what it should. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
float oracle_uniform(uint32_t x);
float oracle_ln(float u);
void oracle_sincos_2pi(uint32_t x, float *sin_out, float *cos_out);
void oracle_normal4(uint64_t seed, int b, int layer, int h, int i, int jq, double z[4]);
uint16_t oracle_f32_to_bf16(float x);
double oracle_bf16_to_f64(uint16_t h);
double oracle_query_scale(int d);
int oracle_build_proxies_at(int B, int Hq, int W, int d, int P, double gamma, int ddof, uint64_t seed, int layer,
                            int b0, int h0, const void *q_win, int dtype, const float *rope_cos_f,
                            const float *rope_sin_f, const float *rope_cos_l, const float *rope_sin_l,
                            uint16_t *proxies, uint16_t *q_last, double *stats);
int oracle_build_proxies(int B, int Hq, int W, int d, int P, double gamma, int ddof, uint64_t seed, int layer,
                         const void *q_win, int dtype, const float *rope_cos_f, const float *rope_sin_f,
                         const float *rope_cos_l, const float *rope_sin_l, uint16_t *proxies, uint16_t *q_last,
                         double *stats);
int oracle_hidden_stats(int B, int T, int D, int ddof, const void *hidden, int dtype, double *stats);
int oracle_hidden_proxies(int B, int D, int P, double gamma, uint64_t seed, int layer, int b0,
                          const double *stats, uint16_t *hp);
int oracle_project_proxies(int B, int P, int D, int Hq, int d, const uint16_t *hp, const uint16_t *wq,
                           const float *rope_cos, const float *rope_sin, uint16_t *proxies, double *pre);
int oracle_score(int B, int Hq, int Hkv, int T, int d, int P, int G, const uint16_t *proxies,
                 const uint16_t *q_last, const void *k, int kdtype, double *group_mass, double *mass,
                 double *anchor);
int oracle_select(int B, int Hkv, int T, int G, int mode, double tau, double lambda, int keep_last, int budget,
                  int c_max, const double *group_mass, const double *mass, const double *anchor, int32_t *idx,
                  int32_t *counts, int32_t *votes, double *score, double *cut_mass, int32_t *cut_size);
int oracle_gather(int B, int H, int T, int64_t row_bytes, int c_max, const void *src, const int32_t *idx,
                  const int32_t *counts, void *dst);
int oracle_decode_check(int B, int Hq, int Hkv, int T, int d, int n_dec, const uint16_t *q_dec, const void *k,
                        int kdtype, const int32_t *idx, const int32_t *counts, int c_max, const void *k_out,
                        const void *v_out, int kvdtype, double *coverage, double *out);
int oracle_window_rows(int B, int Hq, int W, int d, int n, const void *q_win, int dtype, uint16_t *rows);
int oracle_shape_scores(int B, int Hkv, int T, int kind, int window, int pool, int sinks, const double *mass,
                        double *score);
int oracle_num_threads(void);

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (uint32_t)(rng >> 16);
}
static float next_f(void) { return (float)((int)(next_u32() % 20001) - 10000) / 4000.0f; }

static int failures = 0;
static void expect(int got, int want, const char *what) {
    if (got != want) {
        fprintf(stderr, "%s: returned %d, expected %d\n", what, got, want);
        ++failures;
    }
}

static void *xmalloc(size_t n) {
    void *p = malloc(n ? n : 1);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

/* input tensors: fp32 (dtype 0) or bf16 bits (dtype 1), n elements */
static void *make_input(size_t n, int dtype) {
    if (dtype == 0) {
        float *x = xmalloc(n * sizeof(float));
        for (size_t i = 0; i < n; ++i) x[i] = next_f();
        return x;
    }
    uint16_t *x = xmalloc(n * sizeof(uint16_t));
    for (size_t i = 0; i < n; ++i) x[i] = oracle_f32_to_bf16(next_f());
    return x;
}

static float *make_table(int n) {
    float *t = xmalloc((size_t)n * sizeof(float));
    for (int i = 0; i < n; ++i) t[i] = (float)cos(0.1 * (i + 1));
    return t;
}

static void scalar_routines(void) {
    uint32_t ctr[4] = {1u, 2u, 3u, 4u}, key[2] = {5u, 6u}, out[4];
    oracle_philox4x32_10(ctr, key, out);
    float s, c;
    for (int i = 0; i < 64; ++i) {
        const uint32_t x = next_u32();
        (void)oracle_ln(oracle_uniform(x));
        oracle_sincos_2pi(x, &s, &c);
    }
    double z[4];
    oracle_normal4(123u, 1, 2, 3, 4, 5, z);
    (void)oracle_bf16_to_f64(oracle_f32_to_bf16(1.5f));
    (void)oracle_query_scale(128);
    expect(oracle_num_threads() >= 1, 1, "num_threads");
}

static void proxies_and_hidden(void) {
    const int B = 2, Hq = 4, W = 5, d = 8, P = 32;
    for (int dtype = 0; dtype < 2; ++dtype)
        for (int rope = 0; rope < 2; ++rope)
            for (int ddof = 0; ddof < 2; ++ddof) {
                void *q = make_input((size_t)B * Hq * W * d, dtype);
                float *cf = rope ? make_table(d / 2) : NULL, *sf = rope ? make_table(d / 2) : NULL;
                float *cl = rope ? make_table(d / 2) : NULL, *sl = rope ? make_table(d / 2) : NULL;
                uint16_t *prox = xmalloc((size_t)B * Hq * P * d * 2), *ql = xmalloc((size_t)B * Hq * d * 2);
                double *st = xmalloc((size_t)B * Hq * 2 * d * sizeof(double));
                expect(oracle_build_proxies(B, Hq, W, d, P, 2.0, ddof, 7u, 3, q, dtype, cf, sf, cl, sl, prox, ql,
                                            ddof ? NULL : st), 0, "build_proxies");
                expect(oracle_build_proxies_at(B, Hq, W, d, P, 0.0, ddof, 7u, 3, 1, 2, q, dtype, cf, sf, cl, sl,
                                               prox, ql, st), 0, "build_proxies_at");
                uint16_t *rows = xmalloc((size_t)B * Hq * 2 * d * 2);
                expect(oracle_window_rows(B, Hq, W, d, 2, q, dtype, rows), 0, "window_rows");
                free(rows); free(q); free(cf); free(sf); free(cl); free(sl); free(prox); free(ql); free(st);
            }
    expect(oracle_build_proxies(1, 1, 1, 8, 4, 1.0, 1, 0, 0, NULL, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL), -1,
           "build_proxies W - ddof < 1");
    expect(oracle_build_proxies(1, 1, 4, 6, 4, 1.0, 0, 0, 0, NULL, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL), -1,
           "build_proxies d % 4");

    const int T = 7, D = 8, Hh = 2, dh = 8;
    for (int dtype = 0; dtype < 2; ++dtype)
        for (int ddof = 0; ddof < 2; ++ddof) {
            void *h = make_input((size_t)B * T * D, dtype);
            double *st = xmalloc((size_t)B * 2 * D * sizeof(double));
            expect(oracle_hidden_stats(B, T, D, ddof, h, dtype, st), 0, "hidden_stats");
            uint16_t *hp = xmalloc((size_t)B * P * D * 2);
            expect(oracle_hidden_proxies(B, D, P, 3.0, 11u, 1, 0, st, hp), 0, "hidden_proxies");
            uint16_t *wq = make_input((size_t)Hh * dh * D, 1);
            float *cs = make_table(dh / 2), *sn = make_table(dh / 2);
            uint16_t *prox = xmalloc((size_t)B * Hh * P * dh * 2);
            double *pre = xmalloc((size_t)B * Hh * P * dh * sizeof(double));
            expect(oracle_project_proxies(B, P, D, Hh, dh, hp, wq, ddof ? cs : NULL, ddof ? sn : NULL, prox,
                                          ddof ? pre : NULL), 0, "project_proxies");
            free(h); free(st); free(hp); free(wq); free(cs); free(sn); free(prox); free(pre);
        }
    expect(oracle_hidden_stats(1, 1, 8, 1, NULL, 0, NULL), -1, "hidden_stats T - ddof < 1");
}

static void score_select_gather_decode(void) {
    const int B = 2, Hq = 4, Hkv = 2, d = 8, P = 32, G = 2, n_dec = 3;
    const int Ts[3] = {1, 5, 37};
    for (int ti = 0; ti < 3; ++ti)
        for (int kdtype = 0; kdtype < 2; ++kdtype) {
            const int T = Ts[ti];
            uint16_t *prox = make_input((size_t)B * Hq * P * d, 1), *ql = make_input((size_t)B * Hq * d, 1);
            void *k = make_input((size_t)B * Hkv * T * d, kdtype);
            double *gm = xmalloc((size_t)B * Hkv * G * T * sizeof(double));
            double *mass = xmalloc((size_t)B * Hkv * T * sizeof(double)), *an = xmalloc((size_t)B * Hkv * T * sizeof(double));
            expect(oracle_score(B, Hq, Hkv, T, d, P, G, prox, ql, k, kdtype, kdtype ? gm : NULL, mass, an), 0,
                   "score (no group masses)");
            expect(oracle_score(B, Hq, Hkv, T, d, P, G, prox, ql, k, kdtype, gm, mass, an), 0, "score");
            for (int mode = 0; mode < 2; ++mode)
                for (int keep = 0; keep < 2; ++keep) {
                    const int budgets[3] = {1, 4, 64};
                    for (int bi = 0; bi < 3; ++bi) {
                        const int budget = budgets[bi], c_max = budget + 3;
                        int32_t *idx = xmalloc((size_t)B * Hkv * c_max * 4), *cnt = xmalloc((size_t)B * Hkv * 4);
                        int32_t *votes = xmalloc((size_t)B * Hkv * T * 4), *csz = xmalloc((size_t)B * Hkv * G * 4);
                        double *sc = xmalloc((size_t)B * Hkv * T * sizeof(double));
                        double *cm = xmalloc((size_t)B * Hkv * G * sizeof(double));
                        const int full = (bi + mode) & 1;
                        expect(oracle_select(B, Hkv, T, G, mode, bi == 2 ? 1.0 : 0.95, bi == 1 ? 0.0 : 1.0, keep,
                                             budget, c_max, gm, mass, an, idx, cnt, full ? votes : NULL,
                                             full ? sc : NULL, full ? cm : NULL, full ? csz : NULL), 0, "select");
                        /* gather both rows and a 16-byte row of a wider layout */
                        uint8_t *dst = xmalloc((size_t)B * Hkv * c_max * d * 2);
                        expect(oracle_gather(B, Hkv, T, (int64_t)d * 2, c_max, k, idx, cnt, dst), 0, "gather");
                        uint16_t *qd = make_input((size_t)B * Hq * n_dec * d, 1);
                        uint16_t *ko = xmalloc((size_t)B * Hkv * c_max * d * 2), *vo = xmalloc((size_t)B * Hkv * c_max * d * 2);
                        uint16_t *kbf = make_input((size_t)B * Hkv * T * d, 1);
                        expect(oracle_gather(B, Hkv, T, (int64_t)d * 2, c_max, kbf, idx, cnt, ko), 0, "gather k");
                        expect(oracle_gather(B, Hkv, T, (int64_t)d * 2, c_max, kbf, idx, cnt, vo), 0, "gather v");
                        double *cov = xmalloc((size_t)B * Hq * n_dec * sizeof(double));
                        double *out = xmalloc((size_t)B * Hq * n_dec * d * sizeof(double));
                        expect(oracle_decode_check(B, Hq, Hkv, T, d, n_dec, qd, kbf, 1, idx, cnt, c_max, ko, vo, 1,
                                                   cov, out), 0, "decode_check");
                        free(idx); free(cnt); free(votes); free(csz); free(sc); free(cm); free(dst); free(qd);
                        free(ko); free(vo); free(kbf); free(cov); free(out);
                    }
                }
            for (int kind = 0; kind < 3; ++kind) {
                double *sc = xmalloc((size_t)B * Hkv * T * sizeof(double));
                expect(oracle_shape_scores(B, Hkv, T, kind, 3, 5, 2, mass, sc), 0, "shape_scores");
                free(sc);
            }
            free(prox); free(ql); free(k); free(gm); free(mass); free(an);
        }
    expect(oracle_score(1, 3, 2, 4, 8, 32, 2, NULL, NULL, NULL, 1, NULL, NULL, NULL), -1, "score Hq % Hkv");
    expect(oracle_select(1, 1, 4, 1, 0, 0.0, 1.0, 1, 2, 2, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL), -1,
           "select tau = 0");
    expect(oracle_select(1, 1, 4, 1, 0, 0.9, 1.0, 1, 3, 2, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL), -1,
           "select c_max < budget");
    expect(oracle_shape_scores(1, 1, 4, 0, 1, 4, 0, NULL, NULL), -1, "shape_scores even pool");
}

int main(void) {
    scalar_routines();
    proxies_and_hidden();
    score_select_gather_decode();
    if (failures) {
        fprintf(stderr, "%d unexpected return code(s)\n", failures);
        return 1;
    }
    printf("oracle sanitize driver: all calls returned as expected\n");
    return 0;
}
