/*
 * Test driver: calls every exported function of the CPU oracle (drref.c)
 * on small inputs, including the edge cases of each (empty inputs, one
 * element, ties, all selected, the bucketless tiny filter, fewer values
 * than coefficients, chord segmentation, the double exponential, every
 * index policy).  Built together with drref.c by gcc with AddressSanitizer
 * and UndefinedBehaviorSanitizer (host code only) by
 * tests/test_oracle_sanitize.py, which runs it and expects exit status 0
 * and no sanitizer report.  Prints one line per function group.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint32_t drref_murmur3_32(const uint8_t *data, uint64_t len, uint32_t seed);
uint64_t drref_bloom_pos(uint32_t i, uint32_t j, uint64_t m);
void drref_bloom_pos_many(const uint32_t *idx, uint64_t n, uint32_t j, uint64_t m, uint64_t *out);
int drref_bloom_params(uint64_t n, double fpr, uint64_t *m_out, uint32_t *k_out);
int drref_topr(const float *g, uint64_t d, uint64_t r, uint32_t *S_out);
int drref_nonzero(const float *g, uint64_t d, uint32_t *S_out, uint64_t cap, uint64_t *n_out);
int drref_bloom_encode(const uint32_t *S, uint64_t n, uint64_t m, uint32_t k, uint32_t *words);
int drref_bloom_query(const uint32_t *words, uint64_t m, uint32_t k, uint64_t d, uint32_t *P_out, uint64_t cap,
                      uint64_t *n_out);
int drref_sort_desc(const float *V, uint64_t n, uint32_t *perm_out);
int drref_lsq_fit(const double *x, const double *y, uint64_t n, uint32_t D, double *coef_out);
void drref_fit_shape(uint64_t n, uint32_t D, uint32_t S, uint32_t *S_eff, uint32_t *D_eff);
uint32_t drref_sigma_bits(uint64_t n);
uint64_t drref_sigma_words(uint64_t n);
int drref_dexp_fit(const double *t, const double *y, uint64_t n, double *theta_out, double *rss_out);
int drref_segment(const float *C, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, uint64_t *bounds_out,
                  uint32_t *S_eff_out);
uint32_t drref_seg_heuristic(const float *C, uint64_t n, uint32_t D);
int drref_curvefit_encode_ex(const float *V, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, uint32_t model,
                             float *coef_out, double *coef64_out, uint32_t *sigma_out, uint64_t *bounds_out,
                             uint32_t *S_eff_out, uint32_t *D_eff_out, uint32_t *b_out, uint32_t *model_out);
int drref_curvefit_encode_seg(const float *V, uint64_t n, uint32_t D, uint32_t S, uint32_t mode, float *coef_out,
                              double *coef64_out, uint32_t *sigma_out, uint64_t *bounds_out, uint32_t *S_eff_out,
                              uint32_t *D_eff_out, uint32_t *b_out);
int drref_curvefit_encode(const float *V, uint64_t n, uint32_t D, uint32_t S, float *coef_out, double *coef64_out,
                          uint32_t *sigma_out, uint32_t *S_eff_out, uint32_t *D_eff_out, uint32_t *b_out);
int drref_curvefit_decode_ex(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S_eff,
                             const uint64_t *bounds, uint32_t model, float *vals_out);
int drref_curvefit_decode_seg(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S_eff,
                              const uint64_t *bounds, float *vals_out);
int drref_curvefit_decode(const float *coef, const uint32_t *sigma, uint64_t n, uint32_t D, uint32_t S,
                          float *vals_out);
uint32_t drref_perm(uint32_t q, uint64_t N, uint32_t seed);
int drref_policy_slots(uint64_t npos, uint64_t r, uint32_t policy, uint32_t seed, uint32_t *slot_out,
                       uint64_t *ncoded);

#define MAXN 20000
#define MAXS 4096

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(void) /* xorshift64*, top 32 bits */
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}
static float frnd(void) { return ((float)rnd() / 4294967296.0f - 0.5f) * 2e-3f; }

static int fails = 0;
static void expect(int cond, const char *what)
{
    if (!cond) {
        printf("FAIL %s\n", what);
        ++fails;
    }
}

static float g[MAXN], V[MAXN], vals[MAXN], coef[MAXS * 8];
static double coef64[MAXS * 8], x64[MAXN], y64[MAXN];
static uint32_t S[MAXN], P[MAXN], perm[MAXN], sigma[MAXN + 2], slots[MAXN];
static uint64_t bounds[MAXS + 1], pos[MAXN];
static uint32_t words[1 << 16];

static void hashes(void)
{
    const uint8_t msg[] = "Hello, world!";
    expect(drref_murmur3_32(msg, 0, 0) == 0, "murmur empty");
    expect(drref_murmur3_32(msg, 13, 0x9747B28Cu) == 0x24884CBAu, "murmur known answer");
    for (uint64_t len = 0; len <= 13; ++len)
        (void)drref_murmur3_32(msg, len, 7);
    (void)drref_bloom_pos(0, 0, 32);
    (void)drref_bloom_pos(0xFFFFFFFFu, 31, 0xFFFFFFE0u);
    for (uint32_t q = 0; q < 100; ++q)
        S[q] = rnd();
    drref_bloom_pos_many(S, 100, 3, 150784, pos);
    drref_bloom_pos_many(S, 0, 3, 150784, pos);
    uint64_t m;
    uint32_t k;
    expect(drref_bloom_params(10486, 1e-3, &m, &k) == 0 && m == 150784 && k == 10, "bloom params");
    expect(drref_bloom_params(0, 1e-3, &m, &k) == 0 && m == 32, "bloom params n=0");
    expect(drref_bloom_params(10, 0.0, &m, &k) != 0, "bloom params bad rate");
    printf("hashes ok\n");
}

static void select_and_filter(uint64_t d, uint64_t r, double fpr)
{
    for (uint64_t i = 0; i < d; ++i)
        g[i] = (i % 7 == 3) ? 0.0f : frnd();
    if (d > 4) {
        g[1] = g[2]; /* a tie */
        g[3] = -0.0f;
    }
    expect(drref_topr(g, d, r, S) == 0, "topr");
    uint64_t nz = 0;
    expect(drref_nonzero(g, d, S + 0, MAXN, &nz) == 0, "nonzero");
    expect(drref_topr(g, d, r, S) == 0, "topr again");
    uint64_t m;
    uint32_t k;
    expect(drref_bloom_params(r, fpr, &m, &k) == 0, "params");
    if (m / 32 > sizeof words / 4)
        return;
    expect(drref_bloom_encode(S, r, m, k, words) == 0, "bloom encode");
    uint64_t np = 0;
    expect(drref_bloom_query(words, m, k, d, P, MAXN, &np) == 0, "bloom query");
    expect(np >= r, "no false negatives");
    uint64_t np2 = 0;
    (void)drref_bloom_query(words, m, k, d, P, np / 2, &np2); /* capacity too small */
    expect(np2 == np, "query count with a short output");
}

static void fits(uint64_t n, uint32_t D, uint32_t Sg)
{
    for (uint64_t i = 0; i < n; ++i)
        V[i] = (i % 11 == 0) ? V[i / 2] : frnd(); /* ties */
    expect(drref_sort_desc(V, n, perm) == 0, "sort");
    for (uint64_t i = 0; i < n; ++i) {
        x64[i] = (double)i;
        y64[i] = (double)V[i];
    }
    if (n >= D + 1)
        expect(drref_lsq_fit(x64, y64, n, D, coef64) == 0, "lsq fit");
    uint32_t se = 0, de = 0, b = 0, mo = 0;
    drref_fit_shape(n, D, Sg, &se, &de);
    (void)drref_sigma_bits(n);
    (void)drref_sigma_words(n);
    for (uint32_t mode = 0; mode <= 1; ++mode) {
        memset(sigma, 0, sizeof sigma);
        expect(drref_curvefit_encode_ex(V, n, D, Sg, mode, 0, coef, coef64, sigma, bounds, &se, &de, &b, &mo) == 0,
               "encode poly");
        expect(drref_curvefit_decode_ex(coef, sigma, n, D, se, bounds, mo, vals) == 0, "decode poly");
        expect(drref_curvefit_encode_seg(V, n, D, Sg, mode, coef, coef64, sigma, bounds, &se, &de, &b) == 0,
               "encode seg");
        expect(drref_curvefit_decode_seg(coef, sigma, n, D, se, bounds, vals) == 0, "decode seg");
        if (Sg) {
            uint32_t s2 = 0;
            expect(drref_segment(V, n, D, Sg, mode, bounds, &s2) == 0, "segment");
        }
    }
    if (Sg) {
        expect(drref_curvefit_encode(V, n, D, Sg, coef, coef64, sigma, &se, &de, &b) == 0, "encode");
        expect(drref_curvefit_decode(coef, sigma, n, D, Sg, vals) == 0, "decode");
    }
    /* the double exponential (degree 3 rows) */
    expect(drref_curvefit_encode_ex(V, n, 3, Sg ? Sg : 1, 0, 1, coef, coef64, sigma, bounds, &se, &de, &b, &mo) == 0,
           "encode dexp");
    expect(drref_curvefit_decode_ex(coef, sigma, n, 3, se, bounds, mo, vals) == 0, "decode dexp");
    /* the run-count heuristic needs the sorted curve */
    for (uint64_t i = 0; i < n; ++i)
        vals[i] = V[perm[i]];
    (void)drref_seg_heuristic(vals, n, D);
    if (n >= 4) {
        double th[4], rss;
        for (uint64_t i = 0; i < n; ++i)
            x64[i] = n > 1 ? (2.0 * (double)i - (double)(n - 1)) / (double)(n - 1) : 0.0;
        expect(drref_dexp_fit(x64, y64, n, th, &rss) == 0, "dexp fit");
    }
}

static void policies(void)
{
    const uint64_t sizes[] = {0, 1, 2, 3, 17, 1000, 4097};
    for (unsigned a = 0; a < sizeof sizes / sizeof sizes[0]; ++a) {
        uint64_t np = sizes[a];
        for (uint32_t pol = 0; pol <= 4; ++pol) {
            uint64_t nc = 0;
            expect(drref_policy_slots(np, np / 3, pol, 12345u + pol, slots, &nc) == 0, "policy slots");
        }
        for (uint32_t q = 0; q < np && q < 50; ++q)
            (void)drref_perm(q, np, 99u);
    }
    printf("policies ok\n");
}

int main(void)
{
    hashes();
    const uint64_t shapes[][2] = {{0, 0}, {1, 0}, {1, 1}, {5, 5}, {64, 7}, {4097, 41}, {9000, 900}, {20000, 200}};
    for (unsigned s = 0; s < sizeof shapes / sizeof shapes[0]; ++s) {
        select_and_filter(shapes[s][0], shapes[s][1], 1e-3);
        select_and_filter(shapes[s][0], shapes[s][1], 0.3);
    }
    printf("selection and filters ok\n");
    const uint64_t fshapes[][3] = {{0, 5, 8}, {1, 5, 8}, {3, 5, 8}, {6, 5, 1}, {100, 1, 0}, {5000, 5, 8},
                                   {4000, 0, 4096}, {7000, 3, 16}};
    for (unsigned s = 0; s < sizeof fshapes / sizeof fshapes[0]; ++s)
        fits(fshapes[s][0], (uint32_t)fshapes[s][1], (uint32_t)fshapes[s][2]);
    printf("fits ok\n");
    policies();
    if (fails) {
        printf("%d failures\n", fails);
        return 1;
    }
    printf("all ok\n");
    return 0;
}
