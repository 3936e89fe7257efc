/*
 * Native checks of the C oracle, built with AddressSanitizer and
 * UndefinedBehaviorSanitizer by tests/test_sanitizers.py.  Every array has
 * exactly the length the step may touch, so a read or write past a key's
 * end, or into a zero-length key, is reported.
 *   1. The worked example of tests/golden/worked_example.txt (path in
 *      argv[1]): three steps of one element, bit for bit (exact dyadic
 *      values; paper section 3.2.2 and section 4.2).
 *   2. Many shapes against a second, independently written loop of the
 *      same definition (ascending worker sum, then the four fused updates),
 *      bit for bit, both momentum forms.
 *   3. The double-precision, plain SGD and Adam steps over the same shapes
 *      (they must stay finite), and argument errors.
 * Exit status 0 when everything holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_step_f32(int, int, const int64_t *, const float *const *, float *const *,
                    float *const *, float, float, float, int);
int oracle_step_f64(int, int, const int64_t *, const double *const *, double *const *,
                    double *const *, double, double, double, int);
int oracle_step_sgd_f32(int, int, const int64_t *, const float *const *, float *const *, float,
                        float);
int oracle_step_adam_f32(int, int, const int64_t *, const float *const *, float *const *,
                         float *const *, float *const *, float, float, float, float, float,
                         int64_t);

static int failures = 0;

static void check(int ok, const char *what) {
    if (!ok) {
        fprintf(stderr, "FAILED: %s\n", what);
        ++failures;
    }
}

static uint32_t bits(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    return u;
}

/* a small deterministic generator (xorshift), values in [-0.5, 0.5) */
static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static float draw(void) {
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return (float)((double)(rng_state >> 11) / 9007199254740992.0 - 0.5);
}

static float *alloc_f(int64_t n) { return n ? (float *)malloc((size_t)n * sizeof(float)) : NULL; }

static void worked_example(const char *path) {
    FILE *f = fopen(path, "r");
    check(f != NULL, "open the worked example");
    if (!f) return;
    char line[256];
    float g0 = 0, g1 = 0, w0 = 0, m0 = 0, lr = 0, mu = 0, wd = 0;
    int cases = 0;
    while (fgets(line, sizeof line, f)) {
        if (strncmp(line, "inputs ", 7) == 0) {
            check(sscanf(line + 7, "%f %f %f %f %f %f %f", &g0, &g1, &w0, &m0, &lr, &mu, &wd) == 7,
                  "parse the inputs line");
        } else if (strncmp(line, "nesterov ", 9) == 0 || strncmp(line, "plain ", 6) == 0) {
            const int nest = line[0] == 'n';
            int step = 0;
            float we = 0, me = 0;
            check(sscanf(line + (nest ? 9 : 6), "%d %f %f", &step, &we, &me) == 3, "parse a case");
            float *g[2] = {alloc_f(1), alloc_f(1)};
            float *w = alloc_f(1), *m = alloc_f(1);
            g[0][0] = g0;
            g[1][0] = g1;
            w[0] = w0;
            m[0] = m0;
            const int64_t n = 1;
            for (int t = 0; t < step; ++t)
                check(oracle_step_f32(2, 1, &n, (const float *const *)g, &w, &m, lr, mu, wd, nest) == 0,
                      "worked example step");
            check(bits(w[0]) == bits(we) && bits(m[0]) == bits(me), "worked example values");
            free(g[0]);
            free(g[1]);
            free(w);
            free(m);
            ++cases;
        }
    }
    fclose(f);
    check(cases == 6, "six worked-example cases");
}

static void shapes(void) {
    static const int workers[] = {1, 2, 3, 4, 16};
    static const int64_t lens[] = {0, 1, 2, 3, 4, 5, 7, 8, 15, 16, 17, 8191, 8192, 8193};
    const int K = (int)(sizeof lens / sizeof lens[0]);
    for (size_t wi = 0; wi < sizeof workers / sizeof workers[0]; ++wi) {
        const int N = workers[wi];
        for (int nest = 0; nest < 2; ++nest) {
            float **g = (float **)malloc((size_t)N * K * sizeof(float *));
            float **w = (float **)malloc(K * sizeof(float *));
            float **m = (float **)malloc(K * sizeof(float *));
            float **wr = (float **)malloc(K * sizeof(float *));
            float **mr = (float **)malloc(K * sizeof(float *));
            for (int k = 0; k < K; ++k) {
                for (int j = 0; j < N; ++j) {
                    g[j * K + k] = alloc_f(lens[k]);
                    for (int64_t i = 0; i < lens[k]; ++i) g[j * K + k][i] = draw() * 0.02f;
                }
                w[k] = alloc_f(lens[k]);
                m[k] = alloc_f(lens[k]);
                wr[k] = alloc_f(lens[k]);
                mr[k] = alloc_f(lens[k]);
                for (int64_t i = 0; i < lens[k]; ++i) {
                    w[k][i] = wr[k][i] = draw() * 0.1f;
                    m[k][i] = mr[k][i] = draw() * 0.01f;
                }
            }
            const float lr = 0.1f, mu = 0.9f, wd = 1e-4f;
            check(oracle_step_f32(N, K, lens, (const float *const *)g, w, m, lr, mu, wd, nest) == 0,
                  "step over the shapes");
            /* the same definition written again: s in worker order, then fused updates */
            for (int k = 0; k < K; ++k)
                for (int64_t i = 0; i < lens[k]; ++i) {
                    float s = 0.0f;
                    for (int j = 0; j < N; ++j) s = j == 0 ? g[k][i] : s + g[j * K + k][i];
                    const float d = fmaf(wd, wr[k][i], s);
                    const float m1 = fmaf(mu, mr[k][i], d);
                    const float u = nest ? fmaf(mu, m1, d) : m1;
                    wr[k][i] = fmaf(-lr, u, wr[k][i]);
                    mr[k][i] = m1;
                    check(bits(w[k][i]) == bits(wr[k][i]) && bits(m[k][i]) == bits(mr[k][i]),
                          "second loop agrees");
                }
            /* the other steps over the same shapes */
            double **gd = (double **)malloc((size_t)N * K * sizeof(double *));
            double **wd64 = (double **)malloc(K * sizeof(double *));
            double **md64 = (double **)malloc(K * sizeof(double *));
            float **vz = (float **)malloc(K * sizeof(float *));
            for (int k = 0; k < K; ++k) {
                vz[k] = lens[k] ? (float *)calloc((size_t)lens[k], sizeof(float)) : NULL;
                for (int j = 0; j < N; ++j) {
                    gd[j * K + k] = lens[k] ? (double *)malloc((size_t)lens[k] * sizeof(double)) : NULL;
                    for (int64_t i = 0; i < lens[k]; ++i) gd[j * K + k][i] = g[j * K + k][i];
                }
                wd64[k] = lens[k] ? (double *)calloc((size_t)lens[k], sizeof(double)) : NULL;
                md64[k] = lens[k] ? (double *)calloc((size_t)lens[k], sizeof(double)) : NULL;
            }
            check(oracle_step_f64(N, K, lens, (const double *const *)gd, wd64, md64, 0.1, 0.9, 1e-4,
                                  nest) == 0, "double step");
            check(oracle_step_sgd_f32(N, K, lens, (const float *const *)g, w, lr, wd) == 0, "SGD step");
            check(oracle_step_adam_f32(N, K, lens, (const float *const *)g, w, m, vz, 1e-3f, 0.9f,
                                       0.999f, 1e-8f, wd, 1 + nest) == 0, "Adam step");
            for (int k = 0; k < K; ++k)
                for (int64_t i = 0; i < lens[k]; ++i)
                    check(isfinite(w[k][i]) && isfinite(m[k][i]) && isfinite(wd64[k][i]),
                          "finite results");
            for (int k = 0; k < K; ++k) {
                for (int j = 0; j < N; ++j) {
                    free(g[j * K + k]);
                    free(gd[j * K + k]);
                }
                free(w[k]);
                free(m[k]);
                free(wr[k]);
                free(mr[k]);
                free(wd64[k]);
                free(md64[k]);
                free(vz[k]);
            }
            free(vz);
            free(g);
            free(gd);
            free(w);
            free(m);
            free(wr);
            free(mr);
            free(wd64);
            free(md64);
        }
    }
}

static void argument_errors(void) {
    const int64_t n = 4, neg = -1;
    float a[4] = {0}, *p = a;
    const float *cp = a;
    check(oracle_step_f32(0, 1, &n, &cp, &p, &p, 0.1f, 0.9f, 0.0f, 1) == -1, "zero workers");
    check(oracle_step_f32(1, 0, &n, &cp, &p, &p, 0.1f, 0.9f, 0.0f, 1) == -1, "zero keys");
    check(oracle_step_f32(1, 1, &neg, &cp, &p, &p, 0.1f, 0.9f, 0.0f, 1) == -1, "negative length");
    check(oracle_step_f32(1, 1, &n, NULL, &p, &p, 0.1f, 0.9f, 0.0f, 1) == -1, "null gradients");
    check(oracle_step_adam_f32(1, 1, &n, &cp, &p, &p, &p, 0.1f, 1.0f, 0.9f, 0.0f, 0.0f, 1) == -1,
          "beta1 of 1");
    check(oracle_step_adam_f32(1, 1, &n, &cp, &p, &p, &p, 0.1f, 0.9f, 0.9f, 0.0f, 0.0f, 0) == -1,
          "step 0");
}

int main(int argc, char **argv) {
    if (argc < 2) {
        fprintf(stderr, "usage: oracle_check worked_example.txt\n");
        return 2;
    }
    worked_example(argv[1]);
    shapes();
    argument_errors();
    if (failures) fprintf(stderr, "%d checks failed\n", failures);
    else printf("oracle checks passed\n");
    return failures ? 1 : 0;
}
