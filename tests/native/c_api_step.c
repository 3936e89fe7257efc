/*
 * The library driven through its C interface alone (include/phub.h, no
 * Python): a job of 8 workers over ragged keys, three steps with fresh
 * gradients, every key read back through phub_pull and phub_get_state and
 * compared bit for bit with the C oracle (oracle/phub_oracle.c, linked into
 * this test program only).  Exits 0 and prints "c api checks passed", or
 * exits 1 with the first failure.
 */
#include <hip/hip_runtime_api.h>

#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "phub.h"

int oracle_step_f32(int num_workers, int num_keys, const int64_t *key_elems,
                    const float *const *grads, float *const *weights, float *const *moms,
                    float lr, float mu, float wd, int nesterov);

#define N 8
#define K 7
#define STEPS 3

#define CHECK_HIP(x)                                                               \
    do {                                                                           \
        hipError_t e_ = (x);                                                       \
        if (e_ != hipSuccess) {                                                    \
            fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));         \
            return 1;                                                              \
        }                                                                          \
    } while (0)
#define CHECK_PHUB(x)                                                              \
    do {                                                                           \
        int rc_ = (x);                                                             \
        if (rc_ != PHUB_OK) {                                                      \
            fprintf(stderr, "%s returned %d: %s\n", #x, rc_, phub_last_error());   \
            return 1;                                                              \
        }                                                                          \
    } while (0)

/* a small counter-free generator: xorshift32, mapped to [-scale, scale) */
static uint32_t rng = 1805u;
static float uniform(float scale) {
    rng ^= rng << 13;
    rng ^= rng >> 17;
    rng ^= rng << 5;
    return scale * ((float)(rng >> 8) / 8388608.0f - 1.0f);
}

int main(void) {
    const int64_t key_elems[K] = {5, 1024, 8193, 0, 40000, 3, 2 * 8192 + 3};
    const float lr = 0.1f, mu = 0.9f, wd = 1e-4f;
    hipStream_t stream;
    CHECK_HIP(hipStreamCreate(&stream));
    phub_job *job = NULL;
    CHECK_PHUB(phub_init(&job, N, K, key_elems, 32768, lr, mu, wd, 1, stream));

    float *w_host[K], *m_host[K], *g_host[N * K];
    float *g_dev[N * K], *w0_dev[K];
    for (int k = 0; k < K; ++k) {
        const size_t bytes = (size_t)(key_elems[k] > 0 ? key_elems[k] : 1) * sizeof(float);
        w_host[k] = malloc(bytes);
        m_host[k] = calloc(1, bytes);
        if (!w_host[k] || !m_host[k]) return 1;
        for (int64_t i = 0; i < key_elems[k]; ++i) w_host[k][i] = uniform(0.05f);
        CHECK_HIP(hipMalloc((void **)&w0_dev[k], bytes));
        CHECK_HIP(hipMemcpy(w0_dev[k], w_host[k], (size_t)key_elems[k] * sizeof(float),
                            hipMemcpyHostToDevice));
        CHECK_PHUB(phub_set_weights(job, k, w0_dev[k]));
        for (int w = 0; w < N; ++w) {
            g_host[w * K + k] = malloc(bytes);
            if (!g_host[w * K + k]) return 1;
            CHECK_HIP(hipMalloc((void **)&g_dev[w * K + k], bytes));
        }
    }

    for (int t = 0; t < STEPS; ++t) {
        for (int w = 0; w < N; ++w)
            for (int k = 0; k < K; ++k) {
                for (int64_t i = 0; i < key_elems[k]; ++i) g_host[w * K + k][i] = uniform(1e-2f);
                CHECK_HIP(hipMemcpy(g_dev[w * K + k], g_host[w * K + k],
                                    (size_t)key_elems[k] * sizeof(float), hipMemcpyHostToDevice));
            }
        /* pushes in reverse worker order: the sum's order is the worker index */
        for (int w = N - 1; w >= 0; --w)
            for (int k = 0; k < K; ++k) CHECK_PHUB(phub_push(job, w, k, g_dev[w * K + k]));
        CHECK_PHUB(phub_step(job));
        CHECK_PHUB(phub_sync(job));
        if (oracle_step_f32(N, K, key_elems, (const float *const *)g_host, w_host, m_host, lr, mu,
                            wd, 1) != 0)
            return 1;
    }

    for (int k = 0; k < K; ++k) {
        const size_t bytes = (size_t)key_elems[k] * sizeof(float);
        const float *w_pull = NULL, *w_state = NULL, *m_state = NULL;
        CHECK_PHUB(phub_pull(job, k, &w_pull));
        CHECK_PHUB(phub_get_state(job, k, &w_state, &m_state));
        if (w_pull != w_state) {
            fprintf(stderr, "key %d: phub_pull and phub_get_state disagree\n", k);
            return 1;
        }
        if (!bytes) continue;
        float *w = malloc(bytes), *m = malloc(bytes);
        if (!w || !m) return 1;
        CHECK_HIP(hipMemcpy(w, w_pull, bytes, hipMemcpyDeviceToHost));
        CHECK_HIP(hipMemcpy(m, m_state, bytes, hipMemcpyDeviceToHost));
        if (memcmp(w, w_host[k], bytes) || memcmp(m, m_host[k], bytes)) {
            fprintf(stderr, "key %d (%lld elements): GPU state differs from the oracle\n", k,
                    (long long)key_elems[k]);
            return 1;
        }
        free(w);
        free(m);
    }
    /* a step without every push is refused and names what is missing */
    CHECK_PHUB(phub_push(job, 0, 0, g_dev[0]));
    if (phub_step(job) != PHUB_ENOTREADY || !strstr(phub_last_error(), "has not pushed")) {
        fprintf(stderr, "an incomplete step was not refused: %s\n", phub_last_error());
        return 1;
    }
    CHECK_PHUB(phub_destroy(job));
    for (int k = 0; k < K; ++k) {
        free(w_host[k]);
        free(m_host[k]);
        CHECK_HIP(hipFree(w0_dev[k]));
        for (int w = 0; w < N; ++w) {
            free(g_host[w * K + k]);
            CHECK_HIP(hipFree(g_dev[w * K + k]));
        }
    }
    CHECK_HIP(hipStreamDestroy(stream));
    printf("c api checks passed: %d workers, %d keys, %d steps, bit-exact against the oracle\n", N,
           K, STEPS);
    return 0;
}
