/*
 * Oracle for the PHub parameter-exchange step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this.  It is a plain, slow,
 * single-threaded CPU definition of what the exchange step computes and
 * shares no code, header or table with the GPU library.
 *
 * What the step computes (paper, section 3.2.2 "Gradient Aggregation and
 * Optimization", and section 4.2, which names the optimizer):
 *   - aggregation is an elementwise sum, over workers, of the gradients
 *     pushed for one key;
 *   - optimization is an elementwise SGD update with Nesterov's accelerated
 *     gradient, applied to the key's model values with the aggregated
 *     gradient.
 * Chunking a key changes nothing in the result (section 4.2 states that the
 * changes did not alter the computation), so the oracle walks each key as a
 * whole.
 *
 * Readings where the paper is silent (every one is listed with its reason in
 * the design notes):
 *   - the aggregate is the sum, not the mean (section 3.2.2 says aggregation
 *     sums); a caller who wants the mean scales lr by 1/N;
 *   - the sum is a left fold in fp32 in ascending worker index, so that it
 *     does not depend on arrival order;
 *   - weight decay is coupled L2: it is added to the aggregated gradient
 *     before momentum, for every key;
 *   - momentum uses no dampening and starts from zero; Nesterov uses the
 *     reformulated look-ahead form in which the step direction is
 *     d + mu * m' (the form of common framework optimizers);
 *   - each of the four update formulas is evaluated as one correctly
 *     rounded fused multiply-add, and the sum as plain fp32 additions
 *     (round to nearest even, no flush of subnormals);
 *   - single precision throughout, as the paper's aggregation is fp32
 *     (section 3.2.2 counts single-precision adds).
 *
 * Per element, with s the sum, w the weight, m the momentum:
 *     d  = wd * w + s              (fused)
 *     m' = mu * m + d              (fused)
 *     u  = nesterov ? mu * m' + d  (fused)
 *                   : m'
 *     w' = -lr * u + w             (fused)
 *
 * The paper's optimizers are pluggable (section 3.2.2: any optimizer that
 * complies with the API can be used at run time).  Two more are defined
 * below, with the same aggregation: plain SGD (no state) and Adam (two
 * moment arrays).
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fPIC -shared -lm
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL -1

/*
 * One exchange step in fp32.
 *   num_workers  N >= 1
 *   num_keys     K >= 1
 *   key_elems    K element counts (each >= 0)
 *   grads        N*K pointers; grads[w*K + k] holds key k's gradient from worker w
 *   weights      K pointers to the master weights of each key (updated in place)
 *   moms         K pointers to the momentum of each key (updated in place)
 * Returns 0, or -1 on a bad argument (nothing is written then).
 */
int oracle_step_f32(int num_workers, int num_keys, const int64_t *key_elems,
                    const float *const *grads, float *const *weights,
                    float *const *moms, float lr, float mu, float wd,
                    int nesterov)
{
    if (num_workers < 1 || num_keys < 1 || !key_elems || !grads || !weights || !moms)
        return ORACLE_EINVAL;
    for (int k = 0; k < num_keys; ++k)
        if (key_elems[k] < 0)
            return ORACLE_EINVAL;

    for (int k = 0; k < num_keys; ++k) {
        float *w = weights[k];
        float *m = moms[k];
        for (int64_t i = 0; i < key_elems[k]; ++i) {
            /* aggregation: worker 0 first, then each next worker in turn */
            float s = grads[0 * (size_t)num_keys + k][i];
            for (int j = 1; j < num_workers; ++j)
                s = s + grads[(size_t)j * num_keys + k][i];

            /* optimization of the same element */
            float d = fmaf(wd, w[i], s);
            float m1 = fmaf(mu, m[i], d);
            float u = nesterov ? fmaf(mu, m1, d) : m1;
            w[i] = fmaf(-lr, u, w[i]);
            m[i] = m1;
        }
    }
    return ORACLE_OK;
}

/*
 * The same step carried out in double precision, on double arrays.  It is
 * the reference against which the fp32 step's rounding error is bounded.
 */
int oracle_step_f64(int num_workers, int num_keys, const int64_t *key_elems,
                    const double *const *grads, double *const *weights,
                    double *const *moms, double lr, double mu, double wd,
                    int nesterov)
{
    if (num_workers < 1 || num_keys < 1 || !key_elems || !grads || !weights || !moms)
        return ORACLE_EINVAL;
    for (int k = 0; k < num_keys; ++k)
        if (key_elems[k] < 0)
            return ORACLE_EINVAL;

    for (int k = 0; k < num_keys; ++k) {
        double *w = weights[k];
        double *m = moms[k];
        for (int64_t i = 0; i < key_elems[k]; ++i) {
            double s = grads[0 * (size_t)num_keys + k][i];
            for (int j = 1; j < num_workers; ++j)
                s = s + grads[(size_t)j * num_keys + k][i];
            double d = fma(wd, w[i], s);
            double m1 = fma(mu, m[i], d);
            double u = nesterov ? fma(mu, m1, d) : m1;
            w[i] = fma(-lr, u, w[i]);
            m[i] = m1;
        }
    }
    return ORACLE_OK;
}

/*
 * Plain SGD with coupled L2 weight decay, no state, in fp32 (a pluggable
 * optimizer, section 3.2.2).  Per element, with s the sum:
 *     d  = wd * w + s      (fused)
 *     w' = -lr * d + w     (fused)
 */
int oracle_step_sgd_f32(int num_workers, int num_keys, const int64_t *key_elems,
                        const float *const *grads, float *const *weights, float lr, float wd)
{
    if (num_workers < 1 || num_keys < 1 || !key_elems || !grads || !weights)
        return ORACLE_EINVAL;
    for (int k = 0; k < num_keys; ++k)
        if (key_elems[k] < 0)
            return ORACLE_EINVAL;

    for (int k = 0; k < num_keys; ++k) {
        float *w = weights[k];
        for (int64_t i = 0; i < key_elems[k]; ++i) {
            float s = grads[0 * (size_t)num_keys + k][i];
            for (int j = 1; j < num_workers; ++j)
                s = s + grads[(size_t)j * num_keys + k][i];
            float d = fmaf(wd, w[i], s);
            w[i] = fmaf(-lr, d, w[i]);
        }
    }
    return ORACLE_OK;
}

/*
 * Adam (Kingma and Ba) with coupled L2 weight decay and bias correction, in
 * fp32 (a pluggable optimizer, section 3.2.2).  `step` is the number of
 * this step, counted from 1 for each job.  Four scalars are derived from
 * the fp32 hyperparameters once per step, in double, each rounded once to
 * fp32:
 *     c1 = 1 - b1,  c2 = 1 - b2,
 *     k1 = lr / (1 - b1^step),  k2 = 1 / (1 - b2^step).
 * Per element, with s the sum, w the weight, m and v the two moments (zero
 * at the start); every operation is rounded once, and the three marked ones
 * are fused multiply-adds:
 *     d   = wd * w + s               (fused)
 *     m'  = b1 * m + (c1 * d)        (fused)
 *     v'  = b2 * v + (c2 * (d * d))  (fused)
 *     den = sqrt(v' * k2) + eps
 *     w'  = w - (k1 * m') / den
 * (k1 * m' is lr times the bias-corrected first moment; v' * k2 is the
 * bias-corrected second moment.)
 */
static void adam_scalars(float lr, float b1, float b2, int64_t step, float *c1, float *c2,
                         float *k1, float *k2)
{
    *c1 = (float)(1.0 - (double)b1);
    *c2 = (float)(1.0 - (double)b2);
    *k1 = (float)((double)lr / (1.0 - pow((double)b1, (double)step)));
    *k2 = (float)(1.0 / (1.0 - pow((double)b2, (double)step)));
}

int oracle_step_adam_f32(int num_workers, int num_keys, const int64_t *key_elems,
                         const float *const *grads, float *const *weights,
                         float *const *m1s, float *const *m2s, float lr, float b1, float b2,
                         float eps, float wd, int64_t step)
{
    if (num_workers < 1 || num_keys < 1 || !key_elems || !grads || !weights || !m1s || !m2s ||
        step < 1 || !(b1 >= 0.0f && b1 < 1.0f) || !(b2 >= 0.0f && b2 < 1.0f))
        return ORACLE_EINVAL;
    for (int k = 0; k < num_keys; ++k)
        if (key_elems[k] < 0)
            return ORACLE_EINVAL;
    float c1, c2, k1, k2;
    adam_scalars(lr, b1, b2, step, &c1, &c2, &k1, &k2);

    for (int k = 0; k < num_keys; ++k) {
        float *w = weights[k];
        float *m = m1s[k];
        float *v = m2s[k];
        for (int64_t i = 0; i < key_elems[k]; ++i) {
            float s = grads[0 * (size_t)num_keys + k][i];
            for (int j = 1; j < num_workers; ++j)
                s = s + grads[(size_t)j * num_keys + k][i];
            float d = fmaf(wd, w[i], s);
            float mn = fmaf(b1, m[i], c1 * d);
            float dd = d * d;
            float vn = fmaf(b2, v[i], c2 * dd);
            float den = sqrtf(vn * k2) + eps;
            float q = (k1 * mn) / den;
            w[i] = w[i] - q;
            m[i] = mn;
            v[i] = vn;
        }
    }
    return ORACLE_OK;
}
