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
