/*
 * Parameter-server side of Gorila -- plain fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY (like gorila_oracle.c): used by the tests and the
 * benchmark's CPU-baseline leg, never by the product path, and sharing no
 * code with the HIP library.
 *
 * What it computes (Nair et al. 2015):
 *  - Section 4 (parameter server) and Section 4.2 (stability): the server
 *    applies the gradients it receives to theta+ one at a time, each applied
 *    gradient being one update of the server; a gradient whose parameters
 *    are older than a threshold is discarded; the update rule is AdaGrad
 *    (Duchi, Hazan and Singer 2011, diagonal form):
 *        h <- h + g*g,   theta+ <- theta+ - lr * g / (eps + sqrt(h)).
 *  - Section 4.2: each learner keeps a running mean and standard deviation of
 *    its absolute DQN loss and discards a gradient whose absolute loss is
 *    above the mean plus k standard deviations.
 *
 * Readings (the paper states none of these values or forms):
 *  - Staleness: gradient g was computed from theta+ at server version
 *    version[g] (the number of updates applied when the learner copied it).
 *    Gradients are taken in index order; when gradient g's turn comes the
 *    server is at version V (earlier applied gradients of the same call
 *    included), and g is applied iff keep[g] and V - version[g] <= max_delay;
 *    each applied gradient increments V.
 *  - AdaGrad's eps is added to sqrt(h) (the delta of Duchi et al.).
 *  - Loss statistics per learner: (n, mean, var) of x = |loss|.  Before x is
 *    included, the gradient is discarded iff n >= max(warmup, 1), x > mean
 *    and (x - mean)^2 > k^2 var (that is, x > mean + k sd, without a square
 *    root).  Then x is included: with alpha > 0 as an exponentially weighted
 *    mean and variance, d = x - mean, mean += alpha d,
 *    var = (1 - alpha)(var + alpha d^2); with alpha = 0 as the cumulative
 *    mean and (population) variance, n' = n + 1, mean' = mean + d / n',
 *    var' = (n var + d (x - mean')) / n'.  The first loss sets mean = x,
 *    var = 0 in both modes.  Every loss is included, kept or not.
 */
#include <math.h>
#include <stdint.h>

#include "gorila_oracle.h"

int oracle_loss_filter(double* stats, const double* loss, int32_t groups, double alpha,
                       double k, int64_t warmup, uint8_t* keep_out) {
    if (!stats || !loss || !keep_out || groups < 0 || alpha < 0.0 || alpha > 1.0 || k < 0.0)
        return -1;
    for (int32_t g = 0; g < groups; ++g) {
        double* st = stats + 3 * (int64_t)g; /* n, mean, var */
        const double x = fabs(loss[g]);
        const double n = st[0], mean = st[1], var = st[2];
        int discard = 0;
        if (n >= 1.0 && n >= (double)warmup && x > mean) {
            const double d = x - mean;
            discard = d * d > (k * k) * var;
        }
        keep_out[g] = discard ? 0 : 1;
        if (n == 0.0) {
            st[1] = x;
            st[2] = 0.0;
        } else if (alpha > 0.0) {
            const double d = x - mean;
            st[1] = mean + alpha * d;
            st[2] = (1.0 - alpha) * (var + (alpha * d) * d);
        } else {
            const double n1 = n + 1.0;
            const double d = x - mean;
            const double mean1 = mean + d / n1;
            st[1] = mean1;
            st[2] = (n * var + d * (x - mean1)) / n1;
        }
        st[0] = n + 1.0;
    }
    return 0;
}

int oracle_ps_apply(double* theta, double* accum, int64_t n, const double* grads,
                    int32_t groups, const uint8_t* keep, const int64_t* version,
                    int64_t* ps_version, int64_t max_delay, double lr, double eps,
                    uint8_t* applied_out) {
    if (!theta || !accum || !version || !ps_version || !applied_out || n < 0 || groups < 0)
        return -1;
    if (!(eps > 0.0) || !(lr >= 0.0)) return -1; /* eps > 0 keeps 0 / 0 out of the update */
    if (groups > 0 && !grads) return -1;
    int64_t v = *ps_version;
    for (int32_t g = 0; g < groups; ++g) {
        const int ok = (!keep || keep[g]) && v - version[g] <= max_delay;
        applied_out[g] = ok ? 1 : 0;
        if (!ok) continue;
        const double* gr = grads + (int64_t)g * n;
        for (int64_t i = 0; i < n; ++i) {
            accum[i] += gr[i] * gr[i];
            theta[i] -= lr * gr[i] / (eps + sqrt(accum[i]));
        }
        ++v;
    }
    *ps_version = v;
    return 0;
}
