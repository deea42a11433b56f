/*
 * Gorila DQN learner step -- plain fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, by the package smoke check
 * and by the benchmark's CPU-baseline leg.  The product path never calls it.
 * It is written from the paper (Nair et al. 2015) as the plain definition of
 * what the learner step computes, in fp64, with no blocking or fusion, so it
 * can be checked against the paper by eye.  It shares no code with the HIP
 * library.
 *
 * Readings of the paper used here (the paper is silent or garbled on them):
 *  - Network (Section 5.1, experimental set-up): valid cross-correlations,
 *    OIHW weights, biases present, flatten of the last conv in (c, i, j)
 *    order, input bytes scaled by 1/255, ReLU'(0) = 0.
 *  - Loss (eq. (1), Algorithm 1): the target is y = r for a terminal next
 *    state, else y = r + gamma * max_a' Q(s', a'; theta-); the per-sample
 *    loss is the Huber function of delta = y - Q(s, a; theta) with threshold
 *    `clip` (0.5 delta^2 inside, clip*|delta| - 0.5 clip^2 outside), i.e.
 *    the squared error of eq. (1) with its derivative clipped to
 *    [-clip, clip]; clip = +inf gives eq. (1) with a factor 1/2.  The batch
 *    loss is the mean over the minibatch.
 *  - Gradient (eq. (2)): grads = d loss / d theta, which for |delta| <= clip
 *    is minus the minibatch mean of eq. (2)'s g.  No gradient flows into
 *    theta- (the target network is only ever copied).
 *  - epsilon-greedy (Algorithm 1): with probability eps a uniformly random
 *    action, else the lowest-index argmax of Q.  The two uniform draws per
 *    environment come from the SplitMix64 output function (Steele, Lea and
 *    Flood, OOPSLA 2014) evaluated at seed + (2e+1)*G and seed + (2e+2)*G,
 *    G = 0x9E3779B97F4A7C15, all mod 2^64.
 *  - Frame stacking (Section 5.1): the state is the four most recent frames,
 *    oldest in channel 0; a frame that lies before the start of the current
 *    episode is replaced by zeros.  The replay ring (Section 4, replay
 *    memory) has `capacity` slots, `head` is the physical slot of the oldest
 *    frame, and logical position k lives in slot (head + k) mod capacity.
 *    ep_start flags the first frame of an episode; logical 0 counts as one.
 *    A transition sampled at logical k is (stack(k), action[k], reward[k],
 *    stack(k+1)), and it is terminal iff k+1 starts a new episode.
 */
#include "gorila_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Topology and parameter layout                                              */
/* ------------------------------------------------------------------------ */

typedef struct {
    int h1, w1, h2, w2, h3, w3; /* spatial sizes after each convolution */
    int flat;                   /* c3 * h3 * w3 */
    int64_t off[11];            /* W1 b1 W2 b2 W3 b3 W4 b4 W5 b5 total */
} layout;

static int conv_out(int in, int k, int s) {
    if (k <= 0 || s <= 0 || in < k) return -1;
    return (in - k) / s + 1;
}

static int make_layout(const oracle_net* n, layout* L) {
    if (!n || n->in_c <= 0 || n->c1 <= 0 || n->c2 <= 0 || n->c3 <= 0 ||
        n->hidden <= 0 || n->n_actions <= 0)
        return -1;
    L->h1 = conv_out(n->in_h, n->k1, n->s1);
    L->w1 = conv_out(n->in_w, n->k1, n->s1);
    if (L->h1 < 0 || L->w1 < 0) return -1;
    L->h2 = conv_out(L->h1, n->k2, n->s2);
    L->w2 = conv_out(L->w1, n->k2, n->s2);
    if (L->h2 < 0 || L->w2 < 0) return -1;
    L->h3 = conv_out(L->h2, n->k3, n->s3);
    L->w3 = conv_out(L->w2, n->k3, n->s3);
    if (L->h3 < 0 || L->w3 < 0) return -1;
    L->flat = n->c3 * L->h3 * L->w3;
    int64_t sz[10] = {
        (int64_t)n->c1 * n->in_c * n->k1 * n->k1, n->c1,
        (int64_t)n->c2 * n->c1 * n->k2 * n->k2,   n->c2,
        (int64_t)n->c3 * n->c2 * n->k3 * n->k3,   n->c3,
        (int64_t)n->hidden * L->flat,             n->hidden,
        (int64_t)n->n_actions * n->hidden,        n->n_actions};
    L->off[0] = 0;
    for (int t = 0; t < 10; ++t) L->off[t + 1] = L->off[t] + sz[t];
    return 0;
}

int64_t oracle_param_count(const oracle_net* net) {
    layout L;
    if (make_layout(net, &L)) return -1;
    return L.off[10];
}

int oracle_param_offsets(const oracle_net* net, int64_t* off) {
    layout L;
    if (!off || make_layout(net, &L)) return -1;
    for (int t = 0; t < 11; ++t) off[t] = L.off[t];
    return 0;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int oracle_set_num_threads(int32_t n) {
    if (n < 1) return -1;
#ifdef _OPENMP
    omp_set_num_threads(n);
#endif
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Layers, written as their definitions                                      */
/* ------------------------------------------------------------------------ */

/* z[o][i][j] = b[o] + sum_{c,u,v} w[o][c][u][v] * in[c][s*i+u][s*j+v] */
static void conv_forward(const double* in, int C, int H, int W,
                         const double* w, const double* b, int O, int k, int s,
                         int Ho, int Wo, double* z) {
    for (int o = 0; o < O; ++o)
        for (int i = 0; i < Ho; ++i)
            for (int j = 0; j < Wo; ++j) {
                double acc = b[o];
                for (int c = 0; c < C; ++c)
                    for (int u = 0; u < k; ++u)
                        for (int v = 0; v < k; ++v)
                            acc += w[((o * C + c) * k + u) * k + v] *
                                   in[(c * H + s * i + u) * W + s * j + v];
                z[(o * Ho + i) * Wo + j] = acc;
            }
}

/* d_in[c][s*i+u][s*j+v] += w[o][c][u][v] * dz[o][i][j]  (d_in zeroed first) */
static void conv_backward_data(const double* dz, int O, int Ho, int Wo,
                               const double* w, int C, int k, int s, int H,
                               int W, double* d_in) {
    memset(d_in, 0, sizeof(double) * (size_t)C * H * W);
    for (int o = 0; o < O; ++o)
        for (int i = 0; i < Ho; ++i)
            for (int j = 0; j < Wo; ++j) {
                double g = dz[(o * Ho + i) * Wo + j];
                for (int c = 0; c < C; ++c)
                    for (int u = 0; u < k; ++u)
                        for (int v = 0; v < k; ++v)
                            d_in[(c * H + s * i + u) * W + s * j + v] +=
                                w[((o * C + c) * k + u) * k + v] * g;
            }
}

/* y[n] = b[n] + sum_k w[n][k] * x[k] */
static void linear_forward(const double* x, int K, const double* w,
                           const double* b, int N, double* y) {
    for (int n = 0; n < N; ++n) {
        double acc = b[n];
        for (int k = 0; k < K; ++k) acc += w[(int64_t)n * K + k] * x[k];
        y[n] = acc;
    }
}

/* Distance of a layer's pre-activations from the ReLU kink, relative to the
 * size of the terms summed into them: min over units of
 * |z| / (|b| + sum |w| |x|).  A finite-precision evaluation of z errs by a
 * small multiple of that denominator, so units with a small ratio are the ones
 * whose ReLU derivative another precision may decide differently.  A unit
 * whose terms are all zero is exactly zero in any precision and is skipped. */
static double conv_margin(const double* in, int C, int H, int W, const double* w,
                          const double* b, int O, int k, int s, int Ho, int Wo,
                          const double* z) {
    double m = INFINITY;
    for (int o = 0; o < O; ++o)
        for (int i = 0; i < Ho; ++i)
            for (int j = 0; j < Wo; ++j) {
                double scale = fabs(b[o]);
                for (int c = 0; c < C; ++c)
                    for (int u = 0; u < k; ++u)
                        for (int v = 0; v < k; ++v)
                            scale += fabs(w[((o * C + c) * k + u) * k + v]) *
                                     fabs(in[(c * H + s * i + u) * W + s * j + v]);
                if (scale > 0.0) m = fmin(m, fabs(z[(o * Ho + i) * Wo + j]) / scale);
            }
    return m;
}

static double linear_margin(const double* x, int K, const double* w, const double* b, int N,
                            const double* z) {
    double m = INFINITY;
    for (int n = 0; n < N; ++n) {
        double scale = fabs(b[n]);
        for (int k = 0; k < K; ++k) scale += fabs(w[(int64_t)n * K + k]) * fabs(x[k]);
        if (scale > 0.0) m = fmin(m, fabs(z[n]) / scale);
    }
    return m;
}

static void relu(const double* z, double* h, int64_t n) {
    for (int64_t t = 0; t < n; ++t) h[t] = z[t] > 0.0 ? z[t] : 0.0;
}

/* dz = dh * [z > 0]   (the derivative of ReLU at 0 is taken as 0) */
static void relu_backward(const double* dh, const double* z, double* dz,
                          int64_t n) {
    for (int64_t t = 0; t < n; ++t) dz[t] = z[t] > 0.0 ? dh[t] : 0.0;
}

/* Everything one forward + backward pass of one sample keeps. */
typedef struct {
    double *x, *z1, *h1, *z2, *h2, *z3, *h3, *z4, *h4, *q;
    double *dq, *dz4, *dz3, *dz2, *dz1;
} sample_state;

static int64_t sample_doubles(const oracle_net* n, const layout* L) {
    int64_t nx = (int64_t)n->in_c * n->in_h * n->in_w;
    int64_t n1 = (int64_t)n->c1 * L->h1 * L->w1;
    int64_t n2 = (int64_t)n->c2 * L->h2 * L->w2;
    int64_t n3 = L->flat;
    return nx + 3 * n1 + 3 * n2 + 3 * n3 + 3 * n->hidden + 2 * n->n_actions;
}

static void carve(const oracle_net* n, const layout* L, double* base,
                  sample_state* S) {
    int64_t nx = (int64_t)n->in_c * n->in_h * n->in_w;
    int64_t n1 = (int64_t)n->c1 * L->h1 * L->w1;
    int64_t n2 = (int64_t)n->c2 * L->h2 * L->w2;
    int64_t n3 = L->flat;
    double* p = base;
    S->x = p;   p += nx;
    S->z1 = p;  p += n1;
    S->h1 = p;  p += n1;
    S->dz1 = p; p += n1;
    S->z2 = p;  p += n2;
    S->h2 = p;  p += n2;
    S->dz2 = p; p += n2;
    S->z3 = p;  p += n3;
    S->h3 = p;  p += n3;
    S->dz3 = p; p += n3;
    S->z4 = p;  p += n->hidden;
    S->h4 = p;  p += n->hidden;
    S->dz4 = p; p += n->hidden;
    S->q = p;   p += n->n_actions;
    S->dq = p;  p += n->n_actions;
}

/* Q-network forward pass of one state (Section 5.1). */
static void forward(const oracle_net* n, const layout* L, const double* th,
                    const uint8_t* state, sample_state* S) {
    const int64_t* o = L->off;
    int64_t nx = (int64_t)n->in_c * n->in_h * n->in_w;
    for (int64_t t = 0; t < nx; ++t) S->x[t] = (double)state[t] / 255.0;
    conv_forward(S->x, n->in_c, n->in_h, n->in_w, th + o[0], th + o[1], n->c1,
                 n->k1, n->s1, L->h1, L->w1, S->z1);
    relu(S->z1, S->h1, (int64_t)n->c1 * L->h1 * L->w1);
    conv_forward(S->h1, n->c1, L->h1, L->w1, th + o[2], th + o[3], n->c2,
                 n->k2, n->s2, L->h2, L->w2, S->z2);
    relu(S->z2, S->h2, (int64_t)n->c2 * L->h2 * L->w2);
    conv_forward(S->h2, n->c2, L->h2, L->w2, th + o[4], th + o[5], n->c3,
                 n->k3, n->s3, L->h3, L->w3, S->z3);
    relu(S->z3, S->h3, L->flat);
    /* h3 in (c, i, j) order is already the flattened input of layer 4 */
    linear_forward(S->h3, L->flat, th + o[6], th + o[7], n->hidden, S->z4);
    relu(S->z4, S->h4, n->hidden);
    linear_forward(S->h4, n->hidden, th + o[8], th + o[9], n->n_actions, S->q);
}

/* Smallest relative kink margin over the four hidden layers of one sample. */
static double kink_margin(const oracle_net* n, const layout* L, const double* th,
                          const sample_state* S) {
    const int64_t* o = L->off;
    double m = conv_margin(S->x, n->in_c, n->in_h, n->in_w, th + o[0], th + o[1], n->c1,
                           n->k1, n->s1, L->h1, L->w1, S->z1);
    m = fmin(m, conv_margin(S->h1, n->c1, L->h1, L->w1, th + o[2], th + o[3], n->c2, n->k2,
                            n->s2, L->h2, L->w2, S->z2));
    m = fmin(m, conv_margin(S->h2, n->c2, L->h2, L->w2, th + o[4], th + o[5], n->c3, n->k3,
                            n->s3, L->h3, L->w3, S->z3));
    m = fmin(m, linear_margin(S->h3, L->flat, th + o[6], th + o[7], n->hidden, S->z4));
    return m;
}

/* Back-propagate dq through one sample, leaving dz4..dz1 (data gradients
 * of the pre-activations).  Weight gradients are summed afterwards. */
static void backward_data(const oracle_net* n, const layout* L,
                          const double* th, sample_state* S, double* scratch) {
    const int64_t* o = L->off;
    /* dh4[k] = sum_a W5[a][k] dq[a] */
    for (int k = 0; k < n->hidden; ++k) {
        double acc = 0.0;
        for (int a = 0; a < n->n_actions; ++a)
            acc += th[o[8] + (int64_t)a * n->hidden + k] * S->dq[a];
        scratch[k] = acc;
    }
    relu_backward(scratch, S->z4, S->dz4, n->hidden);
    /* df[k] = sum_j W4[j][k] dz4[j] */
    for (int k = 0; k < L->flat; ++k) {
        double acc = 0.0;
        for (int j = 0; j < n->hidden; ++j)
            acc += th[o[6] + (int64_t)j * L->flat + k] * S->dz4[j];
        scratch[k] = acc;
    }
    relu_backward(scratch, S->z3, S->dz3, L->flat);
    conv_backward_data(S->dz3, n->c3, L->h3, L->w3, th + o[4], n->c2, n->k3,
                       n->s3, L->h2, L->w2, scratch);
    relu_backward(scratch, S->z2, S->dz2, (int64_t)n->c2 * L->h2 * L->w2);
    conv_backward_data(S->dz2, n->c2, L->h2, L->w2, th + o[2], n->c1, n->k2,
                       n->s2, L->h1, L->w1, scratch);
    relu_backward(scratch, S->z1, S->dz1, (int64_t)n->c1 * L->h1 * L->w1);
}

/* dW[o][c][u][v] = sum_b sum_{i,j} dz_b[o][i][j] * in_b[c][s*i+u][s*j+v],
 * db[o] = sum_b sum_{i,j} dz_b[o][i][j].  in_sel picks the layer input. */
static void conv_weight_grad(sample_state* S, int B, int which,
                             const oracle_net* n, const layout* L, double* gw,
                             double* gb) {
    int O, C, k, s, H, W, Ho, Wo;
    if (which == 1) {
        O = n->c1; C = n->in_c; k = n->k1; s = n->s1;
        H = n->in_h; W = n->in_w; Ho = L->h1; Wo = L->w1;
    } else if (which == 2) {
        O = n->c2; C = n->c1; k = n->k2; s = n->s2;
        H = L->h1; W = L->w1; Ho = L->h2; Wo = L->w2;
    } else {
        O = n->c3; C = n->c2; k = n->k3; s = n->s3;
        H = L->h2; W = L->w2; Ho = L->h3; Wo = L->w3;
    }
#pragma omp parallel for schedule(static)
    for (int o = 0; o < O; ++o) {
        double bsum = 0.0;
        for (int b = 0; b < B; ++b) {
            const double* dz = which == 1 ? S[b].dz1 : which == 2 ? S[b].dz2 : S[b].dz3;
            for (int t = 0; t < Ho * Wo; ++t) bsum += dz[o * Ho * Wo + t];
        }
        gb[o] = bsum;
        for (int c = 0; c < C; ++c)
            for (int u = 0; u < k; ++u)
                for (int v = 0; v < k; ++v) {
                    double acc = 0.0;
                    for (int b = 0; b < B; ++b) {
                        const double* dz = which == 1 ? S[b].dz1
                                         : which == 2 ? S[b].dz2 : S[b].dz3;
                        const double* in = which == 1 ? S[b].x
                                         : which == 2 ? S[b].h1 : S[b].h2;
                        for (int i = 0; i < Ho; ++i)
                            for (int j = 0; j < Wo; ++j)
                                acc += dz[(o * Ho + i) * Wo + j] *
                                       in[(c * H + s * i + u) * W + s * j + v];
                    }
                    gw[((o * C + c) * k + u) * k + v] = acc;
                }
    }
}

/* dW[j][k] = sum_b dz_b[j] * in_b[k],  db[j] = sum_b dz_b[j] */
static void linear_weight_grad(sample_state* S, int B, int which, int N, int K,
                               double* gw, double* gb) {
#pragma omp parallel for schedule(static)
    for (int j = 0; j < N; ++j) {
        double bsum = 0.0;
        for (int b = 0; b < B; ++b) bsum += which == 4 ? S[b].dz4[j] : S[b].dq[j];
        gb[j] = bsum;
        for (int k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int b = 0; b < B; ++b) {
                double d = which == 4 ? S[b].dz4[j] : S[b].dq[j];
                double x = which == 4 ? S[b].h3[k] : S[b].h4[k];
                acc += d * x;
            }
            gw[(int64_t)j * K + k] = acc;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Entry points                                                              */
/* ------------------------------------------------------------------------ */

int oracle_q_forward(const oracle_net* net, const double* theta,
                     const uint8_t* states, int32_t n, double* q_out) {
    layout L;
    if (make_layout(net, &L) || !theta || n < 0 || (n > 0 && (!states || !q_out)))
        return -1;
    int64_t per = sample_doubles(net, &L);
    int64_t nx = (int64_t)net->in_c * net->in_h * net->in_w;
    int nt = oracle_num_threads();
    double* buf = (double*)malloc(sizeof(double) * (size_t)(per * nt));
    if (!buf) return -2;
#pragma omp parallel for schedule(dynamic)
    for (int b = 0; b < n; ++b) {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        sample_state S;
        carve(net, &L, buf + (int64_t)tid * per, &S);
        forward(net, &L, theta, states + (int64_t)b * nx, &S);
        for (int a = 0; a < net->n_actions; ++a)
            q_out[(int64_t)b * net->n_actions + a] = S.q[a];
    }
    free(buf);
    return 0;
}

/* SplitMix64 output function (Steele, Lea and Flood 2014), mod 2^64. */
static uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

int oracle_act(const oracle_net* net, const double* theta,
               const uint8_t* states, int32_t n, double eps, uint64_t seed,
               int32_t* actions_out, double* q_out) {
    layout L;
    if (make_layout(net, &L) || !(eps >= 0.0 && eps <= 1.0) || n < 0 ||
        (n > 0 && !actions_out))
        return -1;
    int A = net->n_actions;
    double* q = (double*)malloc(sizeof(double) * (size_t)((int64_t)n * A + 1));
    if (!q) return -2;
    int rc = oracle_q_forward(net, theta, states, n, q);
    if (rc) { free(q); return rc; }
    const uint64_t G = 0x9E3779B97F4A7C15ULL;
    /* explore iff a uniform 53-bit integer is below floor(eps * 2^53) */
    uint64_t threshold = (uint64_t)floor(eps * 9007199254740992.0);
    for (int e = 0; e < n; ++e) {
        uint64_t u = splitmix64_mix(seed + (2 * (uint64_t)e + 1) * G);
        uint64_t v = splitmix64_mix(seed + (2 * (uint64_t)e + 2) * G);
        const double* qe = q + (int64_t)e * A;
        int act;
        if ((u >> 11) < threshold) {
            act = (int)(((v >> 32) * (uint64_t)A) >> 32); /* uniform over A */
        } else {
            act = 0; /* lowest index among the maxima */
            for (int a = 1; a < A; ++a)
                if (qe[a] > qe[act]) act = a;
        }
        actions_out[e] = act;
    }
    if (q_out) memcpy(q_out, q, sizeof(double) * (size_t)((int64_t)n * A));
    free(q);
    return 0;
}

int oracle_learner_step(const oracle_net* net, const double* theta,
                        const double* theta_target, const uint8_t* s,
                        const uint8_t* s2, const int32_t* a, const double* r,
                        const uint8_t* term, int32_t B, double gamma,
                        double clip, double* grads_out, double* loss_out,
                        double* q_out, double* q2_out, double* margin_out,
                        double* td_out) {
    layout L;
    if (make_layout(net, &L) || !theta || !theta_target || !s || !s2 || !a ||
        !r || !term || B <= 0 || !grads_out || !loss_out || !(clip > 0.0))
        return -1;
    const int A = net->n_actions;
    for (int b = 0; b < B; ++b)
        if (a[b] < 0 || a[b] >= A) return -1;

    int64_t per = sample_doubles(net, &L);
    int64_t nx = (int64_t)net->in_c * net->in_h * net->in_w;
    int64_t scratch_n = (int64_t)net->c1 * L.h1 * L.w1;
    if (L.flat > scratch_n) scratch_n = L.flat;
    if (net->hidden > scratch_n) scratch_n = net->hidden;
    if ((int64_t)net->c2 * L.h2 * L.w2 > scratch_n) scratch_n = (int64_t)net->c2 * L.h2 * L.w2;
    int nt = oracle_num_threads();

    double* buf = (double*)malloc(sizeof(double) * (size_t)(per * B));
    double* tbuf = (double*)malloc(sizeof(double) * (size_t)((per + scratch_n) * nt));
    double* ell = (double*)malloc(sizeof(double) * (size_t)B);
    sample_state* S = (sample_state*)malloc(sizeof(sample_state) * (size_t)B);
    if (!buf || !tbuf || !ell || !S) {
        free(buf); free(tbuf); free(ell); free(S);
        return -2;
    }

    /* Per sample: online forward, target forward, TD target and error,
     * Huber loss, dLoss/dQ and the data gradients. */
#pragma omp parallel for schedule(dynamic)
    for (int b = 0; b < B; ++b) {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        sample_state T;
        double* tb = tbuf + (int64_t)tid * (per + scratch_n);
        carve(net, &L, tb, &T);
        double* scratch = tb + per;

        carve(net, &L, buf + (int64_t)b * per, &S[b]);
        forward(net, &L, theta, s + (int64_t)b * nx, &S[b]);
        if (margin_out) margin_out[b] = kink_margin(net, &L, theta, &S[b]);
        forward(net, &L, theta_target, s2 + (int64_t)b * nx, &T);

        double m = T.q[0]; /* max_a' Q(s', a'; theta-) */
        for (int k = 1; k < A; ++k)
            if (T.q[k] > m) m = T.q[k];
        double y = term[b] ? r[b] : r[b] + gamma * m; /* Algorithm 1 */
        double delta = y - S[b].q[a[b]];
        double ad = fabs(delta);
        ell[b] = ad <= clip ? 0.5 * delta * delta : clip * ad - 0.5 * clip * clip;
        double g = delta > clip ? clip : (delta < -clip ? -clip : delta);
        for (int k = 0; k < A; ++k) S[b].dq[k] = 0.0;
        /* d ell / d Q(s,a) = -clamp(delta), and the batch loss is a mean */
        S[b].dq[a[b]] = -g / (double)B;
        backward_data(net, &L, theta, &S[b], scratch);

        if (q_out)
            for (int k = 0; k < A; ++k) q_out[(int64_t)b * A + k] = S[b].q[k];
        if (q2_out)
            for (int k = 0; k < A; ++k) q2_out[(int64_t)b * A + k] = T.q[k];
        if (td_out) {
            td_out[(int64_t)b * 4 + 0] = m;
            td_out[(int64_t)b * 4 + 1] = y;
            td_out[(int64_t)b * 4 + 2] = delta;
            td_out[(int64_t)b * 4 + 3] = ell[b];
        }
    }

    double loss = 0.0;
    for (int b = 0; b < B; ++b) loss += ell[b];
    *loss_out = loss / (double)B;

    const int64_t* o = L.off;
    conv_weight_grad(S, B, 1, net, &L, grads_out + o[0], grads_out + o[1]);
    conv_weight_grad(S, B, 2, net, &L, grads_out + o[2], grads_out + o[3]);
    conv_weight_grad(S, B, 3, net, &L, grads_out + o[4], grads_out + o[5]);
    linear_weight_grad(S, B, 4, net->hidden, L.flat, grads_out + o[6], grads_out + o[7]);
    linear_weight_grad(S, B, 5, A, net->hidden, grads_out + o[8], grads_out + o[9]);

    free(buf); free(tbuf); free(ell); free(S);
    return 0;
}

int oracle_gather(const uint8_t* frames, const uint8_t* ep_start,
                  const int32_t* action, const float* reward,
                  int64_t capacity, int64_t head, int32_t hist,
                  int64_t frame_bytes, const int64_t* idx, int32_t n,
                  uint8_t* s_out, uint8_t* s2_out, int64_t* frame_map_out,
                  int32_t* a_out, float* r_out, uint8_t* term_out) {
    if (!frames || !ep_start || !action || !reward || capacity < 2 ||
        head < 0 || head >= capacity || hist <= 0 || frame_bytes <= 0 || n < 0)
        return -1;
    for (int t = 0; t < n; ++t)
        if (idx[t] < 0 || idx[t] > capacity - 2) return -1;
    for (int t = 0; t < n; ++t) {
        for (int which = 0; which < 2; ++which) {
            int64_t k = idx[t] + which; /* s = stack(k), s' = stack(k+1) */
            /* e(k): the latest episode start at or before k (logical 0 is one) */
            int64_t e = k;
            while (e > 0 && !ep_start[(head + e) % capacity]) --e;
            uint8_t* dst = (which == 0 ? s_out : s2_out) + (int64_t)t * hist * frame_bytes;
            for (int j = 0; j < hist; ++j) {
                int64_t l = k - (hist - 1) + j; /* channel j holds frame l */
                int64_t slot = -1;
                if (l >= e) {
                    slot = (head + l) % capacity;
                    memcpy(dst + (int64_t)j * frame_bytes, frames + slot * frame_bytes,
                           (size_t)frame_bytes);
                } else {
                    memset(dst + (int64_t)j * frame_bytes, 0, (size_t)frame_bytes);
                }
                if (frame_map_out)
                    frame_map_out[((int64_t)t * 2 + which) * hist + j] = slot;
            }
        }
        int64_t p = (head + idx[t]) % capacity;
        int64_t p1 = (head + idx[t] + 1) % capacity;
        a_out[t] = action[p];
        r_out[t] = reward[p];
        term_out[t] = ep_start[p1] ? 1 : 0;
    }
    return 0;
}
