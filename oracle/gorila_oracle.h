/*
 * Gorila DQN learner step -- plain fp64 CPU oracle (declarations).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link
 * or call this code: only the tests, the package smoke check and the CPU
 * baseline leg of the benchmark use it.  It shares no code with the HIP
 * library (this header is the oracle's own, written independently of
 * include/gorila.h).
 *
 * What it computes (Nair et al. 2015, "Massively Parallel Methods for Deep
 * Reinforcement Learning"):
 *   - the Q-network of the experimental set-up section (three convolutions,
 *     a 512-unit fully connected layer, a linear action head, ReLU after
 *     every hidden layer), here with a configurable topology so that tiny
 *     networks can be finite-differenced;
 *   - the DQN loss of eq. (1) and its gradient, eq. (2), with the terminal
 *     case of Algorithm 1 and a Huber/clipped TD error (clip = +inf gives
 *     eq. (1) exactly);
 *   - the epsilon-greedy behaviour policy of Algorithm 1;
 *   - frame stacking of the four most recent frames out of a replay ring.
 *
 * All arithmetic is IEEE fp64.  Every entry point returns 0 on success and
 * a negative value on a bad argument (nothing is written in that case).
 */
#ifndef GORILA_ORACLE_H
#define GORILA_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Network topology.  Input is in_c x in_h x in_w uint8, scaled by 1/255.
 * Layer l is a valid (unpadded) cross-correlation with c_l filters of size
 * c_{l-1} x k_l x k_l and stride s_l, followed by ReLU.  Then a ReLU fully
 * connected layer of `hidden` units and a linear layer of n_actions units.
 * The Atari network is {4,84,84, 32,8,4, 64,4,2, 64,3,1, 512, A}. */
typedef struct {
    int32_t in_c, in_h, in_w;
    int32_t c1, k1, s1;
    int32_t c2, k2, s2;
    int32_t c3, k3, s3;
    int32_t hidden;
    int32_t n_actions;
} oracle_net;

/* Number of parameters.  The flat layout is, in this order, W1 [c1,in_c,k1,k1],
 * b1 [c1], W2 [c2,c1,k2,k2], b2, W3 [c3,c2,k3,k3], b3, W4 [hidden, c3*h3*w3],
 * b4 [hidden], W5 [A, hidden], b5 [A]; the flatten of conv3's output is
 * channel-major (c, i, j).  Returns -1 for an invalid topology. */
int64_t oracle_param_count(const oracle_net* net);

/* Offsets of the ten tensors inside the flat vector; off has 11 entries
 * (the 11th is the total). */
int oracle_param_offsets(const oracle_net* net, int64_t* off);

/* Threads the OpenMP loops use, and a way to change it (n >= 1). */
int oracle_num_threads(void);
int oracle_set_num_threads(int32_t n);

/* Q(s, .; theta) for n states [n, in_c, in_h, in_w] -> q_out [n, A]. */
int oracle_q_forward(const oracle_net* net, const double* theta,
                     const uint8_t* states, int32_t n, double* q_out);

/* epsilon-greedy actions (Algorithm 1) with the SplitMix64 draws described
 * in the source; q_out may be NULL. */
int oracle_act(const oracle_net* net, const double* theta,
               const uint8_t* states, int32_t n, double eps, uint64_t seed,
               int32_t* actions_out, double* q_out);

/* One learner step on B stacked transitions (s, a, r, s', terminal).
 * grads_out [P] = d loss / d theta, loss_out [1] = mean Huber loss.
 * q_out / q2_out [B, A] (may be NULL) receive Q(s;theta), Q(s';theta-).
 * margin_out [B] (may be NULL) receives each sample's smallest ReLU kink
 * margin over the online network: min |z| / (|b| + sum |w||x|) over every
 * hidden pre-activation z (units whose terms are all zero are skipped).
 * td_out [B, 4] (may be NULL) receives, per sample, max_a' Q(s', a'; theta-),
 * the TD target y, the TD error delta = y - Q(s, a; theta) and its Huber
 * loss (Algorithm 1, eq. (1)). */
int oracle_learner_step(const oracle_net* net, const double* theta,
                        const double* theta_target, const uint8_t* s,
                        const uint8_t* s2, const int32_t* a, const double* r,
                        const uint8_t* term, int32_t B, double gamma,
                        double clip, double* grads_out, double* loss_out,
                        double* q_out, double* q2_out, double* margin_out,
                        double* td_out);

/* Replay gather: for logical positions idx[n] build s = stack(k) and
 * s' = stack(k+1) (each hist frames of frame_bytes bytes, oldest first),
 * the frame map [n, 2, hist] (physical slot, or -1 where zero-filled),
 * a = action[p(k)], r = reward[p(k)], term = ep_start[p(k+1)]. */
int oracle_gather(const uint8_t* frames, const uint8_t* ep_start,
                  const int32_t* action, const float* reward,
                  int64_t capacity, int64_t head, int32_t hist,
                  int64_t frame_bytes, const int64_t* idx, int32_t n,
                  uint8_t* s_out, uint8_t* s2_out, int64_t* frame_map_out,
                  int32_t* a_out, float* r_out, uint8_t* term_out);

/* ---- Actor side (actor_oracle.c; Algorithm 1, Section 4, Section 5.1) ---- */

/* Store m experience records into a replay ring (Algorithm 1 "store the
 * transition in D"; Section 4 replay memory): record j (frame of frame_bytes
 * bytes, episode-start flag, the action taken at that frame and the reward
 * that followed) goes to logical position size + j, i.e. physical slot
 * (head + size + j) mod capacity; when the ring is full the oldest record is
 * overwritten and head advances.  *head and *size are updated.  m <= capacity. */
int oracle_replay_insert(uint8_t* frames, uint8_t* ep_start, int32_t* action, float* reward,
                         int64_t capacity, int64_t frame_bytes, int64_t* head, int64_t* size,
                         const uint8_t* frames_in, const uint8_t* ep_start_in,
                         const int32_t* action_in, const float* reward_in, int32_t m);

/* Parameter pull / target sync (Algorithm 1: learners and actors update theta
 * from theta+, and every N global updates the learner syncs theta- with
 * theta+; Section 5.1: N = 60K).  For each of `copies` destinations
 * dst[c] ([copies][n], fp32 when to_bf16 == 0, else bf16 bit patterns
 * rounded to nearest even from the fp32 value) with version dst_version[c]:
 * when period == 0, or ps_version / period > dst_version[c] / period
 * (integer division: a multiple of period was crossed), dst[c] = src and
 * dst_version[c] = ps_version; otherwise both are left alone.
 * synced_out[c] = 1 iff copied. */
int oracle_params_sync(const float* src, void* dst, int64_t n, int32_t copies, int32_t to_bf16,
                       int64_t ps_version, int64_t* dst_version, int64_t period,
                       uint8_t* synced_out);

/* bf16 bit pattern of an fp32 value, round to nearest even (NaN stays NaN). */
uint16_t oracle_f32_to_bf16(float x);

/* epsilon of the behaviour policy after `update` global updates (Section 5.1:
 * annealed linearly from eps_start to eps_end over the first anneal_updates
 * updates, constant after). */
double oracle_epsilon(int64_t update, double eps_start, double eps_end, int64_t anneal_updates);

/* ---- Parameter-server side (ps_oracle.c; Section 4 and Section 4.2) ---- */

/* Loss-statistics gradient filter for `groups` learners: stats [groups][3]
 * = (n, mean, var) of each learner's absolute loss, updated in place with
 * loss[g]; keep_out[g] = 0 iff the gradient of that loss is discarded
 * (n >= max(warmup, 1) and |loss| > mean + k sd before the update).  alpha > 0:
 * exponentially weighted statistics; alpha = 0: cumulative. */
int oracle_loss_filter(double* stats, const double* loss, int32_t groups, double alpha,
                       double k, int64_t warmup, uint8_t* keep_out);

/* Apply `groups` gradients grads [groups][n] to theta [n] with AdaGrad
 * (accumulator accum [n]) in index order; gradient g is applied iff keep[g]
 * (keep may be NULL) and *ps_version - version[g] <= max_delay at its turn;
 * every applied gradient increments *ps_version.  applied_out [groups]. */
int oracle_ps_apply(double* theta, double* accum, int64_t n, const double* grads,
                    int32_t groups, const uint8_t* keep, const int64_t* version,
                    int64_t* ps_version, int64_t max_delay, double lr, double eps,
                    uint8_t* applied_out);

#ifdef __cplusplus
}
#endif
#endif
