/*
 * libgorila -- the Gorila DQN learner step and actor inference on one MI355X.
 *
 * Method: Nair et al. 2015, "Massively Parallel Methods for Deep
 * Reinforcement Learning".  The learner's job (Section 4, Learners;
 * Algorithm 1) is: sample a minibatch of transitions (s, a, r, s') from
 * replay memory, form the target y = r for terminal s' and
 * y = r + gamma * max_a' Q(s', a'; theta-) otherwise, take the squared TD
 * error of eq. (1) and compute its gradient, eq. (2), with respect to theta.
 * Actors (Section 4, Actors; Algorithm 1) choose epsilon-greedy actions on
 * Q(s, a; theta).  The Q-network is the one of Section 5.1.
 *
 * Conventions for every call below:
 *  - All array arguments are DEVICE pointers owned by the caller (normally
 *    torch tensors), C-contiguous, on the device the context was made on.
 *    Nothing is allocated or freed inside a call.  Inputs are never modified.
 *  - All work is enqueued on the context's HIP stream and is asynchronous;
 *    outputs are valid once that stream has been synchronised.
 *  - Return value 0 = success; a negative GORILA_E* code otherwise.  Argument
 *    errors are detected on the host before anything is enqueued.  Errors
 *    that only the device can see (an index or an action out of range) set
 *    a sticky flag in the workspace; the kernels then read a zero frame /
 *    action 0 instead of touching memory out of bounds, and the error is
 *    returned by gorila_ctx_check() (or by the next call on the context).
 *  - States are uint8 [n, 4, 84, 84]: four 84x84 luminance frames, oldest
 *    first (Section 5.1).  Network input is state / 255.
 *  - Parameters are one flat vector in this order (weights OIHW / [out, in]):
 *    W1 [32,4,8,8], b1 [32], W2 [64,32,4,4], b2 [64], W3 [64,64,3,3], b3 [64],
 *    W4 [512,3136], b4 [512], W5 [A,512], b5 [A]; the FC input is conv3's
 *    output flattened channel-major.  gorila_param_count(A) elements.
 *  - Not thread-safe per context: calls on one context must not overlap.
 */
#ifndef GORILA_H
#define GORILA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    GORILA_OK = 0,
    GORILA_EINVAL = -1,        /* bad pointer, size, dtype or action count      */
    GORILA_ERANGE = -2,        /* device saw an index or action out of range    */
    GORILA_EWORKSPACE = -3,    /* workspace too small for this call             */
    GORILA_EHIP = -4,          /* HIP runtime or launch error                   */
    GORILA_EUNSUPPORTED = -5   /* valid request the library does not implement */
};

enum { GORILA_F32 = 0, GORILA_BF16 = 1 };
enum { GORILA_REPLAY_STACKED = 0, GORILA_REPLAY_RING = 1 };

/* A parameter set theta (device pointer to the flat layout above).  fp32
 * sets must be 16-byte aligned, bf16 sets 2-byte aligned (so the rows of a
 * [groups, P] bf16 array qualify); states and frame buffers 16-byte aligned.
 * Misalignment is GORILA_EINVAL. */
typedef struct {
    const void* data;     /* fp32 (GORILA_F32) or bf16 bit patterns (GORILA_BF16) */
    int32_t n_actions;    /* A, 1 .. 32 (the Atari action set has 18)             */
    int32_t dtype;
} gorila_params;

/* Replay memory D (Section 4, Experience replay memory).
 *
 * STACKED: `rows` whole transitions; a minibatch index k in [0, rows) names
 *   s = s[k] and s' = s2[k] (uint8 [rows,4,84,84]), action[k], reward[k] and
 *   term[k] (nonzero = s' is terminal).
 * RING: a ring of `capacity` single uint8 84x84 frames holding `size`
 *   frames (0 .. capacity; capacity once the ring has wrapped); `head` is the
 *   slot of the oldest frame and logical position k (0 <= k < size) lives in
 *   slot (head + k) mod capacity.  With rows = R > 1 the arrays hold R rings of
 *   `capacity` slots each ([R][capacity] layout, one ring per actor of
 *   Section 4's bundled mode, filled in lockstep so they share `head`), and a
 *   minibatch index r * capacity + k names logical position k of ring r;
 *   rows 0 or 1 is a single ring.  Frame maps then report global slots
 *   r * capacity + slot.  ep_start[slot] != 0 marks the first frame of an
 *   episode; logical 0 also counts as one.  A minibatch index is a logical
 *   position k in [0, size-2]: s is the stack of frames k-3 .. k and s'
 *   of frames k-2 .. k+1 (oldest first), where any frame before the latest
 *   episode start at or before the stack's newest frame is all zeros (the
 *   paper concatenates the four most recent frames, Section 5.1; zero-fill at
 *   episode starts is this library's reading).  The transition's action and
 *   reward are action[slot(k)], reward[slot(k)]; it is terminal iff k+1
 *   starts an episode.  s, s2 and term are unused.  An index past size-2
 *   (a slot not yet written) is out of range (GORILA_ERANGE).
 * `reserved` is padding (set it to 0). */
typedef struct {
    int32_t kind;
    int32_t reserved;
    const uint8_t* s;
    const uint8_t* s2;
    const uint8_t* term;
    int64_t rows;
    const uint8_t* frames;
    const uint8_t* ep_start;
    int64_t capacity;
    int64_t head;
    int64_t size;            /* RING: frames stored per ring, 0 .. capacity */
    const int32_t* action;   /* [rows] or [capacity] */
    const float* reward;     /* [rows] or [capacity] */
} gorila_replay;

typedef struct gorila_ctx gorila_ctx;

/* Number of elements of a flat parameter vector with A actions, or -1. */
int64_t gorila_param_count(int32_t n_actions);

/* Device workspace bytes needed by learner calls with batch <= max_batch on
 * `groups` parameter sets (1 for the single-learner call), and by forward and
 * act calls on n <= 2 * max_batch * groups states; dtype GORILA_BF16 adds room
 * for fp32 copies of groups + 1 bf16 parameter sets.  0 for invalid
 * arguments (groups outside 1 .. 16 included).  The caller allocates it; the
 * context keeps only the pointer. */
size_t gorila_workspace_bytes(int32_t max_batch, int32_t n_actions, int32_t dtype,
                              int32_t groups);

/* Bind a stream (hipStream_t, may be NULL for the null stream) and a device
 * workspace of ws_bytes (>= gorila_workspace_bytes(1,1,0,1), 256-byte
 * aligned) to a new context on the current device.  The context owns only
 * host bookkeeping; destroy it before freeing the workspace.  Creation runs
 * one small kernel that records which XCD each of 256 workgroups runs on
 * (split reductions are used only if ids equal mod 8 share one), waits for
 * it (a stream synchronisation), then zeroes the workspace's first 8192 bytes
 * (an error word, the counters of split reductions, which every call leaves
 * at zero, and a frame of zeros that no call writes) on the stream; the
 * caller must not write the workspace
 * while the context lives, and calls on one context must not overlap (one
 * stream).  The first context made on a device also sets up that device's
 * no-allocation scratch (gorila_act_noalloc below).  workspace = NULL with
 * ws_bytes = 0 makes a context without a workspace: only gorila_act_noalloc
 * and the calls that use no workspace (replay insert, parameter sync, loss
 * filter, parameter-server apply, gorila_ctx_check) accept it; the others
 * return GORILA_EWORKSPACE. */
int gorila_ctx_create(gorila_ctx** out, void* hip_stream, void* workspace, size_t ws_bytes);
int gorila_ctx_destroy(gorila_ctx* ctx);
/* Point the context at another stream (subsequent calls enqueue there). */
int gorila_ctx_set_stream(gorila_ctx* ctx, void* hip_stream);
/* Synchronise the context's stream and report (then clear) the sticky device
 * error: GORILA_ERANGE if an index or action was out of range. */
int gorila_ctx_check(gorila_ctx* ctx);
const char* gorila_strerror(int code);

/* Kernel timing for benchmarks and profiling.  After
 * gorila_ctx_timing_begin(ctx, stage_mask, max_records), every learner step,
 * forward or act call records a HIP event pair on the context's stream
 * around each stage whose bit (1u << stage) is set in stage_mask, up to
 * max_records pairs in total (events are created here, not in the calls).
 * gorila_ctx_timing_end synchronises the stream, writes for each of the first
 * n_stages stages the summed milliseconds (total_ms) and the number of
 * recorded launches (count), and stops recording.  Stage numbers and names:
 * gorila_stage_name(i) (NULL past the last stage).  Timing does not change
 * any result. */
int gorila_ctx_timing_begin(gorila_ctx* ctx, uint32_t stage_mask, int32_t max_records);
int gorila_ctx_timing_end(gorila_ctx* ctx, double* total_ms, int32_t* count, int32_t n_stages);
const char* gorila_stage_name(int32_t stage);

/* Replay gather (Section 4 replay memory, Section 5.1 frame stacking).
 * For n minibatch indices idx [n] (int64) write s_out, s2_out
 * [n,4,84,84] uint8, frame_map_out [n,2,4] int64 (RING: the slot each
 * channel was copied from, -1 = zero-filled; STACKED: row*4 + channel),
 * a_out [n] int32, r_out [n] float, term_out [n] uint8.  frame_map_out may be
 * NULL.  Uses no workspace beyond the context's header. */
int gorila_gather(const gorila_replay* replay, const int64_t* idx, int32_t n,
                  uint8_t* s_out, uint8_t* s2_out, int64_t* frame_map_out,
                  int32_t* a_out, float* r_out, uint8_t* term_out, gorila_ctx* ctx);

/* Q(s, .; theta) (Section 5.1 network) for states [n,4,84,84] -> q_out [n,A]
 * fp32.  theta may be GORILA_F32 or GORILA_BF16 (widened exactly to fp32).
 * Needs gorila_workspace_bytes(ceil(n/2), A, dtype, 1). */
int gorila_q_forward(const gorila_params* params, const uint8_t* states_u8, int32_t n,
                     float* q_out, gorila_ctx* ctx);

/* epsilon-greedy actions (Algorithm 1): for env e, with probability eps a
 * uniformly random action, else the lowest-index argmax of Q(s_e, .; theta).
 * The two uniform draws per env are u = mix(seed + (2e+1)G) and
 * v = mix(seed + (2e+2)G), G = 0x9E3779B97F4A7C15, mix = the SplitMix64
 * output function (Steele, Lea and Flood 2014), all mod 2^64; explore iff
 * (u >> 11) < floor(eps * 2^53), random action = ((v >> 32) * A) >> 32.
 * actions_out [n] int32; q_out [n,A] fp32 may be NULL.  eps in [0, 1]. */
int gorila_act(const gorila_params* params, const uint8_t* states_u8, int32_t n, float eps,
               uint64_t seed, int32_t* actions_out, float* q_out, gorila_ctx* ctx);

/* One DQN learner step (Algorithm 1; eq. (1) and (2)) on the minibatch
 * idx [batch] drawn from `replay`:
 *   q = Q(s; theta), q' = Q(s'; theta-), y = r + gamma (1 - term) max q',
 *   delta = y - q[a], loss = mean_b huber(delta_b) with threshold clip_delta
 *   (0.5 delta^2 for |delta| <= clip_delta, clip_delta |delta| - 0.5
 *   clip_delta^2 beyond; clip_delta = +INFINITY gives eq. (1) times 1/2),
 *   grads_out [P] fp32 = d loss / d theta (for |delta| <= clip_delta this is
 *   minus the minibatch mean of eq. (2)'s g), loss_out [1] fp32.
 * No gradient flows into theta-.  params and target_params must have the
 * same A and dtype GORILA_F32.  Needs gorila_workspace_bytes(batch, A, 0, 1). */
int gorila_learner_step(const gorila_params* params, const gorila_params* target_params,
                        const gorila_replay* replay, const int64_t* idx, int32_t batch,
                        float gamma, float clip_delta, float* grads_out, float* loss_out,
                        gorila_ctx* ctx);

/* `groups` independent learner steps (Section 4: many learners, each with
 * its own, possibly stale, replica of theta) sharing one target theta-.
 * params points to `groups` (1 .. 16) host-side parameter descriptors, each
 * GORILA_F32 or GORILA_BF16 and all with the target's A; group g is the
 * learner step of gorila_learner_step on params[g] and the minibatch
 * idx[g*batch .. g*batch+batch-1], and writes grads_out[g*P .. g*P+P-1] and
 * loss_out[g] (fp32).  When every set (the target's included) is bf16, the
 * products run on bf16 MFMA operands with fp32 accumulation: forward
 * activations as two bf16 terms (value rounded to bf16, plus the rounded
 * residual), backward operands rounded to bf16, weights exact; gradients
 * then agree with the exact step to a few 1e-3 relative L2 (fp32: ~1e-6).
 * Otherwise bf16 sets are widened exactly to fp32 and the step runs in fp32.  The forward passes of all groups share launches.
 * Needs gorila_workspace_bytes(batch, A, GORILA_BF16 if any set is bf16 else
 * GORILA_F32, groups); EINVAL for groups outside 1 .. 16. */
int gorila_learner_step_grouped(const gorila_params* params, int32_t groups,
                                const gorila_params* target_params, const gorila_replay* replay,
                                const int64_t* idx, int32_t batch, float gamma, float clip_delta,
                                float* grads_out, float* loss_out, gorila_ctx* ctx);

/* For callers that cannot allocate device memory at call time (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * gorila_act without a workspace.  Same arguments, semantics and results as
 * gorila_act (the same kernels run), for n <= GORILA_NOALLOC_MAX_STATES
 * states; larger n returns GORILA_EWORKSPACE.  Intermediate results live in
 * a static device array of at most GORILA_NOALLOC_SCRATCH_MB MiB that each
 * device holds until the process ends (its address is resolved when the first
 * context is made on that device); the call allocates nothing.  Every call on
 * one device shares that array: calls that overlap on one device, from any
 * context or stream, race and must not be issued. */
#define GORILA_NOALLOC_MAX_STATES 256
#define GORILA_NOALLOC_SCRATCH_MB 44
int gorila_act_noalloc(const gorila_params* params, const uint8_t* states_u8, int32_t n,
                       float eps, uint64_t seed, int32_t* actions_out, float* q_out,
                       gorila_ctx* ctx);

/* Per-transition values of the most recent learner call on this context
 * (gorila_learner_step or _grouped; Algorithm 1's target and eq. (1)'s
 * error), in that call's row order (group g's rows g*batch .. g*batch+batch-1):
 *   q_out      [rows, A] fp32: Q(s; theta) of the learner's parameters,
 *   q_next_out [rows, A] fp32: Q(s'; theta-),
 *   td_out     [rows, 4] fp32: max_a' Q(s', a'; theta-), the target y, the
 *              TD error delta = y - Q(s, a; theta) and its Huber loss,
 * with rows = groups * batch.  Any output may be NULL.  The values live in the
 * context's workspace until a forward or act call reuses it: GORILA_EINVAL
 * if no learner call has run since the context was made or since such a
 * call.  Enqueued on the context's stream (device-to-device copies). */
int gorila_learner_td(gorila_ctx* ctx, float* q_out, float* q_next_out, float* td_out);

/* ---- Actor side (Algorithm 1, Section 4 actors and replay memory, Section 5.1) ---- */

/* Store experience in replay rings (Algorithm 1: the actor stores each step's
 * transition in D; Section 4: one replay memory per actor in bundled mode).
 * frames [rings][capacity][84][84] u8, ep_start / action / reward
 * [rings][capacity] (device; the arrays of a gorila_replay RING with
 * rows = rings); all rings share *head and *size (host values, updated at
 * enqueue time: the rings are filled in lockstep).  m records per ring,
 * inputs [m][rings][...] (frames_in [m][rings][84][84], ep_start_in,
 * action_in, reward_in [m][rings], device): record j of ring r is the frame,
 * its episode-start flag, the action taken at it and the reward that
 * followed, and lands in slot (head + size + j) mod capacity of ring r, so
 * once a ring is full each record overwrites the oldest and head advances.
 * Then size = min(size + m, capacity) and head moves by the overflow.
 * EINVAL for m outside 0 .. capacity or capacity < 2; frames and frames_in
 * 16-byte aligned. */
int gorila_replay_insert(uint8_t* frames, uint8_t* ep_start, int32_t* action, float* reward,
                         int64_t capacity, int32_t rings, int64_t* head, int64_t* size,
                         const uint8_t* frames_in, const uint8_t* ep_start_in,
                         const int32_t* action_in, const float* reward_in, int32_t m,
                         gorila_ctx* ctx);

/* Parameter pull and periodic target sync (Algorithm 1: actors and learners
 * update theta from theta+ of the parameter server; every N global updates
 * the learner syncs theta- with theta+; Section 5.1: N = 60K).  src [n] fp32
 * (theta+, device); dst [copies][n] (device, fp32 or, with dst_dtype
 * GORILA_BF16, bf16 bit patterns rounded to nearest even; copies 0 .. 64);
 * dst_version [copies] (int64, device) is the server version each copy
 * holds.  With *ps_version (int64 device scalar) the current version, copy c
 * is due when period == 0 (a pull) or a multiple of period lies in
 * (dst_version[c], *ps_version] (period > 0, versions >= 0: a sync); a due
 * copy receives src and dst_version[c] = *ps_version; synced_out [copies]
 * (u8, may be NULL) reports which were copied.  Everything stays on the
 * device.  EINVAL for a bad dtype, period < 0, copies > 64 or misalignment
 * (fp32 4-byte, bf16 2-byte, int64 8-byte). */
int gorila_params_sync(const float* src, void* dst, int64_t n, int32_t copies, int32_t dst_dtype,
                       const int64_t* ps_version, int64_t* dst_version, int64_t period,
                       uint8_t* synced_out, gorila_ctx* ctx);

/* Behaviour-policy epsilon after `update` global updates (Section 5.1:
 * annealed from 1 to 0.1 over the first million updates): eps_start for
 * update <= 0, eps_end from anneal_updates on, linear in between.  Host
 * arithmetic only; pass it to gorila_act. */
double gorila_epsilon(int64_t update, double eps_start, double eps_end, int64_t anneal_updates);

/* ---- Parameter-server side (Section 4, parameter server; Section 4.2) ---- */

/* Most gradients one gorila_ps_apply call takes. */
#define GORILA_PS_MAX_GROUPS 4096

/* Loss-statistics gradient filter (Section 4.2: each learner keeps a running
 * mean and standard deviation of its absolute DQN loss and discards a
 * gradient whose absolute loss exceeds the mean by more than k standard
 * deviations).  For learner g (0 <= g < groups): x = |loss[g]| (loss [groups]
 * fp32, e.g. the loss_out of gorila_learner_step_grouped) is compared with
 * its statistics stats[g] = (n, mean, var) (fp64 [groups][3], device, 8-byte
 * aligned, caller-owned, zero-initialised before a learner's first loss):
 * keep_out[g] = 0 iff n >= max(warmup, 1), x > mean and (x - mean)^2 > k^2
 * var; then x joins the statistics (kept or not): the first x sets
 * (1, x, 0); after that, alpha > 0 gives exponentially weighted statistics
 * d = x - mean, mean += alpha d, var = (1 - alpha)(var + alpha d^2), and
 * alpha = 0 cumulative ones, mean' = mean + d/(n+1),
 * var' = (n var + d (x - mean')) / (n+1); n += 1.  Every step is one fp64
 * operation rounded once.  EINVAL for alpha outside [0, 1] or k < 0. */
int gorila_loss_filter(double* stats, const float* loss, int32_t groups, double alpha, double k,
                       int64_t warmup, uint8_t* keep_out, gorila_ctx* ctx);

/* Parameter-server apply (Section 4: the server applies learner gradients to
 * theta+; Section 4.2: gradients computed from parameters older than a
 * threshold are discarded, and the update rule is AdaGrad, Duchi, Hazan and
 * Singer 2011).  grads [groups][n] fp32 (e.g. grads_out of the grouped learner
 * step, n = P) are taken in index order; gradient g was computed from theta+
 * at server version grad_version[g] (int64 [groups]); at its turn the server
 * is at version V (*ps_version, int64 device scalar, earlier applied gradients
 * of this call included) and it is applied iff keep[g] (u8 [groups], NULL =
 * all kept, e.g. the keep_out of gorila_loss_filter) and V - grad_version[g]
 * <= max_delay; each applied gradient advances *ps_version by one and updates
 * every element i of theta_plus / accum [n] (fp32, in place):
 *     accum[i] += g_i^2;  theta_plus[i] -= lr * g_i / (eps + sqrt(accum[i])).
 * applied_out [groups] u8 receives the decisions.  All pointers are device
 * pointers; fp32 arrays 4-byte aligned, int64 ones 8-byte aligned.  The
 * decisions and the version stay on the device (no host round trip).
 * EINVAL for eps <= 0, lr < 0, n > 2^31 - 1 or groups outside
 * 0 .. GORILA_PS_MAX_GROUPS.  Uses no workspace. */
int gorila_ps_apply(float* theta_plus, float* accum, int64_t n, const float* grads, int32_t groups,
                    const uint8_t* keep, const int64_t* grad_version, int64_t* ps_version,
                    int64_t max_delay, float lr, float eps, uint8_t* applied_out, gorila_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif
