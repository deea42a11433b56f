// Host-side launchers of the Gorila kernels (internal to libgorila).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gorila.h"
#include "common.h"

namespace gorila {

// Replay source as the kernels see it.
struct ReplayView {
    int kind;
    const uint8_t* s;
    const uint8_t* s2;
    const uint8_t* term;
    int64_t rows;
    const uint8_t* frames;
    const uint8_t* ep_start;
    int64_t capacity;
    int64_t head;
    int64_t size;  // RING: frames stored per ring (valid indices 0 .. size-2)
    const int32_t* action;
    const float* reward;
};


// Materialising gather: s_out / s2_out [n][4][84][84], frame_map [n][2][4]
// (may be null), a, r, term, in one launch (one workgroup per transition).
void launch_gather(const ReplayView& rv, const int64_t* idx, int n, int n_actions,
                   uint8_t* s_out, uint8_t* s2_out, int64_t* frame_map, int32_t* a, float* r,
                   uint8_t* term, unsigned* err, hipStream_t st);

// Replay insert into `rings` rings of `capacity` slots ([rings][capacity]
// layout): record j of ring r (inputs [records / rings][rings]) goes to slot
// (base + j) mod capacity of its ring; base + j never exceeds 2 capacity.
void launch_insert(uint8_t* frames, uint8_t* ep_start, int32_t* action, float* reward,
                   int64_t capacity, int rings, int64_t base, const uint8_t* frames_in,
                   const uint8_t* ep_in, const int32_t* act_in, const float* rew_in, int records,
                   hipStream_t st);

// Transposed conv weights used as MFMA operands.
//  w2t [16][64][32]: W2[o][c][u][v] at [(u,v)][o][c]   (conv2 forward)
//  w3t [9][64][64]:  W3[o][c][u][v] at [(u,v)][o][c]   (conv3 forward)
//  w3d [9][64][64]:  W3[o][c][u][v] at [(u,v)][c][o]   (conv3 data gradient)
//  w2p [4][4][32][64]: W2[o][c][u][v] at [(u/2,v/2)][(u%2,v%2)][c][o]  (conv2 data gradient)
struct WeightViews {
    const float* theta;   // flat parameters
    float* w2t;
    float* w3t;
    float* w3d;           // may be null (forward only)
    float* w2p;           // may be null
    // when not null: the same parameters as bf16 bit patterns, which the
    // transposes read (and widen exactly) instead of theta, so that they need
    // not wait for theta's widened copy
    const uint16_t* theta16 = nullptr;
};
constexpr int MAX_NETS = MAX_LEARNER_GROUPS + 1;  // learner replicas + their shared target
struct WeightViewSet {
    WeightViews v[MAX_NETS];
};

// Block `blk` of `nblk` (256 threads each) of one net's transposes.  Every
// destination is written in index order (coalesced); the scattered reads come
// from the 128 KB of W2 and W3, which stay in L2.
constexpr int PREP_BLOCKS = 64;  // blocks per net
__device__ inline void prep_weights_part(const WeightViews& v, int blk, int nblk) {
    // W2 [o][c][u][v], 64 x 32 x 4 x 4; W3 [o][c][u][v], 64 x 64 x 3 x 3
    auto W2 = [&](int i) {
        return v.theta16 ? __uint_as_float((uint32_t)v.theta16[OFF_W2 + i] << 16) : v.theta[OFF_W2 + i];
    };
    auto W3 = [&](int i) {
        return v.theta16 ? __uint_as_float((uint32_t)v.theta16[OFF_W3 + i] << 16) : v.theta[OFF_W3 + i];
    };
    const int stride = nblk * 256;
    for (int d = blk * 256 + (int)threadIdx.x; d < 16 * 64 * 32; d += stride) {
        {  // w2t[t][o][c], t = u*4 + v
            const int c = d & 31, o = (d >> 5) & 63, t = d >> 11;
            v.w2t[d] = W2(((o * 32 + c) * 4 + (t >> 2)) * 4 + (t & 3));
        }
        if (v.w2p) {  // w2p[tp][phase][c][o]: tap pair (u/2, v/2), stride phase (u%2, v%2)
            const int o = d & 63, c = (d >> 6) & 31, phase = (d >> 11) & 3, tp = d >> 13;
            const int u = (tp >> 1) * 2 + (phase >> 1), vv = (tp & 1) * 2 + (phase & 1);
            v.w2p[d] = W2(((o * 32 + c) * 4 + u) * 4 + vv);
        }
    }
    for (int d = blk * 256 + (int)threadIdx.x; d < 9 * 64 * 64; d += stride) {
        {  // w3t[t][o][c], t = u*3 + v
            const int c = d & 63, o = (d >> 6) & 63, t = d >> 12;
            v.w3t[d] = W3((o * 64 + c) * 9 + t);
        }
        if (v.w3d) {  // w3d[t][c][o]
            const int o = d & 63, c = (d >> 6) & 63, t = d >> 12;
            v.w3d[d] = W3((o * 64 + c) * 9 + t);
        }
    }
}

// Widening of bf16 parameter vectors (bit patterns) to fp32, exact:
// dst[i][k] = src[i][k].
struct WidenSet {
    const uint16_t* src[MAX_NETS];
    float* dst[MAX_NETS];
};
// Elements [lo[0], hi[0]) and [lo[1], hi[1]) of n vectors, widened by extra
// blocks of another launch: blocks_per_net() blocks for each vector.
struct WidenJob {
    WidenSet set;
    int n = 0;
    int64_t lo[2] = {0, 0}, hi[2] = {0, 0};
    int blocks_per_net() const {
        const int64_t c = (hi[0] - lo[0]) + (hi[1] - lo[1]);
        return n ? (int)(c / 4096 < 1 ? 1 : c / 4096 > 256 ? 256 : c / 4096) : 0;
    }
};
// Block blk of nblk (256 threads each) of vector i's widening.
__device__ inline void widen_part(const WidenJob& wj, int i, int blk, int nblk) {
    const uint16_t* src0 = wj.set.src[i];
    float* dst0 = wj.set.dst[i];
    const int64_t tid = (int64_t)blk * 256 + threadIdx.x, stride = (int64_t)nblk * 256;
    for (int r = 0; r < 2; ++r) {
        const int64_t count = wj.hi[r] - wj.lo[r];
        if (count <= 0) continue;
        const uint16_t* src = src0 + wj.lo[r];
        float* dst = dst0 + wj.lo[r];
        // elements before the first 8-byte boundary of the (2-byte aligned)
        // source and after the last whole group of four go one by one
        const int64_t head = min<int64_t>(count, ((8 - ((uintptr_t)src & 7)) & 7) >> 1);
        const int64_t quads = (count - head) >> 2, tail = head + 4 * quads;
        if (tid < head) dst[tid] = __uint_as_float((uint32_t)src[tid] << 16);
        for (int64_t q = tid; q < quads; q += stride) {
            const int64_t e = head + 4 * q;
            const uint2 v = *(const uint2*)(src + e);
            dst[e] = __uint_as_float(v.x << 16);
            dst[e + 1] = __uint_as_float(v.x & 0xffff0000u);
            dst[e + 2] = __uint_as_float(v.y << 16);
            dst[e + 3] = __uint_as_float(v.y & 0xffff0000u);
        }
        if (tail + tid < count) dst[tail + tid] = __uint_as_float((uint32_t)src[tail + tid] << 16);
    }
}

// Minibatch resolution, the weight transposes and the parameter widening in
// one launch (they are independent: transposes of widened sets read the bf16
// source): the first blocks resolve the indices into frame pointers
// ftab[2][n][4] (s then s'; null = zero-filled channel) and a/r/term per row,
// the next the weight transposes of n_nets sets (prep_weights_part), the
// rest wj's widening (wj may be null).
void launch_resolve_prep(const ReplayView& rv, const int64_t* idx, int n, int n_actions,
                         const uint8_t** ftab, int32_t* a, float* r, uint8_t* term,
                         unsigned* err, const WeightViews* nets, int n_nets, const WidenJob* wj,
                         hipStream_t st);

// Forward layers.  `groups` parameter sets; group g owns rows [g*n, (g+1)*n)
// of every activation buffer.  bf16: the parameter sets hold bf16 values
// (widened to fp32) and the products run on bf16 MFMA operands (common.h).
void launch_conv1_fwd(const uint8_t* const* ftab, const GroupPtrs& theta, int groups, int n,
                      float* h1, bool bf16, hipStream_t st);
// Workspace for balancing a launch (TailSplit): ws holds SPLIT_MAX_SLOTS
// partial 64x64 tiles, cnt SPLIT_MAX_TILES counters that are zero between
// launches; ws == nullptr turns splitting off.  The launches on one stream run one after another, so they share it.
// cus is set either way (launch shapes use it).
struct SplitWs {
    float* ws = nullptr;
    int* cnt = nullptr;
    int cus = 0;  // compute units of the device
};
void launch_conv2_fwd(const float* h1, const GroupPtrs& w2t, const GroupPtrs& theta, int groups,
                      int n, float* h2, const SplitWs& sw, bool bf16, hipStream_t st);
void launch_conv3_fwd(const float* h2, const GroupPtrs& w3t, const GroupPtrs& theta, int groups,
                      int n, float* h3, const SplitWs& sw, bool bf16, hipStream_t st);
// fc1 forward as split-K partial sums partial[g][s][b][512]; returns the
// number of splits s (the head kernels finish the layer).  With bf16, W4 is
// read from w4b (the sets' bf16 W4 blocks, 2-byte aligned at least), not theta.
int launch_fc1_fwd(const float* h3, const GroupPtrs& theta, const GroupPtrs16& w4b, int groups,
                   int n, float* partial, bool bf16, hipStream_t st);

// Head: Q values, epsilon-greedy actions, TD error / Huber loss / dLoss.
// Each first finishes the FC-512 layer (splits in order, bias, ReLU).
void launch_q_head(const float* fc1part, int splits, const float* theta, int n, int A, float* q,
                   hipStream_t st);
void launch_act_head(const float* fc1part, int splits, const float* theta, int n, int A, float eps,
                     uint64_t seed, int32_t* actions, float* q_out, hipStream_t st);
// Writes h4 (online rows), q [2n][A], ell, coef = dLoss/dQ(s,a), td [n][4] =
// (max_a' Q(s',a'), y, delta, ell) per learner row, and dz4.
// `groups` learner groups of n rows each (group g: rows g*n .. g*n+n-1, online
// parameters thetas.p[g]); fc1part_online / fc1part_target + g * part_stride
// each hold [splits][n][512] for group g.
void launch_td_head(const float* fc1part_online, const float* fc1part_target, int64_t part_stride,
                    int splits, const GroupPtrs& thetas, int groups, const float* theta_target,
                    int n, int A, const int32_t* a, const float* r, const uint8_t* term,
                    float gamma, float clip, float* h4, float* q, float* ell, float* coef,
                    float* td, float* dz4, hipStream_t st);

// Backward of `groups` learner groups of n rows each (group g: rows
// g*n .. g*n+n-1 of every per-sample tensor, parameters of set g), three
// launches of independent jobs each:
//  fc1: dz3 = [h3 > 0] W4^T dz4 (stored [b][p][o]), dW4 and db4 into
//       grads + g * grads_stride, and row-block partials of dW5, db5 and the
//       loss (returns row blocks per group);
//  conv3: dz2 and split partials of dW3 / db3 (returns splits per group);
//  conv2: dz1 and split partials of dW2 / db2 (returns splits per group).
// kp: dz3 / dz2 partial planes, each groups * n rows long; fc1 writes kp
// planes of dz3, conv3 reads them and writes kp planes of dz2, conv2 reads
// those.
int launch_fc1_backward(const float* dz4, const GroupPtrs& theta, const GroupPtrs16& w4b,
                        int groups, const float* h3,
                        const float* h4, const int32_t* a, const float* coef, const float* ell,
                        int n, int A, float* dz3, float* grads, int64_t grads_stride,
                        float* hpart, int kp, const SplitWs& sw, bool bf16, hipStream_t st);
int launch_conv3_backward(const float* dz3, const GroupPtrs& w3d, int groups, const float* h2,
                          int n, float* dz2, float* partial, float* bias_part, int kp, bool bf16,
                          hipStream_t st);
// dz1: fp32, or (bf16) the values rounded to bf16 in the same [n][20][20][32]
// order, as the conv1 weight gradient below reads it.
int launch_conv2_backward(const float* dz2, const GroupPtrs& w2p, int groups, const float* h1,
                          int n, float* dz1, float* partial, float* bias_part, int kp, bool bf16,
                          hipStream_t st);
// ftab: [groups * n][4] frame pointers of the online states (null: zero-filled);
// zero_frame: FRAME_BYTES of zeros, read in place of a null frame; dz1 as
// launch_conv2_backward wrote it (bf16 bit patterns when bf16).
void launch_conv1_wgrad(const float* dz1, const uint8_t* const* ftab, const uint8_t* zero_frame,
                        int groups, int n,
                        float* partial, float* bias_part, int max_splits, int* splits_out,
                        bool bf16, hipStream_t st);
// Conv weight-gradient partials [group][split][o][(tap, c)], bias partials
// bias_part[layer][group][split][64] (one row per split, written by the
// weight-gradient workgroups of column tile 0) and the head partials
// hpart[group][block][HP_STRIDE], each summed in split / block order into
// grads + g * grads_stride and loss_out[g].
struct ReduceArgs {
    const float* part1;
    const float* part2;
    const float* part3;
    const float* bias_part;
    const float* hpart;
    int s1, s2, s3, head_blocks, n, A, groups;
    int64_t grads_stride;
    float* grads;
    float* loss_out;
};
void launch_grad_reduce(const ReduceArgs& ra, hipStream_t st);

// Parameter-server side (ps.hip).  Loss-statistics filter: stats [groups][3]
// (n, mean, var of |loss|, fp64) updated in place, keep [groups].  Apply:
// decides which of grads [groups][n] to apply (applied [groups], *ps_version
// advanced on the device; one workgroup), then AdaGrad-updates theta / accum
// [n] with them.
void launch_loss_filter(double* stats, const float* loss, int groups, double alpha, double k,
                        int64_t warmup, uint8_t* keep, hipStream_t st);
void launch_ps_apply(float* theta, float* accum, int64_t n, const float* grads, int groups,
                     const uint8_t* keep, const int64_t* version, int64_t* ps_version,
                     int64_t max_delay, float lr, float eps, uint8_t* applied, hipStream_t st);

// Parameter pull / periodic target sync (ps.hip): copies <= 64 destinations
// dst [copies][n] (fp32 or bf16), each copied when due, versions recorded by
// a second launch.
void launch_params_sync(const float* src, void* dst, int64_t n, int copies, bool to_bf16,
                        const int64_t* ps_version, int64_t* dst_version, int64_t period,
                        uint8_t* synced, hipStream_t st);

// Sizes of the split-K / partial buffers the launchers above may use.
constexpr int TARGET_WGS = 1024;             // split-K launches aim at ~4 workgroups per CU
constexpr int FC1_MAX_SPLITS = 14;
constexpr int WG_MAX_SPLITS = 256;
constexpr int CONV3_WG_SPLITS = 114;         // 9 column tiles x 114 splits ~ 1024 workgroups
constexpr int CONV2_WG_SPLITS = 64;          // 8 column tiles x 64 splits
constexpr int CONV1_WG_MAX_SPLITS = 512;
// Small batches split the fc1 and conv3 data gradients over the reduction:
// with B learner rows, dz3 and dz2 arrive as bwd_parts(B) partial planes
// (each already masked by the ReLU, which is linear in them) that the conv3
// and conv2 backward loaders add in plane order.  bwd_split_rows(B) >=
// bwd_parts(B) * B rows are reserved per tensor; it never decreases with B,
// so a workspace sized for a batch serves every smaller one.
__host__ __device__ constexpr int bwd_parts(int64_t rows) { return rows <= 64 ? 4 : rows <= 128 ? 2 : 1; }
__host__ __device__ constexpr int64_t bwd_split_rows(int64_t rows) {
    return rows <= 64 ? 4 * rows : rows <= 256 ? 256 : rows;
}
constexpr int BIAS_PART_STRIDE = 512 * 64;  // floats per layer in bias_part
constexpr int HEAD_MAX_BLOCKS = 16;          // row blocks of the head partials, per group
constexpr int HP_DB5 = MAX_ACTIONS * HID;    // offsets inside one head partial
constexpr int HP_LOSS = HP_DB5 + MAX_ACTIONS;
constexpr int HP_STRIDE = HP_LOSS + 32;

}  // namespace gorila
