// Action head (linear FC 512 -> A, Section 5.1) and what follows it:
//  - Q values;
//  - epsilon-greedy actions (Algorithm 1);
//  - the DQN TD target y = r + gamma (1 - term) max_a' Q(s', a'; theta-),
//    TD error delta = y - Q(s, a; theta), Huber loss and dLoss/dQ (eq. (1),
//    (2); Algorithm 1's terminal case), fused with the action-head backward
//    dz4 = dLoss/dQ(s,a) * W5[a][:] * [h4 > 0].
// One wave64 per sample.  The FC-512 layer arrives as split-K partial sums
// fc1part[g][s][b][512]; lane l adds its 8 columns over the splits in order,
// adds the bias and applies the ReLU, so h4 is finished here.  Each of the A
// dot products is a butterfly sum over the wave, so every lane ends with the
// same bit pattern and nothing depends on scheduling.
#include "common.h"
#include "kernels.h"

namespace gorila {

__device__ inline float dot8(const float* h, f32x4 w0, f32x4 w1) {
    float s = h[0] * w0[0];
    s = fmaf(h[1], w0[1], s);
    s = fmaf(h[2], w0[2], s);
    s = fmaf(h[3], w0[3], s);
    s = fmaf(h[4], w1[0], s);
    s = fmaf(h[5], w1[1], s);
    s = fmaf(h[6], w1[2], s);
    s = fmaf(h[7], w1[3], s);
    return s;
}

// out[j] = b5[k] + sum_i h4[i] W5[k][i] for k = k0 + j, j < HB (k < A
// matter; later ones repeat row A - 1).  All HB rows are loaded before the
// first dot product and the HB butterfly sums are independent, so a block of
// actions costs one memory round trip instead of one per action.
constexpr int HB = 6;
__device__ inline void head_rows(const float* h, const float* W5, const float* b5, int k0, int A,
                                 int lane, float* out) {
    f32x4 w0[HB], w1[HB];
#pragma unroll
    for (int j = 0; j < HB; ++j) {
        const float* w = W5 + min(k0 + j, A - 1) * HID + lane * 8;
        w0[j] = ld4(w);
        w1[j] = ld4(w + 4);
    }
#pragma unroll
    for (int j = 0; j < HB; ++j) out[j] = dot8(h, w0[j], w1[j]);
#pragma unroll
    for (int j = 0; j < HB; ++j) out[j] = wave_sum(out[j]) + b5[min(k0 + j, A - 1)];
}

// h[0..7] = relu(b4[8l..] + sum_s part[s][b][8l..]) for one row b.
__device__ inline void finish_h4(const float* part, int splits, int64_t split_stride,
                                 const float* b4, int lane, float* h) {
    // every split's partial is loaded before the first addition, so the loads
    // overlap instead of waiting for one another
    f32x4 pa[FC1_MAX_SPLITS], pc[FC1_MAX_SPLITS];
#pragma unroll
    for (int s = 0; s < FC1_MAX_SPLITS; ++s)
        if (s < splits) {
            const float* p = part + s * split_stride + lane * 8;
            pa[s] = ld4(p);
            pc[s] = ld4(p + 4);
        }
    f32x4 a = pa[0], c = pc[0];
#pragma unroll
    for (int s = 1; s < FC1_MAX_SPLITS; ++s)
        if (s < splits) {
            a += pa[s];
            c += pc[s];
        }
    const f32x4 ba = ld4(b4 + lane * 8), bc = ld4(b4 + lane * 8 + 4);
    h[0] = fmaxf(a[0] + ba[0], 0.f); h[1] = fmaxf(a[1] + ba[1], 0.f);
    h[2] = fmaxf(a[2] + ba[2], 0.f); h[3] = fmaxf(a[3] + ba[3], 0.f);
    h[4] = fmaxf(c[0] + bc[0], 0.f); h[5] = fmaxf(c[1] + bc[1], 0.f);
    h[6] = fmaxf(c[2] + bc[2], 0.f); h[7] = fmaxf(c[3] + bc[3], 0.f);
}

// SplitMix64 output function (Steele, Lea and Flood 2014).
__device__ inline uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void q_head_kernel(const float* __restrict__ fc1part, int splits,
                                                     const float* __restrict__ theta, int n, int A,
                                                     float* __restrict__ q,
                                                     int32_t* __restrict__ actions,
                                                     uint64_t explore_below, uint64_t seed) {
    const int lane = threadIdx.x & 63, b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= n) return;
    float h[8];
    finish_h4(fc1part + (int64_t)b * HID, splits, (int64_t)n * HID, theta + OFF_B4, lane, h);
    const float* W5 = theta + OFF_W5;
    const float* b5 = theta + off_b5(A);
    float best = 0.0f;
    int best_a = 0;
    for (int k0 = 0; k0 < A; k0 += HB) {
        float qs[HB];
        head_rows(h, W5, b5, k0, A, lane, qs);
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const int k = k0 + j;
            if (k >= A) break;
            const float s = qs[j];
            if (q && lane == 0) q[(int64_t)b * A + k] = s;
            if (k == 0 || s > best) { best = s; best_a = k; }  // lowest index among the maxima
        }
    }
    if (actions && lane == 0) {
        const uint64_t G = 0x9E3779B97F4A7C15ull;
        const uint64_t u = splitmix64_mix(seed + (2ull * (uint64_t)b + 1ull) * G);
        const uint64_t v = splitmix64_mix(seed + (2ull * (uint64_t)b + 2ull) * G);
        const bool explore = (u >> 11) < explore_below;
        actions[b] = explore ? (int32_t)(((v >> 32) * (uint64_t)A) >> 32) : best_a;
    }
}

void launch_q_head(const float* fc1part, int splits, const float* theta, int n, int A, float* q,
                   hipStream_t st) {
    if (n <= 0) return;
    q_head_kernel<<<(n + 3) / 4, 256, 0, st>>>(fc1part, splits, theta, n, A, q, nullptr, 0, 0);
}

void launch_act_head(const float* fc1part, int splits, const float* theta, int n, int A, float eps,
                     uint64_t seed, int32_t* actions, float* q_out, hipStream_t st) {
    if (n <= 0) return;
    // explore iff a uniform 53-bit integer is below floor(eps * 2^53); eps is
    // exact in double and the scaling by 2^53 is exact.
    const uint64_t below = (uint64_t)floor((double)eps * 9007199254740992.0);
    q_head_kernel<<<(n + 3) / 4, 256, 0, st>>>(fc1part, splits, theta, n, A, q_out, actions, below,
                                               seed);
}

// Learner group g (blockIdx.y) owns rows g*n .. g*n+n-1 of a, r, term, h4,
// ell, coef and dz4, and rows 2gn .. 2gn+2n-1 of q (online, then target).
// fc1part_online / fc1part_target + g * part_stride: [splits][n][512] for the
// group's online network (on s) and the target network (on s').
__global__ __launch_bounds__(256) void td_head_kernel(
    const float* __restrict__ fc1part, const float* __restrict__ fc1part_t, int64_t part_stride,
    int splits, GroupPtrs thetas, const float* __restrict__ theta_t, int n, int A,
    const int32_t* __restrict__ a, const float* __restrict__ r, const uint8_t* __restrict__ term,
    float gamma, float clip, float* __restrict__ h4, float* __restrict__ q,
    float* __restrict__ ell, float* __restrict__ coef, float* __restrict__ dz4) {
    const int lane = threadIdx.x & 63, bl = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (bl >= n) return;
    const int grp = blockIdx.y;
    const float* theta = thetas.p[grp];
    const int64_t ss = (int64_t)n * HID;
    float h[8], ht[8];
    finish_h4(fc1part + grp * part_stride + (int64_t)bl * HID, splits, ss, theta + OFF_B4, lane, h);
    finish_h4(fc1part_t + grp * part_stride + (int64_t)bl * HID, splits, ss, theta_t + OFF_B4, lane,
              ht);
    const int64_t b = (int64_t)grp * n + bl;  // learner row
    q += (int64_t)grp * 2 * n * A;
    float* h4row = h4 + b * HID + lane * 8;
    *(f32x4*)h4row = f32x4{h[0], h[1], h[2], h[3]};
    *(f32x4*)(h4row + 4) = f32x4{h[4], h[5], h[6], h[7]};
    const float* W5 = theta + OFF_W5;
    const float* b5 = theta + off_b5(A);
    const float* W5t = theta_t + OFF_W5;
    const float* b5t = theta_t + off_b5(A);
    const int ab = a[b];
    float q_sa = 0.0f, m = 0.0f;
    for (int k0 = 0; k0 < A; k0 += HB) {
        float qs[HB], qt[HB];
        head_rows(h, W5, b5, k0, A, lane, qs);
        head_rows(ht, W5t, b5t, k0, A, lane, qt);
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const int k = k0 + j;
            if (k >= A) break;
            const float s = qs[j], st = qt[j];
            if (lane == 0) {
                q[(int64_t)bl * A + k] = s;
                q[(int64_t)(n + bl) * A + k] = st;
            }
            if (k == ab) q_sa = s;
            m = k == 0 ? st : fmaxf(m, st);  // max_a' Q(s', a'; theta-)
        }
    }
    const float y = term[b] ? r[b] : r[b] + gamma * m;
    const float d = y - q_sa;
    const float ad = fabsf(d);
    const float g = fminf(fmaxf(d, -clip), clip);
    const float cf = -g / (float)n;  // d(mean loss)/dQ(s, a)
    if (lane == 0) {
        ell[b] = ad <= clip ? 0.5f * d * d : clip * ad - 0.5f * clip * clip;
        coef[b] = cf;
    }
    const float* w = W5 + ab * HID + lane * 8;
    float* out = dz4 + b * HID + lane * 8;
    const f32x4 w0 = ld4(w), w1 = ld4(w + 4);
    const f32x4 o0 = {h[0] > 0.f ? cf * w0[0] : 0.f, h[1] > 0.f ? cf * w0[1] : 0.f,
                      h[2] > 0.f ? cf * w0[2] : 0.f, h[3] > 0.f ? cf * w0[3] : 0.f};
    const f32x4 o1 = {h[4] > 0.f ? cf * w1[0] : 0.f, h[5] > 0.f ? cf * w1[1] : 0.f,
                      h[6] > 0.f ? cf * w1[2] : 0.f, h[7] > 0.f ? cf * w1[3] : 0.f};
    *(f32x4*)out = o0;
    *(f32x4*)(out + 4) = o1;
}

void launch_td_head(const float* fc1part_online, const float* fc1part_target, int64_t part_stride,
                    int splits, const GroupPtrs& thetas, int groups, const float* theta_target,
                    int n, int A, const int32_t* a, const float* r, const uint8_t* term,
                    float gamma, float clip, float* h4, float* q, float* ell, float* coef,
                    float* dz4, hipStream_t st) {
    if (n <= 0) return;
    td_head_kernel<<<dim3((n + 3) / 4, groups), 256, 0, st>>>(
        fc1part_online, fc1part_target, part_stride, splits, thetas, theta_target, n, A, a, r, term,
        gamma, clip, h4, q, ell, coef, dz4);
}

}  // namespace gorila
