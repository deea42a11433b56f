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
//
// One workgroup of four waves per learner row, so the row's dependent memory
// round trips overlap: every load that does not depend on h4 (the fc1 split
// partials, this wave's W5 rows of both networks, the W5 row of the chosen
// action) is issued before the first sum.  Waves 0-1 finish the online h4,
// waves 2-3 the target's (four hidden units a thread) into LDS; wave w then
// computes the Q values of actions w, w + 4, ... of both networks (lane l:
// units 8l .. 8l + 7 of one W5 row, then the butterfly sum -- the same
// arithmetic, in the same order, as one wave per row); every thread forms the
// TD error from the Q values in LDS, and waves 0-1 write dz4.
constexpr int TD_JB = 3;  // actions per wave whose W5 rows are loaded together (A <= 12: one round trip)
__global__ __launch_bounds__(256) void td_head_kernel(
    const float* __restrict__ fc1part, const float* __restrict__ fc1part_t, int64_t part_stride,
    int splits, GroupPtrs thetas, const float* __restrict__ theta_t, int n, int A,
    const int32_t* __restrict__ a, const float* __restrict__ r, const uint8_t* __restrict__ term,
    float gamma, float clip, float* __restrict__ h4, float* __restrict__ q,
    float* __restrict__ ell, float* __restrict__ coef, float* __restrict__ td,
    float* __restrict__ dz4) {
    __shared__ __attribute__((aligned(16))) float hs[2][HID];  // online, target h4
    __shared__ float qv[2][MAX_ACTIONS];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bl = blockIdx.x, grp = blockIdx.y;
    const float* theta = thetas.p[grp];
    const int64_t b = (int64_t)grp * n + bl;  // learner row
    const int ab = a[b];
    const float* W5 = theta + OFF_W5;
    const float* b5 = theta + off_b5(A);
    const float* W5t = theta_t + OFF_W5;
    const float* b5t = theta_t + off_b5(A);

    // loads that do not depend on h4: this thread's network and units
    const bool tgt = tid >= 128;
    const int u = 4 * (tid & 127);
    const int64_t ss = (int64_t)n * HID;
    const float* pp = (tgt ? fc1part_t : fc1part) + grp * part_stride + (int64_t)bl * HID + u;
    f32x4 pa[FC1_MAX_SPLITS];
#pragma unroll
    for (int s = 0; s < FC1_MAX_SPLITS; ++s)
        if (s < splits) pa[s] = ld4(pp + s * ss);
    const f32x4 bias = ld4((tgt ? theta_t : theta) + OFF_B4 + u);
    const f32x4 wa = ld4(W5 + ab * HID + u);  // the chosen action's row (online units)
    const int nk = (A - wave + 3) / 4;  // this wave's actions
    f32x4 w0[TD_JB], w1[TD_JB], v0[TD_JB], v1[TD_JB];
#pragma unroll
    for (int j = 0; j < TD_JB; ++j) {
        const int k = min(wave + 4 * j, A - 1);
        w0[j] = ld4(W5 + k * HID + lane * 8);
        w1[j] = ld4(W5 + k * HID + lane * 8 + 4);
        v0[j] = ld4(W5t + k * HID + lane * 8);
        v1[j] = ld4(W5t + k * HID + lane * 8 + 4);
    }

    // h4 = relu(b4 + sum of the split partials in split order)
    f32x4 hv = pa[0];
#pragma unroll
    for (int s = 1; s < FC1_MAX_SPLITS; ++s)
        if (s < splits) hv += pa[s];
    hv = f32x4{fmaxf(hv[0] + bias[0], 0.f), fmaxf(hv[1] + bias[1], 0.f),
               fmaxf(hv[2] + bias[2], 0.f), fmaxf(hv[3] + bias[3], 0.f)};
    *(f32x4*)&hs[tgt][u] = hv;
    if (!tgt) *(f32x4*)(h4 + b * HID + u) = hv;
    __syncthreads();

    // Q of this wave's actions for both networks
    float h[8], hh[8];
    {
        const f32x4 x0 = *(const f32x4*)&hs[0][lane * 8], x1 = *(const f32x4*)&hs[0][lane * 8 + 4];
        const f32x4 y0 = *(const f32x4*)&hs[1][lane * 8], y1 = *(const f32x4*)&hs[1][lane * 8 + 4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            h[e] = x0[e]; h[4 + e] = x1[e];
            hh[e] = y0[e]; hh[4 + e] = y1[e];
        }
    }
    q += (int64_t)grp * 2 * n * A;
    for (int j0 = 0; j0 < nk; j0 += TD_JB) {
        if (j0 > 0) {
#pragma unroll
            for (int j = 0; j < TD_JB; ++j) {
                const int k = min(wave + 4 * (j0 + j), A - 1);
                w0[j] = ld4(W5 + k * HID + lane * 8);
                w1[j] = ld4(W5 + k * HID + lane * 8 + 4);
                v0[j] = ld4(W5t + k * HID + lane * 8);
                v1[j] = ld4(W5t + k * HID + lane * 8 + 4);
            }
        }
        float so[TD_JB], st[TD_JB];
#pragma unroll
        for (int j = 0; j < TD_JB; ++j) {
            so[j] = dot8(h, w0[j], w1[j]);
            st[j] = dot8(hh, v0[j], v1[j]);
        }
#pragma unroll
        for (int j = 0; j < TD_JB; ++j) {
            const int k = wave + 4 * (j0 + j);
            const float qo = wave_sum(so[j]) + b5[min(k, A - 1)];
            const float qt = wave_sum(st[j]) + b5t[min(k, A - 1)];
            if (j0 + j < nk && lane == 0) {
                qv[0][k] = qo;
                qv[1][k] = qt;
                q[(int64_t)bl * A + k] = qo;
                q[(int64_t)(n + bl) * A + k] = qt;
            }
        }
    }
    __syncthreads();

    // TD error, Huber loss and dLoss/dQ(s, a) (every thread, the same values)
    float m = qv[1][0];
    for (int k = 1; k < A; ++k) m = fmaxf(m, qv[1][k]);  // max_a' Q(s', a'; theta-)
    const float q_sa = qv[0][ab];
    const float y = term[b] ? r[b] : r[b] + gamma * m;
    const float d = y - q_sa;
    const float ad = fabsf(d);
    const float g = fminf(fmaxf(d, -clip), clip);
    const float cf = -g / (float)n;  // d(mean loss)/dQ(s, a)
    if (tid == 0) {
        const float l = ad <= clip ? 0.5f * d * d : clip * ad - 0.5f * clip * clip;
        ell[b] = l;
        coef[b] = cf;
        *(f32x4*)(td + 4 * b) = f32x4{m, y, d, l};
    }
    if (!tgt)
        *(f32x4*)(dz4 + b * HID + u) = f32x4{hv[0] > 0.f ? cf * wa[0] : 0.f, hv[1] > 0.f ? cf * wa[1] : 0.f,
                                             hv[2] > 0.f ? cf * wa[2] : 0.f, hv[3] > 0.f ? cf * wa[3] : 0.f};
}

void launch_td_head(const float* fc1part_online, const float* fc1part_target, int64_t part_stride,
                    int splits, const GroupPtrs& thetas, int groups, const float* theta_target,
                    int n, int A, const int32_t* a, const float* r, const uint8_t* term,
                    float gamma, float clip, float* h4, float* q, float* ell, float* coef,
                    float* td, float* dz4, hipStream_t st) {
    if (n <= 0) return;
    static_assert(4 * 128 == HID, "four hidden units a thread, two networks");
    td_head_kernel<<<dim3(n, groups), 256, 0, st>>>(
        fc1part_online, fc1part_target, part_stride, splits, thetas, theta_target, n, A, a, r, term,
        gamma, clip, h4, q, ell, coef, td, dz4);
}

}  // namespace gorila
