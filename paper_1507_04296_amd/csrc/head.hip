// Action head (linear FC 512 -> A, Section 4.1) and what follows it:
//  - Q values;
//  - epsilon-greedy actions (Algorithm 1);
//  - the DQN TD target y = r + gamma (1 - term) max_a' Q(s', a'; theta-),
//    TD error delta = y - Q(s, a; theta), Huber loss and dLoss/dQ (eq. (1),
//    (2); Algorithm 1's terminal case), fused with the action-head backward
//    dz4 = dLoss/dQ(s,a) * W5[a][:] * [h4 > 0].
// One wave64 per sample: lane l holds h4[8l .. 8l+7]; each of the A dot
// products is a butterfly sum over the wave, so every lane ends with the same
// bit pattern and the result does not depend on scheduling.
#include "common.h"
#include "kernels.h"

namespace gorila {

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ inline float dot8(const float* h, const float* w) {
    const f32x4 w0 = ld4(w), w1 = ld4(w + 4);
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

__device__ inline void load8(const float* p, float* h) {
    const f32x4 a = ld4(p), b = ld4(p + 4);
    h[0] = a[0]; h[1] = a[1]; h[2] = a[2]; h[3] = a[3];
    h[4] = b[0]; h[5] = b[1]; h[6] = b[2]; h[7] = b[3];
}

// SplitMix64 output function (Steele, Lea and Flood 2014).
__device__ inline uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void q_head_kernel(const float* __restrict__ h4,
                                                     const float* __restrict__ theta, int n, int A,
                                                     float* __restrict__ q,
                                                     int32_t* __restrict__ actions,
                                                     uint64_t explore_below, uint64_t seed) {
    const int lane = threadIdx.x & 63, b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= n) return;
    float h[8];
    load8(h4 + (int64_t)b * HID + lane * 8, h);
    const float* W5 = theta + OFF_W5;
    const float* b5 = theta + off_b5(A);
    float best = 0.0f;
    int best_a = 0;
    for (int k = 0; k < A; ++k) {
        const float s = wave_sum(dot8(h, W5 + k * HID + lane * 8)) + b5[k];
        if (q && lane == 0) q[(int64_t)b * A + k] = s;
        if (k == 0 || s > best) { best = s; best_a = k; }  // lowest index among the maxima
    }
    if (actions && lane == 0) {
        const uint64_t G = 0x9E3779B97F4A7C15ull;
        const uint64_t u = splitmix64_mix(seed + (2ull * (uint64_t)b + 1ull) * G);
        const uint64_t v = splitmix64_mix(seed + (2ull * (uint64_t)b + 2ull) * G);
        const bool explore = (u >> 11) < explore_below;
        actions[b] = explore ? (int32_t)(((v >> 32) * (uint64_t)A) >> 32) : best_a;
    }
}

void launch_q_head(const float* h4, const float* theta, int n, int A, float* q, hipStream_t st) {
    if (n <= 0) return;
    q_head_kernel<<<(n + 3) / 4, 256, 0, st>>>(h4, theta, n, A, q, nullptr, 0, 0);
}

void launch_act_head(const float* h4, const float* theta, int n, int A, float eps, uint64_t seed,
                     int32_t* actions, float* q_out, hipStream_t st) {
    if (n <= 0) return;
    // explore iff a uniform 53-bit integer is below floor(eps * 2^53); eps is
    // exact in double and the scaling by 2^53 is exact.
    const uint64_t below = (uint64_t)floor((double)eps * 9007199254740992.0);
    q_head_kernel<<<(n + 3) / 4, 256, 0, st>>>(h4, theta, n, A, q_out, actions, below, seed);
}

// h4 holds 2n rows: online rows [0, n) on s, target rows [n, 2n) on s'.
__global__ __launch_bounds__(256) void td_head_kernel(
    const float* __restrict__ h4, const float* __restrict__ theta,
    const float* __restrict__ theta_t, int n, int A, const int32_t* __restrict__ a,
    const float* __restrict__ r, const uint8_t* __restrict__ term, float gamma, float clip,
    float* __restrict__ q, float* __restrict__ ell, float* __restrict__ coef,
    float* __restrict__ dz4) {
    const int lane = threadIdx.x & 63, b = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= n) return;
    float h[8], ht[8];
    load8(h4 + (int64_t)b * HID + lane * 8, h);
    load8(h4 + (int64_t)(n + b) * HID + lane * 8, ht);
    const float* W5 = theta + OFF_W5;
    const float* b5 = theta + off_b5(A);
    const float* W5t = theta_t + OFF_W5;
    const float* b5t = theta_t + off_b5(A);
    const int ab = a[b];
    float q_sa = 0.0f, m = 0.0f;
    for (int k = 0; k < A; ++k) {
        const float s = wave_sum(dot8(h, W5 + k * HID + lane * 8)) + b5[k];
        const float st = wave_sum(dot8(ht, W5t + k * HID + lane * 8)) + b5t[k];
        if (lane == 0) {
            q[(int64_t)b * A + k] = s;
            q[(int64_t)(n + b) * A + k] = st;
        }
        if (k == ab) q_sa = s;
        m = k == 0 ? st : fmaxf(m, st);  // max_a' Q(s', a'; theta-)
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
    float* out = dz4 + (int64_t)b * HID + lane * 8;
    const f32x4 w0 = ld4(w), w1 = ld4(w + 4);
    const f32x4 o0 = {h[0] > 0.f ? cf * w0[0] : 0.f, h[1] > 0.f ? cf * w0[1] : 0.f,
                      h[2] > 0.f ? cf * w0[2] : 0.f, h[3] > 0.f ? cf * w0[3] : 0.f};
    const f32x4 o1 = {h[4] > 0.f ? cf * w1[0] : 0.f, h[5] > 0.f ? cf * w1[1] : 0.f,
                      h[6] > 0.f ? cf * w1[2] : 0.f, h[7] > 0.f ? cf * w1[3] : 0.f};
    *(f32x4*)out = o0;
    *(f32x4*)(out + 4) = o1;
}

void launch_td_head(const float* h4, const float* theta, const float* theta_target, int n, int A,
                    const int32_t* a, const float* r, const uint8_t* term, float gamma, float clip,
                    float* q, float* ell, float* coef, float* dz4, hipStream_t st) {
    if (n <= 0) return;
    td_head_kernel<<<(n + 3) / 4, 256, 0, st>>>(h4, theta, theta_target, n, A, a, r, term, gamma,
                                                clip, q, ell, coef, dz4);
}

// dW5[k][:] = sum_{b: a_b = k} coef_b h4[b][:], db5[k] = sum_{b: a_b = k} coef_b,
// db4 = sum_b dz4[b][:], loss = mean_b ell_b.  Block k < A does row k of dW5;
// block A does db4, db5 and the loss.  Every sum runs over b in order.
__global__ __launch_bounds__(256) void head_reduce_kernel(
    const float* __restrict__ h4, const float* __restrict__ dz4, const int32_t* __restrict__ a,
    const float* __restrict__ coef, const float* __restrict__ ell, int n, int A,
    float* __restrict__ grads, float* __restrict__ loss_out) {
    const int blk = blockIdx.x, tid = threadIdx.x;
    if (blk < A) {
        for (int k = tid; k < HID; k += 256) {
            float s = 0.0f;
            for (int b = 0; b < n; ++b)
                if (a[b] == blk) s = fmaf(coef[b], h4[(int64_t)b * HID + k], s);
            grads[OFF_W5 + (int64_t)blk * HID + k] = s;
        }
        return;
    }
    for (int k = tid; k < HID; k += 256) {
        float s = 0.0f;
        for (int b = 0; b < n; ++b) s += dz4[(int64_t)b * HID + k];
        grads[OFF_B4 + k] = s;
    }
    if (tid < A) {
        float s = 0.0f;
        for (int b = 0; b < n; ++b)
            if (a[b] == tid) s += coef[b];
        grads[off_b5(A) + tid] = s;
    }
    if (tid == 255) {
        double s = 0.0;
        for (int b = 0; b < n; ++b) s += (double)ell[b];
        loss_out[0] = (float)(s / (double)n);
    }
}

void launch_head_reduce(const float* h4, const float* dz4, const int32_t* a, const float* coef,
                        const float* ell, int n, int A, float* grads, float* loss_out,
                        hipStream_t st) {
    if (n <= 0) return;
    head_reduce_kernel<<<A + 1, 256, 0, st>>>(h4, dz4, a, coef, ell, n, A, grads, loss_out);
}

}  // namespace gorila
