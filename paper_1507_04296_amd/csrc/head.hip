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

// Partial sums of the action-head gradients and the loss over blocks of rows:
//   hpart[bb][a*512 + k] = sum_{b in block bb, a_b = a} coef_b h4[b][k]   (dW5)
//   hpart[bb][HP_DB5 + a] = sum_{b in block bb, a_b = a} coef_b           (db5)
//   hpart[bb][HP_LOSS]    = sum_{b in block bb} ell_b                     (loss)
// Grid (8 column tiles, row blocks).  Thread (column kl, lane group bq) adds
// rows bq, bq+4, ... of its block in order into its own LDS slots; the four
// lane groups are added in order, so every sum is deterministic.  The blocks
// are summed in order by the final gradient reduction.
__global__ __launch_bounds__(256) void head_partial_kernel(
    const float* __restrict__ h4, const int32_t* __restrict__ a, const float* __restrict__ coef,
    const float* __restrict__ ell, int n, int A, int rows_per_block, float* __restrict__ hpart) {
    __shared__ float sacc[4][MAX_ACTIONS][64];
    const int tid = threadIdx.x, kl = tid & 63, bq = tid >> 6;
    const int k = blockIdx.x * 64 + kl, bb = blockIdx.y;
    const int b0 = bb * rows_per_block, b1 = min(n, b0 + rows_per_block);
    float* out = hpart + (int64_t)bb * HP_STRIDE;
    for (int j = 0; j < A; ++j) sacc[bq][j][kl] = 0.0f;
    for (int b = b0 + bq; b < b1; b += 4) {
        const int ab = a[b];
        sacc[bq][ab][kl] = fmaf(coef[b], h4[(int64_t)b * HID + k], sacc[bq][ab][kl]);
    }
    __syncthreads();
    for (int e = tid; e < A * 64; e += 256) {
        const int j = e >> 6, kk = e & 63;
        out[j * HID + blockIdx.x * 64 + kk] =
            ((sacc[0][j][kk] + sacc[1][j][kk]) + sacc[2][j][kk]) + sacc[3][j][kk];
    }
    if (blockIdx.x == 0) {
        // wave w: actions j = w, w+4, ...; lane l: rows b0+l, b0+l+64, ...
        const int lane = tid & 63, w = tid >> 6;
        for (int j = w; j < A; j += 4) {
            float s = 0.0f;
            for (int b = b0 + lane; b < b1; b += 64)
                if (a[b] == j) s += coef[b];
            s = wave_sum(s);
            if (lane == 0) out[HP_DB5 + j] = s;
        }
        if (w == 0) {
            float s = 0.0f;
            for (int b = b0 + lane; b < b1; b += 64) s += ell[b];
            s = wave_sum(s);
            if (lane == 0) out[HP_LOSS] = s;
        }
    }
}

int launch_head_partial(const float* h4, const int32_t* a, const float* coef, const float* ell,
                        int n, int A, float* hpart, hipStream_t st) {
    if (n <= 0) return 0;
    int rows = max(32, (n + HEAD_MAX_BLOCKS - 1) / HEAD_MAX_BLOCKS);
    const int blocks = (n + rows - 1) / rows;
    head_partial_kernel<<<dim3(HID / 64, blocks), 256, 0, st>>>(h4, a, coef, ell, n, A, rows, hpart);
    return blocks;
}

}  // namespace gorila
