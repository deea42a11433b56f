// Parameter-server side of the learner loop (Section 4, parameter server;
// Section 4.2, stability): the loss-statistics gradient filter and the
// AdaGrad apply of learner gradients to theta+ with stale-gradient discard.
//
// Both are HBM or latency bound, not matrix work: the apply streams theta+,
// the AdaGrad accumulator and every accepted gradient once (fp32, coalesced
// vectors of up to four elements per lane, many loads per thread in flight),
// applying the accepted gradients in index order to each element.
#include "common.h"
#include "kernels.h"

namespace gorila {

// One thread per learner.  Statistics (n, mean, var) of |loss| in fp64;
// every operation rounds once (no contraction into fused multiply-adds), so
// the decision and the statistics are reproducible operation for operation.
__global__ __launch_bounds__(64) void loss_filter_kernel(double* __restrict__ stats,
                                                         const float* __restrict__ loss, int groups,
                                                         double alpha, double k, int64_t warmup,
                                                         uint8_t* __restrict__ keep) {
#pragma clang fp contract(off)
    const int g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= groups) return;
    double* st = stats + 3 * (int64_t)g;
    const double x = fabs((double)loss[g]);
    const double n = st[0], mean = st[1], var = st[2];
    bool discard = false;
    // x > mean + k sd, written without a square root: (x - mean)^2 > k^2 var
    if (n >= 1.0 && n >= (double)warmup && x > mean) {
        const double d = x - mean;
        discard = d * d > (k * k) * var;
    }
    keep[g] = discard ? 0 : 1;
    double m1, v1;
    if (n == 0.0) {
        m1 = x;
        v1 = 0.0;
    } else if (alpha > 0.0) {  // exponentially weighted
        const double d = x - mean;
        m1 = mean + alpha * d;
        v1 = (1.0 - alpha) * (var + (alpha * d) * d);
    } else {  // cumulative (Welford)
        const double n1 = n + 1.0;
        const double d = x - mean;
        m1 = mean + d / n1;
        v1 = (n * var + d * (x - m1)) / n1;
    }
    st[0] = n + 1.0;
    st[1] = m1;
    st[2] = v1;
}

void launch_loss_filter(double* stats, const float* loss, int groups, double alpha, double k,
                        int64_t warmup, uint8_t* keep, hipStream_t st) {
    if (groups <= 0) return;
    loss_filter_kernel<<<(groups + 63) / 64, 64, 0, st>>>(stats, loss, groups, alpha, k, warmup,
                                                          keep);
}

// Which gradients the server applies, in index order: gradient g is applied
// iff keep[g] and the server version at its turn minus version[g] is within
// max_delay; each applied gradient advances the version.  The decisions form
// a chain: one workgroup loads 256 entries at a time in parallel into LDS, one
// thread walks them into a bit mask in LDS.  Returns the version after the
// walk (to thread 0).
__device__ int64_t plan_chain(const uint8_t* __restrict__ keep, const int64_t* __restrict__ version,
                              int groups, const int64_t* __restrict__ ps_version, int64_t max_delay,
                              uint32_t* mask, int mask_words) {
    __shared__ int64_t sver[256];
    __shared__ uint8_t skeep[256];
    const int tid = threadIdx.x;
    for (int w = tid; w < mask_words; w += 256) mask[w] = 0;
    int64_t v = tid == 0 ? *ps_version : 0;
    for (int g0 = 0; g0 < groups; g0 += 256) {
        const int g = g0 + tid;
        if (g < groups) {
            sver[tid] = version[g];
            skeep[tid] = keep ? keep[g] : 1;
        }
        __syncthreads();
        if (tid == 0) {
            const int m = groups - g0 < 256 ? groups - g0 : 256;
            for (int j = 0; j < m; ++j)
                if (skeep[j] && v - sver[j] <= max_delay) {
                    mask[(g0 + j) >> 5] |= 1u << ((g0 + j) & 31);
                    ++v;
                }
        }
        __syncthreads();
    }
    return v;
}

constexpr int PS_ELEMS = 4;   // elements per thread per pass
constexpr int PS_CHUNK = 4;   // gradients whose values are loaded together
constexpr int PS_MAX_GROUPS = 4096;  // GORILA_PS_MAX_GROUPS
constexpr int PS_MASK_WORDS = PS_MAX_GROUPS / 32;

typedef float f32x2 __attribute__((ext_vector_type(2)));

// Load / store VEC consecutive floats at vector index i (a 32-bit index, so
// a uniform row base plus a per-lane offset addresses every access).
template <int VEC> struct VecIO;
template <> struct VecIO<1> {
    __device__ static void load(const float* p, uint32_t i, float* o) { o[0] = p[i]; }
    __device__ static void store(float* p, uint32_t i, const float* v) { p[i] = v[0]; }
};
template <> struct VecIO<2> {
    __device__ static void load(const float* p, uint32_t i, float* o) {
        const f32x2 v = reinterpret_cast<const f32x2*>(p)[i];
        o[0] = v[0];
        o[1] = v[1];
    }
    __device__ static void store(float* p, uint32_t i, const float* v) {
        reinterpret_cast<f32x2*>(p)[i] = f32x2{v[0], v[1]};
    }
};
template <> struct VecIO<4> {
    __device__ static void load(const float* p, uint32_t i, float* o) {
        const f32x4 v = reinterpret_cast<const f32x4*>(p)[i];
        o[0] = v[0];
        o[1] = v[1];
        o[2] = v[2];
        o[3] = v[3];
    }
    __device__ static void store(float* p, uint32_t i, const float* v) {
        reinterpret_cast<f32x4*>(p)[i] = f32x4{v[0], v[1], v[2], v[3]};
    }
};

// One workgroup: the decisions into applied [groups] and the new version.
__global__ __launch_bounds__(256) void ps_plan_kernel(const uint8_t* __restrict__ keep,
                                                      const int64_t* __restrict__ version,
                                                      int groups, int64_t* __restrict__ ps_version,
                                                      int64_t max_delay,
                                                      uint8_t* __restrict__ applied) {
    __shared__ uint32_t smask[PS_MASK_WORDS];
    const int64_t v = plan_chain(keep, version, groups, ps_version, max_delay, smask,
                                 (groups + 31) / 32);
    __syncthreads();
    for (int g = threadIdx.x; g < groups; g += 256) applied[g] = (smask[g >> 5] >> (g & 31)) & 1u;
    if (threadIdx.x == 0) *ps_version = v;
}

// AdaGrad on each element: for every applied gradient in order,
// h += g^2; theta -= lr g / (eps + sqrt(h)).  A thread owns ILP vectors of VEC
// consecutive elements; the values of up to PS_CHUNK applied gradients are
// loaded before any is used, so many independent loads are in flight.
template <int VEC>
__global__ __launch_bounds__(256) void ps_apply_kernel(float* __restrict__ theta,
                                                       float* __restrict__ accum, int64_t n,
                                                       const float* __restrict__ grads, int groups,
                                                       const uint8_t* __restrict__ applied,
                                                       float lr, float eps) {
    constexpr int ILP = PS_ELEMS / VEC;
    using IO = VecIO<VEC>;
    // n < 2^31 (checked by the caller): every vector index fits 32 bits
    const uint32_t nv = (uint32_t)(n / VEC);  // vectors (n is a multiple of VEC)
    const uint32_t stride = gridDim.x * 256u * ILP;
    for (uint32_t base = blockIdx.x * 256u * ILP + threadIdx.x; base < nv; base += stride) {
        float th[ILP][VEC], h[ILP][VEC];
        uint32_t at[ILP];  // vector index (clamped into range; stores are guarded)
        bool in[ILP];
#pragma unroll
        for (int u = 0; u < ILP; ++u) {
            const uint32_t i = base + u * 256u;
            in[u] = i < nv;
            at[u] = in[u] ? i : 0u;
            IO::load(theta, at[u], th[u]);
            IO::load(accum, at[u], h[u]);
        }
        for (int g0 = 0; g0 < groups; g0 += PS_CHUNK) {
            unsigned mask = 0;  // applied gradients of this chunk (uniform)
#pragma unroll
            for (int j = 0; j < PS_CHUNK; ++j)
                if (g0 + j < groups && applied[g0 + j]) mask |= 1u << j;
            float gv[PS_CHUNK][ILP][VEC];
#pragma unroll
            for (int j = 0; j < PS_CHUNK; ++j) {
                if (!(mask >> j & 1u)) continue;
                const float* gr = grads + (int64_t)(g0 + j) * n;
#pragma unroll
                for (int u = 0; u < ILP; ++u) IO::load(gr, at[u], gv[j][u]);
            }
#pragma unroll
            for (int j = 0; j < PS_CHUNK; ++j) {
                if (!(mask >> j & 1u)) continue;
#pragma unroll
                for (int u = 0; u < ILP; ++u)
#pragma unroll
                    for (int c = 0; c < VEC; ++c) {
                        const float gc = gv[j][u][c];
                        h[u][c] = h[u][c] + gc * gc;
                        th[u][c] = th[u][c] - lr * gc / (eps + sqrtf(h[u][c]));
                    }
            }
        }
#pragma unroll
        for (int u = 0; u < ILP; ++u)
            if (in[u]) {
                IO::store(theta, at[u], th[u]);
                IO::store(accum, at[u], h[u]);
            }
    }
}

void launch_ps_apply(float* theta, float* accum, int64_t n, const float* grads, int groups,
                     const uint8_t* keep, const int64_t* version, int64_t* ps_version,
                     int64_t max_delay, float lr, float eps, uint8_t* applied, hipStream_t st) {
    ps_plan_kernel<<<1, 256, 0, st>>>(keep, version, groups, ps_version, max_delay, applied);
    if (n <= 0 || groups <= 0) return;
    // widest vector that every row and array start allows
    const uintptr_t addr = (uintptr_t)theta | (uintptr_t)accum | (uintptr_t)grads;
    int vec = 1;
    if (n % 4 == 0 && addr % 16 == 0) vec = 4;
    else if (n % 2 == 0 && addr % 8 == 0) vec = 2;
    const int64_t per_block = 256 * (PS_ELEMS / vec);
    int64_t blocks = (n / vec + per_block - 1) / per_block;
    if (blocks > 8192) blocks = 8192;
    if (vec == 4)
        ps_apply_kernel<4><<<(int)blocks, 256, 0, st>>>(theta, accum, n, grads, groups, applied, lr,
                                                         eps);
    else if (vec == 2)
        ps_apply_kernel<2><<<(int)blocks, 256, 0, st>>>(theta, accum, n, grads, groups, applied, lr,
                                                         eps);
    else
        ps_apply_kernel<1><<<(int)blocks, 256, 0, st>>>(theta, accum, n, grads, groups, applied, lr,
                                                         eps);
}

// ---------------------------------------------------------------------------
// Parameter pull / periodic target sync (Algorithm 1: replicas update theta
// from theta+; every N global updates theta- is synced with theta+).  A copy
// is due when period == 0 or a multiple of period lies in (held version,
// current version].  The copy kernel reads src once per element and writes
// every due destination (fp32, or bf16 rounded to nearest even); a second,
// one-workgroup launch then records the versions, so no workgroup can see a
// version updated by another.
// ---------------------------------------------------------------------------
constexpr int SYNC_MAX_COPIES = 64;

__device__ inline bool sync_due(int64_t now, int64_t held, int64_t period) {
    return period == 0 || now / period > held / period;
}

__device__ inline uint16_t f32_to_bf16_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0)
        return (uint16_t)((u >> 16) | 0x0040u);  // NaN stays a quiet NaN
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

template <bool BF16>
__global__ __launch_bounds__(256) void sync_copy_kernel(const float* __restrict__ src,
                                                        void* __restrict__ dst, int64_t n,
                                                        int copies,
                                                        const int64_t* __restrict__ ps_version,
                                                        const int64_t* __restrict__ dst_version,
                                                        int64_t period) {
    __shared__ uint64_t sdue;  // bit c: destination c is due (copies <= 64)
    if (threadIdx.x == 0) {
        const int64_t now = *ps_version;
        uint64_t m = 0;
        for (int c = 0; c < copies; ++c)
            if (sync_due(now, dst_version[c], period)) m |= 1ull << c;
        sdue = m;
    }
    __syncthreads();
    const uint64_t due = sdue;
    if (!due) return;
    constexpr int ILP = 4;
    const int64_t stride = (int64_t)gridDim.x * 256 * ILP;
    for (int64_t base = (int64_t)blockIdx.x * 256 * ILP + threadIdx.x; base < n; base += stride) {
        float v[ILP];
#pragma unroll
        for (int u = 0; u < ILP; ++u) {
            const int64_t i = base + u * 256;
            v[u] = src[i < n ? i : 0];
        }
        for (int c = 0; c < copies; ++c) {
            if (!((due >> c) & 1ull)) continue;
#pragma unroll
            for (int u = 0; u < ILP; ++u) {
                const int64_t i = base + u * 256;
                if (i >= n) continue;
                if (BF16) ((uint16_t*)dst)[(int64_t)c * n + i] = f32_to_bf16_rne(v[u]);
                else ((float*)dst)[(int64_t)c * n + i] = v[u];
            }
        }
    }
}

__global__ void sync_finalize_kernel(int copies, const int64_t* __restrict__ ps_version,
                                     int64_t* __restrict__ dst_version, int64_t period,
                                     uint8_t* __restrict__ synced) {
    const int c = threadIdx.x;
    if (c >= copies) return;
    const int64_t now = *ps_version;
    const bool d = sync_due(now, dst_version[c], period);
    if (d) dst_version[c] = now;
    if (synced) synced[c] = d ? 1 : 0;
}

void launch_params_sync(const float* src, void* dst, int64_t n, int copies, bool to_bf16,
                        const int64_t* ps_version, int64_t* dst_version, int64_t period,
                        uint8_t* synced, hipStream_t st) {
    if (copies <= 0) return;
    if (n > 0) {
        int64_t blocks = (n + 256 * 4 - 1) / (256 * 4);
        if (blocks > 4096) blocks = 4096;
        if (to_bf16)
            sync_copy_kernel<true><<<(int)blocks, 256, 0, st>>>(src, dst, n, copies, ps_version,
                                                                 dst_version, period);
        else
            sync_copy_kernel<false><<<(int)blocks, 256, 0, st>>>(src, dst, n, copies, ps_version,
                                                                  dst_version, period);
    }
    sync_finalize_kernel<<<1, SYNC_MAX_COPIES, 0, st>>>(copies, ps_version, dst_version, period,
                                                        synced);
}

}  // namespace gorila
