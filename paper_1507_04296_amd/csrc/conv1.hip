// First convolution (Section 5.1: 32 filters of 4x8x8, stride 4, ReLU) on the
// raw uint8 frames, forward and weight gradient.  Bytes enter the products as
// exact integers; the 1/255 input scale is applied once in each epilogue.
#include "common.h"
#include "kernels.h"

namespace gorila {

// The layer on v_mfma_f32_32x32x16_bf16 with exact products: the bytes
// (integers 0..255) are exact bf16 values, and W1 enters as WP bf16 planes
// whose sum is W1 exactly -- one plane for bf16 parameter sets; for fp32 sets
// three (w = hi + mid + lo, each the rounded remainder of the previous: 8 + 8
// + 8 significant bits cover fp32's 24; exact for |w| above ~2^-90), so every
// product is exact and only the fp32 accumulation rounds, as in an fp32 GEMM.  A workgroup of 13 waves
// keeps the planes in LDS and walks samples b = blockIdx.x, b + gridDim.x,
// ... of its parameter set: it converts a sample's 4 frames to bf16 once, into
// LDS, fetches the next sample's frames into registers while wave t computes
// pixel tile t (32 pixels x 32 filters; the 13th tile is half full).  One
// 16-wide MFMA step covers two filter rows (c, u) of 8 columns v: lane half h
// takes row 2 * step + h, so a lane's eight operands are eight consecutive
// bf16 pixels of one input row.
constexpr int C1F_WAVES = (P1 + 31) / 32;  // 13
constexpr int C1F_THREADS = 64 * C1F_WAVES;
constexpr int C1F_WLD = 256 + 8;           // W1 row stride in LDS (bf16): 528 bytes
constexpr int C1F_XV = STATE_BYTES / 16;   // 1764 16-byte vectors per sample
constexpr int C1F_XPT = (C1F_XV + C1F_THREADS - 1) / C1F_THREADS;
// resident workgroups: two per CU with one plane (73 KB of LDS), one with three
__host__ __device__ constexpr int c1f_target_wgs(int wp) { return wp == 1 ? 512 : 256; }

template <int WP>
__launch_bounds__(C1F_THREADS) __global__ void conv1_fwd_mfma16_kernel(
    const uint8_t* const* __restrict__ ftab, GroupPtrs theta, int n, float* __restrict__ h1) {
    __shared__ __attribute__((aligned(16))) __bf16 xs[STATE_BYTES];
    __shared__ __attribute__((aligned(16))) __bf16 ws[WP][C1 * C1F_WLD];
    __shared__ float bs[C1];
    const int g = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float* W1 = theta.p[g];

    uint4 xv[C1F_XPT];
    unsigned okm = 0;  // bit k: xv[k] holds frame bytes (else zeros)
    // The sample's 16-byte vectors of this thread.  Branch-free, so all of
    // them are in flight together: the four frame pointers are read first (the
    // same for every thread), a null frame reads W1 instead and is zeroed when
    // converted (not here, which would wait for the loads).
    auto fetch = [&](int b) {
        const uint8_t* const* fr = ftab + ((int64_t)g * n + b) * 4;
        const uint8_t* f0 = fr[0];
        const uint8_t* f1 = fr[1];
        const uint8_t* f2 = fr[2];
        const uint8_t* f3 = fr[3];
#pragma unroll
        for (int k = 0; k < C1F_XPT; ++k) {
            const int e = tid + k * C1F_THREADS;  // vector e: frame e / 441
            const int fi = e / (FRAME_BYTES / 16);
            const uint8_t* f = fi == 0 ? f0 : fi == 1 ? f1 : fi == 2 ? f2 : f3;
            const bool ok = e < C1F_XV && f != nullptr;
            xv[k] = ldg_u4(ok ? (const uint4*)f + (e - fi * (FRAME_BYTES / 16))
                              : (const uint4*)(W1 + OFF_W1));
            okm = k == 0 ? (unsigned)ok : okm | ((unsigned)ok << k);
        }
    };
    fetch(blockIdx.x);

    constexpr int WQ = C1 * 256 / 4;  // 2048 weight quads
    for (int q = tid; q < WQ; q += C1F_THREADS) {
        f32x4 w = ld4(W1 + OFF_W1 + 4 * q);
#pragma unroll
        for (int pl = 0; pl < WP; ++pl) {
            bf16x4 v;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = (__bf16)w[i];
                w[i] -= (float)v[i];  // exact: the remainder has at most 16 significant bits
            }
            *(bf16x4*)(ws[pl] + (q >> 6) * C1F_WLD + 4 * (q & 63)) = v;
        }
    }
    if (tid < C1) bs[tid] = W1[OFF_B1 + tid];
    const int col = lane & 31, h = lane >> 5;

    int m = wave * 32 + (lane & 31);
    if (m >= P1) m = 0;  // padding rows compute on a valid pixel, never stored
    const int i = m / H1, j = m - i * H1;
    const __bf16* xb = xs + (S1 * i) * IN_W + S1 * j;  // 8-byte aligned
    const int wofs = col * C1F_WLD + 8 * h;             // 16-byte aligned

    for (int b = blockIdx.x; b < n; b += gridDim.x) {
#pragma unroll
        for (int k = 0; k < C1F_XPT; ++k) {
            const int e = tid + k * C1F_THREADS;
            if (e < C1F_XV) {
                const uint4 v = (okm >> k) & 1u ? xv[k] : make_uint4(0, 0, 0, 0);
                const uint32_t d[4] = {v.x, v.y, v.z, v.w};
                bf16x8 lo, hi;
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    lo[t] = (__bf16)(float)((d[t >> 2] >> (8 * (t & 3))) & 255u);
                    hi[t] = (__bf16)(float)((d[2 + (t >> 2)] >> (8 * (t & 3))) & 255u);
                }
                *(bf16x8*)(xs + 16 * e) = lo;
                *(bf16x8*)(xs + 16 * e + 8) = hi;
            }
        }
        __syncthreads();
        if (b + (int)gridDim.x < n) fetch(b + gridDim.x);  // in flight during the products

        f32x16 acc = f32x16{};
#pragma unroll
        for (int st = 0; st < 16; ++st) {
            const int cb = 2 * st + h, c = cb >> 3, u = cb & 7;
            const __bf16* px = xb + c * FRAME_BYTES + u * IN_W;
            const bf16x4 x0 = *(const bf16x4*)px, x1 = *(const bf16x4*)(px + 4);
            const bf16x8 x = __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
            for (int pl = 0; pl < WP; ++pl) {
                const bf16x8 w = *(const bf16x8*)(ws[pl] + wofs + 16 * st);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, w, acc, 0, 0, 0);
            }
        }
        float* out = h1 + ((int64_t)g * n + b) * P1 * C1 + (wave * 32 + 4 * h) * C1 + col;
        const float bias = bs[col];
        if (wave < C1F_WAVES - 1) {  // full tiles: no per-store conditions
#pragma unroll
            for (int r = 0; r < 16; ++r)
                out[(8 * (r >> 2) + (r & 3)) * C1] = fmaxf(acc[r] * (1.0f / 255.0f) + bias, 0.0f);
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (wave * 32 + 8 * (r >> 2) + 4 * h + (r & 3) < P1)
                    out[(8 * (r >> 2) + (r & 3)) * C1] = fmaxf(acc[r] * (1.0f / 255.0f) + bias, 0.0f);
        }
        __syncthreads();  // every wave is done with xs before the next sample lands
    }
}

void launch_conv1_fwd(const uint8_t* const* ftab, const GroupPtrs& theta, int groups, int n,
                      float* h1, bool bf16, hipStream_t st) {
    if (n <= 0) return;
    // one round of resident workgroups, each walking its set's samples
    if (bf16) {
        const int per_group = max(1, min(n, c1f_target_wgs(1) / groups));
        conv1_fwd_mfma16_kernel<1><<<dim3(per_group, groups), C1F_THREADS, 0, st>>>(ftab, theta, n, h1);
    } else {
        const int per_group = max(1, min(n, c1f_target_wgs(3) / groups));
        conv1_fwd_mfma16_kernel<3><<<dim3(per_group, groups), C1F_THREADS, 0, st>>>(ftab, theta, n, h1);
    }
}

// The weight gradient on v_mfma_f32_32x32x16_bf16 with exact products:
// dW1[o][n] for the 256 columns n = (c, u, v) is a sum over pixels of
// dz1[pixel][o] * byte.  The bytes are exact bf16 values; dz1 enters as WP
// bf16 planes whose sum is dz1 exactly (three for fp32 steps, as in the
// forward kernel; one, rounded, for bf16 steps), so only the fp32
// accumulation rounds.  The stride-4 columns are made contiguous by staging
// each input row in LDS by phase: xs[c][r][m][s][q] = row r byte 4 (q + s) + m,
// so the bytes of columns v = 4s + m at pixels j .. j+7 are eight consecutive
// entries.  A unit is two output rows of one sample (40 pixels, padded to 2 x
// 24 = 6 groups of 8, with zeros past j = 19); an MFMA step takes two groups
// (lane half h: group 2 step + h), so a unit is three steps.  Each workgroup
// (4 waves; wave w owns columns 64 w .. 64 w + 63) sums a contiguous range of
// units of one parameter set into its partial [32][256]; db1 is summed from
// the fp32 dz1 values as they are staged.  The LDS stage is double buffered
// and the next unit's data is fetched into registers during the products.
constexpr int C1W_UR = 2;                       // output rows per unit
constexpr int C1W_UNITS = H1 / C1W_UR;          // 10 units per sample
constexpr int C1W_JP = 24;                      // padded pixel columns per output row
constexpr int C1W_XR = S1 * (C1W_UR - 1) + K1;  // 12 input rows per unit
constexpr int C1W_DQ = C1W_UR * H1 * C1 / 4;    // 320 dz1 quads per unit
constexpr int C1W_XW = IN_C * C1W_XR * IN_W / 4;  // 1008 input words per unit
constexpr int C1W_TARGET = 512;                 // workgroups: two per CU

template <int WP>
struct C1wStage {
    __bf16 d[WP][C1][C1W_UR * C1W_JP];          // dz1 planes [o][(row, j)]
    __bf16 x[IN_C][C1W_XR][4][2][C1W_JP];      // [c][r][m][s][q]
};

template <int WP>
__global__ __launch_bounds__(256) void conv1_wgrad_mfma16_kernel(
    const float* __restrict__ dz1, const uint8_t* const* __restrict__ ftab, int n,
    float* __restrict__ partial, float* __restrict__ bias_part) {
    __shared__ __attribute__((aligned(16))) C1wStage<WP> stg[2];
    __shared__ float bred[256 / 8][C1];
    const int g = blockIdx.y, S = gridDim.x, x = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int U = n * C1W_UNITS;
    const int u0 = (int)((int64_t)x * U / S), u1 = (int)((int64_t)(x + 1) * U / S);

    for (int e = tid; e < (int)(sizeof(stg) / 16); e += 256) ((uint4*)stg)[e] = make_uint4(0, 0, 0, 0);

    // prefetch registers: two dz1 quads (pixels 2p and 2p + 1 of the unit,
    // channels 4 (t % 8) .. +3; threads t < 160) and four input words
    const bool dz_lane = tid < C1W_DQ / 2;
    const int dq0 = (tid >> 3) * 16 + (tid & 7);  // quad of pixel 2p (8 quads a pixel)
    f32x4 dq[2];
    uint32_t xw[4];
    auto fetch = [&](int u) {
        const int b = u / C1W_UNITS, i0 = (u - b * C1W_UNITS) * C1W_UR;
        const float* dsrc = dz1 + (((int64_t)g * n + b) * P1 + i0 * H1) * C1;
#pragma unroll
        for (int k = 0; k < 2; ++k) dq[k] = ld4(dsrc + 4 * (dz_lane ? dq0 + 8 * k : 0));
        const uint8_t* const* fr = ftab + ((int64_t)g * n + b) * 4;
        const uint8_t* f0 = fr[0];
        const uint8_t* f1 = fr[1];
        const uint8_t* f2 = fr[2];
        const uint8_t* f3 = fr[3];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int w = tid + 256 * k;  // word w: channel w / 252
            const int c = w / (C1W_XW / IN_C);
            const uint8_t* f = c == 0 ? f0 : c == 1 ? f1 : c == 2 ? f2 : f3;
            const bool ok = w < C1W_XW && f != nullptr;
            const int wi = w - c * (C1W_XW / IN_C);
            // branch-free: a null frame or a spare lane reads dz1 instead
            const uint32_t v = ldg_u32(ok ? f + S1 * i0 * IN_W + 4 * wi : (const uint8_t*)dsrc);
            xw[k] = ok ? v : 0u;
        }
    };
    float bsum[4] = {0.f, 0.f, 0.f, 0.f};  // db1 of o = 4 (tid % 8) + e
    auto stage = [&](C1wStage<WP>& sg) {
        if (dz_lane) {  // two pixels, one packed pair of columns per channel and plane
            const int pu = 2 * (tid >> 3), o0 = 4 * (tid & 7);
            const int col = (pu / H1) * C1W_JP + pu % H1;  // even
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float v0 = dq[0][e], v1 = dq[1][e];
                bsum[e] += v0;
                bsum[e] += v1;
#pragma unroll
                for (int pl = 0; pl < WP; ++pl) {
                    const __bf16 h0 = (__bf16)v0, h1 = (__bf16)v1;
                    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
                    *(bf16x2*)&sg.d[pl][o0 + e][col] = bf16x2{h0, h1};
                    v0 -= (float)h0;  // exact remainders
                    v1 -= (float)h1;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int w = tid + 256 * k;
            if (w < C1W_XW) {
                const int c = w / (C1W_XW / IN_C), wi = w - c * (C1W_XW / IN_C);
                const int r = (4 * wi) / IN_W, q0 = ((4 * wi) % IN_W) / 4;
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const __bf16 h = (__bf16)(float)((xw[k] >> (8 * m)) & 255u);
                    sg.x[c][r][m][0][q0] = h;
                    if (q0 > 0) sg.x[c][r][m][1][q0 - 1] = h;
                }
            }
        }
    };

    f32x16 acc[2] = {f32x16{}, f32x16{}};
    const int h = lane >> 5;
    if (u0 < u1) fetch(u0);
    __syncthreads();  // the zero fill is complete
    for (int u = u0; u < u1; ++u) {
        C1wStage<WP>& sg = stg[u & 1];
        stage(sg);
        __syncthreads();
        if (u + 1 < u1) fetch(u + 1);
#pragma unroll
        for (int st = 0; st < 3; ++st) {
            const int grp = 2 * st + h, ir = grp / 3, j0 = 8 * (grp % 3);
            bf16x8 a[WP];
#pragma unroll
            for (int pl = 0; pl < WP; ++pl)
                a[pl] = *(const bf16x8*)&sg.d[pl][lane & 31][ir * C1W_JP + j0];
#pragma unroll
            for (int tt = 0; tt < 2; ++tt) {
                const int nc = 64 * wave + 32 * tt + (lane & 31);
                const int c = nc >> 6, uu = (nc >> 3) & 7, v = nc & 7;
                const bf16x8 bx = *(const bf16x8*)&sg.x[c][S1 * ir + uu][v & 3][v >> 2][j0];
#pragma unroll
                for (int pl = 0; pl < WP; ++pl)
                    acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[pl], bx, acc[tt], 0, 0, 0);
            }
        }
    }

    const int split = g * S + x;
    float* out = partial + (int64_t)split * C1 * 256;
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            out[(8 * (r >> 2) + 4 * h + (r & 3)) * 256 + 64 * wave + 32 * tt + (lane & 31)] =
                acc[tt][r] * (1.0f / 255.0f);
#pragma unroll
    for (int e = 0; e < 4; ++e) bred[tid >> 3][4 * (tid & 7) + e] = bsum[e];
    __syncthreads();
    if (tid < C1) {
        float t = 0.0f;
        for (int k = 0; k < 256 / 8; ++k) t += bred[k][tid];
        bias_part[(int64_t)split * 64 + tid] = t;
    }
}

void launch_conv1_wgrad(const float* dz1, const uint8_t* const* ftab, int groups, int n,
                        float* partial, float* bias_part, int max_splits, int* splits_out,
                        bool bf16, hipStream_t st) {
    if (n <= 0) {
        *splits_out = 0;
        return;
    }
    // splits per group: one round of two workgroups per CU, each over a
    // contiguous range of at least two units (at batch 32 one unit each left
    // the final reduction 320 partials per element: 10 -> 8 us for it, +0.5
    // here); groups * splits stays within max_splits
    const int splits = max(1, min((n * C1W_UNITS + 1) / 2, min(C1W_TARGET, max_splits) / groups));
    *splits_out = splits;
    if (bf16)
        conv1_wgrad_mfma16_kernel<1><<<dim3(splits, groups), 256, 0, st>>>(dz1, ftab, n, partial, bias_part);
    else
        conv1_wgrad_mfma16_kernel<3><<<dim3(splits, groups), 256, 0, st>>>(dz1, ftab, n, partial, bias_part);
}

}  // namespace gorila
