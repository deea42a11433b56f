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

// Weight gradient: dW1[o][(c,u,v)] = (1/255) sum_pixels dz1[pixel][o] * x[c][4i+u][4j+v]
// over every pixel of the n online samples.  Rows o (32), columns (c,u,v)
// (256, two tiles of 128), reduction over pixels split across workgroups;
// partial[split][o][k] is summed in a fixed order afterwards.
struct Conv1WgradA {  // dz1 rows o, RMAJ quads along o at one pixel
    const float* dz1;
    int npix;
    int o0[MAXQ];
    int kk[MAXQ];
    __device__ void init(int j, int row, int k) { o0[j] = row; kk[j] = k; }
    __device__ f32x4 load(int kc, int j) const {
        const int m = kc * BK + kk[j];
        return sel4(m < npix, ld4(dz1 + (int64_t)(m < npix ? m : 0) * C1 + o0[j]));
    }
};

struct Conv1WgradB {  // input bytes rows (c,u,v), RMAJ quads along v at one pixel
    const uint8_t* const* ftab;
    const uint8_t* safe;  // any readable 7056 bytes, read in place of a zero-filled frame
    int npix, col0;
    int chan[MAXQ], off[MAXQ], kk[MAXQ];
    __device__ void init(int j, int row, int k) {
        const int kr = col0 + row;  // (c, u, v0) with v0 in {0, 4}
        chan[j] = kr >> 6;
        off[j] = ((kr >> 3) & 7) * IN_W + (kr & 7);
        kk[j] = k;
    }
    const uint8_t* const* fsample = nullptr;  // this chunk's sample's frame pointers
    int poff = 0;                              // this chunk's pixel within a frame
    __device__ void prep(int kc) {  // the thread's quads share one pixel
        const int m = kc * BK + kk[0];
        const int mm = m < npix ? m : 0;  // past the end: pixel 0 (A is zero there)
        const int b = mm / P1, p = mm - b * P1, i = p / H1, jj = p - i * H1;
        fsample = ftab + (int64_t)b * 4;
        poff = (S1 * i) * IN_W + S1 * jj;
    }
    __device__ f32x4 load(int, int j) const {
        // a zero-filled frame (null pointer) is zeros
        const uint8_t* f = fsample[chan[j]];
        const bool ok = f != nullptr;
        const uint32_t d = ldg_u32((ok ? f : safe) + poff + off[j]);
        return sel4(ok, f32x4{(float)(d & 255u), (float)((d >> 8) & 255u),
                              (float)((d >> 16) & 255u), (float)(d >> 24)});
    }
};

constexpr int C1W_BN = 128;
// The launch aims at one round of three workgroups per CU (the job's register
// budget allows three): 754 workgroups of 17 chunks measured 58 us against
// 65 us for 986 of 13 chunks (1.3 rounds) at batch 512.
constexpr int C1W_TARGET_WGS = 768;

template <int BF>
struct Conv1WgradJob {
    const float* dz1;
    const uint8_t* const* ftab;
    float* partial;
    float* bias_part;
    int n, splits, cps, groups;
    // in bf16 the bytes are exact operands (one plane)
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? 1 : 0;
    using SH = GemmShape<32, C1W_BN, RMAJ, RMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    static constexpr int NCT = 256 / C1W_BN;
    __host__ __device__ int blocks() const { return pad_xcd(NCT * splits * groups); }
    __device__ void run(int bid, float* smem) const {
        const int t = xcd_tile(bid, blocks());
        if (t >= NCT * splits * groups) return;
        // column tiles of a split adjacent; split runs over (group, split)
        const int col0 = (t % NCT) * C1W_BN, split = t / NCT, g = split / splits;
        const int npix = n * P1;
        const int nchunks = (npix + BK - 1) / BK;
        const int ks = split - g * splits;
        const int kc0 = ks * cps, kc1 = min(nchunks, kc0 + cps);
        const int64_t rows = (int64_t)g * n;
        Conv1WgradA la{dz1 + rows * P1 * C1, npix};
        Conv1WgradB lb{ftab + rows * 4, (const uint8_t*)dz1, npix, col0};
        PartialEpi epi{partial + (int64_t)split * C1 * 256, 256, col0, 1.0f / 255.0f};
        float* rs = col0 == 0 ? bias_part + (int64_t)split * 64 : nullptr;
        mfma_gemm<32, C1W_BN, 1, RMAJ, RMAJ, PA, PB>(smem, kc0, kc1, la, lb, epi, rs);
    }
};

void launch_conv1_wgrad(const float* dz1, const uint8_t* const* ftab, int groups, int n,
                        float* partial, float* bias_part, int max_splits, int* splits_out,
                        bool bf16, hipStream_t st) {
    const int nchunks = (n * P1 + BK - 1) / BK;
    int splits = max(1, min(max_splits, C1W_TARGET_WGS / (256 / C1W_BN)) / groups);
    splits = min(splits, nchunks);
    const int cps = (nchunks + splits - 1) / splits;
    splits = (nchunks + cps - 1) / cps;
    *splits_out = splits;
    if (bf16) launch_jobs(st, Conv1WgradJob<1>{dz1, ftab, partial, bias_part, n, splits, cps, groups});
    else      launch_jobs(st, Conv1WgradJob<0>{dz1, ftab, partial, bias_part, n, splits, cps, groups});
}

}  // namespace gorila
