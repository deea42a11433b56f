// First convolution (Section 5.1: 32 filters of 4x8x8, stride 4, ReLU) on the
// raw uint8 frames, forward and weight gradient.  Bytes enter the products as
// exact integers; the 1/255 input scale is applied once in each epilogue.
#include "common.h"
#include "kernels.h"

#include <type_traits>

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
// forward kernel), so only the fp32 accumulation rounds; bf16 steps read dz1
// already rounded to bf16 (one plane).
//
// Work is cut into units of two output rows of one sample (40 pixels, padded
// to 2 x 24 = 6 groups of 8); an MFMA step takes two groups (lane half h:
// group 2 step + h), so a unit is three steps.  Workgroups come in pairs that
// share a range of units, one per channel pair p (input channels 2 p, 2 p + 1:
// four column tiles of 32); each of a workgroup's eight waves walks its own
// contiguous part of the range with a private LDS stage, with no workgroup
// barrier until the end.  A wave splits the dz1 values of its units into
// planes in registers, straight from their coalesced loads (lane o, h: eight
// pixels of channel o), and multiplies them into its four tiles.  Column tile t is (c = 2 p + t / 2,
// s = t % 2) and lane column l % 32 is (u, m) = ((l % 32) / 4, l % 4), i.e.
// v = 4 s + m; its eight operands are the bytes at x = 4 (j + s) + m of input
// row 4 i + u for the group's pixels j, so each input row is staged by phase:
// xs[c][r][m][s][q] = byte 4 (q + s) + m, and a lane's eight bytes are eight
// consecutive entries.  Entries q >= 20 are used only by the padding pixels
// j = 20 .. 23 and hold zeros (written once), so those pixels' dz1 operands
// (pixels 16 .. 19 read again) need no masking.  The next unit's dz1 values
// and bytes are fetched into registers during the products; the frame
// pointers (wave-uniform, scalar loads) one unit before the fetch that uses
// them, and a null (zero-filled) frame is read from a frame of zeros.  db1 is
// summed from the dz1 values as loaded (kept by the workgroup of channel pair
// 0).  At the end the eight waves are added in a fixed order in LDS and each
// workgroup writes its channel pair's half of one partial [32][256].
constexpr int C1W_UR = 2;                       // output rows per unit
constexpr int C1W_UNITS = H1 / C1W_UR;          // 10 units per sample
constexpr int C1W_Q = 24;                       // phase entries per staged row (pixels padded to 24)
constexpr int C1W_QR = 20;                      // entries that can be non-zero (real pixels)
// LDS stride of a staged (row, m, s) line: 28 entries = 14 dwords, so the 8
// (u, m) lines that 8 neighbouring lanes read (lines 2 (4 u + m) + s, 28
// dwords apart) start on 8 distinct 4-bank groups (with 24 they would share 4)
constexpr int C1W_QS = 28;
constexpr int C1W_XR = S1 * (C1W_UR - 1) + K1;  // 12 input rows per unit
constexpr int C1W_CPW = 2;                      // input channels per wave
constexpr int C1W_WAVES = 8;                    // per workgroup, all on one channel pair
constexpr int C1W_TASKS = C1W_XR * (C1W_QR / 2);  // 120 staging tasks per channel and unit
constexpr int C1W_WGS = 256;                    // workgroups: one per CU

struct C1wStage {
    __bf16 x[C1W_CPW][C1W_XR][4][2][C1W_QS];  // [c][r][m][s][q], q < 24 used; 10.5 KB
};
constexpr int C1W_CH = C1W_XR * 4 * 2 * C1W_QS;  // stage elements per channel
constexpr int C1W_PLANE = 4 * 16 * 64;  // floats: one wave's accumulators
constexpr size_t C1W_SMEM = C1W_WAVES * sizeof(C1wStage) > 4 * C1W_WAVES * C1W_PLANE
                                ? C1W_WAVES * sizeof(C1wStage) : 4 * C1W_WAVES * C1W_PLANE;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// dz1 of a bf16 step (WP = 1) arrives rounded to bf16 ([n][20][20][32] bit
// patterns); it is widened exactly as it is loaded.
template <int WP>
using C1wDz = std::conditional_t<WP == 1, uint16_t, float>;
__device__ inline float c1w_value(float v) { return v; }
__device__ inline float c1w_value(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

template <int WP>
__global__ __launch_bounds__(64 * C1W_WAVES) void conv1_wgrad_mfma16_kernel(
    const C1wDz<WP>* __restrict__ dz1, const uint8_t* const* __restrict__ ftab,
    const uint8_t* __restrict__ zero_frame, int n, int SP, float* __restrict__ partial,
    float* __restrict__ bias_part) {
    __shared__ __attribute__((aligned(16))) char smem[C1W_SMEM];
    __shared__ float bred[C1W_WAVES][2][C1];
    // block b runs on XCD b % 8, so the two workgroups of pair xp (channel
    // pairs 0 and 1, blocks 8 apart) share an L2 and read dz1 from HBM once
    const int g = blockIdx.y, b8 = blockIdx.x / NUM_XCD;
    const int cp = b8 & 1, xp = (b8 >> 1) * NUM_XCD + blockIdx.x % NUM_XCD;  // channel pair, pair
    if (xp >= SP) return;  // padding of the last group of eight pairs
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar unit walk
    const int h = lane >> 5, o = lane & 31;
    C1wStage& sg = ((C1wStage*)smem)[wave];
    __bf16* xs = &sg.x[0][0][0][0][0];

    // this wave's units: a contiguous share of the workgroup pair's share
    const int64_t U = (int64_t)n * C1W_UNITS, W = (int64_t)SP * C1W_WAVES;
    const int64_t wi = (int64_t)xp * C1W_WAVES + wave;
    const int u0 = (int)(wi * U / W), u1 = (int)((wi + 1) * U / W);

    // entries q >= 20 of every staged line stay zero
    for (int e = lane; e < C1W_CPW * C1W_XR * 4 * 2 * (C1W_Q - C1W_QR); e += 64) {
        const int line = e / (C1W_Q - C1W_QR), q = C1W_QR + e % (C1W_Q - C1W_QR);
        xs[line * C1W_QS + q] = (__bf16)0.0f;
    }

    // Staging slots: slot k of this lane is (c, r, qp) = (k / 2, rq / 10,
    // rq % 10) with rq = lane + 64 (k % 2), so a slot's bytes come from one
    // frame for the whole wave (channel 2 p + c); rq >= 120 (lanes 56..63 of
    // the odd slots) repeat task 119: the same bytes to the same place.
    uint32_t toff[2];  // byte offset of dword 2 qp of row r, relative to row 4 i0
    int tlds[2];       // element offset of [0][r][0][0][2 qp] in the stage
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int rq = min(lane + 64 * k, C1W_TASKS - 1);
        const int r = rq / (C1W_QR / 2), qp = rq - r * (C1W_QR / 2);
        toff[k] = (uint32_t)(r * IN_W + 8 * qp);
        tlds[k] = (r * 4) * 2 * C1W_QS + 2 * qp;
    }
    // dz1 byte offsets (relative to the unit's first pixel) of this lane's
    // eight pixels in step st: pixel p0 + t, where (ir, j0) is the lane half's
    // pixel group; a group with j0 = 16 has padding pixels t >= 4, which read
    // pixels 16..19 again (finite values that meet zero bytes).
    using T = C1wDz<WP>;
    uint32_t dlo[3], dhi[3];
#pragma unroll
    for (int st = 0; st < 3; ++st) {
        const int grp = 2 * st + h, ir = grp / 3, j0 = 8 * (grp % 3);
        const int p0 = ir * H1 + j0;
        dlo[st] = (uint32_t)((p0 * C1 + o) * sizeof(T));
        dhi[st] = (uint32_t)(((j0 + 8 > H1 ? p0 : p0 + 4) * C1 + o) * sizeof(T));
    }
    const T* dzg = dz1 + (int64_t)g * n * P1 * C1;

    float av[3][8];          // dz1 of a unit's three steps (this lane's pixels)
    uint32_t xw[4][3];       // three input dwords per staging slot of the next unit
    const uint8_t* fnext[C1W_CPW];  // wave-uniform: frames 2 p, 2 p + 1 of the next fetch's sample
    auto load_ptrs = [&](int u) {
        const int b = u / C1W_UNITS;
        const uint8_t* const* fp = ftab + ((int64_t)g * n + b) * IN_C + C1W_CPW * cp;
#pragma unroll
        for (int c = 0; c < C1W_CPW; ++c) fnext[c] = fp[c];
    };
    auto fetch_dz = [&](int u, int st) {
        const int b = u / C1W_UNITS, i0 = (u - b * C1W_UNITS) * C1W_UR;
        const char* d = (const char*)(dzg + ((int64_t)b * P1 + i0 * H1) * C1);  // wave-uniform
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            av[st][t] = c1w_value(*(const T*)(d + dlo[st] + t * C1 * sizeof(T)));
            av[st][t + 4] = c1w_value(*(const T*)(d + dhi[st] + t * C1 * sizeof(T)));
        }
    };
    auto fetch_bytes = [&](int u) {
        const int i0 = (u % C1W_UNITS) * C1W_UR;
        const uint8_t* fr[C1W_CPW];
#pragma unroll
        for (int c = 0; c < C1W_CPW; ++c) fr[c] = fnext[c] ? fnext[c] + S1 * i0 * IN_W : zero_frame;
        load_ptrs(min(u + 1, u1 - 1));
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int dd = 0; dd < 3; ++dd)  // dwords <= 20: in the row
                xw[k][dd] = ldg_u32(fr[k >> 1] + toff[k & 1] + 4 * dd);
    };
    auto stage = [&]() {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t w0 = xw[k][0], w1 = xw[k][1], w2 = xw[k][2];
            __bf16* dst = xs + (k >> 1) * C1W_CH + tlds[k & 1];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const __bf16 b0 = (__bf16)(float)((w0 >> (8 * m)) & 255u);
                const __bf16 b1 = (__bf16)(float)((w1 >> (8 * m)) & 255u);
                const __bf16 b2 = (__bf16)(float)((w2 >> (8 * m)) & 255u);
                // s = 0: entries q, q + 1 (bytes of dwords q, q + 1); s = 1: bytes of q + 1, q + 2
                *(bf16x2*)(dst + (2 * m) * C1W_QS) = bf16x2{b0, b1};
                *(bf16x2*)(dst + (2 * m + 1) * C1W_QS) = bf16x2{b1, b2};
            }
        }
    };

    f32x16 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = f32x16{};
    float bsum = 0.0f;
    const int col = lane & 31, uu = col >> 2, mm = col & 3;

    // One MFMA step: the operands of its four column tiles from the stage,
    // and the planes of its eight dz1 values (summed into db1 on the way:
    // real pixels only; j0 is 0, 8 or 16).
    auto read_bx = [&](int st, bf16x8 (&bx)[4]) {
        const int grp = 2 * st + h, ir = grp / 3, j0 = 8 * (grp % 3);
#pragma unroll
        for (int t = 0; t < 4; ++t)
            bx[t] = *(const bf16x8*)&sg.x[t >> 1][S1 * ir + uu][mm][t & 1][j0];
    };
    // planes of the eight values, two at a time: a packed round to bf16, the
    // two rounded values widened back, the exact remainders
    auto planes = [&](int st, bf16x8 (&a)[WP]) {
        const int j0 = 8 * ((2 * st + h) % 3);
#pragma unroll
        for (int t = 0; t < 8; t += 2) {
            float v0 = av[st][t], v1 = av[st][t + 1];
            if (t < 4 || j0 + t < H1) {
                bsum += v0;
                bsum += v1;
            }
#pragma unroll
            for (int pl = 0; pl < WP; ++pl) {
                const bf16x2 hp = __builtin_convertvector(f32x2{v0, v1}, bf16x2);
                a[pl][t] = hp[0];
                a[pl][t + 1] = hp[1];
                if (pl + 1 < WP) {
                    const uint32_t bits = __builtin_bit_cast(uint32_t, hp);
                    v0 -= __uint_as_float(bits << 16);
                    v1 -= __uint_as_float(bits & 0xffff0000u);
                }
            }
        }
    };
    auto products = [&](const bf16x8 (&a)[WP], const bf16x8 (&bx)[4]) {
#pragma unroll
        for (int pl = 0; pl < WP; ++pl)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[pl], bx[t], acc[t], 0, 0, 0);
    };

    // Software pipeline over the steps: while a step's products run, the next
    // step's operands are read and its planes split, and each dz1 register is
    // refilled with the next unit's value right after its split (one set of
    // dz1 registers, no copies).  Unit u enters with its step 0 operands and
    // planes ready and leaves with unit u + 1's; the next unit's bytes are
    // staged beside the last step's products, after every operand read of
    // this unit (LDS serves a wave in order).  Fetches past the wave's last
    // unit read that unit again (in bounds, unused).
    if (u0 < u1) {
        const int last = u1 - 1;
        load_ptrs(u0);
#pragma unroll
        for (int st = 0; st < 3; ++st) fetch_dz(u0, st);
        fetch_bytes(u0);
        stage();
        fetch_bytes(min(u0 + 1, last));
        bf16x8 a0[WP], b0[4], a1[WP], b1[4];  // planes and operands of two steps
        read_bx(0, b0);
        planes(0, a0);
        fetch_dz(min(u0 + 1, last), 0);
        // Each region between scheduling barriers runs one step's products
        // beside the next step's operand reads and split; the refills close
        // their region, so they are issued as early as their registers allow.
        auto unit = [&](int u, auto more) {
            constexpr bool MORE = decltype(more)::value;
            products(a0, b0);
            read_bx(1, b1);
            planes(1, a1);
            fetch_dz(min(u + 1, last), 1);
            __builtin_amdgcn_sched_barrier(0);
            products(a1, b1);
            read_bx(2, b0);
            planes(2, a0);
            fetch_dz(min(u + 1, last), 2);
            __builtin_amdgcn_sched_barrier(0);
            products(a0, b0);
            if constexpr (MORE) {
                stage();  // unit u + 1
                fetch_bytes(min(u + 2, last));
                read_bx(0, b0);
                planes(0, a0);
                fetch_dz(min(u + 2, last), 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        for (int u = u0; u < last; ++u) unit(u, std::true_type{});
        unit(last, std::false_type{});
    }

    // Add the eight waves in LDS: each stores its accumulators as one plane
    // laid out [tile][register][lane] (every store 64 consecutive floats),
    // then each thread sums one quad of four columns over the planes in a
    // fixed order and writes it; the two workgroups of a pair write the two
    // column halves of one partial [32][256].
    __syncthreads();  // every wave is done with its stage
    float* red = (float*)smem;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[wave * C1W_PLANE + (t * 16 + r) * 64 + lane] = acc[t][r];
    bred[wave][h][o] = bsum;
    __syncthreads();
    const int split = g * SP + xp;
    float* out = partial + (int64_t)split * C1 * 256 + cp * 128;
    for (int e = tid; e < C1 * 128 / 4; e += 64 * C1W_WAVES) {
        // quad e: row (filter o), column tile c of the pair, quad q = (u, s);
        // register r and lane half of that row in the accumulator layout
        const int row = e >> 5, c = (e >> 4) & 1, q = e & 15, ue = q >> 1, s = q & 1;
        const int r = 4 * (row >> 3) + (row & 3), hh = (row >> 2) & 1;
        const int off = ((2 * c + s) * 16 + r) * 64 + hh * 32 + ue * 4;
        f32x4 sum = *(const f32x4*)(red + off);
#pragma unroll
        for (int w = 1; w < C1W_WAVES; ++w) sum += *(const f32x4*)(red + w * C1W_PLANE + off);
        *(f32x4*)(out + row * 256 + c * 64 + ue * 8 + 4 * s) = sum * (1.0f / 255.0f);
    }
    if (cp == 0 && tid < C1) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < C1W_WAVES; ++w) t += bred[w][0][tid] + bred[w][1][tid];
        bias_part[(int64_t)split * 64 + tid] = t;
    }
}

void launch_conv1_wgrad(const float* dz1, const uint8_t* const* ftab, const uint8_t* zero_frame,
                        int groups, int n, float* partial, float* bias_part, int max_splits,
                        int* splits_out, bool bf16, hipStream_t st) {
    if (n <= 0) {
        *splits_out = 0;
        return;
    }
    // workgroup pairs (one workgroup per channel pair) per group: one
    // workgroup per CU in all, each of whose waves gets at least one unit;
    // groups * pairs stays within max_splits (a pair writes one partial)
    const int splits = max(1, min((n * C1W_UNITS + C1W_WAVES - 1) / C1W_WAVES,
                                  min(C1W_WGS / 2, max_splits) / groups));
    *splits_out = splits;
    // the pairs in groups of eight: 16 blocks each, the kernel's block order
    const int blocks = 2 * pad_xcd(splits);
    if (bf16)
        conv1_wgrad_mfma16_kernel<1><<<dim3(blocks, groups), 64 * C1W_WAVES, 0, st>>>(
            (const uint16_t*)dz1, ftab, zero_frame, n, splits, partial, bias_part);
    else
        conv1_wgrad_mfma16_kernel<3><<<dim3(blocks, groups), 64 * C1W_WAVES, 0, st>>>(
            dz1, ftab, zero_frame, n, splits, partial, bias_part);
}

}  // namespace gorila
