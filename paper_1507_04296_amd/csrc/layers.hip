// Convolution 2/3 and FC-512 layers, forward and backward, as implicit GEMMs
// on the fp32 MFMA tile engine (common.h).  Shapes follow Section 5.1 of the
// paper; the backward pass is the exact gradient of those layers (eq. (2)
// needs grad_theta Q(s, a; theta)).
//
// Every layer below is written as C[row][col] = sum_k A[row][k] * B[col][k]
// plus an epilogue.  Reduction indices of convolutions are ordered
// (tap (u,v), channel): one reduction chunk of 32 is one tap and 32 channels,
// so activation quads are 16 contiguous bytes of an NHWC pixel.
#include "common.h"
#include "kernels.h"

#include <type_traits>

namespace gorila {

// Output positions of an N x N data-gradient grid (kernel K taps per axis
// over an IN x IN input, stride-1 form) in decreasing order of valid taps,
// then raster order.  The data-gradient workgroups of a launch go longest
// first, so the short border positions fill in at the end instead of long
// interior ones trailing the launch.
template <int N, int K, int IN>
struct LongestFirst {
    unsigned char pos[N * N];
    static constexpr int taps(int y) {
        return (y < K - 1 ? y : K - 1) - (y - (IN - 1) > 0 ? y - (IN - 1) : 0) + 1;
    }
    constexpr LongestFirst() : pos() {
        int r = 0;
        for (int want = K * K; want >= 1; --want)
            for (int p = 0; p < N * N; ++p)
                if (taps(p / N) * taps(p % N) == want) pos[r++] = (unsigned char)p;
    }
};

// Gradients handed from one backward launch to the next (dz3, dz2): fp32, or
// in bf16 steps whose reductions are not cut into parts (KP = 1) bf16,
// rounded once by the producer to the precision the consumer's products take
// them in (half the bytes written and read).
template <int BF, int KP> using GradT = std::conditional_t<BF == 1 && KP == 1, uint16_t, float>;
__device__ inline f32x4 ldq(const float* p) { return ld4(p); }
__device__ inline f32x4 ldq(const uint16_t* p) {  // four bf16 values, widened exactly
    const uint2 v = *(const uint2*)p;
    return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                 __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u)};
}
__device__ inline void stg(float* p, float v) { *p = v; }
__device__ inline void stg(uint16_t* p, float v) { *p = __builtin_bit_cast(uint16_t, (__bf16)v); }

// Quad at p summed over the KP partial planes p, p + ps, ... in plane order.
template <int KP, class T>
__device__ __forceinline__ f32x4 ld4_parts(const T* p, int64_t ps) {
    f32x4 v = ldq(p);
#pragma unroll
    for (int s = 1; s < KP; ++s) v += ldq(p + s * ps);
    return v;
}

// ---------------------------------------------------------------------------
// conv2 forward: h2[m][o] = relu(b2[o] + sum_{u,v,c} W2[o][c][u][v] h1[b][2i+u][2j+v][c])
// rows m = (b,i,j) of one group, cols o; 16 chunks = 16 taps x 32 channels.
// ---------------------------------------------------------------------------
struct Conv2FwdA {
    const float* h1;
    int rows, m0;
    const float* base[MAXQ];
    __device__ void init(int j, int row, int k) {
        const int m = m0 + row;
        const int mm = m < rows ? m : 0;
        const int b = mm / P2, p = mm - b * P2, i = p / H2, jj = p - i * H2;
        base[j] = h1 + (((int64_t)b * H1 + S2 * i) * H1 + S2 * jj) * C1 + k;
    }
    // rows past the end read row 0 (finite values) and are never stored
    __device__ f32x4 load(int kc, int j) const {
        const int u = kc >> 2, v = kc & 3;
        return ld4(base[j] + (u * H1 + v) * C1);
    }
};
// Transposed weights w[tap][row][k] with LDK k per row (LDK / BK chunks per
// tap) and ROWS rows per tap.
template <int LDK, int ROWS>
struct WtapB {
    static constexpr int PER_TAP = LDK / BK;
    const float* w;
    const float* base[MAXQ];
    __device__ void init(int j, int row, int k) { base[j] = w + row * LDK + k; }
    __device__ f32x4 load(int kc, int j) const {
        const int t = kc / PER_TAP, part = kc - t * PER_TAP;
        return ld4(base[j] + t * (ROWS * LDK) + part * BK);
    }
};
struct BiasReluStore {
    float* out;
    const float* bias;
    int rows, m0, ld;
    __device__ float pre(int, int col) const { return bias[col]; }
    __device__ void operator()(int row, int col, float v, float b) const {
        const int m = m0 + row;
        if (m < rows) out[(int64_t)m * ld + col] = fmaxf(v + b, 0.0f);
    }
};

// The fp32 job keeps one LDS stage (16 KB): with 80 registers six workgroups
// are resident on a compute unit, so at batch 512 (1296 tiles, 5 a unit and
// 16 over) the whole tiles take one round and the last 16 tiles run as
// reduction pieces beside them, instead of a second round on 16 units.
template <int BF, bool SPLIT = false>
struct Conv2FwdJob {
    const float* h1;
    GroupPtrs w2t, theta;
    float* h2;
    int n, groups;
    TailSplit ts;
    static constexpr int PA = BF ? BF_ACT_FWD : 0, PB = BF ? BF_WEIGHT : 0, CHUNKS = 16;
    static constexpr bool SB = BF == 0;
    static constexpr int MIN_WGS = SB ? 6 : 1;  // 80 registers at most
    using SH = GemmShape<64, 64, KMAJ, KMAJ, PA, PB, SB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int tiles() const { return (n * P2 + 63) / 64; }
    __host__ __device__ int blocks() const {
        return SPLIT ? ts.blocks(tiles() * groups) : pad_xcd(tiles() * groups);
    }
    __device__ void run(int bid, float* smem) const {
        int t, k0 = 0, k1 = CHUNKS;
        SplitPiece sp;
        if constexpr (SPLIT) {
            if (!ts.map(bid, tiles() * groups, CHUNKS, t, k0, k1, sp)) return;
        } else {
            t = xcd_tile(bid, blocks());
            if (t >= tiles() * groups) return;
        }
        const int g = t / tiles(), m0 = (t % tiles()) * 64;
        const int rows = n * P2;
        Conv2FwdA la{h1 + (int64_t)g * n * P1 * C1, rows, m0};
        WtapB<C1, C2> lb{w2t.p[g]};
        BiasReluStore epi{h2 + (int64_t)g * n * P2 * C2, theta.p[g] + OFF_B2, rows, m0, C2};
        if (sp.np == 1) mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB, SB>(smem, 0, CHUNKS, la, lb, epi);
        else mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB, SB>(smem, k0, k1, la, lb, epi, nullptr, sp);
    }
};

void launch_conv2_fwd(const float* h1, const GroupPtrs& w2t, const GroupPtrs& theta, int groups,
                      int n, float* h2, const SplitWs& sw, bool bf16, hipStream_t st) {
    if (n <= 0) return;
    if (bf16) {
        launch_jobs(st, Conv2FwdJob<1>{h1, w2t, theta, h2, n, groups});
        return;
    }
    const int T = (n * P2 + 63) / 64 * groups;
    const TailSplit ts = plan_split(sw.ws, sw.cnt, sw.cus, T, T, Conv2FwdJob<0>::CHUNKS, 6);
    if (ts.tail) launch_jobs(st, Conv2FwdJob<0, true>{h1, w2t, theta, h2, n, groups, ts});
    else launch_jobs(st, Conv2FwdJob<0>{h1, w2t, theta, h2, n, groups, ts});
}

// ---------------------------------------------------------------------------
// conv3 forward, computed transposed so the channel-major (flatten-order)
// output is stored along pixels: h3[b][o][p] = relu(b3[o] + sum W3 h2[b][i+u][j+v][c]).
// rows o (64), cols m = (b,p) of one group; 18 chunks = 9 taps x 2 halves of c.
// ---------------------------------------------------------------------------
struct Conv3FwdB {
    const float* h2;
    int rows, m0;
    const float* base[MAXQ];
    __device__ void init(int j, int row, int k) {
        const int m = m0 + row;
        const int mm = m < rows ? m : 0;
        const int b = mm / P3, p = mm - b * P3, i = p / H3, jj = p - i * H3;
        base[j] = h2 + (((int64_t)b * H2 + i) * H2 + jj) * C2 + k;
    }
    // columns past the end read pixel 0 (finite values) and are never stored
    __device__ f32x4 load(int kc, int j) const {
        const int t = kc >> 1, u = t / 3, v = t - u * 3;
        return ld4(base[j] + (u * H2 + v) * C2 + (kc & 1) * BK);
    }
};
struct Conv3FwdStore {  // row = o, col = pixel index within the tile
    float* out;
    const float* bias;
    int rows, m0;
    __device__ float pre(int row, int) const { return bias[row]; }
    __device__ void operator()(int row, int col, float v, float b3) const {
        const int m = m0 + col;
        if (m >= rows) return;
        const int b = m / P3, p = m - b * P3;
        out[(int64_t)b * FLAT + row * P3 + p] = fmaxf(v + b3, 0.0f);
    }
};

// SPLIT: the launch runs some tiles as reduction pieces (TailSplit); the
// unsplit instantiation carries none of the hand-off code.
template <int BF, bool SPLIT = false>
struct Conv3FwdJob {
    const float* h2;
    GroupPtrs w3t, theta;
    float* h3;
    int n, groups;
    TailSplit ts;
    static constexpr int PA = BF ? BF_WEIGHT : 0, PB = BF ? BF_ACT_FWD : 0, CHUNKS = 18;
    using SH = GemmShape<64, 64, KMAJ, KMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int tiles() const { return (n * P3 + 63) / 64; }
    __host__ __device__ int blocks() const {
        return SPLIT ? ts.blocks(tiles() * groups) : pad_xcd(tiles() * groups);
    }
    __device__ void run(int bid, float* smem) const {
        int t, k0 = 0, k1 = CHUNKS;
        SplitPiece sp;
        if constexpr (SPLIT) {
            if (!ts.map(bid, tiles() * groups, CHUNKS, t, k0, k1, sp)) return;
        } else {
            t = xcd_tile(bid, blocks());
            if (t >= tiles() * groups) return;
        }
        const int g = t / tiles(), m0 = (t % tiles()) * 64;
        const int rows = n * P3;
        WtapB<C2, C3> la{w3t.p[g]};
        Conv3FwdB lb{h2 + (int64_t)g * n * P2 * C2, rows, m0};
        Conv3FwdStore epi{h3 + (int64_t)g * n * FLAT, theta.p[g] + OFF_B3, rows, m0};
        if (sp.np == 1) mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB>(smem, 0, CHUNKS, la, lb, epi);
        else mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB>(smem, k0, k1, la, lb, epi, nullptr, sp);
    }
};

void launch_conv3_fwd(const float* h2, const GroupPtrs& w3t, const GroupPtrs& theta, int groups,
                      int n, float* h3, const SplitWs& sw, bool bf16, hipStream_t st) {
    if (n <= 0) return;
    const int T = (n * P3 + 63) / 64 * groups;
    const TailSplit ts = plan_split(sw.ws, sw.cnt, sw.cus, T, T, Conv3FwdJob<0>::CHUNKS);
    if (bf16 && ts.tail) launch_jobs(st, Conv3FwdJob<1, true>{h2, w3t, theta, h3, n, groups, ts});
    else if (bf16) launch_jobs(st, Conv3FwdJob<1>{h2, w3t, theta, h3, n, groups, ts});
    else if (ts.tail) launch_jobs(st, Conv3FwdJob<0, true>{h2, w3t, theta, h3, n, groups, ts});
    else launch_jobs(st, Conv3FwdJob<0>{h2, w3t, theta, h3, n, groups, ts});
}

// ---------------------------------------------------------------------------
// fc1 forward, split over the 3136-long reduction: partial[g][s][b][o].  The
// action-head kernel adds the splits in order, the bias and the ReLU.
// ---------------------------------------------------------------------------
struct RowMajorK {  // rows of a row-major [rows][ld] matrix, quads along k
    const float* a;
    int rows, r0, ld;
    const float* base[MAXQ];
    // rows past the end read row 0 (finite values); they are output rows or
    // columns that are never stored
    __device__ void init(int j, int row, int k) {
        base[j] = a + (int64_t)(r0 + row < rows ? r0 + row : 0) * ld + k;
    }
    __device__ f32x4 load(int kc, int j) const { return ld4(base[j] + kc * BK); }
};
// bf16 weights read in place and widened exactly: a quad is 4 values at a
// multiple of 4 along a row of W4, so its alignment is that of the matrix,
// which the parameter layout only guarantees to 2 bytes; `al` (8, 4 or 2)
// picks one, two or four loads per quad.
__device__ inline int align_of(const uint16_t* p) {
    const uintptr_t a = (uintptr_t)p;
    return (a & 7) == 0 ? 8 : (a & 3) == 0 ? 4 : 2;
}
__device__ inline f32x4 ld4_bf16(const uint16_t* p, int al) {
    uint32_t a, b;
    if (al == 8) {
        const uint2 v = *(const uint2*)p;
        a = v.x;
        b = v.y;
    } else if (al == 4) {
        a = *(const uint32_t*)p;
        b = *(const uint32_t*)(p + 2);
    } else {
        a = p[0] | ((uint32_t)p[1] << 16);
        b = p[2] | ((uint32_t)p[3] << 16);
    }
    return f32x4{__uint_as_float(a << 16), __uint_as_float(a & 0xffff0000u),
                 __uint_as_float(b << 16), __uint_as_float(b & 0xffff0000u)};
}
struct RowMajorK16 {  // RowMajorK over a bf16 matrix
    const uint16_t* a;
    int rows, r0, ld;
    const uint16_t* base[MAXQ];
    int al = 8;
    __device__ void init(int j, int row, int k) {
        base[j] = a + (int64_t)(r0 + row < rows ? r0 + row : 0) * ld + k;
        al = align_of(a);
    }
    __device__ f32x4 load(int kc, int j) const { return ld4_bf16(base[j] + kc * BK, al); }
};

struct PlainStore {
    float* out;
    int rows, r0, c0, ld;
    __device__ float pre(int, int) const { return 0.0f; }
    __device__ void operator()(int row, int col, float v, float) const {
        if (r0 + row < rows) out[(int64_t)(r0 + row) * ld + c0 + col] = v;
    }
};

constexpr int FC1_CHUNKS = FLAT / BK;  // 98

// Logical tile order (group, split, column tile, row tile): the row tiles that
// share a block of W4 are neighbours and so share an XCD's L2.
template <int BF>
struct Fc1FwdJob {
    const float* h3;
    GroupPtrs theta;
    GroupPtrs16 w4b;  // bf16 steps: W4 of each set, read in place
    float* partial;
    int n, groups, splits, cps;
    static constexpr int PA = BF ? BF_ACT_FWD : 0, PB = BF ? BF_WEIGHT : 0;
    using SH = GemmShape<64, 64, KMAJ, KMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int mt() const { return (n + 63) / 64; }
    __host__ __device__ int tiles() const { return mt() * (HID / 64) * groups * splits; }
    __host__ __device__ int blocks() const { return pad_xcd(tiles()); }
    __device__ void run(int bid, float* smem) const {
        int t = xcd_tile(bid, blocks());
        if (t >= tiles()) return;
        const int r0 = (t % mt()) * 64;
        t /= mt();
        const int c0 = (t % (HID / 64)) * 64;
        t /= HID / 64;
        const int s = t % splits, g = t / splits;
        RowMajorK la{h3 + (int64_t)g * n * FLAT, n, r0, FLAT};
        PlainStore epi{partial + ((int64_t)g * splits + s) * n * HID, n, r0, c0, HID};
        const int kc0 = s * cps, kc1 = min(FC1_CHUNKS, kc0 + cps);
        if constexpr (BF > 0) {
            RowMajorK16 lb{w4b.p[g], HID, c0, FLAT};
            mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB>(smem, kc0, kc1, la, lb, epi);
        } else {
            RowMajorK lb{theta.p[g] + OFF_W4, HID, c0, FLAT};
            mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB>(smem, kc0, kc1, la, lb, epi);
        }
    }
};

int launch_fc1_fwd(const float* h3, const GroupPtrs& theta, const GroupPtrs16& w4b, int groups,
                   int n, float* partial, bool bf16, hipStream_t st) {
    if (n <= 0) return 0;
    const int mt = (n + 63) / 64, tiles = mt * (HID / 64) * groups;
    int splits = min(FC1_MAX_SPLITS, max(1, (TARGET_WGS + tiles - 1) / tiles));
    const int cps = (FC1_CHUNKS + splits - 1) / splits;
    splits = (FC1_CHUNKS + cps - 1) / cps;
    if (bf16) launch_jobs(st, Fc1FwdJob<1>{h3, theta, w4b, partial, n, groups, splits, cps});
    else      launch_jobs(st, Fc1FwdJob<0>{h3, theta, w4b, partial, n, groups, splits, cps});
    return splits;
}

// ---------------------------------------------------------------------------
// fc1 data gradient: dz3 = [h3 > 0] * (W4^T dz4), rows b, cols k (3136 = 49
// tiles), reduction o (16 chunks); dz3 is written as [b][p][o].
// ---------------------------------------------------------------------------
// B[col][k] = M[k][c0 + col] of a row-major [k][ld] matrix (RMAJ quads).
// Reduction indices k >= kmax read row 0; ZERO makes them zeros (one operand
// of a padded reduction must be zero there, the other only finite).
template <bool ZERO>
struct RowMajorR {
    const float* a;
    int c0, ld, kmax;
    const float* base[MAXQ];
    int kk[MAXQ];
    __device__ void init(int j, int row, int k) { base[j] = a + c0 + row; kk[j] = k; }
    __device__ f32x4 load(int kc, int j) const {
        const int k = kc * BK + kk[j];
        const f32x4 v = ld4(base[j] + (int64_t)(k < kmax ? k : 0) * ld);
        return ZERO ? sel4(k < kmax, v) : v;
    }
};

struct RowMajorR16 {  // RowMajorR<false> over a bf16 matrix
    const uint16_t* a;
    int c0, ld, kmax;
    const uint16_t* base[MAXQ];
    int kk[MAXQ];
    int al = 8;
    __device__ void init(int j, int row, int k) {
        base[j] = a + c0 + row;
        kk[j] = k;
        al = align_of(a);
    }
    __device__ f32x4 load(int kc, int j) const {
        const int k = kc * BK + kk[j];
        return ld4_bf16(base[j] + (int64_t)(k < kmax ? k : 0) * ld, al);
    }
};

// df is produced in the FC input's flatten order k = o*49 + p; dz3 is stored
// pixel-major ([b][p][o], like the other activation gradients) so that the
// conv3 backward kernels read it in 16-byte quads.
struct Dz3NhwcStore {
    static constexpr bool MASK = true;
    float* dz3;       // fp32 dz3, or null
    uint16_t* dz3h;   // bf16 dz3 (bf16 steps, one part), or null
    const float* h3;
    int rows, r0, c0;
    __device__ float pre(int row, int col) const {
        const int b = r0 + row;
        return h3[(int64_t)(b < rows ? b : 0) * FLAT + c0 + col];
    }
    __device__ void operator()(int row, int col, float v, float m) const {
        const int b = r0 + row;
        if (b >= rows) return;
        const int k = c0 + col, o = k / P3, p = k - o * P3;
        const float r = m > 0.0f ? v : 0.0f;
        if (dz3h) stg(dz3h + (int64_t)b * FLAT + p * C3 + o, r);
        else stg(dz3 + (int64_t)b * FLAT + p * C3 + o, r);
    }
};

// kp > 1 cuts the reduction over the 512 hidden units into kp parts, each
// writing its masked dz3 plane (the ReLU mask is linear in the parts).
template <int BF, bool SPLIT = false>  // SPLIT as for Conv3FwdJob (kp == 1 only)
struct Fc1DgradJob {
    const float* dz4;
    GroupPtrs theta;
    GroupPtrs16 w4b;  // bf16 steps: W4 of each set, read in place
    const float* h3;
    float* dz3;
    int n, groups, kp;  // kp reduction parts, each writing its own dz3 plane
    TailSplit ts;       // kp == 1 only
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? BF_WEIGHT : 0, CHUNKS = HID / BK;
    using SH = GemmShape<64, 64, KMAJ, RMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int tiles() const { return ((n + 63) / 64) * (FLAT / 64); }
    __host__ __device__ int blocks() const {
        return SPLIT ? ts.blocks(tiles() * groups) : pad_xcd(tiles() * groups * kp);
    }
    __device__ void run(int bid, float* smem) const {
        int t, part = 0, kc0 = 0, kc1 = CHUNKS;  // HID is a whole number of chunks
        SplitPiece sp;
        if constexpr (SPLIT) {
            if (!ts.map(bid, tiles() * groups, CHUNKS, t, kc0, kc1, sp)) return;
        } else {
            t = xcd_tile(bid, blocks());
            if (t >= tiles() * groups * kp) return;
            part = t / (tiles() * groups);
            t -= part * tiles() * groups;
            kc0 = part * CHUNKS / kp;
            kc1 = (part + 1) * CHUNKS / kp;
        }
        const int g = t / tiles();
        t -= g * tiles();
        const int mt = (n + 63) / 64;
        const int r0 = (t % mt) * 64, c0 = (t / mt) * 64;  // row tiles of one W4 column block adjacent
        const int64_t rows = (int64_t)g * n;
        RowMajorK la{dz4 + rows * HID, n, r0, HID};
        const bool half = BF == 1 && kp == 1;  // dz3 as GradT<BF, kp>
        Dz3NhwcStore epi{half ? nullptr : dz3 + part * (int64_t)groups * n * FLAT + rows * FLAT,
                         half ? (uint16_t*)dz3 + rows * FLAT : nullptr, h3 + rows * FLAT, n, r0, c0};
        // small-batch parts keep runtime bounds; whole tiles compile-time ones
        auto gemm = [&](auto& lb) {
            if (SPLIT && sp.np > 1)
                mfma_gemm<64, 64, 2, KMAJ, RMAJ, PA, PB>(smem, kc0, kc1, la, lb, epi, nullptr, sp);
            else if (kp > 1)
                mfma_gemm<64, 64, 2, KMAJ, RMAJ, PA, PB>(smem, kc0, kc1, la, lb, epi);
            else
                mfma_gemm<64, 64, 2, KMAJ, RMAJ, PA, PB>(smem, 0, CHUNKS, la, lb, epi);
        };
        if constexpr (BF > 0) {
            RowMajorR16 lb{w4b.p[g], c0, FLAT, HID};
            gemm(lb);
        } else {
            RowMajorR<false> lb{theta.p[g] + OFF_W4, c0, FLAT, HID};
            gemm(lb);
        }
    }
};

// ---------------------------------------------------------------------------
// fc1 weight gradient: dW4[o][k] = sum_b dz4[b][o] h3[b][k]  (written in place)
// rows o (512), cols k (3136), reduction b.
// ---------------------------------------------------------------------------
template <int BF>
struct Fc1WgradJob {
    const float* dz4;
    const float* h3;
    float* grads;
    int64_t grads_stride;
    int n, groups;
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? BF_ACT_WGRAD : 0;
    using SH = GemmShape<64, 64, RMAJ, RMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int tiles() const { return (HID / 64) * (FLAT / 64); }
    __host__ __device__ int blocks() const { return pad_xcd(tiles() * groups); }
    __device__ void run(int bid, float* smem) const {
        int t = xcd_tile(bid, blocks());
        if (t >= tiles() * groups) return;
        const int g = t / tiles();
        t -= g * tiles();
        const int r0 = (t % (HID / 64)) * 64, c0 = (t / (HID / 64)) * 64;
        const int64_t rows = (int64_t)g * n;
        float* gr = grads + g * grads_stride;
        RowMajorR<true> la{dz4 + rows * HID, r0, HID, n};
        RowMajorR<false> lb{h3 + rows * FLAT, c0, FLAT, n};
        PlainStore epi{gr + OFF_W4, HID, r0, c0, FLAT};
        // db4[o] = sum_b dz4[b][o]: the row sums of this GEMM's A operand
        float* rs = c0 == 0 ? gr + OFF_B4 + r0 : nullptr;
        mfma_gemm<64, 64, 2, RMAJ, RMAJ, PA, PB>(smem, 0, (n + BK - 1) / BK, la, lb, epi, rs);
    }
};

// Row-block partial sums of the action-head gradients and of the loss:
//   hpart[bb][a*512 + k] = sum_{b in block bb, a_b = a} coef_b h4[b][k]   (dW5)
//   hpart[bb][HP_DB5 + a] = sum_{b in block bb, a_b = a} coef_b           (db5)
//   hpart[bb][HP_LOSS]    = sum_{b in block bb} ell_b                     (loss)
// Block (column tile kt, row block bb).  Thread (column kl, lane group bq)
// adds rows bq, bq+4, ... of its block in order into its own LDS slots; the
// four lane groups are added in order, so every sum is deterministic.  The row
// blocks are summed in order by the final gradient reduction.
struct HeadPartialJob {
    const float* h4;
    const int32_t* a;
    const float* coef;
    const float* ell;
    float* hpart;
    int n, A, rows_per_block, row_blocks, groups;
    static constexpr int SMEM = 4 * MAX_ACTIONS * 64;
    __host__ __device__ int blocks() const { return pad_xcd((HID / 64) * row_blocks * groups); }
    __device__ void run(int bid, float* smem) const {
        if (bid >= (HID / 64) * row_blocks * groups) return;
        float (*sacc)[MAX_ACTIONS][64] = (float (*)[MAX_ACTIONS][64])smem;
        const int tid = threadIdx.x, kl = tid & 63, bq = tid >> 6;
        const int kt = bid % (HID / 64), gbb = bid / (HID / 64);
        const int g = gbb / row_blocks, bb = gbb - g * row_blocks;
        const int k = kt * 64 + kl;
        // rows of group g, block bb (learner rows g*n + b0 .. g*n + b1 - 1)
        const int b0 = g * n + bb * rows_per_block, b1 = g * n + min(n, (bb + 1) * rows_per_block);
        float* out = hpart + (int64_t)gbb * HP_STRIDE;
        for (int j = 0; j < A; ++j) sacc[bq][j][kl] = 0.0f;
        int b = b0 + bq;
        for (; b + 12 < b1; b += 16) {  // four rows a trip, their loads issued together
            int ab[4];
            float cf[4], hv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                ab[u] = a[b + 4 * u];
                cf[u] = coef[b + 4 * u];
                hv[u] = h4[(int64_t)(b + 4 * u) * HID + k];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                sacc[bq][ab[u]][kl] = fmaf(cf[u], hv[u], sacc[bq][ab[u]][kl]);
        }
        for (; b < b1; b += 4) {
            const int ab = a[b];
            sacc[bq][ab][kl] = fmaf(coef[b], h4[(int64_t)b * HID + k], sacc[bq][ab][kl]);
        }
        __syncthreads();
        for (int e = tid; e < A * 64; e += 256) {
            const int j = e >> 6, kk = e & 63;
            out[j * HID + kt * 64 + kk] =
                ((sacc[0][j][kk] + sacc[1][j][kk]) + sacc[2][j][kk]) + sacc[3][j][kk];
        }
        if (kt == 0) {
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
};

int launch_fc1_backward(const float* dz4, const GroupPtrs& theta, const GroupPtrs16& w4b,
                        int groups, const float* h3,
                        const float* h4, const int32_t* a, const float* coef, const float* ell,
                        int n, int A, float* dz3, float* grads, int64_t grads_stride,
                        float* hpart, int kp, const SplitWs& sw, bool bf16, hipStream_t st) {
    if (n <= 0) return 0;
    const int rows = max(32, (n + HEAD_MAX_BLOCKS - 1) / HEAD_MAX_BLOCKS);
    const int row_blocks = (n + rows - 1) / rows;
    const HeadPartialJob hp{h4, a, coef, ell, hpart, n, A, rows, row_blocks, groups};
    // the two GEMMs balance as one launch of equal tiles when their chunk
    // counts agree (the batch rounds up to the 512 hidden units)
    TailSplit ts;
    const int wt = (HID / 64) * (FLAT / 64) * groups, dt = ((n + 63) / 64) * (FLAT / 64) * groups;
    if (kp == 1 && (n + BK - 1) / BK == HID / BK)
        ts = plan_split(sw.ws, sw.cnt, sw.cus, wt + dt, dt, HID / BK);
    // Dispatch order: when the launch runs several rounds of workgroups per
    // compute unit and the data-gradient tiles are the longer ones (many
    // learner groups of a few rows each), those go first so that the short
    // weight-gradient tiles fill in behind them instead of trailing them.
    // Otherwise (one round, or equal tiles whose last data-gradient tiles are
    // split) the weight gradient goes first, which measured faster at batches
    // 32 and 512.
    const bool dgrad_first = (n + BK - 1) / BK < HID / BK / kp && wt + dt > 4 * sw.cus;
    auto go = [&](auto bf) {
        constexpr int BF = decltype(bf)::value;
        const Fc1WgradJob<BF> w{dz4, h3, grads, grads_stride, n, groups};
        const Fc1DgradJob<BF> d{dz4, theta, w4b, h3, dz3, n, groups, kp, ts};
        if (dgrad_first) launch_jobs(st, d, w, hp);
        else if (ts.tail) launch_jobs(st, w, Fc1DgradJob<BF, true>{dz4, theta, w4b, h3, dz3, n, groups, kp, ts}, hp);
        else launch_jobs(st, w, d, hp);
    };
    if (bf16) go(std::integral_constant<int, 1>{});
    else go(std::integral_constant<int, 0>{});
    return row_blocks;
}

// ---------------------------------------------------------------------------
// conv3 data gradient (stride 1): dh2[b][y][x][c] = sum_{u,v,o} W3[o][c][u][v]
// dz3[b][y-u][x-v][o] over in-range (y-u, x-v); then dz2 = dh2 * [h2 > 0].
// A workgroup owns one output position (y, x) for 64 samples, so the taps that
// fall outside the 7x7 input are the same for every row and are left out of
// the reduction: only the 1..9 valid taps x 64 channels are multiplied.
// rows b, cols c (64), reduction (valid tap, o) in chunks of 32 o.
// ---------------------------------------------------------------------------
template <int KP, class T>
struct Conv3DgradA {  // KMAJ quads dz3[b][p][o..o+3] at p = (y-u)*7 + (x-v)
    const T* dz3;
    int n, b0, y, x, u0, v0, nv;
    int64_t ps;  // KP planes of dz3, ps elements apart
    const T* base[MAXQ];
    __device__ void init(int j, int row, int k) {
        const int b = b0 + row;
        base[j] = dz3 + (int64_t)(b < n ? b : 0) * FLAT + k;  // rows past n: never stored
    }
    __device__ f32x4 load(int kc, int j) const {
        const int t = kc >> 1, u = u0 + t / nv, v = v0 + t % nv;
        return ld4_parts<KP>(base[j] + ((y - u) * H3 + (x - v)) * C3 + (kc & 1) * BK, ps);
    }
};
struct Conv3DgradB {  // w3d[(u,v)][c][o], rows c, quads along o
    const float* w3d;
    int u0, v0, nv;
    const float* base[MAXQ];
    __device__ void init(int j, int row, int k) { base[j] = w3d + row * C3 + k; }
    __device__ f32x4 load(int kc, int j) const {
        const int t = kc >> 1, tap = (u0 + t / nv) * K3 + v0 + t % nv;
        return ld4(base[j] + tap * C2 * C3 + (kc & 1) * BK);
    }
};
template <class T>
struct Conv3DgradStore {
    static constexpr bool MASK = true;
    T* dz2;
    const float* h2;
    int n, b0, pos;
    __device__ float pre(int row, int col) const {
        const int b = b0 + row;
        return h2[((int64_t)(b < n ? b : 0) * P2 + pos) * C2 + col];
    }
    __device__ void operator()(int row, int col, float v, float m) const {
        const int b = b0 + row;
        if (b >= n) return;
        stg(dz2 + ((int64_t)b * P2 + pos) * C2 + col, m > 0.0f ? v : 0.0f);
    }
};

// dz3 arrives as KP partial planes, and KP > 1 also cuts the reduction over
// (tap, o) into KP parts, each writing its own masked dz2 plane.
template <int BF, int KP>
struct Conv3DgradJob {
    const float* dz3;
    GroupPtrs w3d;
    const float* h2;
    float* dz2;
    int n, groups;
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? BF_WEIGHT : 0;
    using SH = GemmShape<64, 64, KMAJ, KMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int tiles() const { return P2 * ((n + 63) / 64); }
    __host__ __device__ int blocks() const { return pad_xcd(tiles() * groups * KP); }
    __device__ void run(int bid, float* smem) const {
        int t = xcd_tile(bid, blocks());
        if (t >= tiles() * groups * KP) return;
        const int part = t / (tiles() * groups);
        t -= part * tiles() * groups;
        const int g = t / tiles();
        t -= g * tiles();
        const int64_t rows = (int64_t)g * n, plane = (int64_t)groups * n;
        constexpr LongestFirst<H2, K3, H3> ORDER{};
        // the position is uniform over the workgroup: keep it (and what derives
        // from it) in scalar registers
        const int pos = __builtin_amdgcn_readfirstlane(ORDER.pos[t % P2]);
        const int y = pos / H2, x = pos - y * H2, b0 = (t / P2) * 64;
        const int u0 = max(0, y - (H3 - 1)), u1 = min(K3 - 1, y);
        const int v0 = max(0, x - (H3 - 1)), v1 = min(K3 - 1, x);
        const int nv = v1 - v0 + 1, taps = (u1 - u0 + 1) * nv;
        using G = GradT<BF, KP>;
        Conv3DgradA<KP, G> la{(const G*)dz3 + rows * FLAT, n, b0, y, x, u0, v0, nv, plane * FLAT};
        Conv3DgradB lb{w3d.p[g], u0, v0, nv};
        Conv3DgradStore<G> epi{(G*)dz2 + (part * plane + rows) * P2 * C2, h2 + rows * P2 * C2, n, b0, pos};
        mfma_gemm<64, 64, 2, KMAJ, KMAJ, PA, PB>(smem, part * 2 * taps / KP, (part + 1) * 2 * taps / KP,
                                                 la, lb, epi);
    }
};

// ---------------------------------------------------------------------------
// conv3 weight gradient: dW3[o][c][u][v] = sum_{b,i,j} dz3[b][i][j][o] h2[b][i+u][j+v][c]
// rows o (64), cols (tap, c): one tap of 64 channels per column tile,
// reduction over the n*49 output pixels, split across workgroups.
// partial[s][o][tap*64 + c].
// ---------------------------------------------------------------------------
template <int KP, class T>
struct Conv3WgradA {  // RMAJ quads dz3[b][p][o0..o0+3] at one output pixel m = (b, p)
    const T* dz3;
    int npix;
    int64_t ps;  // KP planes of dz3, ps elements apart
    int o0[MAXQ], kk[MAXQ];
    __device__ void init(int j, int row, int k) { o0[j] = row; kk[j] = k; }
    __device__ f32x4 load(int kc, int j) const {
        const int m = kc * BK + kk[j];
        return sel4(m < npix, ld4_parts<KP>(dz3 + (int64_t)(m < npix ? m : 0) * C3 + o0[j], ps));
    }
};
struct Conv3WgradB {  // RMAJ quads: 4 channels of h2 at one (pixel, tap)
    const float* h2;
    int npix, tap;
    int c0[MAXQ], kk[MAXQ];
    const float* pix = nullptr;  // h2 at this chunk's (pixel, tap), set by prep
    __device__ void init(int j, int row, int k) { c0[j] = row; kk[j] = k; }
    __device__ void prep(int kc) {  // the thread's quads share one pixel
        const int m = kc * BK + kk[0];
        const int mm = m < npix ? m : 0;  // past the end: pixel 0 (A is zero there)
        const int b = mm / P3, p = mm - b * P3, i = p / H3, jj = p - i * H3;
        const int u = tap / 3, v = tap - u * 3;
        pix = h2 + (((int64_t)b * H2 + i + u) * H2 + jj + v) * C2;
    }
    __device__ f32x4 load(int, int j) const { return ld4(pix + c0[j]); }
};

template <int BF, int KP>
struct Conv3WgradJob {
    const float* dz3;
    const float* h2;
    float* partial;
    float* bias_part;
    int n, splits, cps, groups;
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? BF_ACT_WGRAD : 0;
    using SH = GemmShape<64, 64, RMAJ, RMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int blocks() const { return pad_xcd(9 * splits * groups); }
    __device__ void run(int bid, float* smem) const {
        const int t = xcd_tile(bid, blocks());
        if (t >= 9 * splits * groups) return;
        // the nine taps of one split share dz3 rows; s runs over (group, split)
        const int tap = t % 9, s = t / 9, g = s / splits;
        const int npix = n * P3, nchunks = (npix + BK - 1) / BK;
        const int64_t rows = (int64_t)g * n;
        const int ks = s - g * splits;
        using G = GradT<BF, KP>;
        Conv3WgradA<KP, G> la{(const G*)dz3 + rows * FLAT, npix, (int64_t)groups * n * FLAT};
        Conv3WgradB lb{h2 + rows * P2 * C2, npix, tap};
        PartialEpi epi{partial + (int64_t)s * C3 * 9 * C2, 9 * C2, tap * C2, 1.0f};
        float* rs = tap == 0 ? bias_part + (int64_t)s * 64 : nullptr;
        mfma_gemm<64, 64, 2, RMAJ, RMAJ, PA, PB>(smem, ks * cps, min(nchunks, (ks + 1) * cps), la, lb, epi, rs);
    }
};

// Splits per group shrink with the group count so one launch stays near the
// same number of workgroups; groups * splits stays within WG_MAX_SPLITS.
template <int BF, int KP>
static void conv3_backward_jobs(const float* dz3, const GroupPtrs& w3d, int groups, const float* h2,
                                int n, float* dz2, float* partial, float* bias_part, int splits,
                                int cps, hipStream_t st) {
    launch_jobs(st, Conv3DgradJob<BF, KP>{dz3, w3d, h2, dz2, n, groups},
                Conv3WgradJob<BF, KP>{dz3, h2, partial, bias_part, n, splits, cps, groups});
}

// f(integral_constant<int, k>) for the plane count k in {1, 2, 4}
template <class F>
static void with_parts(int k, F&& f) {
    if (k == 4) f(std::integral_constant<int, 4>{});
    else if (k == 2) f(std::integral_constant<int, 2>{});
    else f(std::integral_constant<int, 1>{});
}

int launch_conv3_backward(const float* dz3, const GroupPtrs& w3d, int groups, const float* h2,
                          int n, float* dz2, float* partial, float* bias_part, int kp, bool bf16,
                          hipStream_t st) {
    if (n <= 0) return 0;
    const int nchunks = (n * P3 + BK - 1) / BK;
    int splits = min(min(WG_MAX_SPLITS / groups, nchunks), max(1, CONV3_WG_SPLITS / groups));
    const int cps = (nchunks + splits - 1) / splits;
    splits = (nchunks + cps - 1) / cps;
    with_parts(kp, [&](auto k) {
        if (bf16)
            conv3_backward_jobs<1, k.value>(dz3, w3d, groups, h2, n, dz2, partial, bias_part, splits,
                                            cps, st);
        else
            conv3_backward_jobs<0, k.value>(dz3, w3d, groups, h2, n, dz2, partial, bias_part, splits,
                                            cps, st);
    });
    return splits;
}

// ---------------------------------------------------------------------------
// conv2 data gradient (stride 2).  Output pixel (2y'+py, 2x'+px) receives
// taps u = py + 2du, v = px + 2dv from dz2[y'-du][x'-dv], du, dv in {0, 1}, so
// the four stride phases (py, px) of one (y', x') read the same four dz2
// pixels with different weights and no inserted zeros are multiplied.  A
// workgroup owns one (y', x') for 64 samples and two or all four phases as
// its columns (phase, c); taps that fall outside the 9x9 input are the same
// for every row and column and are skipped.  Reduction (valid tap, o) in
// chunks of 32 o; dz1 = dh1 * [h1 > 0].
// ---------------------------------------------------------------------------
template <int KP, class T>
struct Conv2DgradA {  // KMAJ quads dz2[b][i][j][o..o+3]
    const T* dz2;
    int n, b0, yy, xx, du0, dv0, ndv;
    int64_t ps;  // KP planes of dz2, ps elements apart
    const T* base[MAXQ];
    __device__ void init(int j, int row, int k) {
        const int b = b0 + row;
        base[j] = dz2 + (int64_t)(b < n ? b : 0) * P2 * C2 + k;  // rows past n: never stored
    }
    __device__ f32x4 load(int kc, int j) const {
        const int t = kc >> 1, du = du0 + t / ndv, dv = dv0 + t % ndv;
        return ld4_parts<KP>(base[j] + ((yy - du) * H2 + (xx - dv)) * C2 + (kc & 1) * BK, ps);
    }
};
struct Conv2DgradB {  // w2p[(du,dv)][phase][c][o], rows (phase, c), quads along o
    const float* w2p;
    int du0, dv0, ndv;
    const float* base[MAXQ];
    __device__ void init(int j, int row, int k) { base[j] = w2p + row * C2 + k; }
    __device__ f32x4 load(int kc, int j) const {
        const int t = kc >> 1, tp = (du0 + t / ndv) * 2 + dv0 + t % ndv;
        return ld4(base[j] + tp * 4 * C1 * C2 + (kc & 1) * BK);
    }
};
// bf16 steps store dz1 rounded to bf16 (the precision the conv1 weight
// gradient multiplies it in), half the bytes of the fp32 steps' dz1.
template <int BF>
struct Conv2DgradStore {
    static constexpr bool MASK = true;
    using T = std::conditional_t<BF == 1, uint16_t, float>;
    T* dz1;
    const float* h1;
    int n, b0, yy, xx, c0;  // c0: the tile's first column (phase, c)
    __device__ int64_t at(int b, int col) const {
        const int phase = (c0 + col) >> 5, c = col & 31;
        const int y = 2 * yy + (phase >> 1), x = 2 * xx + (phase & 1);
        return (((int64_t)b * H1 + y) * H1 + x) * C1 + c;
    }
    __device__ float pre(int row, int col) const {
        const int b = b0 + row;
        return h1[at(b < n ? b : 0, col)];
    }
    __device__ void operator()(int row, int col, float v, float m) const {
        const int b = b0 + row;
        if (b >= n) return;
        const float r = m > 0.0f ? v : 0.0f;
        if constexpr (BF == 1) dz1[at(b, col)] = __builtin_bit_cast(uint16_t, (__bf16)r);
        else dz1[at(b, col)] = r;
    }
};

template <int BF, int KP>
struct Conv2DgradJob {
    const float* dz2;
    GroupPtrs w2p;
    const float* h1;
    float* dz1;
    int n, groups;
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? BF_WEIGHT : 0;
    // fp32: two phases per tile (more, smaller workgroups measured faster:
    // 69 -> 67 us at batch 512, 19 -> 14.5 us at batch 32); bf16: all four
    static constexpr int BN = BF ? 128 : 64, NCT = 128 / BN;
    using SH = GemmShape<64, BN, KMAJ, KMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int tiles() const { return 100 * NCT * ((n + 63) / 64); }
    __host__ __device__ int blocks() const { return pad_xcd(tiles() * groups); }
    __device__ void run(int bid, float* smem) const {
        int t = xcd_tile(bid, blocks());
        if (t >= tiles() * groups) return;
        const int g = t / tiles();
        t -= g * tiles();
        const int64_t rows = (int64_t)g * n;
        // the column tiles of one position adjacent, positions longest first
        constexpr LongestFirst<10, 2, H2> ORDER{};
        const int ct = t % NCT, b0 = (t / (100 * NCT)) * 64;
        const int pos = __builtin_amdgcn_readfirstlane(ORDER.pos[(t / NCT) % 100]);  // uniform
        const int yy = pos / 10, xx = pos % 10;
        const int du0 = max(0, yy - (H2 - 1)), du1 = min(1, yy);
        const int dv0 = max(0, xx - (H2 - 1)), dv1 = min(1, xx);
        const int ndv = dv1 - dv0 + 1, taps = (du1 - du0 + 1) * ndv;
        using G = GradT<BF, KP>;
        Conv2DgradA<KP, G> la{(const G*)dz2 + rows * P2 * C2, n, b0, yy, xx, du0, dv0, ndv,
                              (int64_t)groups * n * P2 * C2};
        Conv2DgradB lb{w2p.p[g] + ct * BN * C2, du0, dv0, ndv};
        Conv2DgradStore<BF> epi{(typename Conv2DgradStore<BF>::T*)dz1 + rows * P1 * C1, h1 + rows * P1 * C1,
                                n, b0, yy, xx, ct * BN};
        mfma_gemm<64, BN, 2, KMAJ, KMAJ, PA, PB>(smem, 0, 2 * taps, la, lb, epi);
    }
};

// ---------------------------------------------------------------------------
// conv2 weight gradient: dW2[o][c][u][v] = sum_{b,i,j} dz2[b][i][j][o] h1[b][2i+u][2j+v][c]
// rows o (64), cols (tap, c) with two taps per 64-column tile, reduction over
// the n*81 output pixels split across workgroups.  partial[s][o][tap*32 + c].
// ---------------------------------------------------------------------------
template <int KP, class T>
struct Conv2WgradA {  // dz2 quads along o at one pixel
    const T* dz2;
    int npix;
    int64_t ps;  // KP planes of dz2, ps elements apart
    int o0[MAXQ], kk[MAXQ];
    __device__ void init(int j, int row, int k) { o0[j] = row; kk[j] = k; }
    __device__ f32x4 load(int kc, int j) const {
        const int m = kc * BK + kk[j];
        return sel4(m < npix, ld4_parts<KP>(dz2 + (int64_t)(m < npix ? m : 0) * C2 + o0[j], ps));
    }
};
struct Conv2WgradB {  // h1 quads along c at one (pixel, tap)
    const float* h1;
    int npix, tap0;
    int off[MAXQ], kk[MAXQ];
    __device__ void init(int j, int row, int k) {
        const int t = tap0 + (row >> 5), c0 = row & 31;
        off[j] = ((t >> 2) * H1 + (t & 3)) * C1 + c0;
        kk[j] = k;
    }
    const float* pix = nullptr;  // h1 at this chunk's pixel, set by prep
    __device__ void prep(int kc) {  // the thread's quads share one pixel
        const int m = kc * BK + kk[0];
        const int mm = m < npix ? m : 0;  // past the end: pixel 0 (A is zero there)
        const int b = mm / P2, p = mm - b * P2, i = p / H2, jj = p - i * H2;
        pix = h1 + (((int64_t)b * H1 + S2 * i) * H1 + S2 * jj) * C1;
    }
    __device__ f32x4 load(int, int j) const { return ld4(pix + off[j]); }
};

template <int BF, int KP>
struct Conv2WgradJob {
    const float* dz2;
    const float* h1;
    float* partial;
    float* bias_part;
    int n, splits, cps, groups;
    static constexpr int PA = BF ? BF_GRAD : 0, PB = BF ? BF_ACT_WGRAD : 0;
    using SH = GemmShape<64, 64, RMAJ, RMAJ, PA, PB>;
    static constexpr int SMEM = SH::SMEM_FLOATS;
    __host__ __device__ int blocks() const { return pad_xcd(8 * splits * groups); }
    __device__ void run(int bid, float* smem) const {
        const int t = xcd_tile(bid, blocks());
        if (t >= 8 * splits * groups) return;
        // the column tiles of one split share dz2 rows; s runs over (group, split)
        const int tap0 = (t % 8) * 2, s = t / 8, g = s / splits;
        const int npix = n * P2, nchunks = (npix + BK - 1) / BK;
        const int64_t rows = (int64_t)g * n;
        const int ks = s - g * splits;
        using G = GradT<BF, KP>;
        Conv2WgradA<KP, G> la{(const G*)dz2 + rows * P2 * C2, npix, (int64_t)groups * n * P2 * C2};
        Conv2WgradB lb{h1 + rows * P1 * C1, npix, tap0};
        PartialEpi epi{partial + (int64_t)s * C2 * 16 * C1, 16 * C1, tap0 * C1, 1.0f};
        float* rs = tap0 == 0 ? bias_part + (int64_t)s * 64 : nullptr;
        mfma_gemm<64, 64, 2, RMAJ, RMAJ, PA, PB>(smem, ks * cps, min(nchunks, (ks + 1) * cps), la, lb, epi, rs);
    }
};

// the weight-gradient workgroups are the longer ones (21 chunks against at
// most 8 at batch 512): dispatched first, they do not trail the launch
template <int BF, int KP>
static void conv2_backward_jobs(const float* dz2, const GroupPtrs& w2p, int groups, const float* h1,
                                int n, float* dz1, float* partial, float* bias_part, int splits,
                                int cps, hipStream_t st) {
    launch_jobs(st, Conv2WgradJob<BF, KP>{dz2, h1, partial, bias_part, n, splits, cps, groups},
                Conv2DgradJob<BF, KP>{dz2, w2p, h1, dz1, n, groups});
}

int launch_conv2_backward(const float* dz2, const GroupPtrs& w2p, int groups, const float* h1,
                          int n, float* dz1, float* partial, float* bias_part, int kp, bool bf16,
                          hipStream_t st) {
    if (n <= 0) return 0;
    const int nchunks = (n * P2 + BK - 1) / BK;
    int splits = min(min(WG_MAX_SPLITS / groups, nchunks), max(1, CONV2_WG_SPLITS / groups));
    const int cps = (nchunks + splits - 1) / splits;
    splits = (nchunks + cps - 1) / cps;
    with_parts(kp, [&](auto k) {
        if (bf16)
            conv2_backward_jobs<1, k.value>(dz2, w2p, groups, h1, n, dz1, partial, bias_part, splits,
                                            cps, st);
        else
            conv2_backward_jobs<0, k.value>(dz2, w2p, groups, h1, n, dz1, partial, bias_part, splits,
                                            cps, st);
    });
    return splits;
}

// ---------------------------------------------------------------------------
// Final reduction.  Every output element is a sum of partials (split partials
// of the conv weight gradients, bias partials, row-block partials of dW5, db5
// and the loss) scattered to its place in the flat layout.  Two kernels:
//
// One learner group (many partials per element: tens to hundreds of
// splits): a block owns 64 consecutive elements of the list below; its four
// waves each add every fourth partial, sixteen loads in flight, then one wave
// adds the four sums in wave order.
//   [0, N1)            dW1   (partials already in [o][c][u][v] order)
//   [.., +N2)          dW2   (partials [o][(u*4+v)*32 + c])
//   [.., +N3)          dW3   (partials [o][(u*3+v)*64 + c])
//   [.., +160)         db1, db2, db3
//   [.., +A*512)       dW5
//   [.., +A)           db5
//   [.., +1)           loss (divided by the batch size)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void grad_reduce_kernel(ReduceArgs ra) {
    constexpr int N1 = C1 * 256, N2 = C2 * 16 * C1, N3 = C3 * 9 * C2;
    constexpr int E0 = N1 + N2 + N3, E1 = E0 + C1 + C2 + C3;
    const int E2 = E1 + ra.A * HID, E3 = E2 + ra.A;
    __shared__ float red[4][64];
    const int el = threadIdx.x & 63, sq = threadIdx.x >> 6;
    const int e = blockIdx.x * 64 + el;
    // learner group blockIdx.y: its own partial blocks, gradient and loss
    const int g = blockIdx.y;
    ra.part1 += (int64_t)g * ra.s1 * N1;
    ra.part2 += (int64_t)g * ra.s2 * N2;
    ra.part3 += (int64_t)g * ra.s3 * N3;
    ra.hpart += (int64_t)g * ra.head_blocks * HP_STRIDE;
    ra.grads += g * ra.grads_stride;
    ra.loss_out += g;
    const float* src = nullptr;
    int nsplit = 0, stride = 0;
    float* dst = nullptr;
    float scale = 1.0f;
    if (e < N1) {
        src = ra.part1 + e; nsplit = ra.s1; stride = N1; dst = ra.grads + OFF_W1 + e;
    } else if (e < N1 + N2) {
        const int p = e - N1;
        src = ra.part2 + p; nsplit = ra.s2; stride = N2;
        const int o = p >> 9, t = (p >> 5) & 15, c = p & 31;
        dst = ra.grads + OFF_W2 + ((o * C1 + c) * K2 + (t >> 2)) * K2 + (t & 3);
    } else if (e < E0) {
        const int p = e - N1 - N2;
        src = ra.part3 + p; nsplit = ra.s3; stride = N3;
        const int o = p / 576, t = (p / 64) % 9, c = p & 63;
        dst = ra.grads + OFF_W3 + ((o * C2 + c) * K3 + t / 3) * K3 + t % 3;
    } else if (e < E1) {
        const int q = e - E0;
        int layer = 2, o = q - C1 - C2;
        if (q < C1) { layer = 0; o = q; }
        else if (q < C1 + C2) { layer = 1; o = q - C1; }
        nsplit = layer == 0 ? ra.s1 : layer == 1 ? ra.s2 : ra.s3;
        src = ra.bias_part + (int64_t)layer * BIAS_PART_STRIDE + (int64_t)g * nsplit * 64 + o;
        stride = 64;
        dst = ra.grads + (layer == 0 ? OFF_B1 : layer == 1 ? OFF_B2 : OFF_B3) + o;
    } else if (e < E2) {
        const int q = e - E1;
        src = ra.hpart + q; nsplit = ra.head_blocks; stride = HP_STRIDE;
        dst = ra.grads + OFF_W5 + q;
    } else if (e < E3) {
        const int q = e - E2;
        src = ra.hpart + HP_DB5 + q; nsplit = ra.head_blocks; stride = HP_STRIDE;
        dst = ra.grads + off_b5(ra.A) + q;
    } else if (e == E3) {
        src = ra.hpart + HP_LOSS; nsplit = ra.head_blocks; stride = HP_STRIDE;
        dst = ra.loss_out;
        scale = 1.0f / (float)ra.n;
    }
    // partials s = sq, sq + 4, ... added in that order; sixteen of them are
    // loaded before the first is added, so the loads overlap
    float acc = 0.0f;
    if (dst) {
        for (int s0 = sq; s0 < nsplit; s0 += 4 * 16) {
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int s = s0 + 4 * u;
                v[u] = s < nsplit ? src[(int64_t)s * stride] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (s0 + 4 * u < nsplit) acc += v[u];
        }
    }
    red[sq][el] = acc;
    __syncthreads();
    if (sq == 0 && dst) *dst = (((red[0][el] + red[1][el]) + red[2][el]) + red[3][el]) * scale;
}


// Several learner groups (a few partials per element, many elements): the
// elements of each group form the segments below; a segment with n partials
// per element gives each element `sq` split lanes (the smallest power of two
// with n / sq <= RED_LOADS), each thread reading 16-byte quads of four
// consecutive elements, so a block covers up to 1024 elements.  Lane j adds
// partials j, j + sq, j + 2 sq, ... in order and the lane sums are then added
// in lane order.  (Measured: with one group the first kernel is faster, 9.7
// against 11.7 us at batch 512; with 16 groups of 64 rows this one, 14.4
// against 26.8 us.)
//   dW1   partials already in [o][c][u][v] order
//   dW2   partials [o][(u*4+v)*32 + c]
//   dW3   partials [o][(u*3+v)*64 + c]
//   db1, db2, db3, dW5, db5
//   loss  divided by the batch size
// ---------------------------------------------------------------------------
enum { SEG_W1, SEG_W2, SEG_W3, SEG_B1, SEG_B2, SEG_B3, SEG_W5, SEG_B5, SEG_LOSS, NSEG };
constexpr int RED_LOADS = 8;
struct ReduceSeg {
    const float* src;  // group 0, split 0, element 0
    int gstride;       // floats between groups
    int sstride;       // floats between splits
    int nsplit, nel, width, lsq, block0;  // 1 << lsq split lanes
};
struct ReducePlan {
    ReduceSeg seg[NSEG];
    float* grads;
    int64_t grads_stride;
    float* loss_out;
    float inv_n;
    int A;
};

__device__ inline int64_t reduce_dst(int kind, int e, int A) {
    switch (kind) {
    case SEG_W1: return OFF_W1 + e;
    case SEG_W2: {
        const int o = e >> 9, t = (e >> 5) & 15, c = e & 31;
        return OFF_W2 + ((o * C1 + c) * K2 + (t >> 2)) * K2 + (t & 3);
    }
    case SEG_W3: {
        const int o = e / 576, t = (e / 64) % 9, c = e & 63;
        return OFF_W3 + ((o * C2 + c) * K3 + t / 3) * K3 + t % 3;
    }
    case SEG_B1: return OFF_B1 + e;
    case SEG_B2: return OFF_B2 + e;
    case SEG_B3: return OFF_B3 + e;
    case SEG_W5: return OFF_W5 + e;
    default: return off_b5(A) + e;  // SEG_B5
    }
}

__global__ __launch_bounds__(256) void grad_reduce_grouped_kernel(ReducePlan rp) {
    __shared__ f32x4 red[256];
    // every segment's fields are read at once and this block's selected, so
    // the argument loads are one round trip (indexing the table by a value
    // computed from other arguments would be two)
    int kind = 0;
    ReduceSeg sg = rp.seg[0];
#pragma unroll
    for (int k = 1; k < NSEG; ++k) {
        const ReduceSeg c = rp.seg[k];
        const bool take = (int)blockIdx.x >= c.block0;
        kind = take ? k : kind;
        sg.src = take ? c.src : sg.src;
        sg.gstride = take ? c.gstride : sg.gstride;
        sg.sstride = take ? c.sstride : sg.sstride;
        sg.nsplit = take ? c.nsplit : sg.nsplit;
        sg.nel = take ? c.nel : sg.nel;
        sg.width = take ? c.width : sg.width;
        sg.lsq = take ? c.lsq : sg.lsq;
        sg.block0 = take ? c.block0 : sg.block0;
    }
    const int t = threadIdx.x, lq = 8 - sg.lsq, qpb = 1 << lq, qi = t & (qpb - 1), lane = t >> lq;
    const int sq = 1 << sg.lsq;
    const int e0 = (((int)blockIdx.x - sg.block0) * qpb + qi) * sg.width;
    const int g = blockIdx.y;
    const float* src = sg.src + g * sg.gstride + e0;
    f32x4 acc = {};
    if (e0 < sg.nel) {
        for (int s0 = lane; s0 < sg.nsplit; s0 += RED_LOADS * sq) {
            f32x4 v[RED_LOADS];
#pragma unroll
            for (int u = 0; u < RED_LOADS; ++u) {
                const int s = s0 + u * sq;
                v[u] = f32x4{};
                if (s < sg.nsplit) {
                    if (sg.width == 4) v[u] = ld4(src + s * sg.sstride);
                    else v[u][0] = src[s * sg.sstride];
                }
            }
#pragma unroll
            for (int u = 0; u < RED_LOADS; ++u)
                if (s0 + u * sq < sg.nsplit) acc += v[u];
        }
    }
    red[t] = acc;
    __syncthreads();
    if (lane != 0 || e0 >= sg.nel) return;
    // the lane sums in lane order, eight LDS reads in flight at a time
    f32x4 sum = {};
    for (int j0 = 0; j0 < sq; j0 += 8) {
        f32x4 r[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) r[u] = j0 + u < sq ? red[((j0 + u) << lq) + qi] : f32x4{};
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (j0 + u < sq) sum += r[u];
    }
    if (kind == SEG_LOSS) {
        rp.loss_out[g] = sum[0] * rp.inv_n;
        return;
    }
    float* grads = rp.grads + g * rp.grads_stride;
    for (int i = 0; i < sg.width && e0 + i < sg.nel; ++i) grads[reduce_dst(kind, e0 + i, rp.A)] = sum[i];
}

void launch_grad_reduce(const ReduceArgs& ra, hipStream_t st) {
    if (ra.groups == 1) {
        const int total = C1 * 256 + C2 * 16 * C1 + C3 * 9 * C2 + C1 + C2 + C3 + ra.A * HID + ra.A + 1;
        grad_reduce_kernel<<<dim3((total + 63) / 64, 1), 256, 0, st>>>(ra);
        return;
    }
    ReducePlan rp{};
    auto set = [&](int kind, const float* src, int64_t gstride, int sstride, int nsplit, int nel,
                   int width) {
        ReduceSeg& sg = rp.seg[kind];
        sg.src = src;
        sg.gstride = (int)gstride;  // < 2^31: at most 512 splits of 36864 floats
        sg.sstride = sstride;
        sg.nsplit = nsplit;
        sg.nel = nel;
        sg.width = width;
        sg.lsq = 0;
        while (sg.lsq < 6 && (RED_LOADS << sg.lsq) < nsplit) ++sg.lsq;
    };
    constexpr int N1 = C1 * 256, N2 = C2 * 16 * C1, N3 = C3 * 9 * C2;
    set(SEG_W1, ra.part1, (int64_t)ra.s1 * N1, N1, ra.s1, N1, 4);
    set(SEG_W2, ra.part2, (int64_t)ra.s2 * N2, N2, ra.s2, N2, 4);
    set(SEG_W3, ra.part3, (int64_t)ra.s3 * N3, N3, ra.s3, N3, 4);
    set(SEG_B1, ra.bias_part, (int64_t)ra.s1 * 64, 64, ra.s1, C1, 4);
    set(SEG_B2, ra.bias_part + BIAS_PART_STRIDE, (int64_t)ra.s2 * 64, 64, ra.s2, C2, 4);
    set(SEG_B3, ra.bias_part + 2 * BIAS_PART_STRIDE, (int64_t)ra.s3 * 64, 64, ra.s3, C3, 4);
    const int64_t hg = (int64_t)ra.head_blocks * HP_STRIDE;
    set(SEG_W5, ra.hpart, hg, HP_STRIDE, ra.head_blocks, ra.A * HID, 4);
    set(SEG_B5, ra.hpart + HP_DB5, hg, HP_STRIDE, ra.head_blocks, ra.A, 1);
    set(SEG_LOSS, ra.hpart + HP_LOSS, hg, HP_STRIDE, ra.head_blocks, 1, 1);
    int blocks = 0;
    for (int k = 0; k < NSEG; ++k) {
        ReduceSeg& sg = rp.seg[k];
        sg.block0 = blocks;
        const int quads = (sg.nel + sg.width - 1) / sg.width, qpb = 256 >> sg.lsq;
        blocks += (quads + qpb - 1) / qpb;
    }
    rp.grads = ra.grads;
    rp.grads_stride = ra.grads_stride;
    rp.loss_out = ra.loss_out;
    rp.inv_n = 1.0f / (float)ra.n;
    rp.A = ra.A;
    grad_reduce_grouped_kernel<<<dim3(blocks, ra.groups), 256, 0, st>>>(rp);
}

}  // namespace gorila
