// Shared device-side definitions for the Gorila learner-step kernels (gfx950).
//
// Network (Nair et al. 2015, Section 5.1): 4x84x84 uint8 input scaled by
// 1/255, conv 32@8x8 stride 4 -> 20x20, conv 64@4x4 stride 2 -> 9x9,
// conv 64@3x3 stride 1 -> 7x7, FC 3136 -> 512, linear FC 512 -> A, ReLU after
// every hidden layer.  Parameters are one flat fp32 vector: W1 [32,4,8,8],
// b1, W2 [64,32,4,4], b2, W3 [64,64,3,3], b3, W4 [512,3136], b4, W5 [A,512], b5.
//
// Activation layouts in the workspace (chosen so every producer stores and
// every consumer loads whole 16-byte vectors):
//   h1, dz1 : [n][20][20][32]  pixel-major, channel-minor (NHWC)
//   h2, dz2 : [n][9][9][64]    NHWC
//   h3      : [n][64][49]      channel-major: the flatten order of the FC input
//   dz3     : [n][49][64]      NHWC
//   h4, dz4 : [n][512]
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace gorila {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int IN_C = 4, IN_H = 84, IN_W = 84;
constexpr int FRAME_BYTES = IN_H * IN_W;          // 7056 = 441 x 16 bytes
constexpr int STATE_BYTES = IN_C * FRAME_BYTES;   // 28224
constexpr int C1 = 32, K1 = 8, S1 = 4, H1 = 20, P1 = H1 * H1;  // 400 pixels
constexpr int C2 = 64, K2 = 4, S2 = 2, H2 = 9, P2 = H2 * H2;   // 81
constexpr int C3 = 64, K3 = 3, H3 = 7, P3 = H3 * H3;           // 49
constexpr int FLAT = C3 * P3;                                  // 3136
constexpr int HID = 512;
constexpr int MAX_ACTIONS = 32;

constexpr int64_t OFF_W1 = 0, OFF_B1 = 8192, OFF_W2 = 8224, OFF_B2 = 40992,
                  OFF_W3 = 41056, OFF_B3 = 77920, OFF_W4 = 77984,
                  OFF_B4 = 1683616, OFF_W5 = 1684128;
__host__ __device__ constexpr int64_t off_b5(int A) { return OFF_W5 + (int64_t)HID * A; }
__host__ __device__ constexpr int64_t param_count(int A) { return off_b5(A) + A; }

// Up to MAX_GROUPS parameter sets per launch, passed by value.
constexpr int MAX_GROUPS = 32;
// Learner groups per grouped step: their online and target forward passes
// (2 per group) share the forward launches.
constexpr int MAX_LEARNER_GROUPS = MAX_GROUPS / 2;
struct GroupPtrs {
    const float* p[MAX_GROUPS];
};
struct GroupPtrs16 {  // bf16 bit patterns
    const uint16_t* p[MAX_GROUPS];
};

// Sticky device error bits (workspace word 0).
constexpr unsigned ERR_IDX_RANGE = 1u, ERR_ACTION_RANGE = 2u;

// ---------------------------------------------------------------------------
// fp32 MFMA tile engine.
//
// One 256-thread workgroup (4 wave64s) computes a BM x BN tile of
// C = sum_k A[row][k] * B[col][k] with v_mfma_f32_32x32x2_f32.  The reduction
// runs in chunks of BK = 32 that are staged through LDS, double buffered, one
// barrier per chunk.  Each operand tile lives in LDS in one of two layouts:
//   KMAJ: [rows][BK]       (reduction index contiguous; read as one b128;
//                           the 8 quads of row r are stored XOR-permuted by
//                           (r ^ r >> 3) & 7, so 16 consecutive rows read or
//                           written at one quad cover every LDS bank once)
//   RMAJ: [BK][rows + 4]   (row index contiguous; read as four b32)
// and is filled from global memory in 16-byte quads that are contiguous in
// the operand's natural global layout: along k for KMAJ, along rows for RMAJ.
//
// Inside every group of 8 reduction indices, lane half h (lane / 32) feeds
// indices 4h .. 4h+3 to four consecutive MFMAs, so a lane's four values are
// one contiguous LDS vector.  A and B use the same permutation, so the sum is
// unchanged.
//
// Accumulator element r of lane l in a 32x32 tile is row 8*(r/4) + 4*(l/32)
// + r%4, column l%32, so each epilogue store of a wave writes two runs of 32
// consecutive columns.
// ---------------------------------------------------------------------------
constexpr int BK = 32;
enum { KMAJ = 0, RMAJ = 1 };

template <int ROWS, int MODE>
struct LdsTile {
    static constexpr int LD = MODE == KMAJ ? BK : ROWS + 4;
    __device__ static inline int swz(int row, int k) {  // KMAJ: k of quad (k / 4) in LDS
        return (((k >> 2) ^ (row ^ (row >> 3))) & 7) << 2;
    }
    static constexpr int SIZE = MODE == KMAJ ? ROWS * LD : BK * LD;  // floats
    static constexpr int QUADS = ROWS * BK / 4;
    static constexpr int NQ = (QUADS + 255) / 256;   // quads per thread

    // Tile coordinates (row, k) of the first element of quad j of thread t.
    // RMAJ: all NQ quads of a thread share one k (rows 4s, 4(s + S), ... with
    // S = ROWS / (4 NQ) threads per k), so a loader can decompose the
    // reduction index once per chunk for all of them.
    __device__ static inline void quad_coord(int t, int j, int& row, int& k) {
        if (MODE == KMAJ) {
            const int e = t + 256 * j;
            row = e / (BK / 4);
            k = (e % (BK / 4)) * 4;
        } else {
            constexpr int S = ROWS / 4 / NQ;  // threads per k
            k = t / S;
            row = ((t % S) + S * j) * 4;
        }
    }
    __device__ static inline void put(float* s, int row, int k, f32x4 v) {
        if (MODE == KMAJ) *(f32x4*)(s + row * LD + swz(row, k)) = v;
        else              *(f32x4*)(s + k * LD + row) = v;
    }
    // Values (row r, k = kb .. kb+3).
    __device__ static inline f32x4 get(const float* s, int r, int kb) {
        if (MODE == KMAJ) return *(const f32x4*)(s + r * LD + swz(r, kb));
        f32x4 v;
        v[0] = s[(kb + 0) * LD + r];
        v[1] = s[(kb + 1) * LD + r];
        v[2] = s[(kb + 2) * LD + r];
        v[3] = s[(kb + 3) * LD + r];
        return v;
    }
};

// Loaders keep per-quad state in arrays of MAXQ entries.  A loader may also
// have prep(kc), called once per chunk before its load(kc, j) calls (an RMAJ
// loader's quads share one k, so per-k work can be done there once).
constexpr int MAXQ = 4;
template <class T, class = void> struct HasPrep : std::false_type {};
template <class T>
struct HasPrep<T, std::void_t<decltype(std::declval<T&>().prep(0))>> : std::true_type {};
// An epilogue with `static constexpr bool MASK = true` only tests pre > 0.
template <class T, class = void> struct IsMaskEpi : std::false_type {};
template <class T>
struct IsMaskEpi<T, std::void_t<decltype(T::MASK)>> : std::bool_constant<T::MASK> {};

// ---------------------------------------------------------------------------
// bf16 operands (v_mfma_f32_32x32x16_bf16, fp32 accumulation).
//
// With P > 0 the engine below keeps an operand in LDS as P planes of bf16
// instead of fp32: plane 0 holds each value rounded to the nearest bf16, and
// with P = 2 plane 1 holds the rounding residual, itself rounded to bf16, so
// that hi + lo carries about 16 significant bits and the engine adds both
// products hi*B and lo*B.  The loaders still deliver fp32 quads; they are
// converted as they are stored to LDS.  A plane is [rows][BK] bf16 (64 bytes
// a row) whose four 16-byte chunks are stored XOR-permuted by (r >> 2) & 3:
// rows r and r + 4k share LDS banks, and the permutation spreads them
// (measured: no bank conflicts for k-contiguous operands, against 0.33-0.6
// of LDS cycles for permutations by the low row bits or none).  Lane l of an MFMA supplies row l % 32 and the
// eight reduction indices 8 (l / 32) .. +7 of its 16-wide step; the
// accumulator layout is that of the fp32 instruction.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

template <int ROWS, int PL>
struct Bf16Tile {
    static constexpr int PLANE = ROWS * BK * 2;  // bytes
    static constexpr int BYTES = PL * PLANE;
    __device__ static inline int chunk(int row, int c) {
        return row * (BK * 2) + (((c ^ (row >> 2)) & 3) << 4);
    }
    // Quad v of a MODE-laid operand at tile coordinates (row, k): KMAJ quads
    // are 4 reduction indices of one row, RMAJ quads 4 rows at one index.
    template <int MODE>
    __device__ static inline void put(char* s, int row, int k, f32x4 v) {
        // two values per rounding instruction; a rounded pair widens back by
        // moving each half to the top of a word, and the residual is exact
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const bf16x2 h01 = __builtin_convertvector(f32x2{v[0], v[1]}, bf16x2);
        const bf16x2 h23 = __builtin_convertvector(f32x2{v[2], v[3]}, bf16x2);
        const bf16x4 hi = __builtin_shufflevector(h01, h23, 0, 1, 2, 3);
        bf16x4 lo;
        if (PL == 2) {
            const uint32_t b01 = __builtin_bit_cast(uint32_t, h01);
            const uint32_t b23 = __builtin_bit_cast(uint32_t, h23);
            const bf16x2 l01 = __builtin_convertvector(
                f32x2{v[0] - __uint_as_float(b01 << 16), v[1] - __uint_as_float(b01 & 0xffff0000u)},
                bf16x2);
            const bf16x2 l23 = __builtin_convertvector(
                f32x2{v[2] - __uint_as_float(b23 << 16), v[3] - __uint_as_float(b23 & 0xffff0000u)},
                bf16x2);
            lo = __builtin_shufflevector(l01, l23, 0, 1, 2, 3);
        }
        if (MODE == KMAJ) {
            const int off = chunk(row, k >> 3) + ((k & 4) << 1);
            *(bf16x4*)(s + off) = hi;
            if (PL == 2) *(bf16x4*)(s + PLANE + off) = lo;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int off = chunk(row + e, k >> 3) + ((k & 7) << 1);
                *(__bf16*)(s + off) = hi[e];
                if (PL == 2) *(__bf16*)(s + PLANE + off) = lo[e];
            }
        }
    }
    __device__ static inline bf16x8 get(const char* s, int plane, int row, int c) {
        return *(const bf16x8*)(s + plane * PLANE + chunk(row, c));
    }
};

// Planes per operand role when a step runs on bf16 parameters.  Forward
// activations are split: the TD error is a small difference of Q values, so
// Q needs more than bf16's 8 bits (rounding every activation to bf16 leaves
// gradients several percent off, split activations about 0.2 %).  Weights are
// bf16 values already, exact in one plane; the backward pass rounds both its
// gradients and the activations its weight gradients read (measured: worst
// tensor 2.5e-3 relative L2 either way; the split weight-gradient operand
// only moved W2-W4 from 0.9-2.4e-3 to 0.3-1.9e-3, at two MFMAs instead of one).
constexpr int BF_ACT_FWD = 2, BF_WEIGHT = 1, BF_GRAD = 1, BF_ACT_WGRAD = 1;

// PA, PB: bf16 planes of A and B (0 and 0: the fp32 engine).
// SB: one LDS stage instead of two (half the LDS, so more workgroups are
// resident on a compute unit, at two barriers a chunk instead of one).
template <int BM, int BN, int AMODE, int BMODE, int PA = 0, int PB = 0, bool SB = false>
struct GemmShape {
    static_assert((PA > 0) == (PB > 0) && PA <= 2 && PB <= 2, "both operands fp32, or both bf16");
    using LA = LdsTile<BM, AMODE>;
    using LB = LdsTile<BN, BMODE>;
    using TA = Bf16Tile<BM, PA ? PA : 1>;
    using TB = Bf16Tile<BN, PB ? PB : 1>;
    static constexpr int STAGE_FLOATS = PA ? (TA::BYTES + TB::BYTES) / 4 : LA::SIZE + LB::SIZE;
    static constexpr int SMEM_FLOATS = (SB ? 1 : 2) * STAGE_FLOATS;
};

// One piece of a tile whose reduction is cut into np pieces run by different
// workgroups (np == 1: the whole tile, no hand-off).  Each piece stores its
// accumulators to ws[piece] (tile-private, np * BM * BN floats) and counts
// itself in *cnt; the piece that counts last adds the np partial tiles in
// piece order, so the sum does not depend on which piece finishes last, runs
// the epilogue and sets *cnt back to 0 for the next launch.  No piece waits
// for another.
//
// All pieces of a tile run on one XCD (TailSplit places them so: workgroup
// ids that agree mod 8 share an XCD whenever a partition dispatches
// round-robin over 1, 2, 4 or 8 XCDs, which gorila_ctx_create checks on the
// device), so the pieces, on different compute units, share one L2: the
// coherence point of the compiler's own protocol for workgroups whose waves
// span compute units (workgroup scope with thread-group split), which the
// hand-off follows:
//  - release: every thread waits until its stores have completed (they write
//    through the per-unit L1 to that L2), a barrier, then one atomic add on
//    the tile's counter (performed in the L2);
//  - acquire: the piece that counted last invalidates its compute unit's L1
//    (buffer_inv sc0) before it loads the other pieces' tiles, so they come
//    from the L2; the asm statement also keeps the compiler from moving the
//    loads above it.
// The agent-scope forms (an L2 write-back before the add and an L2
// invalidation or L2-bypassing loads after it) would make the exchange
// coherent across XCDs too, but they write back or drop every other
// workgroup's lines in the L2, and measured slower (see the design notes).
constexpr int SPLIT_MAX_TILES = 128, SPLIT_MAX_PIECES = 16, SPLIT_MAX_SLOTS = 512;
constexpr int SPLIT_TILE_FLOATS = 64 * 64;
struct SplitPiece {
    float* ws = nullptr;
    int* cnt = nullptr;
    int piece = 0, np = 1;
};

// Loaders: `la.init(j, row, k)` is called once per quad slot j of this thread
// with the quad's tile coordinates; `la.load(kc, j)` returns the quad for
// reduction chunk kc (zeros where the operand is zero-padded).
// If rowsum_out is not null, rowsum_out[t] (t < BM) receives sum_k A[t][k]
// over this workgroup's reduction range: wave w adds the k of every chunk in
// [8w, 8w + 8) for rows lane < BM (so the four waves carry equal extra work),
// and the four wave sums are added in wave order at the end (BM <= 64 only).
//
// Epilogue protocol: epi.pre(row, col) returns a value the epilogue needs for
// that output element (a ReLU mask, a bias, or 0 when it needs none); it is
// called for every accumulator element before the reduction loop, so its
// loads overlap the loop instead of waiting behind the epilogue's own stores.
// epi(row, col, value, pre) then writes the element.  A mask epilogue's
// values are kept as one bit per element (pre > 0), 16 bits per accumulator
// tile instead of 16 registers, and handed back as 1 or 0.
//
// The chunk loop is unrolled by two so that the LDS buffer and the register
// set of every access are compile-time constants: LDS is then addressed with
// ds_read/ds_write, and each global load is waited for only where its data is
// stored to LDS, one chunk later.
template <int BM, int BN, int WAVES_M, int AMODE, int BMODE, int PA = 0, int PB = 0,
          bool SB = false, class LoadA, class LoadB, class Epi>
__device__ __forceinline__ void mfma_gemm(float* smem, int kc_begin, int kc_end,
                                          LoadA& la, LoadB& lb, Epi& epi,
                                          float* rowsum_out = nullptr,
                                          const SplitPiece& sp = SplitPiece{}) {
    using SH = GemmShape<BM, BN, AMODE, BMODE, PA, PB, SB>;
    using LA = typename SH::LA;
    using LB = typename SH::LB;
    using TA = typename SH::TA;
    using TB = typename SH::TB;
    constexpr bool BF = PA > 0;
    constexpr int WAVES_N = 4 / WAVES_M;
    constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int STAGE = SH::STAGE_FLOATS;  // floats per LDS buffer
    static_assert(TM * 32 == WM && TN * 32 == WN, "wave tile must be a multiple of 32");
    static_assert(LA::NQ <= MAXQ && LB::NQ <= MAXQ, "loader state arrays hold MAXQ quads");
    static_assert(LA::QUADS % 256 == 0 && LB::QUADS % 256 == 0, "every thread owns whole quads");
    static_assert((AMODE == KMAJ || (BM / 4) % LA::NQ == 0) && (BMODE == KMAJ || (BN / 4) % LB::NQ == 0),
                  "RMAJ tiles split each k's quads evenly over a thread's quads");

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WAVES_M, wn = wave / WAVES_M;

    int qa_row[LA::NQ], qa_k[LA::NQ], qb_row[LB::NQ], qb_k[LB::NQ];
#pragma unroll
    for (int j = 0; j < LA::NQ; ++j) {
        LA::quad_coord(tid, j, qa_row[j], qa_k[j]);
        la.init(j, qa_row[j], qa_k[j]);
    }
#pragma unroll
    for (int j = 0; j < LB::NQ; ++j) {
        LB::quad_coord(tid, j, qb_row[j], qb_k[j]);
        lb.init(j, qb_row[j], qb_k[j]);
    }

    constexpr bool MASK = IsMaskEpi<Epi>::value;
    f32x16 acc[TM][TN], pre[TM][TN];
    uint32_t bits[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            acc[i][j] = f32x16{};
#pragma unroll
            for (int r = 0; r < 16; ++r)
                pre[i][j][r] = epi.pre(wm * WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3),
                                       wn * WN + j * 32 + (lane & 31));
        }
    auto pack_mask = [&]() {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                uint32_t b = 0;
#pragma unroll
                for (int r = 0; r < 16; ++r) b |= (pre[i][j][r] > 0.0f ? 1u : 0u) << r;
                bits[i][j] = b;
            }
    };

    // Register sets 0/1 hold chunks fetched ahead; set s always holds chunks
    // with (kc - kc_begin) % 2 == s.
    f32x4 ra0[LA::NQ], rb0[LB::NQ], ra1[LA::NQ], rb1[LB::NQ];
    auto gload = [&](int kc, f32x4* ra, f32x4* rb) {
        if constexpr (HasPrep<LoadA>::value) la.prep(kc);
        if constexpr (HasPrep<LoadB>::value) lb.prep(kc);
#pragma unroll
        for (int j = 0; j < LA::NQ; ++j) ra[j] = la.load(kc, j);
#pragma unroll
        for (int j = 0; j < LB::NQ; ++j) rb[j] = lb.load(kc, j);
    };
    auto sstore = [&](float* buf, const f32x4* ra, const f32x4* rb) {
        if constexpr (BF) {
#pragma unroll
            for (int j = 0; j < LA::NQ; ++j)
                TA::template put<AMODE>((char*)buf, qa_row[j], qa_k[j], ra[j]);
#pragma unroll
            for (int j = 0; j < LB::NQ; ++j)
                TB::template put<BMODE>((char*)buf + TA::BYTES, qb_row[j], qb_k[j], rb[j]);
        } else {
#pragma unroll
            for (int j = 0; j < LA::NQ; ++j) LA::put(buf, qa_row[j], qa_k[j], ra[j]);
#pragma unroll
            for (int j = 0; j < LB::NQ; ++j) LB::put(buf + LA::SIZE, qb_row[j], qb_k[j], rb[j]);
        }
    };

    const bool do_rowsum = rowsum_out != nullptr;  // uniform over the workgroup
    float rowsum = 0.0f;
    auto compute_bf16 = [&](const float* buf) {
        const char* sa = (const char*)buf;
        const char* sb = sa + TA::BYTES;
#pragma unroll
        for (int st = 0; st < BK / 16; ++st) {
            const int c = 2 * st + (lane >> 5);
            bf16x8 a0[TM], a1[TM], b0[TN], b1[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                a0[i] = TA::get(sa, 0, wm * WM + i * 32 + (lane & 31), c);
                if (PA == 2) a1[i] = TA::get(sa, 1, wm * WM + i * 32 + (lane & 31), c);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                b0[j] = TB::get(sb, 0, wn * WN + j * 32 + (lane & 31), c);
                if (PB == 2) b1[j] = TB::get(sb, 1, wn * WN + j * 32 + (lane & 31), c);
            }
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[i], b0[j], acc[i][j], 0, 0, 0);
                    if (PA == 2)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[i], b0[j], acc[i][j], 0, 0, 0);
                    if (PB == 2)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[i], b1[j], acc[i][j], 0, 0, 0);
                }
        }
        if (BM <= 64 && do_rowsum && lane < BM) {  // chunk `wave` of row `lane`: k = 8w .. 8w+7
            float t = 0.0f;
#pragma unroll
            for (int pl = 0; pl < PA; ++pl) {
                const bf16x8 v = TA::get(sa, pl, lane, wave);
                t += (((float)v[0] + (float)v[1]) + ((float)v[2] + (float)v[3])) +
                     (((float)v[4] + (float)v[5]) + ((float)v[6] + (float)v[7]));
            }
            rowsum += t;
        }
    };
    auto compute = [&](const float* buf) {
        if constexpr (BF) {
            compute_bf16(buf);
            return;
        }
        const float* sa = buf;
        const float* sb = buf + LA::SIZE;
#pragma unroll
        for (int g = 0; g < BK / 8; ++g) {
            const int kb = 8 * g + 4 * (lane >> 5);
            f32x4 av[TM], bv[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) av[i] = LA::get(sa, wm * WM + i * 32 + (lane & 31), kb);
#pragma unroll
            for (int j = 0; j < TN; ++j) bv[j] = LB::get(sb, wn * WN + j * 32 + (lane & 31), kb);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][q], bv[j][q], acc[i][j], 0, 0, 0);
        }
        if (BM <= 64 && do_rowsum && lane < BM) {
            const f32x4 v0 = LA::get(sa, lane, 8 * wave), v1 = LA::get(sa, lane, 8 * wave + 4);
            rowsum += (((v0[0] + v0[1]) + (v0[2] + v0[3])) + ((v1[0] + v1[1]) + (v1[2] + v1[3])));
        }
    };

    if constexpr (SB) {
        // One LDS stage: a chunk is stored, then multiplied, with the next
        // chunk's global loads in flight meanwhile.
        if (kc_begin < kc_end) gload(kc_begin, ra0, rb0);
        // the mask loads were issued before the first chunk's, so packing
        // them here does not wait for that chunk
        if constexpr (MASK) pack_mask();
        int kc = kc_begin;
        for (; kc + 1 < kc_end; kc += 2) {
            sstore(smem, ra0, rb0);
            gload(kc + 1, ra1, rb1);
            __syncthreads();
            compute(smem);
            __syncthreads();
            sstore(smem, ra1, rb1);
            if (kc + 2 < kc_end) gload(kc + 2, ra0, rb0);
            __syncthreads();
            compute(smem);
            __syncthreads();
        }
        if (kc < kc_end) {
            sstore(smem, ra0, rb0);
            __syncthreads();
            compute(smem);
            __syncthreads();
        }
    } else {
        if (kc_begin < kc_end) {
            gload(kc_begin, ra0, rb0);
            if (kc_begin + 1 < kc_end) gload(kc_begin + 1, ra1, rb1);
            sstore(smem, ra0, rb0);
        }
        // the mask loads were issued before the first chunk's, whose data is in
        // LDS by now, so packing them here waits for nothing more
        if constexpr (MASK) pack_mask();
        __syncthreads();
        // One exit, so the accumulators stay in the same registers on every trip
        // (an exit between the two halves makes the compiler copy them).
        int kc = kc_begin;
        for (; kc + 1 < kc_end; kc += 2) {
            // even chunk: LDS buffer 0, refill register set 0 with chunk kc+2
            if (kc + 2 < kc_end) gload(kc + 2, ra0, rb0);
            compute(smem);
            sstore(smem + STAGE, ra1, rb1);
            __syncthreads();
            // odd chunk: LDS buffer 1, refill register set 1 with chunk kc+3
            if (kc + 3 < kc_end) gload(kc + 3, ra1, rb1);
            compute(smem + STAGE);
            if (kc + 2 < kc_end) sstore(smem, ra0, rb0);
            __syncthreads();
        }
        if (kc < kc_end) {  // an odd chunk count ends in buffer 0
            compute(smem);
            __syncthreads();
        }
    }
    if (BM <= 64 && do_rowsum) {
        // the LDS buffers are free after the loop's last barrier
        if (lane < BM) smem[wave * 64 + lane] = rowsum;
        __syncthreads();
        if (tid < BM) rowsum_out[tid] = ((smem[tid] + smem[64 + tid]) + smem[128 + tid]) + smem[192 + tid];
    }
    // hand-off between the pieces of one tile (never with a row sum; tiles up
    // to SPLIT_TILE_FLOATS elements)
    constexpr int NV = TM * TN * 4;  // f32x4 per thread: 256 * NV * 4 == BM * BN
    static_assert(256 * NV * 4 == BM * BN, "four waves hold the tile");
    if (BM * BN <= SPLIT_TILE_FLOATS && sp.np > 1) {
        f32x4* mine = (f32x4*)sp.ws + ((int64_t)sp.piece * 256 + tid) * NV;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    mine[(i * TN + j) * 4 + q] = f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1],
                                                       acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        __builtin_amdgcn_s_waitcnt(0);  // release: the partial tile is in the L2 before it is counted
        __syncthreads();
        int* flag = (int*)smem;  // the LDS buffers are free after the loop's last barrier
        if (tid == 0)
            flag[0] = __hip_atomic_fetch_add(sp.cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        if (flag[0] != sp.np - 1) return;
        // acquire: drop this unit's L1 so every partial tile is read from the L2
        asm volatile("buffer_inv sc0" ::: "memory");
        // add every piece's partial tile (this one's included, read back) in
        // piece order, two pieces' loads in flight at a time
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
        for (int p0 = 0; p0 < sp.np; p0 += 2) {
            f32x4 part[2][NV];
#pragma unroll
            for (int q = 0; q < 2; ++q)
                if (p0 + q < sp.np) {
                    const f32x4* src = (const f32x4*)sp.ws + ((int64_t)(p0 + q) * 256 + tid) * NV;
#pragma unroll
                    for (int v = 0; v < NV; ++v) part[q][v] = src[v];
                }
#pragma unroll
            for (int q = 0; q < 2; ++q)
                if (p0 + q < sp.np) {
#pragma unroll
                    for (int i = 0; i < TM; ++i)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
#pragma unroll
                            for (int r = 0; r < 16; ++r)
                                acc[i][j][r] += part[q][(i * TN + j) * 4 + r / 4][r % 4];
                }
        }
        if (tid == 0) *sp.cnt = 0;
    }

    // The epilogue's element coordinates come from an opaque copy of the
    // lane index, so its address arithmetic is redone here instead of being
    // shared with the prologue's pre() and held in registers across the loop.
    int elane = lane;
    asm volatile("" : "+v"(elane));
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                int row = wm * WM + i * 32 + 8 * (r >> 2) + 4 * (elane >> 5) + (r & 3);
                int col = wn * WN + j * 32 + (elane & 31);
                if constexpr (MASK)
                    epi(row, col, acc[i][j][r], (bits[i][j] >> r) & 1u ? 1.0f : 0.0f);
                else
                    epi(row, col, acc[i][j][r], pre[i][j][r]);
            }
}

// Epilogue writing scale * C into a row-major [rows][ld] buffer at column col0.
struct PartialEpi {
    float* out;
    int ld, col0;
    float scale;
    __device__ float pre(int, int) const { return 0.0f; }
    __device__ void operator()(int row, int col, float v, float) const {
        out[(int64_t)row * ld + col0 + col] = v * scale;
    }
};

// Butterfly sum over a wave64: every lane ends with the same bit pattern.
__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Workgroups are dispatched to the eight XCDs round-robin by workgroup id, and
// each XCD has its own L2.  Every job pads its block count to a multiple of 8
// (so every job starts at a multiple of 8 in its launch) and maps its block
// index through xcd_tile, which sends logical tiles [k*n/8, (k+1)*n/8) to XCD
// k: tiles that are neighbours in logical order, and share operands, then
// share an L2.  Logical tiles >= the real count are idle.
constexpr int NUM_XCD = 8;
__host__ __device__ inline int pad_xcd(int n) { return (n + NUM_XCD - 1) / NUM_XCD * NUM_XCD; }
__device__ inline int xcd_tile(int bid, int padded) {
    return (bid % NUM_XCD) * (padded / NUM_XCD) + bid / NUM_XCD;
}

// Balancing a launch over the compute units.  When a launch of T equal tiles
// puts k tiles on every compute unit and r = T mod CUs more on a few of them,
// those few run a whole tile longer than the rest; when T is at most half the
// unit count, most units idle while a few walk each tile's whole reduction.
// A job's TailSplit keeps its first `full` tiles whole (one XCD-mapped
// workgroup each) and runs its last `tail` tiles as `pieces` reduction pieces
// each (SplitPiece), dispatched after the whole tiles, so that work is spread
// over more units.
// Tail tile s goes to XCD s % 8 with all of its pieces: tail block j runs on
// XCD j % 8 and is that XCD's (j / 8)-th piece.  ws holds tail * pieces <=
// SPLIT_MAX_SLOTS partial tiles of SPLIT_TILE_FLOATS floats, cnt one counter per
// tail tile (zero between launches).
struct TailSplit {
    float* ws = nullptr;
    int* cnt = nullptr;
    int full = -1, tail = 0, pieces = 1;  // full < 0: the whole job unsplit
    __host__ __device__ int blocks(int tiles) const {
        return tail ? pad_xcd(full) + NUM_XCD * ((tail + NUM_XCD - 1) / NUM_XCD) * pieces
                    : pad_xcd(tiles);
    }
    // Workgroup bid of the job: its tile t, chunk range [k0, k1) of `chunks`,
    // and its piece (np == 1 for a whole tile); false for an idle workgroup.
    __device__ bool map(int bid, int tiles, int chunks, int& t, int& k0, int& k1,
                        SplitPiece& sp) const {
        k0 = 0;
        k1 = chunks;
        if (!tail) {
            t = xcd_tile(bid, pad_xcd(tiles));
            return t < tiles;
        }
        const int head = pad_xcd(full);
        if (bid < head) {
            t = xcd_tile(bid, head);
            return t < full;
        }
        const int j = bid - head, k = j / NUM_XCD, p = k % pieces;
        const int s = (k / pieces) * NUM_XCD + j % NUM_XCD;  // same XCD as every other piece of s
        if (s >= tail) return false;
        t = full + s;
        k0 = p * chunks / pieces;
        k1 = (p + 1) * chunks / pieces;
        sp.ws = ws + (int64_t)s * pieces * SPLIT_TILE_FLOATS;
        sp.cnt = cnt + s;
        sp.piece = p;
        sp.np = pieces;
        return true;
    }
};
// The split for a job of job_tiles tiles of `chunks` chunks that closes a
// launch of launch_tiles equal tiles on `cus` compute units, in pieces of at
// least two chunks:
//  - a small launch (at most half a tile per unit): every tile of the job in
//    two pieces.  A workgroup costs ~5 us before its first chunk and after
//    its last (per-workgroup timestamps at batch 32), and each further piece
//    adds a round trip to the hand-off, so more pieces measured slower;
//  - otherwise the r = launch_tiles mod cus excess tiles, taken from this
//    job, in up to 16 pieces, about one per unit -- only when the whole tiles
//    fit in one round of `slots` workgroups per unit (the residency of the
//    kernel: four for the double-buffered GEMMs here), so that the pieces
//    start alongside them: behind a full round they would only start as whole
//    tiles finish (measured no faster).
inline TailSplit plan_split(float* ws, int* cnt, int cus, int launch_tiles, int job_tiles,
                            int chunks, int slots = 4) {
    TailSplit ts;
    ts.ws = ws;
    ts.cnt = cnt;
    if (!ws || !cnt || cus < 1 || launch_tiles < 1) return ts;
    int r, p = SPLIT_MAX_PIECES;
    if (chunks / 2 < p) p = chunks / 2;
    if (2 * launch_tiles <= cus) {
        r = job_tiles;
        if (p > 2) p = 2;
    } else {
        if (launch_tiles < cus) return ts;
        r = launch_tiles % cus;
        if (r == 0 || r > job_tiles || launch_tiles - r > slots * cus) return ts;
        if (cus / r < p) p = cus / r;
    }
    if (p < 2 || r > SPLIT_MAX_TILES || r * p > SPLIT_MAX_SLOTS) return ts;
    ts.full = job_tiles - r;
    ts.tail = r;
    ts.pieces = p;
    return ts;
}

// Several independent jobs in one launch: blocks [0, a.blocks()) run job a,
// the next b.blocks() run job b, the rest job c.  A job is a struct with
// SMEM (floats of shared memory), blocks() and run(block, smem).
struct NoJob {
    static constexpr int SMEM = 1;
    __host__ __device__ int blocks() const { return 0; }
    __device__ void run(int, float*) const {}
};
constexpr int cmax(int a, int b) { return a > b ? a : b; }
// A job may ask for a minimum residency (workgroups per compute unit), which
// caps the registers the compiler gives it: `static constexpr int MIN_WGS`.
template <class T, class = void> struct MinWgs : std::integral_constant<int, 1> {};
template <class T>
struct MinWgs<T, std::void_t<decltype(T::MIN_WGS)>> : std::integral_constant<int, T::MIN_WGS> {};
template <class J1, class J2, class J3>
__global__ __launch_bounds__(256, cmax(MinWgs<J1>::value, cmax(MinWgs<J2>::value, MinWgs<J3>::value)))
void jobs_kernel(J1 a, J2 b, J3 c) {
    __shared__ __attribute__((aligned(16))) float smem[cmax(J1::SMEM, cmax(J2::SMEM, J3::SMEM))];
    int bid = blockIdx.x;
    const int na = a.blocks();
    if (bid < na) { a.run(bid, smem); return; }
    bid -= na;
    const int nb = b.blocks();
    if (bid < nb) { b.run(bid, smem); return; }
    c.run(bid - nb, smem);
}
template <class J1, class J2 = NoJob, class J3 = NoJob>
inline void launch_jobs(hipStream_t st, const J1& a, const J2& b = J2{}, const J3& c = J3{}) {
    const int blocks = a.blocks() + b.blocks() + c.blocks();
    if (blocks > 0) jobs_kernel<J1, J2, J3><<<blocks, 256, 0, st>>>(a, b, c);
}

__device__ inline f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }
__device__ inline f32x4 sel4(bool ok, f32x4 v) {
    return f32x4{ok ? v[0] : 0.f, ok ? v[1] : 0.f, ok ? v[2] : 0.f, ok ? v[3] : 0.f};
}
__device__ inline f32x4 ld4(const float* p) { return *(const f32x4*)p; }

// Loads through a pointer that was itself read from memory (the replay frame
// tables) would otherwise use the flat address space, whose loads also count
// against the LDS wait counter, so every wait for LDS data would wait for them
// too; these state that the data lives in global memory.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const uint32_t global_u32;
typedef __attribute__((address_space(1))) const u32x4 global_u32x4;
__device__ inline uint32_t ldg_u32(const uint8_t* p) { return *(global_u32*)p; }
__device__ inline uint4 ldg_u4(const uint4* p) {
    const u32x4 v = *(global_u32x4*)p;
    return make_uint4(v[0], v[1], v[2], v[3]);
}

}  // namespace gorila
