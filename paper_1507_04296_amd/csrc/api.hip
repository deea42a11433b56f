// C-ABI entry points of libgorila (declared in include/gorila.h): argument
// validation, the workspace plan and the launch sequence of each call.
#include <math.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "common.h"
#include "kernels.h"

using namespace gorila;

namespace {
// Stages of the calls, in launch order (bits of the timing mask).  The
// minibatch resolution (or a forward call's frame table) shares the prep
// launch.
enum Stage {
    ST_PREP, ST_CONV1_FWD, ST_CONV2_FWD, ST_CONV3_FWD, ST_FC1_FWD, ST_HEAD,
    ST_FC1_BWD, ST_CONV3_BWD, ST_CONV2_BWD, ST_CONV1_WGRAD, ST_GRAD_REDUCE, ST_COUNT
};
const char* const STAGE_NAMES[ST_COUNT] = {
    "prep_weights", "conv1_fwd", "conv2_fwd", "conv3_fwd", "fc1_fwd", "head",
    "fc1_bwd", "conv3_bwd", "conv2_bwd", "conv1_wgrad", "grad_reduce"};
struct TimingRecord {
    int stage;
    hipEvent_t start, stop;
};
}  // namespace

struct gorila_ctx {
    hipStream_t stream;
    char* ws;
    size_t ws_bytes;
    int device;
    int cus = 0;  // compute units of the device
    bool split_ok = false;  // workgroup placement allows split reductions
    uint32_t timing_mask = 0;
    std::vector<TimingRecord> records;  // events created by timing_begin
    size_t used = 0;
    // Where the most recent learner call left its per-row TD values (q of
    // both networks, td rows); valid until a forward or act call reuses the
    // workspace.
    bool td_valid = false;
    int td_b = 0, td_groups = 0, td_actions = 0;
    size_t td_q = 0, td_rows = 0;
    char* scratch = nullptr;  // this device's no-allocation scratch (device address)
};

namespace {
// Records an event pair around one stage when its timing bit is set.
struct StageTimer {
    gorila_ctx* c;
    TimingRecord* rec = nullptr;
    StageTimer(gorila_ctx* ctx, int stage) : c(ctx) {
        if ((c->timing_mask >> stage) & 1u && c->used < c->records.size()) {
            rec = &c->records[c->used++];
            rec->stage = stage;
            (void)hipEventRecord(rec->start, c->stream);
        }
    }
    ~StageTimer() {
        if (rec) (void)hipEventRecord(rec->stop, c->stream);
    }
};
}  // namespace

namespace {

constexpr size_t ALIGN = 256;
constexpr size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// Byte offsets of every workspace region for fwd_rows forward rows (all
// parameter sets together), bwd_rows learner rows, `online` learner parameter
// sets plus one target set, and `widened` fp32 copies of bf16 parameter sets.
constexpr size_t W2T_BYTES = 4 * 16 * 64 * 32, W3T_BYTES = 4 * 9 * 64 * 64;
struct Plan {
    size_t err, zero, ftab, a, r, term;
    size_t theta32, theta32_stride;
    size_t w2t, w3t, w3d, w2p;  // bases of per-set arrays (stride W2T_BYTES / W3T_BYTES)
    size_t h1, h2, h3, h4, q, ell, coef, td;
    size_t dz4, dz3, dz2, dz1;
    size_t fc1part, part1, part2, part3, bpart, hpart;
    size_t split;  // TailSplit partial tiles
    size_t total;
};

// The zeroed head of the workspace (WS_HEAD bytes, cleared when a context is
// created): the sticky error word, then the TailSplit counters at
// SPLIT_CNT_OFFSET (every launch leaves them at zero).  Right after it, at the
// same offset in every plan, ZERO_BYTES that are zeroed at creation and never
// written: a zero frame that kernels read in place of a zero-filled channel.
constexpr size_t WS_HEAD = 1024, SPLIT_CNT_OFFSET = 256, ZERO_BYTES = 7168;
static_assert(ZERO_BYTES >= FRAME_BYTES && ZERO_BYTES % 256 == 0, "a whole frame of zeros");
static_assert(SPLIT_CNT_OFFSET + 4 * SPLIT_MAX_TILES <= WS_HEAD, "counters fit the zeroed head");

constexpr Plan make_plan(int64_t fwd_rows, int64_t bwd_rows, int A, int online = 1,
                         int widened = 0) {
    Plan p{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o += up(bytes); return at; };
    const int64_t F = fwd_rows, B = bwd_rows;
    p.err = take(WS_HEAD);
    p.zero = take(ZERO_BYTES);
    p.ftab = take(sizeof(void*) * 2 * (size_t)(F > 2 * B ? F : 2 * B) * 4);
    p.a = take(4 * (size_t)B);
    p.r = take(4 * (size_t)B);
    p.term = take((size_t)B);
    p.theta32_stride = up(4 * (size_t)param_count(A));
    p.theta32 = take(p.theta32_stride * (size_t)widened);
    p.w2t = take(W2T_BYTES * (size_t)(online + 1));
    p.w3t = take(W3T_BYTES * (size_t)(online + 1));
    p.w3d = take(W3T_BYTES * (size_t)online);
    p.w2p = take(W2T_BYTES * (size_t)online);
    p.h1 = take(4 * (size_t)F * P1 * C1);
    p.h2 = take(4 * (size_t)F * P2 * C2);
    p.h3 = take(4 * (size_t)F * FLAT);
    p.h4 = take(4 * (size_t)F * HID);
    p.q = take(4 * (size_t)F * A);
    p.fc1part = take(4 * (size_t)F * HID * FC1_MAX_SPLITS);
    p.ell = take(4 * (size_t)B);
    p.coef = take(4 * (size_t)B);
    p.td = take(16 * (size_t)B);
    p.dz4 = take(4 * (size_t)B * HID);
    p.dz3 = take(4 * (size_t)bwd_split_rows(B) * FLAT);  // bwd_parts(B) partial planes
    p.dz2 = take(4 * (size_t)bwd_split_rows(B) * P2 * C2);
    p.dz1 = take(4 * (size_t)B * P1 * C1);
    p.part1 = B ? take(4 * (size_t)CONV1_WG_MAX_SPLITS * C1 * 256) : o;
    p.part2 = B ? take(4 * (size_t)WG_MAX_SPLITS * C2 * 16 * C1) : o;
    p.part3 = B ? take(4 * (size_t)WG_MAX_SPLITS * C3 * 9 * C2) : o;
    p.bpart = B ? take(4 * (size_t)3 * BIAS_PART_STRIDE) : o;
    p.hpart = B ? take(4 * (size_t)online * HEAD_MAX_BLOCKS * HP_STRIDE) : o;
    p.split = take(4 * (size_t)SPLIT_MAX_SLOTS * SPLIT_TILE_FLOATS);
    p.total = o;
    return p;
}

template <class T>
T* at(gorila_ctx* c, size_t off) { return (T*)(c->ws + off); }

// Split-reduction workspace of a plan laid out from `base` (the context's
// workspace, or the no-allocation scratch).
SplitWs split_ws(gorila_ctx* c, char* base, const Plan& p) {
    SplitWs sw;
    sw.cus = c->cus;
    sw.ws = c->split_ok ? (float*)(base + p.split) : nullptr;  // null: every tile whole
    sw.cnt = (int*)(base + p.err + SPLIT_CNT_OFFSET);
    return sw;
}
SplitWs split_ws(gorila_ctx* c, const Plan& p) { return split_ws(c, c->ws, p); }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_launch() {
    return hipGetLastError() == hipSuccess ? GORILA_OK : GORILA_EHIP;
}

int check_ctx(gorila_ctx* c) {
    if (!c) return GORILA_EINVAL;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return GORILA_EHIP;
    return dev == c->device ? GORILA_OK : GORILA_EINVAL;
}

// fp32 sets are read with 16-byte loads; bf16 sets only by the widening kernel.
int check_params(const gorila_params* p, bool allow_bf16) {
    if (!p || !p->data) return GORILA_EINVAL;
    if (p->n_actions < 1 || p->n_actions > MAX_ACTIONS) return GORILA_EINVAL;
    if (p->dtype == GORILA_BF16) {
        if ((uintptr_t)p->data & 1u) return GORILA_EINVAL;
        return allow_bf16 ? GORILA_OK : GORILA_EUNSUPPORTED;
    }
    if (p->dtype != GORILA_F32 || !aligned16(p->data)) return GORILA_EINVAL;
    return GORILA_OK;
}

// fp32 view of a parameter set: the caller's vector, or its exact widening
// into the next free fp32 slot of the workspace (queued on the stream).
const float* fp32_params(gorila_ctx* c, const Plan& p, const gorila_params* prm, WidenSet& ws,
                         int& n_widen) {
    if (prm->dtype == GORILA_F32) return (const float*)prm->data;
    float* dst = at<float>(c, p.theta32 + (size_t)n_widen * p.theta32_stride);
    ws.src[n_widen] = (const uint16_t*)prm->data;
    ws.dst[n_widen] = dst;
    ++n_widen;
    return dst;
}

int check_replay(const gorila_replay* rv) {
    if (!rv || !rv->action || !rv->reward) return GORILA_EINVAL;
    if (rv->kind == GORILA_REPLAY_STACKED) {
        if (!rv->s || !rv->s2 || !rv->term || rv->rows < 1) return GORILA_EINVAL;
        if (!aligned16(rv->s) || !aligned16(rv->s2)) return GORILA_EINVAL;
        return GORILA_OK;
    }
    if (rv->kind == GORILA_REPLAY_RING) {
        if (!rv->frames || !rv->ep_start || rv->capacity < 2 || rv->rows < 0) return GORILA_EINVAL;
        if (rv->head < 0 || rv->head >= rv->capacity || !aligned16(rv->frames)) return GORILA_EINVAL;
        if (rv->size < 0 || rv->size > rv->capacity) return GORILA_EINVAL;
        return GORILA_OK;
    }
    return GORILA_EINVAL;
}

ReplayView view_of(const gorila_replay* rv) {
    return ReplayView{rv->kind,     rv->s,        rv->s2,       rv->term,
                      rv->rows,     rv->frames,   rv->ep_start, rv->capacity,
                      rv->head,     rv->size,     rv->action,   rv->reward};
}

// Forward-only calls: the first tblocks workgroups write the frame table of
// n stacked states, the next PREP_BLOCKS the weight transposes of one set and
// the rest widen a bf16 set (independent, so one launch).
__global__ __launch_bounds__(256) void states_prep_kernel(const uint8_t* states, int n,
                                                          const uint8_t** ftab, WeightViews wv,
                                                          int tblocks, unsigned* zero_head,
                                                          WidenJob wj, int wpn) {
    if ((int)blockIdx.x >= tblocks + PREP_BLOCKS) {
        widen_part(wj, 0, blockIdx.x - tblocks - PREP_BLOCKS, wpn);
        return;
    }
    if ((int)blockIdx.x >= tblocks) {
        prep_weights_part(wv, blockIdx.x - tblocks, PREP_BLOCKS);
        return;
    }
    // a scratch that other calls share starts each call with a zero head
    // (error word, split-reduction counters); the split launches come later
    if (zero_head && blockIdx.x == 0)
        for (int i = threadIdx.x; i < (int)(WS_HEAD / 4); i += blockDim.x) zero_head[i] = 0u;
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e < n * 4) ftab[e] = states + (int64_t)(e >> 2) * STATE_BYTES + (int64_t)(e & 3) * FRAME_BYTES;
}

// Forward pass of n states through one parameter set up to h4, with the
// plan's regions laid out from `base`; *theta32 receives the fp32 parameters
// the head must use.  zero_head: clear the plan's head first.
int forward_one(gorila_ctx* c, char* base, const Plan& p, const gorila_params* prm,
                const uint8_t* states, int n, const float** theta32, int* fc1_splits,
                bool zero_head) {
    hipStream_t st = c->stream;
    auto fp = [&](size_t off) { return (float*)(base + off); };
    const uint8_t** ftab = (const uint8_t**)(base + p.ftab);
    WidenJob wj;
    const float* theta = (const float*)prm->data;
    if (prm->dtype != GORILA_F32) {  // exact widening into the plan's fp32 slot
        wj.set.src[0] = (const uint16_t*)prm->data;
        wj.set.dst[0] = fp(p.theta32);
        wj.n = 1;
        wj.hi[0] = param_count(prm->n_actions);
        theta = wj.set.dst[0];
    }
    *theta32 = theta;
    WeightViews wv{theta, fp(p.w2t), fp(p.w3t), nullptr, nullptr};
    if (wj.n) wv.theta16 = wj.set.src[0];
    {
        StageTimer t(c, ST_PREP);
        const int tblocks = (n * 4 + 255) / 256, wpn = wj.blocks_per_net();
        states_prep_kernel<<<tblocks + PREP_BLOCKS + wpn, 256, 0, st>>>(
            states, n, ftab, wv, tblocks, zero_head ? (unsigned*)(base + p.err) : nullptr, wj,
            wpn > 0 ? wpn : 1);
    }
    GroupPtrs th{}, w2t{}, w3t{};
    th.p[0] = theta;
    w2t.p[0] = wv.w2t;
    w3t.p[0] = wv.w3t;
    // forward-only calls compute in fp32 (bf16 parameters are widened exactly)
    { StageTimer t(c, ST_CONV1_FWD); launch_conv1_fwd(ftab, th, 1, n, fp(p.h1), false, st); }
    const SplitWs sw = split_ws(c, base, p);
    { StageTimer t(c, ST_CONV2_FWD); launch_conv2_fwd(fp(p.h1), w2t, th, 1, n, fp(p.h2), sw, false, st); }
    { StageTimer t(c, ST_CONV3_FWD); launch_conv3_fwd(fp(p.h2), w3t, th, 1, n, fp(p.h3), sw, false, st); }
    { StageTimer t(c, ST_FC1_FWD); *fc1_splits = launch_fc1_fwd(fp(p.h3), th, GroupPtrs16{}, 1, n, fp(p.fc1part), false, st); }
    return check_launch();
}

// ---- The no-allocation actor call's scratch ----
// Forward rows of the largest call, one fp32 slot for a widened bf16 set and
// the largest action count, then WS_HEAD bytes for the placement probe of
// contexts made without a workspace.
constexpr Plan NOALLOC_PLAN = make_plan(GORILA_NOALLOC_MAX_STATES, 0, MAX_ACTIONS, 1, 1);
constexpr size_t NOALLOC_PROBE = NOALLOC_PLAN.total;
constexpr size_t NOALLOC_BYTES = NOALLOC_PROBE + WS_HEAD;
static_assert(NOALLOC_BYTES <= (size_t)GORILA_NOALLOC_SCRATCH_MB << 20, "stated scratch size");
}  // namespace

// Each device holds its own copy for the life of the process.  Host code
// never uses this name as an address: it uses the per-device address that
// hipGetSymbolAddress returns (noalloc_scratch below).
static __device__ __align__(256) char scratch[NOALLOC_BYTES];

namespace {

// Per device ordinal: the scratch's device address, resolved once with that
// device current, and its head zeroed.
constexpr int NOALLOC_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char* g_scratch[NOALLOC_MAX_DEVICES] = {};

__global__ __launch_bounds__(256) void zero_words_kernel(unsigned* p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

int noalloc_scratch(int dev, hipStream_t st, char** out) {
    if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return GORILA_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return GORILA_EHIP;
        zero_words_kernel<<<1, 256, 0, st>>>((unsigned*)ptr, (int)((WS_HEAD + ZERO_BYTES) / 4));
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(st) != hipSuccess)
            return GORILA_EHIP;
        g_scratch[dev] = (char*)ptr;
    }
    *out = g_scratch[dev];
    return GORILA_OK;
}

}  // namespace

extern "C" {

int64_t gorila_param_count(int32_t n_actions) {
    if (n_actions < 1 || n_actions > MAX_ACTIONS) return -1;
    return param_count(n_actions);
}

size_t gorila_workspace_bytes(int32_t max_batch, int32_t n_actions, int32_t dtype, int32_t groups) {
    if (max_batch < 1 || n_actions < 1 || n_actions > MAX_ACTIONS || groups < 1) return 0;
    if (dtype != GORILA_F32 && dtype != GORILA_BF16) return 0;
    if (groups > MAX_LEARNER_GROUPS) return 0;
    const int64_t B = (int64_t)max_batch * groups;
    const int widened = dtype == GORILA_BF16 ? groups + 1 : 0;
    return make_plan(2 * B, B, n_actions, groups, widened).total;
}

// Thread 0 of workgroup b writes the XCD it runs on (hardware register
// XCC_ID) to out[b].
static __global__ __launch_bounds__(64) void xcd_probe_kernel(unsigned* out) {
    if (threadIdx.x == 0) out[blockIdx.x] = __builtin_amdgcn_s_getreg((31 << 11) | 20) & 15u;
}

// The split reductions exchange partial tiles through one XCD's L2, so they
// need every workgroup id to share an XCD with the ids equal to it mod 8
// (round-robin dispatch over 1, 2, 4 or 8 XCDs).  Checked once per context on
// WS_HEAD / 4 workgroups, using the workspace head as the record; where it
// does not hold, every tile runs whole.
static int probe_split_placement(gorila_ctx* c, char* rec) {
    constexpr int N = (int)(WS_HEAD / 4);
    unsigned xcc[N];
    xcd_probe_kernel<<<N, 64, 0, c->stream>>>((unsigned*)rec);
    if (hipGetLastError() != hipSuccess) return GORILA_EHIP;
    if (hipMemcpyAsync(xcc, rec, sizeof xcc, hipMemcpyDeviceToHost, c->stream) != hipSuccess ||
        hipStreamSynchronize(c->stream) != hipSuccess)
        return GORILA_EHIP;
    c->split_ok = true;
    for (int b = NUM_XCD; b < N; ++b)
        if (xcc[b] != xcc[b % NUM_XCD]) c->split_ok = false;
    return GORILA_OK;
}

int gorila_ctx_create(gorila_ctx** out, void* hip_stream, void* workspace, size_t ws_bytes) {
    if (!out || !aligned16(workspace)) return GORILA_EINVAL;
    if (!workspace && ws_bytes != 0) return GORILA_EINVAL;
    if (workspace && ws_bytes < make_plan(1, 1, 1).zero + ZERO_BYTES) return GORILA_EWORKSPACE;
    int dev = -1, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GORILA_EHIP;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return GORILA_EHIP;
    gorila_ctx* c = new (std::nothrow) gorila_ctx;
    if (c) {
        c->stream = (hipStream_t)hip_stream;
        c->ws = (char*)workspace;
        c->ws_bytes = ws_bytes;
        c->device = dev;
        c->cus = cus;
    }
    if (!c) return GORILA_EINVAL;
    int rc = noalloc_scratch(dev, c->stream, &c->scratch);
    if (rc == GORILA_OK) rc = probe_split_placement(c, c->ws ? c->ws : c->scratch + NOALLOC_PROBE);
    if (rc != GORILA_OK ||
        (c->ws && hipMemsetAsync(c->ws, 0, WS_HEAD + ZERO_BYTES, c->stream) != hipSuccess)) {
        delete c;
        return GORILA_EHIP;
    }
    *out = c;
    return GORILA_OK;
}

int gorila_ctx_destroy(gorila_ctx* ctx) {
    if (!ctx) return GORILA_EINVAL;
    for (auto& r : ctx->records) {
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
    }
    delete ctx;
    return GORILA_OK;
}

int gorila_ctx_set_stream(gorila_ctx* ctx, void* hip_stream) {
    if (!ctx) return GORILA_EINVAL;
    ctx->stream = (hipStream_t)hip_stream;
    return GORILA_OK;
}

int gorila_ctx_check(gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (hipStreamSynchronize(ctx->stream) != hipSuccess) return GORILA_EHIP;
    if (!ctx->ws) return GORILA_OK;  // no workspace, no device error word
    unsigned word = 0;
    if (hipMemcpy(&word, ctx->ws, sizeof(word), hipMemcpyDeviceToHost) != hipSuccess) return GORILA_EHIP;
    if (word == 0) return GORILA_OK;
    if (hipMemset(ctx->ws, 0, sizeof(word)) != hipSuccess) return GORILA_EHIP;
    return GORILA_ERANGE;
}

const char* gorila_strerror(int code) {
    switch (code) {
        case GORILA_OK: return "success";
        case GORILA_EINVAL: return "invalid argument";
        case GORILA_ERANGE: return "minibatch index or action out of range (seen on the device)";
        case GORILA_EWORKSPACE: return "workspace too small";
        case GORILA_EHIP: return "HIP runtime error";
        case GORILA_EUNSUPPORTED: return "not supported by this library";
        default: return "unknown error";
    }
}

int gorila_ctx_timing_begin(gorila_ctx* ctx, uint32_t stage_mask, int32_t max_records) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (max_records < 0) return GORILA_EINVAL;
    for (auto& r : ctx->records) {
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
    }
    ctx->records.clear();
    ctx->used = 0;
    ctx->timing_mask = 0;
    for (int32_t i = 0; i < max_records; ++i) {
        TimingRecord r{0, nullptr, nullptr};
        if (hipEventCreate(&r.start) != hipSuccess) return GORILA_EHIP;
        if (hipEventCreate(&r.stop) != hipSuccess) {
            (void)hipEventDestroy(r.start);
            return GORILA_EHIP;
        }
        ctx->records.push_back(r);
    }
    ctx->timing_mask = stage_mask;
    return GORILA_OK;
}

int gorila_ctx_timing_end(gorila_ctx* ctx, double* total_ms, int32_t* count, int32_t n_stages) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (n_stages < 0 || (n_stages > 0 && (!total_ms || !count))) return GORILA_EINVAL;
    ctx->timing_mask = 0;
    if (hipStreamSynchronize(ctx->stream) != hipSuccess) return GORILA_EHIP;
    for (int32_t i = 0; i < n_stages; ++i) {
        total_ms[i] = 0.0;
        count[i] = 0;
    }
    for (size_t i = 0; i < ctx->used; ++i) {
        const TimingRecord& r = ctx->records[i];
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) return GORILA_EHIP;
        if (r.stage < n_stages) {
            total_ms[r.stage] += ms;
            count[r.stage] += 1;
        }
    }
    for (auto& r : ctx->records) {
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
    }
    ctx->records.clear();
    ctx->used = 0;
    return GORILA_OK;
}

const char* gorila_stage_name(int32_t stage) {
    return stage >= 0 && stage < ST_COUNT ? STAGE_NAMES[stage] : nullptr;
}

int gorila_gather(const gorila_replay* replay, const int64_t* idx, int32_t n, uint8_t* s_out,
                  uint8_t* s2_out, int64_t* frame_map_out, int32_t* a_out, float* r_out,
                  uint8_t* term_out, gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if ((rc = check_replay(replay))) return rc;
    if (n < 0 || (n > 0 && (!idx || !s_out || !s2_out || !a_out || !r_out || !term_out)))
        return GORILA_EINVAL;
    if (!aligned16(s_out) || !aligned16(s2_out)) return GORILA_EINVAL;
    if (!ctx->ws) return GORILA_EWORKSPACE;
    if (n == 0) return GORILA_OK;
    launch_gather(view_of(replay), idx, n, 0x7fffffff, s_out, s2_out, frame_map_out, a_out, r_out,
                  term_out, at<unsigned>(ctx, make_plan(1, 0, 1).err), ctx->stream);
    return check_launch();
}

int gorila_q_forward(const gorila_params* params, const uint8_t* states_u8, int32_t n,
                     float* q_out, gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if ((rc = check_params(params, true))) return rc;
    if (n < 0 || (n > 0 && (!states_u8 || !q_out)) || !aligned16(states_u8)) return GORILA_EINVAL;
    if (n == 0) return GORILA_OK;
    const Plan p = make_plan(n, 0, params->n_actions, 1, params->dtype == GORILA_BF16);
    if (!ctx->ws || p.total > ctx->ws_bytes) return GORILA_EWORKSPACE;
    const float* theta = nullptr;
    int splits = 0;
    ctx->td_valid = false;  // the forward rows overwrite a learner call's q
    if ((rc = forward_one(ctx, ctx->ws, p, params, states_u8, n, &theta, &splits, false))) return rc;
    {
        StageTimer t(ctx, ST_HEAD);
        launch_q_head(at<float>(ctx, p.fc1part), splits, theta, n, params->n_actions, q_out,
                      ctx->stream);
    }
    return check_launch();
}

int gorila_act(const gorila_params* params, const uint8_t* states_u8, int32_t n, float eps,
               uint64_t seed, int32_t* actions_out, float* q_out, gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if ((rc = check_params(params, true))) return rc;
    if (n < 0 || (n > 0 && (!states_u8 || !actions_out)) || !aligned16(states_u8)) return GORILA_EINVAL;
    if (!(eps >= 0.0f && eps <= 1.0f)) return GORILA_EINVAL;
    if (n == 0) return GORILA_OK;
    const Plan p = make_plan(n, 0, params->n_actions, 1, params->dtype == GORILA_BF16);
    if (!ctx->ws || p.total > ctx->ws_bytes) return GORILA_EWORKSPACE;
    const float* theta = nullptr;
    int splits = 0;
    ctx->td_valid = false;  // the forward rows overwrite a learner call's q
    if ((rc = forward_one(ctx, ctx->ws, p, params, states_u8, n, &theta, &splits, false))) return rc;
    {
        StageTimer t(ctx, ST_HEAD);
        launch_act_head(at<float>(ctx, p.fc1part), splits, theta, n, params->n_actions, eps, seed,
                        actions_out, q_out, ctx->stream);
    }
    return check_launch();
}

int gorila_act_noalloc(const gorila_params* params, const uint8_t* states_u8, int32_t n,
                       float eps, uint64_t seed, int32_t* actions_out, float* q_out,
                       gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if ((rc = check_params(params, true))) return rc;
    if (n < 0 || (n > 0 && (!states_u8 || !actions_out)) || !aligned16(states_u8)) return GORILA_EINVAL;
    if (!(eps >= 0.0f && eps <= 1.0f)) return GORILA_EINVAL;
    if (n > GORILA_NOALLOC_MAX_STATES) return GORILA_EWORKSPACE;
    if (!ctx->scratch) return GORILA_EHIP;
    if (n == 0) return GORILA_OK;
    const Plan p = make_plan(n, 0, params->n_actions, 1, params->dtype == GORILA_BF16);
    if (p.total > NOALLOC_PROBE) return GORILA_EWORKSPACE;  // cannot happen: the plan grows with n, A
    const float* theta = nullptr;
    int splits = 0;
    if ((rc = forward_one(ctx, ctx->scratch, p, params, states_u8, n, &theta, &splits, true)))
        return rc;
    {
        StageTimer t(ctx, ST_HEAD);
        launch_act_head((const float*)(ctx->scratch + p.fc1part), splits, theta, n,
                        params->n_actions, eps, seed, actions_out, q_out, ctx->stream);
    }
    return check_launch();
}

}  // extern "C"

namespace {

// Shared launch sequence of the learner calls: G learner groups of b
// transitions each, group g on parameter set params[g] and minibatch
// idx[g*b .. g*b+b-1], all against one target set.
int learner_steps(gorila_ctx* ctx, const gorila_params* params, int G, bool allow_bf16,
                  const gorila_params* target_params, const gorila_replay* replay,
                  const int64_t* idx, int b, float gamma, float clip_delta, float* grads_out,
                  float* loss_out) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (G < 1 || G > MAX_LEARNER_GROUPS || !params) return GORILA_EINVAL;
    if ((rc = check_params(target_params, allow_bf16))) return rc;
    const int A = target_params->n_actions;
    int n_bf16 = target_params->dtype == GORILA_BF16;
    for (int g = 0; g < G; ++g) {
        if ((rc = check_params(&params[g], allow_bf16))) return rc;
        if (params[g].n_actions != A) return GORILA_EINVAL;
        n_bf16 += params[g].dtype == GORILA_BF16;
    }
    if ((rc = check_replay(replay))) return rc;
    if (b < 1 || !idx || !grads_out || !loss_out) return GORILA_EINVAL;
    if ((int64_t)b * G > (int64_t)1 << 30) return GORILA_EINVAL;
    if (!(gamma >= 0.0f && gamma <= 1.0f) || !(clip_delta > 0.0f)) return GORILA_EINVAL;
    const int B = b * G;  // all learner rows
    // bf16 MFMA products when every parameter set is bf16, fp32 otherwise
    const bool bf16 = n_bf16 == G + 1;
    const Plan p = make_plan(2 * (int64_t)B, B, A, G, n_bf16);
    if (!ctx->ws || p.total > ctx->ws_bytes) return GORILA_EWORKSPACE;
    hipStream_t st = ctx->stream;
    const int64_t P = param_count(A);

    // ftab [2][B][4]: rows g*b .. g*b+b-1 of the s half are group g's states,
    // the same rows of the s' half its next states
    const uint8_t** ftab = at<const uint8_t*>(ctx, p.ftab);
    int32_t* a = at<int32_t>(ctx, p.a);
    float* r = at<float>(ctx, p.r);
    uint8_t* term = at<uint8_t>(ctx, p.term);

    WidenSet widen{};
    int n_widen = 0;
    const float* theta[MAX_LEARNER_GROUPS];
    for (int g = 0; g < G; ++g) theta[g] = fp32_params(ctx, p, &params[g], widen, n_widen);
    const float* theta_t = fp32_params(ctx, p, target_params, widen, n_widen);
    WeightViews wv[MAX_NETS];
    for (int g = 0; g <= G; ++g) {
        wv[g].theta = g < G ? theta[g] : theta_t;
        wv[g].w2t = at<float>(ctx, p.w2t + (size_t)g * W2T_BYTES);
        wv[g].w3t = at<float>(ctx, p.w3t + (size_t)g * W3T_BYTES);
        wv[g].w3d = g < G ? at<float>(ctx, p.w3d + (size_t)g * W3T_BYTES) : nullptr;
        wv[g].w2p = g < G ? at<float>(ctx, p.w2p + (size_t)g * W2T_BYTES) : nullptr;
    }
    // bf16 steps read W4 in place (the fc1 kernels widen it as they load), so
    // only the other tensors are widened
    GroupPtrs16 w4b{};
    if (bf16)
        for (int g = 0; g <= G; ++g)
            w4b.p[g] = (const uint16_t*)(g < G ? params[g].data : target_params->data) + OFF_W4;
    WidenJob wj;
    wj.set = widen;
    wj.n = n_widen;
    wj.hi[0] = bf16 ? OFF_W4 : P;
    if (bf16) {
        wj.lo[1] = OFF_B4;
        wj.hi[1] = P;
    }
    // the transposes of a widened set read its bf16 source, so the minibatch
    // resolution, the transposes and the widening share one launch
    for (int g = 0; g <= G; ++g) {
        const gorila_params& src = g < G ? params[g] : *target_params;
        if (src.dtype == GORILA_BF16) wv[g].theta16 = (const uint16_t*)src.data;
    }
    {
        StageTimer t(ctx, ST_PREP);
        launch_resolve_prep(view_of(replay), idx, B, A, ftab, a, r, term, at<unsigned>(ctx, p.err), wv,
                            G + 1, n_widen ? &wj : nullptr, st);
    }
    // forward groups 0 .. G-1: online nets on s; G .. 2G-1: the target on s'
    GroupPtrs th{}, w2t{}, w3t{};
    GroupPtrs16 w4f{};
    for (int g = 0; g < 2 * G; ++g) {
        const int net = g < G ? g : G;
        th.p[g] = wv[net].theta;
        w2t.p[g] = wv[net].w2t;
        w3t.p[g] = wv[net].w3t;
        w4f.p[g] = w4b.p[net];
    }
    float* h1 = at<float>(ctx, p.h1);
    float* h2 = at<float>(ctx, p.h2);
    float* h3 = at<float>(ctx, p.h3);
    float* h4 = at<float>(ctx, p.h4);
    float* fc1part = at<float>(ctx, p.fc1part);
    { StageTimer t(ctx, ST_CONV1_FWD); launch_conv1_fwd(ftab, th, 2 * G, b, h1, bf16, st); }
    const SplitWs sw = split_ws(ctx, p);
    { StageTimer t(ctx, ST_CONV2_FWD); launch_conv2_fwd(h1, w2t, th, 2 * G, b, h2, sw, bf16, st); }
    { StageTimer t(ctx, ST_CONV3_FWD); launch_conv3_fwd(h2, w3t, th, 2 * G, b, h3, sw, bf16, st); }
    int S = 0;
    { StageTimer t(ctx, ST_FC1_FWD); S = launch_fc1_fwd(h3, th, w4f, 2 * G, b, fc1part, bf16, st); }

    float* dz4 = at<float>(ctx, p.dz4);
    float* dz3 = at<float>(ctx, p.dz3);
    float* dz2 = at<float>(ctx, p.dz2);
    float* dz1 = at<float>(ctx, p.dz1);
    float* ell = at<float>(ctx, p.ell);
    float* coef = at<float>(ctx, p.coef);
    float* q = at<float>(ctx, p.q);
    float* bpart = at<float>(ctx, p.bpart);
    GroupPtrs on{}, w3d{}, w2p{};
    for (int g = 0; g < G; ++g) {
        on.p[g] = theta[g];
        w3d.p[g] = wv[g].w3d;
        w2p.p[g] = wv[g].w2p;
    }
    const int64_t part_stride = (int64_t)S * b * HID;  // fc1 partials of one forward group
    {
        StageTimer t(ctx, ST_HEAD);
        launch_td_head(fc1part, fc1part + G * part_stride, part_stride, S, on, G, theta_t, b, A, a,
                       r, term, gamma, clip_delta, h4, q, ell, coef, at<float>(ctx, p.td), dz4, st);
    }
    ctx->td_valid = true;
    ctx->td_b = b;
    ctx->td_groups = G;
    ctx->td_actions = A;
    ctx->td_q = p.q;
    ctx->td_rows = p.td;
    int head_blocks = 0, s1 = 0, s2 = 0, s3 = 0;
    const int kp = bwd_parts(B);
    {
        StageTimer t(ctx, ST_FC1_BWD);
        head_blocks = launch_fc1_backward(dz4, on, w4b, G, h3, h4, a, coef, ell, b, A, dz3, grads_out, P,
                                          at<float>(ctx, p.hpart), kp, sw, bf16, st);
    }
    {
        StageTimer t(ctx, ST_CONV3_BWD);
        s3 = launch_conv3_backward(dz3, w3d, G, h2, b, dz2, at<float>(ctx, p.part3),
                                   bpart + 2 * BIAS_PART_STRIDE, kp, bf16, st);
    }
    {
        StageTimer t(ctx, ST_CONV2_BWD);
        s2 = launch_conv2_backward(dz2, w2p, G, h1, b, dz1, at<float>(ctx, p.part2),
                                   bpart + BIAS_PART_STRIDE, kp, bf16, st);
    }
    {
        StageTimer t(ctx, ST_CONV1_WGRAD);
        launch_conv1_wgrad(dz1, ftab, at<uint8_t>(ctx, p.zero), G, b, at<float>(ctx, p.part1), bpart,
                           CONV1_WG_MAX_SPLITS, &s1, bf16, st);
    }
    {
        StageTimer t(ctx, ST_GRAD_REDUCE);
        ReduceArgs ra{at<float>(ctx, p.part1), at<float>(ctx, p.part2), at<float>(ctx, p.part3),
                      bpart, at<float>(ctx, p.hpart), s1, s2, s3, head_blocks, b, A, G, P,
                      grads_out, loss_out};
        launch_grad_reduce(ra, st);
    }
    return check_launch();
}

}  // namespace

extern "C" {

int gorila_learner_step(const gorila_params* params, const gorila_params* target_params,
                        const gorila_replay* replay, const int64_t* idx, int32_t batch,
                        float gamma, float clip_delta, float* grads_out, float* loss_out,
                        gorila_ctx* ctx) {
    return learner_steps(ctx, params, 1, false, target_params, replay, idx, batch, gamma,
                         clip_delta, grads_out, loss_out);
}

int gorila_learner_step_grouped(const gorila_params* params, int32_t groups,
                                const gorila_params* target_params, const gorila_replay* replay,
                                const int64_t* idx, int32_t batch, float gamma, float clip_delta,
                                float* grads_out, float* loss_out, gorila_ctx* ctx) {
    return learner_steps(ctx, params, groups, true, target_params, replay, idx, batch, gamma,
                         clip_delta, grads_out, loss_out);
}

int gorila_learner_td(gorila_ctx* ctx, float* q_out, float* q_next_out, float* td_out) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (!ctx->td_valid) return GORILA_EINVAL;
    const size_t b = (size_t)ctx->td_b, G = (size_t)ctx->td_groups, A = (size_t)ctx->td_actions;
    const size_t row = b * A * sizeof(float);  // one group's Q block of one network
    // q region: [group][online, target][b][A]
    const char* q = ctx->ws + ctx->td_q;
    if (q_out && hipMemcpy2DAsync(q_out, row, q, 2 * row, row, G, hipMemcpyDeviceToDevice,
                                  ctx->stream) != hipSuccess)
        return GORILA_EHIP;
    if (q_next_out && hipMemcpy2DAsync(q_next_out, row, q + row, 2 * row, row, G,
                                       hipMemcpyDeviceToDevice, ctx->stream) != hipSuccess)
        return GORILA_EHIP;
    if (td_out && hipMemcpyAsync(td_out, ctx->ws + ctx->td_rows, 16 * b * G,
                                 hipMemcpyDeviceToDevice, ctx->stream) != hipSuccess)
        return GORILA_EHIP;
    return GORILA_OK;
}

int gorila_replay_insert(uint8_t* frames, uint8_t* ep_start, int32_t* action, float* reward,
                         int64_t capacity, int32_t rings, int64_t* head, int64_t* size,
                         const uint8_t* frames_in, const uint8_t* ep_start_in,
                         const int32_t* action_in, const float* reward_in, int32_t m,
                         gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (!head || !size || capacity < 2 || rings < 1 || m < 0 || m > capacity) return GORILA_EINVAL;
    if (*head < 0 || *head >= capacity || *size < 0 || *size > capacity) return GORILA_EINVAL;
    if ((int64_t)m * rings > INT32_MAX) return GORILA_EINVAL;
    if (m == 0) return GORILA_OK;
    if (!frames || !ep_start || !action || !reward || !frames_in || !ep_start_in || !action_in ||
        !reward_in)
        return GORILA_EINVAL;
    if (!aligned16(frames) || !aligned16(frames_in)) return GORILA_EINVAL;
    const int64_t base = (*head + *size) % capacity;
    launch_insert(frames, ep_start, action, reward, capacity, rings, base, frames_in, ep_start_in,
                  action_in, reward_in, m * rings, ctx->stream);
    if ((rc = check_launch())) return rc;
    const int64_t total = *size + m;
    if (total <= capacity) {
        *size = total;
    } else {
        *head = (*head + (total - capacity)) % capacity;
        *size = capacity;
    }
    return GORILA_OK;
}

int gorila_params_sync(const float* src, void* dst, int64_t n, int32_t copies, int32_t dst_dtype,
                       const int64_t* ps_version, int64_t* dst_version, int64_t period,
                       uint8_t* synced_out, gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (n < 0 || copies < 0 || copies > 64 || period < 0) return GORILA_EINVAL;
    if (dst_dtype != GORILA_F32 && dst_dtype != GORILA_BF16) return GORILA_EINVAL;
    if (copies == 0) return GORILA_OK;
    if (!ps_version || !dst_version || (n > 0 && (!src || !dst))) return GORILA_EINVAL;
    if (((uintptr_t)src & 3u) || ((uintptr_t)dst & (dst_dtype == GORILA_BF16 ? 1u : 3u)))
        return GORILA_EINVAL;
    if (((uintptr_t)ps_version | (uintptr_t)dst_version) & 7u) return GORILA_EINVAL;
    launch_params_sync(src, dst, n, copies, dst_dtype == GORILA_BF16, ps_version, dst_version,
                       period, synced_out, ctx->stream);
    return check_launch();
}

double gorila_epsilon(int64_t update, double eps_start, double eps_end, int64_t anneal_updates) {
    if (update <= 0) return eps_start;
    if (anneal_updates <= 0 || update >= anneal_updates) return eps_end;
    return eps_start + (eps_end - eps_start) * ((double)update / (double)anneal_updates);
}

int gorila_loss_filter(double* stats, const float* loss, int32_t groups, double alpha, double k,
                       int64_t warmup, uint8_t* keep_out, gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (groups < 0 || (groups > 0 && (!stats || !loss || !keep_out))) return GORILA_EINVAL;
    if (((uintptr_t)stats & 7u) != 0) return GORILA_EINVAL;
    if (!(alpha >= 0.0 && alpha <= 1.0) || !(k >= 0.0)) return GORILA_EINVAL;
    launch_loss_filter(stats, loss, groups, alpha, k, warmup, keep_out, ctx->stream);
    return check_launch();
}

int gorila_ps_apply(float* theta_plus, float* accum, int64_t n, const float* grads, int32_t groups,
                    const uint8_t* keep, const int64_t* grad_version, int64_t* ps_version,
                    int64_t max_delay, float lr, float eps, uint8_t* applied_out, gorila_ctx* ctx) {
    int rc = check_ctx(ctx);
    if (rc) return rc;
    if (n < 0 || n > INT32_MAX || groups < 0 || groups > GORILA_PS_MAX_GROUPS) return GORILA_EINVAL;
    if (!ps_version || (groups > 0 && (!grad_version || !applied_out))) return GORILA_EINVAL;
    if (n > 0 && (!theta_plus || !accum || (groups > 0 && !grads))) return GORILA_EINVAL;
    if (((uintptr_t)theta_plus | (uintptr_t)accum | (uintptr_t)grads) & 3u) return GORILA_EINVAL;
    if (((uintptr_t)grad_version | (uintptr_t)ps_version) & 7u) return GORILA_EINVAL;
    if (!(eps > 0.0f) || !(lr >= 0.0f) || !(lr < INFINITY)) return GORILA_EINVAL;
    launch_ps_apply(theta_plus, accum, n, grads, groups, keep, grad_version, ps_version, max_delay,
                    lr, eps, applied_out, ctx->stream);
    return check_launch();
}

}  // extern "C"
