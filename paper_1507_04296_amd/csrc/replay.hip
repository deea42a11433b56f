// Replay minibatch resolution, the materialising gather and the replay insert.
//
// Frame stacking (Section 5.1): a state is the four most recent frames,
// oldest in channel 0.  Out of a ring of single frames, channel j of the
// stack ending at logical frame k holds frame l = k - 3 + j, or zeros when l
// lies before the latest episode start at or before k (logical 0 counts as a
// start).  Only starts in (l, k] matter, so at most three flags are read.
#include "common.h"
#include "kernels.h"

#include <type_traits>

namespace gorila {

// Frame pointers (null = zero frame) and physical slots (-1) of s = stack(k)
// and s' = stack(k+1), plus the transition's action, reward and terminal flag.
// An index or action out of range sets a bit of the sticky error word (when
// err is not null) and yields zero stacks / action 0, never an out-of-bounds
// access.
// Slot of head + l for 0 <= head < cap and 0 <= l < cap (no 64-bit division).
__device__ inline int64_t wrap(int64_t x, int64_t cap) { return x >= cap ? x - cap : x; }

struct Resolved {
    const uint8_t* ptr[2][4];
    int64_t slot[2][4];
    int32_t act;
    float rew;
    uint8_t term;
};

__device__ Resolved resolve_one(const ReplayView& rv, int64_t k, int n_actions,
                                unsigned* __restrict__ err) {
    Resolved o;
#pragma unroll
    for (int w = 0; w < 2; ++w)
    #pragma unroll
        for (int c = 0; c < 4; ++c) {
            o.ptr[w][c] = nullptr;
            o.slot[w][c] = -1;
        }
    o.act = 0;
    o.rew = 0.f;
    o.term = 1;
    if (rv.kind == GORILA_REPLAY_STACKED) {
        if (k < 0 || k >= rv.rows) {
            if (err) atomicOr(err, ERR_IDX_RANGE);
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                o.ptr[0][c] = rv.s + k * STATE_BYTES + (int64_t)c * FRAME_BYTES;
                o.ptr[1][c] = rv.s2 + k * STATE_BYTES + (int64_t)c * FRAME_BYTES;
                o.slot[0][c] = o.slot[1][c] = k * 4 + c;
            }
            o.act = rv.action[k];
            o.rew = rv.reward[k];
            o.term = rv.term[k] ? 1 : 0;
        }
    } else {
        const int64_t cap = rv.capacity;
        // rows > 1: that many rings of `capacity` slots sharing `head`, and
        // index r * capacity + k names logical position k of ring r
        const int64_t rings = rv.rows > 1 ? rv.rows : 1;
        const int64_t r = rings > 1 && k >= 0 ? k / cap : 0;
        if (rings > 1) k -= r * cap;
        const int64_t ring0 = r * cap;  // first slot of ring r
        if (k < 0 || k > rv.size - 2 || r >= rings) {  // size <= cap
            if (err) atomicOr(err, ERR_IDX_RANGE);
        } else {
#pragma unroll
            for (int w = 0; w < 2; ++w) {
                const int64_t kn = k + w;  // newest frame of the stack
                // start[d] = frame kn-d begins an episode (d = 0, 1, 2)
                bool start[3];
    #pragma unroll
                for (int d = 0; d < 3; ++d) {
                    const int64_t l = kn - d;
                    start[d] = l >= 0 && rv.ep_start[ring0 + wrap(rv.head + l, cap)] != 0;
                }
    #pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t l = kn - 3 + j;
                    bool zero = l < 0;
                    // any start in (l, kn]: frames kn-d for d = 0 .. 2-j
        #pragma unroll
                    for (int d = 0; d <= 2 - j; ++d) zero = zero || start[d];
                    if (!zero) {
                        const int64_t p = ring0 + wrap(rv.head + l, cap);
                        o.ptr[w][j] = rv.frames + p * FRAME_BYTES;
                        o.slot[w][j] = p;
                    }
                }
            }
            const int64_t p = ring0 + wrap(rv.head + k, cap);
            o.act = rv.action[p];
            o.rew = rv.reward[p];
            o.term = rv.ep_start[ring0 + wrap(rv.head + k + 1, cap)] ? 1 : 0;
        }
    }
    if (o.act < 0 || o.act >= n_actions) {
        if (err) atomicOr(err, ERR_ACTION_RANGE);
        o.act = 0;
    }
    return o;
}

// W: WidenJob, or NoWiden when no set is widened (a smaller argument block)
struct NoWiden {};
template <class W>
__global__ __launch_bounds__(256) void resolve_prep_kernel(
    ReplayView rv, const int64_t* __restrict__ idx, int n, int n_actions,
    const uint8_t** __restrict__ ftab, int32_t* __restrict__ a_out, float* __restrict__ r_out,
    uint8_t* __restrict__ term_out, unsigned* __restrict__ err, WeightViewSet set, int rblocks,
    int pblocks, W wj, int wpn) {
    if constexpr (!std::is_same_v<W, NoWiden>) {
        if ((int)blockIdx.x >= rblocks + pblocks) {
            const int q = blockIdx.x - rblocks - pblocks;
            widen_part(wj, q / wpn, q % wpn, wpn);
            return;
        }
    }
    if ((int)blockIdx.x >= rblocks) {
        const int q = blockIdx.x - rblocks;
        prep_weights_part(set.v[q / PREP_BLOCKS], q % PREP_BLOCKS, PREP_BLOCKS);
        return;
    }
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= n) return;
    const Resolved o = resolve_one(rv, idx[b], n_actions, err);
    for (int w = 0; w < 2; ++w)
        for (int c = 0; c < 4; ++c) ftab[((int64_t)w * n + b) * 4 + c] = o.ptr[w][c];
    a_out[b] = o.act;
    r_out[b] = o.rew;
    term_out[b] = o.term;
}

void launch_resolve_prep(const ReplayView& rv, const int64_t* idx, int n, int n_actions,
                         const uint8_t** ftab, int32_t* a, float* r, uint8_t* term,
                         unsigned* err, const WeightViews* nets, int n_nets, const WidenJob* wj,
                         hipStream_t st) {
    WeightViewSet set{};
    for (int i = 0; i < n_nets && i < MAX_NETS; ++i) set.v[i] = nets[i];
    const int rblocks = n > 0 ? (n + 255) / 256 : 0;
    const int pblocks = PREP_BLOCKS * min(n_nets, MAX_NETS);
    const int wpn = wj ? wj->blocks_per_net() : 0;
    const int blocks = rblocks + pblocks + wpn * (wj ? min(wj->n, MAX_NETS) : 0);
    if (blocks <= 0) return;
    if (wpn > 0)
        resolve_prep_kernel<<<blocks, 256, 0, st>>>(rv, idx, n, n_actions, ftab, a, r, term, err,
                                                    set, rblocks, pblocks, *wj, wpn);
    else
        resolve_prep_kernel<<<blocks, 256, 0, st>>>(rv, idx, n, n_actions, ftab, a, r, term, err,
                                                    set, rblocks, pblocks, NoWiden{}, 1);
}

// The materialising gather: workgroup (b, f) resolves transition b (every
// thread reads the same few flags) and copies one frame of its stacks, so a
// launch has 5n (ring) or 8n (stacked) workgroups in flight.  From a ring,
// logical frame k-3+f (f = 0 .. 4) is read once and written to s (channel f)
// and s' (channel f-1), or zeros where a stack zero-fills it; stacked rows
// copy s (f < 4) and s' (f >= 4) separately.  Workgroup (b, 0) writes the
// frame map, action, reward and terminal flag.
__global__ __launch_bounds__(256) void gather_kernel(ReplayView rv, const int64_t* __restrict__ idx,
                                                     int n, int n_actions, uint8_t* __restrict__ s_out,
                                                     uint8_t* __restrict__ s2_out,
                                                     int64_t* __restrict__ fmap,
                                                     int32_t* __restrict__ a_out,
                                                     float* __restrict__ r_out,
                                                     uint8_t* __restrict__ term_out,
                                                     unsigned* __restrict__ err) {
    const int b = blockIdx.x, f = blockIdx.y, tid = threadIdx.x;
    const bool lead = f == 0 && tid == 0;
    const Resolved o = resolve_one(rv, idx[b], n_actions, lead ? err : nullptr);
    if (lead) {
        a_out[b] = o.act;
        r_out[b] = o.rew;
        term_out[b] = o.term;
        if (fmap)
#pragma unroll
            for (int j = 0; j < 8; ++j) fmap[(int64_t)b * 8 + j] = o.slot[j >> 2][j & 3];
    }
    constexpr int VEC = FRAME_BYTES / 16;  // 441
    uint4* ds = (uint4*)(s_out + (int64_t)b * STATE_BYTES);
    uint4* ds2 = (uint4*)(s2_out + (int64_t)b * STATE_BYTES);
    // Source and destinations of this workgroup's frame, chosen with constant
    // indices (the pointers are uniform over the workgroup).
    const uint8_t* in_s = nullptr;   // frame as channel cs of s (null: zeros)
    const uint8_t* in_s2 = nullptr;  // frame as channel cs2 of s'
    uint4* out_s = nullptr;
    uint4* out_s2 = nullptr;
    if (rv.kind == GORILA_REPLAY_RING) {
        switch (f) {
            case 0: in_s = o.ptr[0][0]; break;
            case 1: in_s = o.ptr[0][1]; in_s2 = o.ptr[1][0]; break;
            case 2: in_s = o.ptr[0][2]; in_s2 = o.ptr[1][1]; break;
            case 3: in_s = o.ptr[0][3]; in_s2 = o.ptr[1][2]; break;
            default: in_s2 = o.ptr[1][3]; break;
        }
        if (f < 4) out_s = ds + f * VEC;
        if (f > 0) out_s2 = ds2 + (f - 1) * VEC;
    } else {
        switch (f) {
            case 0: in_s = o.ptr[0][0]; break;
            case 1: in_s = o.ptr[0][1]; break;
            case 2: in_s = o.ptr[0][2]; break;
            case 3: in_s = o.ptr[0][3]; break;
            case 4: in_s2 = o.ptr[1][0]; break;
            case 5: in_s2 = o.ptr[1][1]; break;
            case 6: in_s2 = o.ptr[1][2]; break;
            default: in_s2 = o.ptr[1][3]; break;
        }
        if (f < 4) out_s = ds + f * VEC;
        else out_s2 = ds2 + (f - 4) * VEC;
    }
    // masks rather than selects between vectors, which the compiler would
    // route through private memory
    const uint4* src = (const uint4*)(in_s ? in_s : in_s2);  // one slot when both are set
    const uint32_t ms = in_s ? ~0u : 0u, ms2 = in_s2 ? ~0u : 0u;
    const uint4 z = make_uint4(0, 0, 0, 0);
    if (src) {
        uint4 v[2];
        const int q0 = tid, q1 = tid + 256;
        v[0] = src[q0];
        if (q1 < VEC) v[1] = src[q1];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int q = tid + 256 * u;
            if (q >= VEC) break;
            if (out_s) out_s[q] = make_uint4(v[u].x & ms, v[u].y & ms, v[u].z & ms, v[u].w & ms);
            if (out_s2)
                out_s2[q] = make_uint4(v[u].x & ms2, v[u].y & ms2, v[u].z & ms2, v[u].w & ms2);
        }
    } else {
        for (int q = tid; q < VEC; q += 256) {
            if (out_s) out_s[q] = z;
            if (out_s2) out_s2[q] = z;
        }
    }
}

void launch_gather(const ReplayView& rv, const int64_t* idx, int n, int n_actions,
                   uint8_t* s_out, uint8_t* s2_out, int64_t* frame_map, int32_t* a, float* r,
                   uint8_t* term, unsigned* err, hipStream_t st) {
    if (n <= 0) return;
    const int frames = rv.kind == GORILA_REPLAY_RING ? 5 : 8;
    gather_kernel<<<dim3(n, frames), 256, 0, st>>>(rv, idx, n, n_actions, s_out, s2_out, frame_map,
                                                   a, r, term, err);
}

// Replay insert: record j of ring r (frames_in [m][rings][84*84] etc.) goes to
// slot (base + j) mod capacity of ring r; one workgroup per record.
__global__ __launch_bounds__(256) void insert_kernel(uint8_t* __restrict__ frames,
                                                     uint8_t* __restrict__ ep_start,
                                                     int32_t* __restrict__ action,
                                                     float* __restrict__ reward, int64_t capacity,
                                                     int rings, int64_t base,
                                                     const uint8_t* __restrict__ frames_in,
                                                     const uint8_t* __restrict__ ep_in,
                                                     const int32_t* __restrict__ act_in,
                                                     const float* __restrict__ rew_in) {
    const int rec = blockIdx.x;  // = j * rings + r
    const int j = rec / rings, r = rec - j * rings;
    const int64_t slot = (int64_t)r * capacity + wrap(base + j, capacity);
    constexpr int VEC = FRAME_BYTES / 16;
    const uint4* src = (const uint4*)(frames_in + (int64_t)rec * FRAME_BYTES);
    uint4* dst = (uint4*)(frames + slot * FRAME_BYTES);
    for (int q = threadIdx.x; q < VEC; q += 256) dst[q] = src[q];
    if (threadIdx.x == 0) {
        ep_start[slot] = ep_in[rec] ? 1 : 0;
        action[slot] = act_in[rec];
        reward[slot] = rew_in[rec];
    }
}

void launch_insert(uint8_t* frames, uint8_t* ep_start, int32_t* action, float* reward,
                   int64_t capacity, int rings, int64_t base, const uint8_t* frames_in,
                   const uint8_t* ep_in, const int32_t* act_in, const float* rew_in, int records,
                   hipStream_t st) {
    if (records <= 0) return;
    insert_kernel<<<records, 256, 0, st>>>(frames, ep_start, action, reward, capacity, rings, base,
                                           frames_in, ep_in, act_in, rew_in);
}

}  // namespace gorila
