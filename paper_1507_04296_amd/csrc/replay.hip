// Replay minibatch resolution and the materialising gather.
//
// Frame stacking (Section 5.1): a state is the four most recent frames,
// oldest in channel 0.  Out of a ring of single frames, channel j of the
// stack ending at logical frame k holds frame l = k - 3 + j, or zeros when l
// lies before the latest episode start at or before k (logical 0 counts as a
// start).  Only starts in (l, k] matter, so at most three flags are read.
#include "common.h"
#include "kernels.h"

namespace gorila {

__global__ __launch_bounds__(256) void resolve_kernel(ReplayView rv, const int64_t* __restrict__ idx,
                                                      int n, int n_actions,
                                                      const uint8_t** __restrict__ ftab,
                                                      int32_t* __restrict__ a_out,
                                                      float* __restrict__ r_out,
                                                      uint8_t* __restrict__ term_out,
                                                      int64_t* __restrict__ fmap,
                                                      unsigned* __restrict__ err) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= n) return;
    const int64_t k = idx[b];
    const uint8_t* ptr[2][4] = {};
    int64_t slot[2][4] = {{-1, -1, -1, -1}, {-1, -1, -1, -1}};
    int32_t act = 0;
    float rew = 0.f;
    uint8_t term = 1;
    if (rv.kind == GORILA_REPLAY_STACKED) {
        if (k < 0 || k >= rv.rows) {
            atomicOr(err, ERR_IDX_RANGE);
        } else {
            for (int c = 0; c < 4; ++c) {
                ptr[0][c] = rv.s + k * STATE_BYTES + (int64_t)c * FRAME_BYTES;
                ptr[1][c] = rv.s2 + k * STATE_BYTES + (int64_t)c * FRAME_BYTES;
                slot[0][c] = slot[1][c] = k * 4 + c;
            }
            act = rv.action[k];
            rew = rv.reward[k];
            term = rv.term[k] ? 1 : 0;
        }
    } else {
        const int64_t cap = rv.capacity;
        if (k < 0 || k > cap - 2) {
            atomicOr(err, ERR_IDX_RANGE);
        } else {
            for (int w = 0; w < 2; ++w) {
                const int64_t kn = k + w;  // newest frame of the stack
                // start[d] = frame kn-d begins an episode (d = 0, 1, 2)
                bool start[3];
                for (int d = 0; d < 3; ++d) {
                    const int64_t l = kn - d;
                    start[d] = l >= 0 && rv.ep_start[(rv.head + l) % cap] != 0;
                }
                for (int j = 0; j < 4; ++j) {
                    const int64_t l = kn - 3 + j;
                    bool zero = l < 0;
                    // any start in (l, kn]: frames kn-d for d = 0 .. 2-j
                    for (int d = 0; d <= 2 - j; ++d) zero = zero || start[d];
                    if (!zero) {
                        const int64_t p = (rv.head + l) % cap;
                        ptr[w][j] = rv.frames + p * FRAME_BYTES;
                        slot[w][j] = p;
                    }
                }
            }
            const int64_t p = (rv.head + k) % cap;
            act = rv.action[p];
            rew = rv.reward[p];
            term = rv.ep_start[(rv.head + k + 1) % cap] ? 1 : 0;
        }
    }
    if (act < 0 || act >= n_actions) {
        atomicOr(err, ERR_ACTION_RANGE);
        act = 0;
    }
    for (int w = 0; w < 2; ++w)
        for (int c = 0; c < 4; ++c) {
            ftab[((int64_t)w * n + b) * 4 + c] = ptr[w][c];
            if (fmap) fmap[((int64_t)b * 2 + w) * 4 + c] = slot[w][c];
        }
    a_out[b] = act;
    r_out[b] = rew;
    term_out[b] = term;
}

void launch_resolve(const ReplayView& rv, const int64_t* idx, int n, int n_actions,
                    const uint8_t** ftab, int32_t* a, float* r, uint8_t* term,
                    int64_t* frame_map, unsigned* err, hipStream_t st) {
    if (n <= 0) return;
    resolve_kernel<<<(n + 255) / 256, 256, 0, st>>>(rv, idx, n, n_actions, ftab, a, r, term,
                                                    frame_map, err);
}

// One workgroup per (transition, s|s'): four frames of 441 16-byte vectors.
__global__ __launch_bounds__(256) void materialize_kernel(const uint8_t* const* __restrict__ ftab,
                                                          int n, uint8_t* __restrict__ s_out,
                                                          uint8_t* __restrict__ s2_out) {
    const int b = blockIdx.x, w = blockIdx.y;
    uint4* dst = (uint4*)((w ? s2_out : s_out) + (int64_t)b * STATE_BYTES);
    constexpr int VEC = FRAME_BYTES / 16;  // 441
    for (int e = threadIdx.x; e < 4 * VEC; e += 256) {
        const int c = e / VEC, q = e - c * VEC;
        const uint4* src = (const uint4*)ftab[((int64_t)w * n + b) * 4 + c];
        dst[e] = src ? src[q] : make_uint4(0, 0, 0, 0);
    }
}

void launch_materialize(const uint8_t* const* ftab, int n, uint8_t* s_out, uint8_t* s2_out,
                        hipStream_t st) {
    if (n <= 0) return;
    materialize_kernel<<<dim3(n, 2), 256, 0, st>>>(ftab, n, s_out, s2_out);
}

}  // namespace gorila
