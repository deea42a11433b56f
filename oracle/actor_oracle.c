/*
 * Actor side of Gorila -- plain CPU oracle (replay insert, epsilon schedule).
 *
 * TEST INFRASTRUCTURE ONLY (like gorila_oracle.c): used by the tests, never by
 * the product path, and sharing no code with the HIP library.
 *
 * What it computes (Nair et al. 2015):
 *  - Algorithm 1: each step the actor stores its experience in the replay
 *    memory D; Section 4: a replay memory per actor (bundled mode) of
 *    Section 5.1's one million frames.  Readings: D holds single frames in a
 *    ring; record j of a call (frame, episode-start flag, action taken at the
 *    frame, reward that followed) is appended at logical position size + j;
 *    once the ring is full every new record overwrites the oldest one and the
 *    head (physical slot of logical 0) moves on.
 *  - Section 5.1: epsilon is annealed from 1 to 0.1 over the first million
 *    global updates.  Reading: linearly in the update count, constant after.
 *  - Algorithm 1: actors and learners update theta from theta+ of the
 *    parameter server, and every N global updates (Section 5.1: 60K) the
 *    learner syncs theta- with theta+.  Reading: a copy whose destination
 *    remembers the server version it holds; a periodic sync copies when a
 *    multiple of N lies in (held version, current version]; a bf16 replica is
 *    the round-to-nearest-even image of the fp32 value.
 */
#include <stdint.h>
#include <string.h>

#include "gorila_oracle.h"

int oracle_replay_insert(uint8_t* frames, uint8_t* ep_start, int32_t* action, float* reward,
                         int64_t capacity, int64_t frame_bytes, int64_t* head, int64_t* size,
                         const uint8_t* frames_in, const uint8_t* ep_start_in,
                         const int32_t* action_in, const float* reward_in, int32_t m) {
    if (!frames || !ep_start || !action || !reward || !head || !size || capacity < 1 ||
        frame_bytes < 1 || m < 0 || m > capacity)
        return -1;
    if (*head < 0 || *head >= capacity || *size < 0 || *size > capacity) return -1;
    for (int32_t j = 0; j < m; ++j) {
        int64_t slot;
        if (*size < capacity) {
            slot = (*head + *size) % capacity; /* append */
            *size += 1;
        } else {
            slot = *head; /* overwrite the oldest record */
            *head = (*head + 1) % capacity;
        }
        memcpy(frames + slot * frame_bytes, frames_in + (int64_t)j * frame_bytes,
               (size_t)frame_bytes);
        ep_start[slot] = ep_start_in[j] ? 1 : 0;
        action[slot] = action_in[j];
        reward[slot] = reward_in[j];
    }
    return 0;
}

double oracle_epsilon(int64_t update, double eps_start, double eps_end, int64_t anneal_updates) {
    if (update <= 0) return eps_start;
    if (anneal_updates <= 0 || update >= anneal_updates) return eps_end;
    return eps_start + (eps_end - eps_start) * ((double)update / (double)anneal_updates);
}

uint16_t oracle_f32_to_bf16(float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0)
        return (uint16_t)((u >> 16) | 0x0040u); /* NaN: keep it a (quiet) NaN */
    /* drop 16 bits, rounding to nearest with ties to the even result */
    const uint32_t lsb = (u >> 16) & 1u;
    return (uint16_t)((u + 0x7fffu + lsb) >> 16);
}

int oracle_params_sync(const float* src, void* dst, int64_t n, int32_t copies, int32_t to_bf16,
                       int64_t ps_version, int64_t* dst_version, int64_t period,
                       uint8_t* synced_out) {
    if (!src || !dst || !dst_version || !synced_out || n < 0 || copies < 0 || period < 0)
        return -1;
    for (int32_t c = 0; c < copies; ++c) {
        const int due = period == 0 || ps_version / period > dst_version[c] / period;
        synced_out[c] = due ? 1 : 0;
        if (!due) continue;
        if (to_bf16) {
            uint16_t* d = (uint16_t*)dst + (int64_t)c * n;
            for (int64_t i = 0; i < n; ++i) d[i] = oracle_f32_to_bf16(src[i]);
        } else {
            float* d = (float*)dst + (int64_t)c * n;
            for (int64_t i = 0; i < n; ++i) d[i] = src[i];
        }
        dst_version[c] = ps_version;
    }
    return 0;
}
