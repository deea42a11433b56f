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
