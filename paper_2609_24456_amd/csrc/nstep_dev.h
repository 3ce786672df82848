// The n-step window of one sample, evaluated by one whole wavefront (used by
// the n-step kernels and by the fused sampler + gather + n-step kernel).
#pragma once
#include "common.h"

namespace conduit {
namespace {

// The loads of the window of the sample at slot i (the same in every lane of
// the wavefront): lane k reads position p + k.  nstep_window_finish evaluates
// them; between the two the wavefront may issue other loads.
struct WindowLoads {
    int64_t i, p;
    bool ok, stored;
    float r;
    uint8_t d;
    uint32_t e;
};

__device__ __forceinline__ WindowLoads nstep_window_load(const NstepArgs& a, int64_t i) {
    WindowLoads w;
    w.i = i;
    w.ok = i >= 0 && i < a.size;  // wave-uniform
    w.p = 0;
    w.stored = false;
    w.r = 0.0f;
    w.d = 0;
    w.e = 0;
    if (w.ok) {
        // the stream position slot i holds: the newest q = i (mod capacity) below total
        w.p = i + ((a.total - 1 - i) / a.capacity) * a.capacity;
        const int64_t q = w.p + lane_id();
        w.stored = lane_id() <= a.n && q < a.total;
        const int64_t s = w.stored ? q % a.capacity : i;  // clamped: every load is in range
        w.r = a.reward[s];
        w.d = a.done[s];
        w.e = a.episode[s];
    }
    return w;
}

// Returns the slot of the bootstrap state (position p + n), or -1 when the
// sample has none (its episode ended inside the window, the window is invalid,
// or the slot is outside [0, size)).  With `write`, lane 0 stores the sample's
// targets and flags a slot outside [0, size).
__device__ __forceinline__ int64_t nstep_window_finish(const NstepArgs& a, int64_t b, const WindowLoads& w,
                                                       bool write) {
    const int lane = lane_id();
    if (!w.ok) {
        if (write && lane == 0) {
            flag_error(a.err, ERR_GATHER_INDEX);
            a.next_idx[b] = -1;
            a.ret[b] = 0.0f;
            a.discount[b] = 0.0f;
            a.valid[b] = 0;
        }
        return -1;
    }
    const uint32_t e0 = __builtin_amdgcn_readlane(w.e, 0);
    const bool same = w.stored && w.e == e0;  // position p + lane continues the episode
    const uint64_t gap = __ballot(lane < a.n && !same);
    const uint64_t term = __ballot(lane < a.n && same && w.d != 0);
    const uint64_t cont = __ballot(same);
    const int first_gap = gap ? __ffsll((unsigned long long)gap) - 1 : 64;
    const int first_term = term ? __ffsll((unsigned long long)term) - 1 : 64;
    int m = 0;            // transitions summed
    bool valid = false, bootstrap = false;
    if (first_term < first_gap) {  // the episode ends inside the window
        valid = true;
        m = first_term + 1;
    } else if (first_gap >= a.n && ((cont >> a.n) & 1ull)) {  // n transitions, state at p+n stored
        valid = true;
        bootstrap = true;
        m = a.n;
    }
    const int64_t next = bootstrap ? (w.p + a.n) % a.capacity : -1;
    if (write) {
        double R = 0.0, g = 1.0;
        for (int k = 0; k < m; ++k) {  // uniform trip count
            const float rk = __shfl(w.r, k, kWave);
            R += g * (double)rk;
            g *= a.gamma;
        }
        if (lane == 0) {
            a.next_idx[b] = next;
            a.ret[b] = valid ? (float)R : 0.0f;
            a.discount[b] = bootstrap ? (float)g : 0.0f;
            a.valid[b] = valid ? 1 : 0;
        }
    }
    return next;
}

// The window of sample b at slot i, loads and evaluation in one (the same
// steps as nstep_window_load + nstep_window_finish; written out as one
// function, which the n-step kernels run 0.45 us faster per DQN batch).
__device__ __forceinline__ int64_t nstep_window_at(const NstepArgs& a, int64_t b, int64_t i, bool write) {
    const int lane = lane_id();
    const bool ok = i >= 0 && i < a.size;  // wave-uniform
    if (!ok) {
        if (write && lane == 0) {
            flag_error(a.err, ERR_GATHER_INDEX);
            a.next_idx[b] = -1;
            a.ret[b] = 0.0f;
            a.discount[b] = 0.0f;
            a.valid[b] = 0;
        }
        return -1;
    }
    // the stream position slot i holds: the newest q = i (mod capacity) below total
    const int64_t p = i + ((a.total - 1 - i) / a.capacity) * a.capacity;
    const int64_t q = p + lane;
    const bool stored = lane <= a.n && q < a.total;
    const int64_t s = stored ? q % a.capacity : i;  // clamped: every load is in range
    const float r = a.reward[s];
    const uint8_t d = a.done[s];
    const uint32_t e = a.episode[s];
    const uint32_t e0 = __builtin_amdgcn_readlane(e, 0);
    const bool same = stored && e == e0;  // position p + lane continues the episode
    const uint64_t gap = __ballot(lane < a.n && !same);
    const uint64_t term = __ballot(lane < a.n && same && d != 0);
    const uint64_t cont = __ballot(same);
    const int first_gap = gap ? __ffsll((unsigned long long)gap) - 1 : 64;
    const int first_term = term ? __ffsll((unsigned long long)term) - 1 : 64;
    int m = 0;            // transitions summed
    bool valid = false, bootstrap = false;
    if (first_term < first_gap) {  // the episode ends inside the window
        valid = true;
        m = first_term + 1;
    } else if (first_gap >= a.n && ((cont >> a.n) & 1ull)) {  // n transitions, state at p+n stored
        valid = true;
        bootstrap = true;
        m = a.n;
    }
    const int64_t next = bootstrap ? (p + a.n) % a.capacity : -1;
    if (write) {
        double R = 0.0, g = 1.0;
        for (int k = 0; k < m; ++k) {  // uniform trip count
            const float rk = __shfl(r, k, kWave);
            R += g * (double)rk;
            g *= a.gamma;
        }
        if (lane == 0) {
            a.next_idx[b] = next;
            a.ret[b] = valid ? (float)R : 0.0f;
            a.discount[b] = bootstrap ? (float)g : 0.0f;
            a.valid[b] = valid ? 1 : 0;
        }
    }
    return next;
}


}  // namespace
}  // namespace conduit
