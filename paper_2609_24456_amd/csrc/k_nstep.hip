// n-step return targets of sampled slots (off-policy delivery materialising
// training-ready transitions, Sec. 2.2; the n-step Q-learning target of the
// DQN line of work the paper builds on): for the slot holding stream position
// p, R = sum_k gamma^k r_{p+k} over the window p, p+1, ... that stops after
// the first done (no bootstrap) or after n transitions (bootstrap from the
// state at p+n, discount gamma^n).  A window that meets a position not yet
// stored, or another episode without a done, is invalid.
//
// One wavefront per sample: lane k reads position p+k (k = 0..n, n <= 63), the
// first gap and the first terminal come from two ballots, and the return is
// summed in fp64 in ascending k from register shuffles, so every lane agrees.
#include "common.h"

namespace conduit {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;

__global__ __launch_bounds__(kThreads) void k_nstep(NstepArgs a) {
    const int64_t b = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (b >= a.batch) return;  // wave-uniform
    const int lane = lane_id();
    const int64_t i = a.idx[b];
    const bool ok = i >= 0 && i < a.size;  // wave-uniform
    if (!ok) {
        if (lane == 0) {
            flag_error(a.err, ERR_GATHER_INDEX);
            a.next_idx[b] = -1;
            a.ret[b] = 0.0f;
            a.discount[b] = 0.0f;
            a.valid[b] = 0;
        }
        return;
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
    double R = 0.0, g = 1.0;
    for (int k = 0; k < m; ++k) {  // uniform trip count
        const float rk = __shfl(r, k, kWave);
        R += g * (double)rk;
        g *= a.gamma;
    }
    if (lane == 0) {
        a.next_idx[b] = bootstrap ? (p + a.n) % a.capacity : -1;
        a.ret[b] = valid ? (float)R : 0.0f;
        a.discount[b] = bootstrap ? (float)g : 0.0f;
        a.valid[b] = valid ? 1 : 0;
    }
}

}  // namespace

hipError_t launch_nstep(const NstepArgs& a, hipStream_t s) {
    const int64_t blocks = (a.batch + kWaves - 1) / kWaves;
    hipLaunchKernelGGL(k_nstep, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
