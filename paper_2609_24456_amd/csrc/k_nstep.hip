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
// With the bootstrap frame stacks requested, k_nstep_gather evaluates the
// windows inside the gather's own workgroups (one launch); otherwise k_nstep.
#include "gather_dev.h"

namespace conduit {

namespace {

constexpr int kNstepWaves = 4;
constexpr int kNstepThreads = kNstepWaves * kWave;

// The window of sample b by one whole wavefront.  Returns the slot of the
// bootstrap state (position p + n), or -1 when the sample has none (its episode
// ended inside the window, the window is invalid, or the index is out of
// range).  With `write`, lane 0 stores the sample's targets and flags a bad
// index.
__device__ __forceinline__ int64_t nstep_window(const NstepArgs& a, int64_t b, bool write) {
    const int lane = lane_id();
    const int64_t i = a.idx[b];
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

__global__ __launch_bounds__(kNstepThreads) void k_nstep(NstepArgs a) {
    const int64_t b = (int64_t)blockIdx.x * kNstepWaves + threadIdx.x / kWave;
    if (b >= a.batch) return;  // wave-uniform
    (void)nstep_window(a, b, true);
}

// Targets and bootstrap frame stacks in one launch, for rows of a few work
// items: W workgroups per sample (two items each), whose first wavefront
// evaluates the sample's window itself -- the first of the W also stores the
// targets -- and whose four wavefronts then gather the stack of the bootstrap
// state (a zero row where there is none), as the fused sampler + gather does
// after its descent.
template <int XF>
__global__ __launch_bounds__(kThreads) void k_nstep_gather(NstepArgs na, GatherArgs a, int32_t bpf, int32_t wgs) {
    __shared__ uint16_t lut[(XF == CONDUIT_XF_U8_BF16_NORM) ? 4 * 256 : 1];
    __shared__ int64_t s_slot;
    const int64_t b = (int64_t)blockIdx.x / wgs;
    const int part = (int)((int64_t)blockIdx.x - b * wgs);
    if (threadIdx.x < kWave) {
        const int64_t next = nstep_window(na, b, part == 0);
        if (threadIdx.x == 0) s_slot = next;
    } else if constexpr (XF == CONDUIT_XF_U8_BF16_NORM) {
        build_lut(a, lut, kWave, kThreads - kWave);
    }
    __syncthreads();
    gather_row<XF>(a, b, part, wgs, bpf, s_slot, lut, threadIdx.x);
}

template <int XF>
hipError_t launch_nstep_gather_xf(const NstepArgs& na, const GatherArgs& ga, int64_t bpf, int64_t wgs,
                                  hipStream_t s) {
    hipLaunchKernelGGL((k_nstep_gather<XF>), dim3((unsigned)(na.batch * wgs)), dim3(kThreads), 0, s, na, ga,
                       (int32_t)bpf, (int32_t)wgs);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_nstep(const NstepArgs& a, hipStream_t s) {
    const int64_t blocks = (a.batch + kNstepWaves - 1) / kNstepWaves;
    hipLaunchKernelGGL(k_nstep, dim3((unsigned)blocks), dim3(kNstepThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_nstep_gather(const NstepArgs& na, const GatherArgs& ga, hipStream_t s) {
    const bool c16 = copy16(ga);
    const int64_t units = ga.row_bytes >> (c16 ? 4 : 2);
    const int64_t bpf = ga.out && units > 0 ? (units + kUnitsPerBlock - 1) / kUnitsPerBlock : 0;
    const int64_t per_row = bpf * ga.stack;
    if (na.batch <= 0 || ga.n != na.batch || ga.ncols != 0 || ga.weights.w || per_row < 1 ||
        per_row > kFusedMaxItemsPerRow)
        return hipErrorNotSupported;
    const int64_t wgs = per_row > 2 ? (per_row + 1) / 2 : 1;  // two items per workgroup
    if (c16) return launch_nstep_gather_xf<kXfCopy16>(na, ga, bpf, wgs, s);
    switch (ga.xform) {
        case CONDUIT_XF_NONE: return launch_nstep_gather_xf<CONDUIT_XF_NONE>(na, ga, bpf, wgs, s);
        case CONDUIT_XF_U8_F32: return launch_nstep_gather_xf<CONDUIT_XF_U8_F32>(na, ga, bpf, wgs, s);
        case CONDUIT_XF_U8_BF16_NORM: return launch_nstep_gather_xf<CONDUIT_XF_U8_BF16_NORM>(na, ga, bpf, wgs, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace conduit
