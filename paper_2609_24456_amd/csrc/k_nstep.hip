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
#include "nstep_dev.h"

namespace conduit {

namespace {

constexpr int kNstepWaves = 4;
constexpr int kNstepThreads = kNstepWaves * kWave;

// The window of sample b, at the slot its index names.
__device__ __forceinline__ int64_t nstep_window(const NstepArgs& a, int64_t b, bool write) {
    return nstep_window_at(a, b, a.idx[b], write);
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
