// Batched, deterministic priority update (the learner's priority callback,
// paper App. C Invariant 2; proportional prioritised replay, Schaul et al.).
//
// Semantics: updates apply as if one after another in array order, so the last
// occurrence of a repeated index wins.  One workgroup of 1024 lanes walks the
// update list in chunks of 1024:
//   1. an LDS open-addressing table (2048 entries) keyed by slot keeps the
//      largest position of every slot within the chunk (LDS atomicMax), which
//      selects exactly one winner per distinct slot;
//   2. winners compute the exact leaf L(p), swap it into the leaf array and push
//      delta = new - old up the 64-ary tree: levels with few nodes are
//      accumulated in LDS bins (flushed once at the end), large levels receive
//      64-bit global atomics directly;
//   3. chunks run in order, so a later chunk reads the leaves an earlier one
//      wrote (same workgroup, separated by a barrier).
// All tree arithmetic is integer modulo 2^64: exact and independent of the
// order in which atomics land.  Sizes of the paper's workloads (256 to 1024
// updates per call) take a single chunk.
//
// Latency: barriers that only order LDS traffic use an LDS-only fence, so the
// global tree atomics issued by the winners are never waited for inside the
// kernel (they drain at its end, overlapping the flush); only the barrier that
// starts a later chunk orders global memory, because that chunk reads leaves
// the previous one wrote.
#include "update_dev.h"

namespace conduit {

namespace {

__global__ __launch_bounds__(kUpdateThreads) void k_update(UpdateArgs a) {
    __shared__ uint32_t keys[kTable];
    __shared__ int32_t owner[kTable];
    __shared__ unsigned long long bins[kBins];
    const uint32_t pmax = update_pass(a, keys, owner, bins);
    flush_bins(a.tree, bins);
    // running maximum priority: one atomic per wavefront
    const uint32_t wm = wave_max_u32(pmax);
    if (lane_id() == 0 && wm > 0) atomicMax(&a.state->max_prio, wm);
}

}  // namespace

hipError_t launch_update(const UpdateArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_update, dim3(1), dim3(kUpdateThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
