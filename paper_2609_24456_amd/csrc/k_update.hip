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

// One tree level recomputed from the level below it (level 1 from the
// leaves): one wavefront per node, lane j loading child 64 * node + j, the
// wavefront's integer sum stored by lane 0.  Every level is zero-padded to a
// multiple of 64 entries and nodes(l) = ceil(nodes(l - 1) / 64), so every
// child index is inside the padded level.
constexpr int kRebuildThreads = 256;

__global__ __launch_bounds__(kRebuildThreads) void k_tree_level(const uint32_t* leaves, const uint64_t* below,
                                                                uint64_t* out, int64_t nodes) {
    const int64_t node = ((int64_t)blockIdx.x * kRebuildThreads + threadIdx.x) / kWave;
    if (node >= nodes) return;  // whole wavefronts leave together
    const int64_t c = node * kWave + lane_id();
    const uint64_t x = leaves ? (uint64_t)leaves[c] : below[c];
    const uint64_t sum = readlane_u64(wave_inclusive_scan_u64(x), kWave - 1);
    if (lane_id() == 0) out[node] = sum;
}

}  // namespace

hipError_t launch_tree_rebuild(const TreeView& t, hipStream_t s) {
    for (int l = 1; l <= t.depth; ++l) {
        const int64_t threads = t.nodes[l] * kWave;
        const int64_t grid = (threads + kRebuildThreads - 1) / kRebuildThreads;
        hipLaunchKernelGGL(k_tree_level, dim3((unsigned)grid), dim3(kRebuildThreads), 0, s, l == 1 ? t.leaves : nullptr,
                           l == 1 ? nullptr : t.level[l - 1], t.level[l], t.nodes[l]);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_update(const UpdateArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_update, dim3(1), dim3(kUpdateThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
