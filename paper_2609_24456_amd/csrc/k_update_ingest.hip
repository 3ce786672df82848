// Fused priority update + ingest: the learner's new priorities for the last
// batch (App. C Invariant 2) and then the actor's next transitions (Sec. 2.2
// off-policy ingestion), with the effects of conduit_update_priorities
// followed by conduit_ingest, in one launch whose parts run concurrently.
//
// In that order the ingest overwrites the leaf of every slot it evicts, so an
// update of such a slot changes nothing but the running maximum priority; and
// the new rows enter with the running maximum raised by the update's
// priorities, which is max(current, every valid update priority).  Hence:
//   * block 0 (1024 lanes) runs the update pass (update_dev.h) skipping the
//     slots the ingest evicts, flushes its LDS bins and raises the running
//     maximum;
//   * every other block is four ingest sub-blocks of 256 lanes (ingest_dev.h):
//     the new rows' columns, leaves and per-wavefront tree deltas, each
//     wavefront computing the raised running maximum from the update list
//     itself, and the payload copy.
// The two sets of leaves are disjoint and every tree change is an integer
// atomic add, so the result equals the two calls made one after the other.
#include "ingest_dev.h"
#include "update_dev.h"

namespace conduit {

namespace {

constexpr int kSubs = kUpdateThreads / kIngestThreads;

template <typename V>
__global__ __launch_bounds__(kUpdateThreads) void k_update_ingest(UpdateArgs u, IngestArgs a, int64_t meta_subs,
                                                                  int64_t copy_subs) {
    __shared__ uint32_t keys[kTable];
    __shared__ int32_t owner[kTable];
    __shared__ unsigned long long bins[kBins];
    if (blockIdx.x == 0) {
        const uint32_t pmax = update_pass(u, keys, owner, bins, a.head, a.n);
        flush_bins(u.tree, bins);
        const uint32_t wm = wave_max_u32(pmax);
        if (lane_id() == 0 && wm > 0) atomicMax(&u.state->max_prio, wm);
        return;
    }
    const int64_t sub = (int64_t)(blockIdx.x - 1) * kSubs + threadIdx.x / kIngestThreads;
    const int tid = (int)(threadIdx.x % kIngestThreads);
    if (sub < meta_subs) {
        // the update block may already have raised the stored maximum with the
        // same priorities: raised_max takes max() over both, so the order of
        // the two parts does not matter
        ingest_meta(a, sub, tid, RaiseList{u.idx, u.prio, u.n, u.size});
    } else if (sub - meta_subs < copy_subs) {
        copy_dense<V>(a, sub - meta_subs, tid);
    }
}

}  // namespace

hipError_t launch_update_ingest(const UpdateArgs& u, const IngestArgs& a, hipStream_t s) {
    const int64_t lanes = [&] {
        const int64_t n1 = a.n < a.capacity - a.head ? a.n : a.capacity - a.head;
        return (n1 + kWave - 1) / kWave * kWave + (a.n - n1 + kWave - 1) / kWave * kWave;
    }();
    const int64_t meta_subs = (lanes + kIngestThreads - 1) / kIngestThreads;
    const uintptr_t al = reinterpret_cast<uintptr_t>(a.src_obs) | reinterpret_cast<uintptr_t>(a.obs) |
                         (uintptr_t)a.row_bytes;
    int vec = (al & 15) == 0 ? 16 : (al & 7) == 0 ? 8 : (al & 3) == 0 ? 4 : 1;
    if (a.row_bytes == 0) vec = 16;
    const int64_t total_vec = a.n * (a.row_bytes / vec);
    const int64_t copy_subs = (total_vec + kIngestThreads * kCopyUnroll - 1) / (kIngestThreads * kCopyUnroll);
    const dim3 grid((unsigned)(1 + (meta_subs + copy_subs + kSubs - 1) / kSubs)), block(kUpdateThreads);
    switch (vec) {
        case 16: hipLaunchKernelGGL((k_update_ingest<u32x4>), grid, block, 0, s, u, a, meta_subs, copy_subs); break;
        case 8: hipLaunchKernelGGL((k_update_ingest<u32x2>), grid, block, 0, s, u, a, meta_subs, copy_subs); break;
        case 4: hipLaunchKernelGGL((k_update_ingest<uint32_t>), grid, block, 0, s, u, a, meta_subs, copy_subs); break;
        default: hipLaunchKernelGGL((k_update_ingest<uint8_t>), grid, block, 0, s, u, a, meta_subs, copy_subs); break;
    }
    return hipGetLastError();
}

}  // namespace conduit
