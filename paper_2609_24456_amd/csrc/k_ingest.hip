// Ring-buffer ingest: copy n transitions into slots (head + j) mod capacity and
// bring the priority sum tree up to date, in one launch.
//
// Off-policy ingestion adds transitions to the long-lived replay store and
// keeps the per-slot bookkeeping that sampling and eviction need (paper
// Sec. 2.2); new transitions enter with the running maximum priority unless the
// caller gives one (proportional prioritised replay, Schaul et al.).
//
// One grid, three block roles:
//   * copy blocks   -- dense observations as one flat, coalesced vector copy of
//                      n*row_bytes bytes whose destination wraps once at the
//                      end of the ring (16-byte vectors when aligned);
//   * ragged blocks -- one block per variable-length sequence;
//   * meta blocks   -- one lane per transition: scalar columns, exact leaf
//                      L(p), and the leaf delta pushed up the 64-ary tree.
// Tree update: each wavefront covers 64 consecutive slots (the lanes are
// arranged so that a wavefront never straddles the ring's wrap point), so at any
// level its slots fall under at most two nodes; the wavefront reduces its deltas
// per node and issues at most two 64-bit integer atomics per level.  Integer
// addition modulo 2^64 is exact and order-independent, so the tree is
// deterministic and equal to the sum of its leaves after the kernel.
#include "ingest_dev.h"

namespace conduit {

namespace {

// The metadata/tree workgroups come first in the grid: their chain of
// dependent memory operations (old leaf, quantiser, tree atomics) is the
// longest, so they start with the first wave of dispatched workgroups and
// overlap the payload copy.
template <typename V, bool RAGGED>
__global__ __launch_bounds__(kIngestThreads) void k_ingest(IngestArgs a, int64_t meta_blocks) {
    const int64_t b = blockIdx.x;
    if (b < meta_blocks) {
        ingest_meta(a, b, threadIdx.x);
    } else {
        if constexpr (RAGGED) copy_ragged(a, b - meta_blocks, threadIdx.x);
        else copy_dense<V>(a, b - meta_blocks, threadIdx.x);
    }
}

}  // namespace

hipError_t launch_ingest(const IngestArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    const int64_t n1 = a.n < a.capacity - a.head ? a.n : a.capacity - a.head;
    const int64_t n2 = a.n - n1;
    const int64_t lanes = (n1 + kWave - 1) / kWave * kWave + (n2 + kWave - 1) / kWave * kWave;
    const int64_t meta_blocks = (lanes + kIngestThreads - 1) / kIngestThreads;
    if (a.length) {  // ragged
        const int64_t grid = a.n + meta_blocks;
        hipLaunchKernelGGL((k_ingest<uint32_t, true>), dim3((unsigned)grid), dim3(kIngestThreads), 0, s, a, meta_blocks);
        return hipGetLastError();
    }
    const uintptr_t al = reinterpret_cast<uintptr_t>(a.src_obs) | reinterpret_cast<uintptr_t>(a.obs) |
                         (uintptr_t)a.row_bytes;
    int vec = (al & 15) == 0 ? 16 : (al & 7) == 0 ? 8 : (al & 3) == 0 ? 4 : 1;
    if (a.row_bytes == 0) vec = 16;
    const int64_t total_vec = a.n * (a.row_bytes / vec);
    const int64_t copy_blocks = (total_vec + kIngestThreads * kCopyUnroll - 1) / (kIngestThreads * kCopyUnroll);
    const dim3 grid((unsigned)(copy_blocks + meta_blocks));
    switch (vec) {
        case 16: hipLaunchKernelGGL((k_ingest<u32x4, false>), grid, dim3(kIngestThreads), 0, s, a, meta_blocks); break;
        case 8: hipLaunchKernelGGL((k_ingest<u32x2, false>), grid, dim3(kIngestThreads), 0, s, a, meta_blocks); break;
        case 4: hipLaunchKernelGGL((k_ingest<uint32_t, false>), grid, dim3(kIngestThreads), 0, s, a, meta_blocks); break;
        default: hipLaunchKernelGGL((k_ingest<uint8_t, false>), grid, dim3(kIngestThreads), 0, s, a, meta_blocks); break;
    }
    return hipGetLastError();
}

}  // namespace conduit
