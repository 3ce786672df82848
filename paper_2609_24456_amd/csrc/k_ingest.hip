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

// Episode id and step of the rows of a single stream, from their done flags
// (the caller gave none): transition t + 1 continues t's episode one step on,
// unless t ended it (done), when t + 1 starts the next episode at step 0; the
// first transition ever is episode 0, step 0.  So for row j, with the
// previous transition (position total - 1, in the slot before head) as row -1:
//   episode(j) = episode(-1) + #{done among rows -1 .. j-1}
//   step(j)    = j - start(j),  start(j) = 1 + the last row k < j with done,
//                or, without one, -(step(-1) + 1) (the episode continues).
// One workgroup: each lane counts the dones of its contiguous share of rows,
// the lanes' counts and last done rows are scanned in LDS, then every lane
// walks its share again writing both columns into the ring.
constexpr int kDeriveThreads = 1024;

__global__ __launch_bounds__(kDeriveThreads) void k_derive_meta(IngestArgs a) {
    __shared__ int64_t s_cnt[2][kDeriveThreads];
    __shared__ int64_t s_last[2][kDeriveThreads];
    __shared__ uint32_t s_ep0;
    __shared__ int64_t s_start0;
    const int tid = threadIdx.x;
    const int64_t per = (a.n + kDeriveThreads - 1) / kDeriveThreads;
    const int64_t lo = (int64_t)tid * per < a.n ? (int64_t)tid * per : a.n;
    const int64_t hi = lo + per < a.n ? lo + per : a.n;
    if (tid == 0) {  // row -1: read before any slot is rewritten (the barriers below)
        uint32_t ep0 = 0;
        int64_t start0 = 0;
        if (a.total > 0) {
            const int64_t ps = (a.head + a.capacity - 1) % a.capacity;
            const bool pd = a.done[ps] != 0;
            ep0 = a.episode[ps] + (pd ? 1u : 0u);
            start0 = pd ? 0 : -((int64_t)a.step[ps] + 1);
        }
        s_ep0 = ep0;
        s_start0 = start0;
    }
    int64_t cnt = 0, last = -1;
    if (a.src_done) {
        for (int64_t j = lo; j < hi; ++j) {
            if (a.src_done[j]) {
                ++cnt;
                last = j;
            }
        }
    }
    // inclusive scans over the lanes (sum of counts, max of last done rows),
    // ping-ponging between two LDS rows
    int cur = 0;
    s_cnt[0][tid] = cnt;
    s_last[0][tid] = last;
    __syncthreads();
    for (int d = 1; d < kDeriveThreads; d <<= 1) {
        const int64_t c = s_cnt[cur][tid] + (tid >= d ? s_cnt[cur][tid - d] : 0);
        const int64_t l0 = s_last[cur][tid], l1 = tid >= d ? s_last[cur][tid - d] : -1;
        s_cnt[cur ^ 1][tid] = c;
        s_last[cur ^ 1][tid] = l0 > l1 ? l0 : l1;
        cur ^= 1;
        __syncthreads();
    }
    const int64_t excl_cnt = tid > 0 ? s_cnt[cur][tid - 1] : 0;
    const int64_t excl_last = tid > 0 ? s_last[cur][tid - 1] : -1;
    uint32_t ep = s_ep0 + (uint32_t)excl_cnt;
    int64_t start = excl_last >= 0 ? excl_last + 1 : s_start0;
    for (int64_t j = lo; j < hi; ++j) {
        const int64_t slot = (a.head + j) % a.capacity;
        if (a.derive & kDeriveEpisode) a.episode[slot] = ep;
        if (a.derive & kDeriveStep) a.step[slot] = (int32_t)(j - start);
        if (a.src_done && a.src_done[j]) {
            ++ep;
            start = j + 1;
        }
    }
}

}  // namespace

hipError_t launch_derive_meta(const IngestArgs& a, hipStream_t s) {
    if (a.n <= 0 || !a.derive) return hipSuccess;
    hipLaunchKernelGGL(k_derive_meta, dim3(1), dim3(kDeriveThreads), 0, s, a);
    return hipGetLastError();
}

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
