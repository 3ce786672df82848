// Priority-update device code shared by the update kernel and the fused
// update + ingest kernel.
#pragma once
#include "common.h"

namespace conduit {

namespace {

constexpr int kUpdateThreads = 1024;
constexpr int kTable = 2048;   // power of two, at least 2x the chunk size
constexpr int kBins = 2048;    // u64 LDS bins for small tree levels

__device__ __forceinline__ uint32_t slot_hash(uint32_t key) { return (key * 0x9E3779B1u) >> (32 - 11); }

// workgroup barrier ordering LDS only (no wait for outstanding global memory)
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The update pass of one workgroup of kUpdateThreads lanes: leaves swapped,
// deltas of large levels sent as global atomics and those of levels kept in
// LDS (tree.lds_offset) accumulated in `bins` (zeroed here).  Returns the
// lane's largest priority; the caller flushes the bins and raises the running
// maximum.  Ends with an LDS-only barrier: the leaf writes are not waited for.
// Slots in the ring range [ev_head, ev_head + ev_n) are about to be
// overwritten by an ingest of the same launch: their leaf and tree work is
// skipped (the ingest replaces the leaf), their priority still counts.
__device__ uint32_t update_pass(const UpdateArgs& a, uint32_t* keys, int32_t* owner, unsigned long long* bins,
                                int64_t ev_head = 0, int64_t ev_n = 0) {
    const int tid = threadIdx.x;
    const TreeView& tr = a.tree;

    uint32_t pmax = 0;
    // the first chunk's index and priority loads are issued before the LDS set-up
    int64_t k = tid;
    int64_t slot_next = k < a.n ? a.idx[k] : -1;
    uint32_t p_next = k < a.n ? a.prio[k] : 0u;
    for (int i = tid; i < kBins; i += kUpdateThreads) bins[i] = 0ull;

    for (int64_t base = 0; base < a.n; base += kUpdateThreads) {
        for (int i = tid; i < kTable; i += kUpdateThreads) {
            keys[i] = 0u;
            owner[i] = -1;
        }
        // orders global memory too: a later chunk reads leaves this one's
        // predecessors wrote
        __syncthreads();
        k = base + tid;
        bool valid = k < a.n;
        const int64_t slot = slot_next;
        const uint32_t p = p_next;
        if (valid && (slot < 0 || slot >= a.size)) {
            flag_error(a.err, ERR_UPDATE_INDEX);
            valid = false;
        }
        // the old leaf is needed only by the winner, but its load is issued now so
        // it overlaps the LDS dedupe and the quantiser (chunks before this one
        // finished their leaf writes before the barrier above); unconditional,
        // from slot 0 for an invalid entry, so that no select of its value makes
        // the lane wait for it here
        const uint32_t old = tr.leaves[valid ? slot : 0];
        uint32_t h = 0;
        if (valid) {
            pmax = p > pmax ? p : pmax;
            const uint32_t key = (uint32_t)slot + 1u;  // 0 marks an empty entry
            h = slot_hash(key);
            while (true) {
                const uint32_t prev = atomicCAS(&keys[h], 0u, key);
                if (prev == 0u || prev == key) break;
                h = (h + 1) & (kTable - 1);
            }
            atomicMax(&owner[h], tid);
        }
        // the next chunk's loads overlap this chunk's dedupe and leaf work
        const int64_t kn = base + kUpdateThreads + tid;
        slot_next = kn < a.n ? a.idx[kn] : -1;
        p_next = kn < a.n ? a.prio[kn] : 0u;
        lds_barrier();
        const int64_t cap = tr.nodes[0];
        const bool evicted = ev_n > 0 && valid && (slot - ev_head + cap) % cap < ev_n;
        if (valid && owner[h] == tid && !evicted) {
            const uint32_t q = quantise_leaf(p, tr.alpha_num, tr.alpha_den, tr.frac_bits);
            tr.leaves[slot] = q;
            const uint64_t delta = (uint64_t)q - (uint64_t)old;  // modulo 2^64
            if (delta) {
                // unrolled over the largest depth: the per-level arguments are
                // loaded together rather than one level at a time
#pragma unroll
                for (int l = 1; l <= kMaxLevels; ++l) {
                    if (l > tr.depth) break;
                    const uint64_t node = (uint64_t)slot >> (kFanoutLog2 * l);
                    const int off = tr.lds_offset[l];
                    if (off >= 0) atomicAdd(&bins[off + node], (unsigned long long)delta);
                    else atomicAdd(reinterpret_cast<unsigned long long*>(tr.level[l] + node), delta);
                }
            }
        }
        lds_barrier();  // bins complete; the table may be cleared again
    }
    return pmax;
}

// Flush the LDS-accumulated levels into the tree (after an LDS barrier).
__device__ void flush_bins(const TreeView& tr, const unsigned long long* bins) {
#pragma unroll
    for (int l = 1; l <= kMaxLevels; ++l) {
        if (l > tr.depth) break;
        const int off = tr.lds_offset[l];
        if (off < 0) continue;
        const int nodes = (int)tr.nodes[l];
        for (int i = threadIdx.x; i < nodes; i += kUpdateThreads) {
            const unsigned long long v = bins[off + i];
            if (v) atomicAdd(reinterpret_cast<unsigned long long*>(tr.level[l] + i), v);
        }
    }
}


}  // namespace
}  // namespace conduit
