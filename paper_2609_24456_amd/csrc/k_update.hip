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
#include "common.h"

namespace conduit {

namespace {

constexpr int kThreads = 1024;
constexpr int kTable = 2048;   // power of two, at least 2x the chunk size
constexpr int kBins = 2048;    // u64 LDS bins for small tree levels

__device__ __forceinline__ uint32_t slot_hash(uint32_t key) { return (key * 0x9E3779B1u) >> (32 - 11); }

// workgroup barrier ordering LDS only (no wait for outstanding global memory)
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__global__ __launch_bounds__(kThreads) void k_update(UpdateArgs a) {
    __shared__ uint32_t keys[kTable];
    __shared__ int32_t owner[kTable];
    __shared__ unsigned long long bins[kBins];
    const int tid = threadIdx.x;
    const TreeView& tr = a.tree;

    uint32_t pmax = 0;
    // the first chunk's index and priority loads are issued before the LDS set-up
    int64_t k = tid;
    int64_t slot_next = k < a.n ? a.idx[k] : -1;
    uint32_t p_next = k < a.n ? a.prio[k] : 0u;
    for (int i = tid; i < kBins; i += kThreads) bins[i] = 0ull;

    for (int64_t base = 0; base < a.n; base += kThreads) {
        for (int i = tid; i < kTable; i += kThreads) {
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
        // finished their leaf writes before the barrier above)
        const uint32_t old = valid ? tr.leaves[slot] : 0u;
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
        const int64_t kn = base + kThreads + tid;
        slot_next = kn < a.n ? a.idx[kn] : -1;
        p_next = kn < a.n ? a.prio[kn] : 0u;
        lds_barrier();
        if (valid && owner[h] == tid) {
            const uint32_t q = quantise_leaf(p, tr.alpha_num, tr.alpha_den, tr.frac_bits);
            tr.leaves[slot] = q;
            const uint64_t delta = (uint64_t)q - (uint64_t)old;  // modulo 2^64
            if (delta) {
                for (int l = 1; l <= tr.depth; ++l) {
                    const uint64_t node = (uint64_t)slot >> (kFanoutLog2 * l);
                    const int off = tr.lds_offset[l];
                    if (off >= 0) atomicAdd(&bins[off + node], (unsigned long long)delta);
                    else atomicAdd(reinterpret_cast<unsigned long long*>(tr.level[l] + node), delta);
                }
            }
        }
        lds_barrier();  // bins complete; the table may be cleared again
    }
    // flush the LDS-accumulated levels
    for (int l = 1; l <= tr.depth; ++l) {
        const int off = tr.lds_offset[l];
        if (off < 0) continue;
        const int nodes = (int)tr.nodes[l];
        for (int i = tid; i < nodes; i += kThreads) {
            const unsigned long long v = bins[off + i];
            if (v) atomicAdd(reinterpret_cast<unsigned long long*>(tr.level[l] + i), v);
        }
    }
    // running maximum priority: one atomic per wavefront
    const uint32_t wm = wave_max_u32(pmax);
    if (lane_id() == 0 && wm > 0) atomicMax(&a.state->max_prio, wm);
}

}  // namespace

hipError_t launch_update(const UpdateArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_update, dim3(1), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
