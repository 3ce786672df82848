// Ring-buffer ingest: copy n transitions into slots (head + j) mod capacity and
// bring the priority sum tree up to date, in one launch.
//
// Off-policy ingestion inserts transitions into a persistent replay dataset and
// keeps the indices and metadata needed for sampling and eviction (paper
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
#include "common.h"

namespace conduit {

namespace {

constexpr int kThreads = 256;
constexpr int kCopyUnroll = 4;
constexpr int kActWords = 8;  // action words of a row held in registers
constexpr int kRaggedUnroll = 8;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void pin(u32x4& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin(u32x2& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin(uint32_t& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void pin(uint8_t& x) {
    uint32_t w = x;
    asm volatile("" : "+v"(w));
    x = (uint8_t)w;
}

template <typename V>
__device__ void copy_dense(const IngestArgs& a, int64_t block) {
    const int64_t vec_per_row = a.row_bytes / (int64_t)sizeof(V);
    const int64_t total = a.n * vec_per_row;
    const int64_t ring = a.capacity * vec_per_row;
    const int64_t head_v = a.head * vec_per_row;
    const V* __restrict__ src = reinterpret_cast<const V*>(a.src_obs);
    V* __restrict__ dst = reinterpret_cast<V*>(a.obs);
    const int64_t base = block * (kThreads * kCopyUnroll) + threadIdx.x;
    // every load is unconditional (out-of-range lanes re-read the last vector) so
    // all kCopyUnroll loads of a lane are in flight at once
    V v[kCopyUnroll];
#pragma unroll
    for (int r = 0; r < kCopyUnroll; ++r) {
        const int64_t i = base + (int64_t)r * kThreads;
        v[r] = src[i < total ? i : total - 1];
    }
    // the empty asm statements keep every load ahead of the first store: the
    // compiler would otherwise sink loads into the stores' range checks and
    // wait between stores (vmcnt counts both)
#pragma unroll
    for (int r = 0; r < kCopyUnroll; ++r) pin(v[r]);
#pragma unroll
    for (int r = 0; r < kCopyUnroll; ++r) {
        const int64_t i = base + (int64_t)r * kThreads;
        if (i < total) {
            int64_t d = head_v + i;
            if (d >= ring) d -= ring;
            dst[d] = v[r];
        }
    }
}

__device__ void copy_ragged(const IngestArgs& a, int64_t j) {
    int64_t slot = a.head + j;
    if (slot >= a.capacity) slot -= a.capacity;
    int64_t len = a.src_offsets[j + 1] - a.src_offsets[j];
    if (len < 0) len = 0;
    if (len > a.max_len) len = a.max_len;  // flagged by the meta lane of row j
    const int64_t off = a.src_offsets[j];
    if (len == 0) return;
    const uint32_t* __restrict__ s = reinterpret_cast<const uint32_t*>(a.src_obs) + off;
    uint32_t* __restrict__ d = reinterpret_cast<uint32_t*>(a.obs + slot * a.row_bytes);
    const bool aux = a.aux && a.src_aux;
    const uint32_t* __restrict__ sa = aux ? reinterpret_cast<const uint32_t*>(a.src_aux) + off : s;
    uint32_t* __restrict__ da = aux ? reinterpret_cast<uint32_t*>(a.aux) + slot * a.max_len : nullptr;
    // kRaggedUnroll elements per lane per pass, every load (clamped to the last
    // element) ahead of the stores
    for (int64_t t0 = threadIdx.x; t0 < len; t0 += (int64_t)kThreads * kRaggedUnroll) {
        uint32_t v[kRaggedUnroll], w[kRaggedUnroll];
#pragma unroll
        for (int r = 0; r < kRaggedUnroll; ++r) {
            const int64_t t = t0 + (int64_t)r * kThreads;
            const int64_t tc = t < len ? t : len - 1;
            v[r] = s[tc];
            w[r] = sa[tc];
        }
#pragma unroll
        for (int r = 0; r < kRaggedUnroll; ++r) {
            pin(v[r]);
            pin(w[r]);
        }
#pragma unroll
        for (int r = 0; r < kRaggedUnroll; ++r) {
            const int64_t t = t0 + (int64_t)r * kThreads;
            if (t < len) {
                d[t] = v[r];
                if (aux) da[t] = w[r];
            }
        }
    }
}

__device__ void ingest_meta(const IngestArgs& a, int64_t block) {
    // rows [0, n1) go to slots head.., rows [n1, n) to slots 0..; each segment
    // starts on a wavefront boundary
    const int64_t n1 = a.n < a.capacity - a.head ? a.n : a.capacity - a.head;
    const int64_t lanes_a = (n1 + kWave - 1) / kWave * kWave;
    const int64_t t = block * kThreads + threadIdx.x;
    int64_t j, slot;
    bool valid;
    if (t < lanes_a) {
        j = t;
        slot = a.head + t;
        valid = t < n1;
    } else {
        j = n1 + (t - lanes_a);
        slot = t - lanes_a;
        valid = j < a.n;
    }
    const uint64_t any_valid = __ballot(valid);
    if (any_valid == 0) return;  // whole wavefront past the end (wave-uniform)

    // every load of the lane's row is issued before its first store (lanes past
    // the end read row 0 and store nothing): one memory round trip in all
    uint64_t delta = 0;
    uint32_t p_seen = 0;
    const int64_t jj = valid ? j : 0;
    const uint32_t old = (valid && a.prioritized) ? a.tree.leaves[slot] : 0u;
    const uint32_t p = !a.prioritized ? 0u : a.src_prio ? a.src_prio[jj] : a.state->max_prio;
    const float rew = a.src_reward ? a.src_reward[jj] : 0.0f;
    const uint8_t dn = a.src_done ? a.src_done[jj] : (uint8_t)0;
    const uint32_t ep = a.src_episode ? a.src_episode[jj] : 0u;
    const int32_t st = a.src_step ? a.src_step[jj] : 0;
    const int64_t len = a.length ? a.src_offsets[jj + 1] - a.src_offsets[jj] : 0;
    const bool act_words = a.src_action && (a.action_bytes & 3) == 0;
    const int words = act_words ? a.action_bytes >> 2 : 0;
    uint32_t w[kActWords];
#pragma unroll
    for (int c = 0; c < kActWords; ++c)
        w[c] = c < words ? reinterpret_cast<const uint32_t*>(a.src_action + jj * a.action_bytes)[c] : 0u;
    if (valid) {
        if (a.action_bytes > 0) {
            uint8_t* dst = a.action + slot * a.action_bytes;
            if (act_words) {
#pragma unroll
                for (int c = 0; c < kActWords; ++c)
                    if (c < words) reinterpret_cast<uint32_t*>(dst)[c] = w[c];
                for (int c = kActWords; c < words; ++c)  // long actions: the rest word by word
                    reinterpret_cast<uint32_t*>(dst)[c] = reinterpret_cast<const uint32_t*>(a.src_action + j * a.action_bytes)[c];
            } else if (a.src_action) {
                for (int c = 0; c < a.action_bytes; ++c) dst[c] = a.src_action[j * a.action_bytes + c];
            } else {
                for (int c = 0; c < a.action_bytes; ++c) dst[c] = 0;
            }
        }
        a.reward[slot] = rew;
        a.done[slot] = dn;
        a.episode[slot] = ep;
        a.step[slot] = st;
        if (a.length) {
            int64_t l = len;
            if (l < 0 || l > a.max_len) {
                flag_error(a.err, ERR_SEQ_LENGTH);
                l = l < 0 ? 0 : a.max_len;
            }
            a.length[slot] = (int32_t)l;
        }
        if (a.prioritized) {
            p_seen = p;
            const uint32_t q = quantise_leaf(p, a.tree.alpha_num, a.tree.alpha_den, a.tree.frac_bits);
            a.tree.leaves[slot] = q;
            delta = (uint64_t)q - (uint64_t)old;  // modulo 2^64
        }
    }
    if (!a.prioritized) return;
    const int lane = lane_id();
    if (a.src_prio) {
        const uint32_t m = wave_max_u32(p_seen);
        if (lane == 0 && m > 0) atomicMax(&a.state->max_prio, m);
    }
    // The wavefront's valid lanes hold consecutive slots slot0, slot0 + 1, ...
    // (lane 0 is valid whenever any lane is: segments start on wave boundaries),
    // so at level l the lanes [0, s) fall under node slot0 >> 6l and the rest
    // under the next node.  One inclusive scan of the deltas gives both sums.
    const uint64_t incl = wave_inclusive_scan_u64(delta);
    const uint64_t slot0 = (uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)slot);
    const uint64_t total = readlane_u64(incl, 63);
    for (int l = 1; l <= a.tree.depth; ++l) {
        const int shift = kFanoutLog2 * l;
        const uint64_t k0 = slot0 >> shift;
        const uint64_t span = ((k0 + 1) << shift) - slot0;  // lanes under node k0
        const uint64_t sa = span >= 64 ? total : readlane_u64(incl, (int)span - 1);
        const uint64_t sb = total - sa;
        if (lane == 0) {
            if (sa) atomicAdd(reinterpret_cast<unsigned long long*>(a.tree.level[l] + k0), sa);
            if (span < 64 && sb) atomicAdd(reinterpret_cast<unsigned long long*>(a.tree.level[l] + k0 + 1), sb);
        }
    }
}

// The metadata/tree workgroups come first in the grid: their chain of
// dependent memory operations (old leaf, quantiser, tree atomics) is the
// longest, so they start with the first wave of dispatched workgroups and
// overlap the payload copy.
template <typename V, bool RAGGED>
__global__ __launch_bounds__(kThreads) void k_ingest(IngestArgs a, int64_t meta_blocks) {
    const int64_t b = blockIdx.x;
    if (b < meta_blocks) {
        ingest_meta(a, b);
    } else {
        if constexpr (RAGGED) copy_ragged(a, b - meta_blocks);
        else copy_dense<V>(a, b - meta_blocks);
    }
}

}  // namespace

hipError_t launch_ingest(const IngestArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    const int64_t n1 = a.n < a.capacity - a.head ? a.n : a.capacity - a.head;
    const int64_t n2 = a.n - n1;
    const int64_t lanes = (n1 + kWave - 1) / kWave * kWave + (n2 + kWave - 1) / kWave * kWave;
    const int64_t meta_blocks = (lanes + kThreads - 1) / kThreads;
    if (a.length) {  // ragged
        const int64_t grid = a.n + meta_blocks;
        hipLaunchKernelGGL((k_ingest<uint32_t, true>), dim3((unsigned)grid), dim3(kThreads), 0, s, a, meta_blocks);
        return hipGetLastError();
    }
    const uintptr_t al = reinterpret_cast<uintptr_t>(a.src_obs) | reinterpret_cast<uintptr_t>(a.obs) |
                         (uintptr_t)a.row_bytes;
    int vec = (al & 15) == 0 ? 16 : (al & 7) == 0 ? 8 : (al & 3) == 0 ? 4 : 1;
    if (a.row_bytes == 0) vec = 16;
    const int64_t total_vec = a.n * (a.row_bytes / vec);
    const int64_t copy_blocks = (total_vec + kThreads * kCopyUnroll - 1) / (kThreads * kCopyUnroll);
    const dim3 grid((unsigned)(copy_blocks + meta_blocks));
    switch (vec) {
        case 16: hipLaunchKernelGGL((k_ingest<u32x4, false>), grid, dim3(kThreads), 0, s, a, meta_blocks); break;
        case 8: hipLaunchKernelGGL((k_ingest<u32x2, false>), grid, dim3(kThreads), 0, s, a, meta_blocks); break;
        case 4: hipLaunchKernelGGL((k_ingest<uint32_t, false>), grid, dim3(kThreads), 0, s, a, meta_blocks); break;
        default: hipLaunchKernelGGL((k_ingest<uint8_t, false>), grid, dim3(kThreads), 0, s, a, meta_blocks); break;
    }
    return hipGetLastError();
}

}  // namespace conduit
