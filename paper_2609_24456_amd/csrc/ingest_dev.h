// Ingest device code shared by the ingest kernel and the fused update + ingest
// kernel: the payload copies, the scalar columns and the per-wavefront tree
// deltas of new transitions.  Every function takes its lane's index within an
// ingest block of kIngestThreads lanes explicitly.
#pragma once
#include "common.h"

namespace conduit {

namespace {

constexpr int kIngestThreads = 256;  // threads of one ingest (sub-)block
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
__device__ void copy_dense(const IngestArgs& a, int64_t block, int tid) {
    const int64_t vec_per_row = a.row_bytes / (int64_t)sizeof(V);
    const int64_t total = a.n * vec_per_row;
    const int64_t ring = a.capacity * vec_per_row;
    const int64_t head_v = a.head * vec_per_row;
    const V* __restrict__ src = reinterpret_cast<const V*>(a.src_obs);
    V* __restrict__ dst = reinterpret_cast<V*>(a.obs);
    const int64_t base = block * (kIngestThreads * kCopyUnroll) + tid;
    // every load is unconditional (out-of-range lanes re-read the last vector) so
    // all kCopyUnroll loads of a lane are in flight at once.  Loads and stores
    // are non-temporal: a copy that streams through the caches moves 10% more
    // bytes per second here (347 MB: 6.4 against 5.8 TB/s)
    V v[kCopyUnroll];
#pragma unroll
    for (int r = 0; r < kCopyUnroll; ++r) {
        const int64_t i = base + (int64_t)r * kIngestThreads;
        v[r] = __builtin_nontemporal_load(src + (i < total ? i : total - 1));
    }
    // the empty asm statements keep every load ahead of the first store: the
    // compiler would otherwise sink loads into the stores' range checks and
    // wait between stores (vmcnt counts both)
#pragma unroll
    for (int r = 0; r < kCopyUnroll; ++r) pin(v[r]);
#pragma unroll
    for (int r = 0; r < kCopyUnroll; ++r) {
        const int64_t i = base + (int64_t)r * kIngestThreads;
        if (i < total) {
            int64_t d = head_v + i;
            if (d >= ring) d -= ring;
            __builtin_nontemporal_store(v[r], dst + d);
        }
    }
}

// Source span [*off, *off + *len) of ragged row j.  Offsets that decrease or
// leave [0, src_elems] give an empty span (ok = false: the metadata lane of the
// row flags it), so no element outside the source is ever read.
__device__ __forceinline__ bool ragged_span(const IngestArgs& a, int64_t j, int64_t* off, int64_t* len) {
    const int64_t b = a.src_offsets[j], e = a.src_offsets[j + 1];
    const bool ok = 0 <= b && b <= e && e <= a.src_elems;
    *off = ok ? b : 0;
    *len = ok ? e - b : 0;
    return ok;
}

__device__ inline void copy_ragged(const IngestArgs& a, int64_t j, int tid) {
    int64_t slot = a.head + j;
    if (slot >= a.capacity) slot -= a.capacity;
    int64_t off, len;
    ragged_span(a, j, &off, &len);
    if (len > a.max_len) len = a.max_len;  // flagged by the meta lane of row j
    if (len == 0) return;
    const uint32_t* __restrict__ s = reinterpret_cast<const uint32_t*>(a.src_obs) + off;
    uint32_t* __restrict__ d = reinterpret_cast<uint32_t*>(a.obs + slot * a.row_bytes);
    const bool aux = a.aux && a.src_aux;
    const uint32_t* __restrict__ sa = aux ? reinterpret_cast<const uint32_t*>(a.src_aux) + off : s;
    uint32_t* __restrict__ da = aux ? reinterpret_cast<uint32_t*>(a.aux) + slot * a.max_len : nullptr;
    // kRaggedUnroll elements per lane per pass, every load (clamped to the last
    // element) ahead of the stores
    for (int64_t t0 = tid; t0 < len; t0 += (int64_t)kIngestThreads * kRaggedUnroll) {
        uint32_t v[kRaggedUnroll], w[kRaggedUnroll];
#pragma unroll
        for (int r = 0; r < kRaggedUnroll; ++r) {
            const int64_t t = t0 + (int64_t)r * kIngestThreads;
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
            const int64_t t = t0 + (int64_t)r * kIngestThreads;
            if (t < len) {
                d[t] = v[r];
                if (aux) da[t] = w[r];
            }
        }
    }
}

// Rows of the ingest as lanes: rows [0, n1) go to slots head.., rows [n1, n)
// to slots 0..; each segment starts on a wavefront boundary, so a wavefront
// never straddles the ring's wrap point.
__device__ __forceinline__ int64_t ingest_lanes(const IngestArgs& a) {
    const int64_t n1 = a.n < a.capacity - a.head ? a.n : a.capacity - a.head;
    return (n1 + kWave - 1) / kWave * kWave + (a.n - n1 + kWave - 1) / kWave * kWave;
}

__device__ __forceinline__ void ingest_row(const IngestArgs& a, int64_t t, int64_t* j, int64_t* slot, bool* valid) {
    const int64_t n1 = a.n < a.capacity - a.head ? a.n : a.capacity - a.head;
    const int64_t lanes_a = (n1 + kWave - 1) / kWave * kWave;
    if (t < lanes_a) {
        *j = t;
        *slot = a.head + t;
        *valid = t < n1;
    } else {
        *j = n1 + (t - lanes_a);
        *slot = t - lanes_a;
        *valid = *j < a.n;
    }
}

// The wavefront's deltas for 64 consecutive slots (lane 0 holds slot0 when any
// lane is valid) pushed up the tree: at level l the lanes [0, s) fall under
// node slot0 >> 6l and the rest under the next node, so one inclusive scan
// gives both sums; lane 0 adds them (`add(level, node, value)`).
template <typename Add>
__device__ __forceinline__ void push_wave_deltas(const TreeView& tr, int64_t slot, uint64_t delta, Add&& add) {
    const uint64_t incl = wave_inclusive_scan_u64(delta);
    const uint64_t slot0 = (uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)slot);
    const uint64_t total = readlane_u64(incl, 63);
    for (int l = 1; l <= tr.depth; ++l) {
        const int shift = kFanoutLog2 * l;
        const uint64_t k0 = slot0 >> shift;
        const uint64_t span = ((k0 + 1) << shift) - slot0;  // lanes under node k0
        const uint64_t sa = span >= 64 ? total : readlane_u64(incl, (int)span - 1);
        const uint64_t sb = total - sa;
        if (lane_id() == 0) {
            if (sa) add(l, k0, sa);
            if (span < 64 && sb) add(l, k0 + 1, sb);
        }
    }
}

constexpr int kRaiseUnroll = 8;  // update entries per lane per pass, all loads in flight

// An update list whose priorities raise the running maximum (n = 0: none).
struct RaiseList {
    const int64_t* idx;
    const uint32_t* prio;
    int64_t n;
    int64_t size;  // valid indices are [0, size)
};

// max(stored running maximum, every valid priority of u) by one wavefront: the
// running maximum after the update list has been applied.  A list of up to 512
// entries is one memory round trip.
__device__ __forceinline__ uint32_t raised_max(const DeviceState* state, const RaiseList& u) {
    const uint32_t cur = state->max_prio;
    uint32_t m = 0;
    for (int64_t base = 0; base < u.n; base += (int64_t)kWave * kRaiseUnroll) {
        int64_t s[kRaiseUnroll];
        uint32_t p[kRaiseUnroll];
#pragma unroll
        for (int r = 0; r < kRaiseUnroll; ++r) {
            const int64_t k = base + (int64_t)r * kWave + lane_id();
            s[r] = k < u.n ? u.idx[k] : -1;
            p[r] = k < u.n ? u.prio[k] : 0u;
        }
#pragma unroll
        for (int r = 0; r < kRaiseUnroll; ++r)
            if (s[r] >= 0 && s[r] < u.size && p[r] > m) m = p[r];
    }
    m = wave_max_u32(m);
    return cur > m ? cur : m;
}

// The scalar columns, leaf and tree deltas of one lane's row.  Rows without a
// caller priority enter with the running maximum: the stored one, raised by the
// priorities of `raise` when it is not empty (an update applied in the same
// launch); those loads go out together with the row's own.
__device__ __forceinline__ void ingest_meta(const IngestArgs& a, int64_t block, int tid,
                                            const RaiseList raise = RaiseList{nullptr, nullptr, 0, 0}) {
    const int64_t t = block * kIngestThreads + tid;
    int64_t j, slot;
    bool valid;
    ingest_row(a, t, &j, &slot, &valid);
    const bool tree = a.prioritized;
    const uint64_t any_valid = __ballot(valid);
    if (any_valid == 0) return;  // whole wavefront past the end (wave-uniform)

    // every load of the lane's row is issued before its first store (lanes past
    // the end read row 0 and store nothing): one memory round trip in all.  The
    // old leaf is read unconditionally (slot 0 for lanes past the end) so that
    // no select of its value waits for it here.
    uint64_t delta = 0;
    uint32_t p_seen = 0;
    const int64_t jj = valid ? j : 0;
    const uint32_t old = tree ? a.tree.leaves[valid ? slot : 0] : 0u;
    const uint32_t p_row = tree && a.src_prio ? a.src_prio[jj] : 0u;
    const bool raised = raise.n > 0;
    const uint32_t p_state = tree && !a.src_prio && !raised ? a.state->max_prio : 0u;
    const float rew = a.src_reward ? a.src_reward[jj] : 0.0f;
    const uint8_t dn = a.src_done ? a.src_done[jj] : (uint8_t)0;
    const uint32_t ep = a.src_episode ? a.src_episode[jj] : 0u;
    const int32_t st = a.src_step ? a.src_step[jj] : 0;
    int64_t len = 0, off_unused;
    const bool span_ok = a.length ? ragged_span(a, jj, &off_unused, &len) : true;
    const bool act_words = a.src_action && (a.action_bytes & 3) == 0;
    const int words = act_words ? a.action_bytes >> 2 : 0;
    uint32_t w[kActWords];
#pragma unroll
    for (int c = 0; c < kActWords; ++c)
        w[c] = c < words ? reinterpret_cast<const uint32_t*>(a.src_action + jj * a.action_bytes)[c] : 0u;
    const uint32_t p = !tree ? 0u : a.src_prio ? p_row : raised ? raised_max(a.state, raise) : p_state;
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
        if (!(a.derive & kDeriveEpisode)) a.episode[slot] = ep;  // else written by the derive pass
        if (!(a.derive & kDeriveStep)) a.step[slot] = st;
        if (a.length) {
            int64_t l = len;
            if (!span_ok) flag_error(a.err, ERR_OFFSETS);
            if (l > a.max_len) {
                flag_error(a.err, ERR_SEQ_LENGTH);
                l = a.max_len;
            }
            a.length[slot] = (int32_t)l;
        }
        if (tree) {
            p_seen = p;
            const uint32_t q = quantise_leaf(p, a.tree.alpha_num, a.tree.alpha_den, a.tree.frac_bits);
            a.tree.leaves[slot] = q;
            delta = (uint64_t)q - (uint64_t)old;  // modulo 2^64
        }
    }
    if (!tree) return;
    if (a.src_prio) {
        const uint32_t m = wave_max_u32(p_seen);
        if (lane_id() == 0 && m > 0) atomicMax(&a.state->max_prio, m);
    }
    push_wave_deltas(a.tree, slot, delta, [&](int l, uint64_t node, uint64_t v) {
        atomicAdd(reinterpret_cast<unsigned long long*>(a.tree.level[l] + node), v);
    });
}

}  // namespace
}  // namespace conduit
