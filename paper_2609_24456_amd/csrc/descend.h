// Stratified inverse-CDF descent of the 64-ary integer sum tree by one
// wavefront (proportional prioritised replay, Schaul et al.; the paper's
// off-policy delivery draws from the replay store, Sec. 2.2).
// Shared by the sampler kernel and the fused sampler + gather.
#pragma once
#include "common.h"

namespace conduit {
namespace {

// Division by the batch size B as a multiply and shifts (Granlund and
// Montgomery, "Division by invariant integers using multiplication", PLDI 1994,
// Fig. 4.1): with l = ceil(log2 B) and m = floor(2^64 (2^l - B) / B) + 1,
// floor(n / B) = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0), t = mulhi(m, n),
// for every 64-bit n.  The host computes m and the shifts once per launch.
struct DivB {
    uint64_t m;
    int32_t sh1, sh2;
    uint64_t d;
};

inline DivB make_divb(uint64_t d) {
    int l = 0;
    while (l < 64 && (1ull << l) < d) ++l;  // ceil(log2 d), d <= 2^20
    const unsigned __int128 num = ((unsigned __int128)1 << 64) * (((unsigned __int128)1 << l) - d);
    DivB r;
    r.m = (uint64_t)(num / d) + 1;
    r.sh1 = l < 1 ? l : 1;
    r.sh2 = l - 1 > 0 ? l - 1 : 0;
    r.d = d;
    return r;
}

__device__ __forceinline__ uint64_t div_b(const DivB& v, uint64_t n) {
    const uint64_t t = __umul64hi(v.m, n);
    return (t + ((n - t) >> v.sh1)) >> v.sh2;
}

struct Descent {
    int64_t slot;   // sampled slot, -1 if the tree is empty
    uint32_t leaf;  // its quantised priority
    bool lost;      // no child exceeded the target (never expected)
};

// Stratum k of B: target t = floor((k*Q + floor(u*Q / 2^64)) / B), evaluated
// without 128-bit division by splitting Q and the high product word into
// quotient and remainder by B (every term fits 64 bits since k < B <= 2^20),
// each division a multiply-shift (DivB).
// At each level the 64 lanes load the 64 children of the current node, take an
// inclusive wavefront prefix sum, and the first lane whose prefix exceeds the
// target (ballot + find-first-set) names the child; its exclusive prefix is
// subtracted from the target.  This is "first slot whose inclusive prefix sum
// exceeds t" with half-open intervals, so zero leaves are never chosen.
//
// Latency is one memory round trip per level.  The total, the uniform and the
// root's children are independent loads and go out together.  With PRE > 0 the
// level below the root's children -- at most PRE groups of 64 entries, one
// group per child of the root -- is loaded in that same round trip and the
// descent selects the group in registers, saving one round trip (the launcher
// picks PRE from the tree's shape).  The tree's depth is a template parameter
// (the launcher dispatches on it): every level pointer is then read from the
// kernel arguments at a constant offset, all at kernel start, where a depth
// known only at run time made each level's pointer a dependent load in front
// of that level's nodes (about 0.5 us of a DQN batch's descent).  All lanes
// return the same result.
template <int PRE, int DEPTH>
__device__ __forceinline__ Descent tree_descend(const TreeView& tr, const uint64_t* uniforms, int64_t k, const DivB& dv) {
    static_assert(DEPTH >= 1 && DEPTH <= kMaxLevels, "tree depth");
    static_assert(PRE == 0 || DEPTH >= 2, "the prefetched level lies two below the root");
    constexpr int top = DEPTH;
    const int lane = lane_id();
    const uint64_t Q = tr.level[top][0];
    const uint64_t u = uniforms[k];
    uint64_t v = top == 1 ? (uint64_t)tr.leaves[lane] : tr.level[top - 1][lane];
    uint64_t pre[PRE > 0 ? PRE : 1];
    if constexpr (PRE > 0) {
        // 1 <= nodes[top - 1] <= PRE (launcher); groups past the last re-read
        // group 0 so that every load is unconditional
        const int groups = (int)tr.nodes[top - 1];
#pragma unroll
        for (int g = 0; g < PRE; ++g) {
            const int64_t c = (int64_t)(g < groups ? g : 0) * kFanout + lane;
            if constexpr (top == 2) pre[g] = (uint64_t)tr.leaves[c];
            else pre[g] = tr.level[top - 2][c];
        }
    }
    Descent r{-1, 0u, false};
    if (Q == 0ull) return r;
    const uint64_t h = __umul64hi(u, Q);
    const uint64_t kk = (uint64_t)k;
    const uint64_t qQ = div_b(dv, Q), rQ = Q - qQ * dv.d;
    const uint64_t qh = div_b(dv, h), rh = h - qh * dv.d;
    uint64_t t = kk * qQ + qh + div_b(dv, kk * rQ + rh);
    uint64_t node = 0;
#pragma unroll
    for (int l = top; l >= 1; --l) {
        if (l != top) {
            if (PRE > 0 && l == top - 1) {
                v = pre[0];
#pragma unroll
                for (int g = 1; g < (PRE > 0 ? PRE : 1); ++g) v = node == (uint64_t)g ? pre[g] : v;
            } else {
                const uint64_t child = node * kFanout + (uint64_t)lane;
                v = l == 1 ? (uint64_t)tr.leaves[child] : tr.level[l - 1][child];
            }
        }
        const uint64_t incl = wave_inclusive_scan_u64(v);
        const uint64_t mask = __ballot(incl > t);
        int sel = 63;
        if (mask) sel = __ffsll((unsigned long long)mask) - 1; else r.lost = true;
        t -= readlane_u64(incl - v, sel);  // exclusive prefix of the chosen child
        node = node * kFanout + (uint64_t)sel;
        if (l == 1) r.leaf = (uint32_t)readlane_u64(v, sel);
    }
    r.slot = (int64_t)node;
    return r;
}

// Depths a capacity of at most 2^31 - 1 slots gives a 64-ary tree.
constexpr int kMaxDescentDepth = 6;

// Calls f.template operator()<PRE, DEPTH>() for the tree's prefetch width and
// depth (compile-time values for tree_descend).
template <typename F>
hipError_t with_descent_shape(const TreeView& tr, int pre, F&& f) {
    switch (tr.depth) {
        case 1: return f.template operator()<0, 1>();
#define CONDUIT_DEPTH_CASE(D)                                        \
        case D:                                                      \
            if (pre == 4) return f.template operator()<4, D>();      \
            if (pre == 16) return f.template operator()<16, D>();    \
            return f.template operator()<0, D>();
        CONDUIT_DEPTH_CASE(2)
        CONDUIT_DEPTH_CASE(3)
        CONDUIT_DEPTH_CASE(4)
        CONDUIT_DEPTH_CASE(5)
        CONDUIT_DEPTH_CASE(6)
#undef CONDUIT_DEPTH_CASE
        default: return hipErrorInvalidValue;
    }
}

// The PRE of tree_descend for a tree: how many groups of the level under the
// root's children to fetch with them (0: none).
inline int descend_prefetch(const TreeView& tr) {
    const int64_t groups = tr.depth >= 2 ? tr.nodes[tr.depth - 1] : 0;
    return groups >= 1 && groups <= 4 ? 4 : groups >= 1 && groups <= 16 ? 16 : 0;
}

}  // namespace
}  // namespace conduit
