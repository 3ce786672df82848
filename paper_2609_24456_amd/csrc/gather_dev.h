// Device pieces of the gather / transform shared by the gather kernels and the
// fused sampler + gather: exact pixel transforms, the work-item decode, the
// load and store halves of an item, and the scalar-column lanes.
//
// A work item is (sample, frame, part) of up to 1792 units of 4 source bytes; a
// workgroup of 256 lanes moves 7 units per lane, 256 lanes apart, so each load
// instruction of a wavefront reads 256 contiguous bytes and each store writes a
// contiguous run (1 KiB for fp32 output).  Frame-stack validity needs the
// episode/step of two slots; those loads are unconditional and issued with the
// payload loads (which depend only on the sample index), so the metadata round
// trip overlaps the payload fetch.
//
// Transforms are exact:
//   U8_F32:  q0 = x * r (r = fp32(1/255)), e = fma(-q0, 255, x), fma(e, r, q0)
//            equals the correctly rounded x/255 for every x in 0..255 (checked
//            exhaustively against exact rational rounding);
//   U8_BF16_NORM: a per-workgroup LDS table of 256 entries per plane, each
//            computed with IEEE single division/subtraction and bf16
//            round-to-nearest-even.
#pragma once
#include "common.h"

namespace conduit {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 7;  // 1792 units per item: one 84x84 frame per item
constexpr int kUnitsPerBlock = kThreads * kUnroll;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Internal transform code (not part of the ABI): XF_NONE on rows whose size is
// a multiple of 16 bytes, moved in 16-byte units, so a wavefront's load or
// store covers 1 KiB instead of 256 bytes.
constexpr int kXfCopy16 = 16;

// the unit an item is made of: 4 bytes, or 16 for kXfCopy16
template <int XF> struct UnitOf {
    typedef uint32_t T;
    static constexpr int kShift = 2;
};
template <> struct UnitOf<kXfCopy16> {
    typedef u32x4 T;
    static constexpr int kShift = 4;
};

#pragma clang fp contract(off)
__device__ __forceinline__ float u8_unit_f32(uint32_t x) {
    const float r = 0x1.010102p-8f;  // nearest float to 1/255
    const float xf = (float)x;
    const float q0 = xf * r;
    const float e = __builtin_fmaf(-q0, 255.0f, xf);
    return __builtin_fmaf(e, r, q0);
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40u);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// One lane per output row.  Every load of the row (clamped to slot 0 when the
// index is out of range, so all are unconditional) is issued before the first
// store: one memory round trip after the index instead of one per column.
constexpr int kScalarWords = 8;  // action words held in registers per pass

__device__ inline void gather_scalars(const GatherArgs& a, int64_t block) {
    const int64_t b = block * kThreads + threadIdx.x;
    if (b >= a.n) return;
    const int64_t i = a.idx[b];
    const bool ok = i >= 0 && i < a.limit;
    const int64_t s = ok ? i : 0;
    const bool act = a.out_action && a.action_bytes > 0;
    const bool act_words = (a.action_bytes & 3) == 0;
    const int words = act && act_words ? a.action_bytes >> 2 : 0;
    uint32_t w[kScalarWords];
#pragma unroll
    for (int c = 0; c < kScalarWords; ++c)
        w[c] = c < words ? reinterpret_cast<const uint32_t*>(a.action + s * a.action_bytes)[c] : 0u;
    const float rew = a.out_reward ? a.reward[s] : 0.0f;
    const uint8_t dn = a.out_done ? a.done[s] : (uint8_t)0;
    float col[kMaxCols];
#pragma unroll
    for (int c = 0; c < kMaxCols; ++c) col[c] = c < a.ncols ? a.cols[c][s] : 0.0f;
    if (act) {
        uint8_t* dst = a.out_action + b * a.action_bytes;
        if (act_words) {
#pragma unroll
            for (int c = 0; c < kScalarWords; ++c)
                if (c < words) reinterpret_cast<uint32_t*>(dst)[c] = ok ? w[c] : 0u;
            for (int c = kScalarWords; c < words; ++c)  // long actions: the rest word by word
                reinterpret_cast<uint32_t*>(dst)[c] = ok ? reinterpret_cast<const uint32_t*>(a.action + s * a.action_bytes)[c] : 0u;
        } else {
            for (int c = 0; c < a.action_bytes; ++c) dst[c] = ok ? a.action[s * a.action_bytes + c] : (uint8_t)0;
        }
    }
    if (a.out_reward) a.out_reward[b] = ok ? rew : 0.0f;
    if (a.out_done) a.out_done[b] = ok ? dn : (uint8_t)0;
#pragma unroll
    for (int c = 0; c < kMaxCols; ++c)
        if (c < a.ncols) a.cols_out[c][b] = ok ? col[c] : 0.0f;
}

// per-workgroup table of the exact u8 -> bf16 normalisation, 256 entries per
// plane, built by lanes [first, first + count)
__device__ __forceinline__ void build_lut(const GatherArgs& a, uint16_t* lut, int first = 0, int count = kThreads) {
    const int planes = (int)((a.row_bytes >> 2) / a.plane_units);
    for (int e = (int)threadIdx.x - first; e < planes * 256; e += count) {
        const int c = e >> 8;
        const float v = u8_unit_f32((uint32_t)(e & 255));
        const float centred = v - a.mean[c];
        lut[e] = bf16_rne(__fdiv_rn(centred, a.stdv[c]));
    }
}

// One work item = (row b, frame k, part) = up to kUnitsPerBlock units of 4
// bytes (16 for kXfCopy16).
struct Item {
    int64_t b;   // output row
    int k;       // frame within the stack (0 = oldest)
    int part;    // chunk of the frame
    int d;       // frames back from the sampled slot
    int64_t j;   // source slot
    bool ok;     // sample index in range
};

__device__ __forceinline__ Item decode(const GatherArgs& a, int64_t it, int bpf, int64_t i) {
    Item t;
    const int64_t frame = it / bpf;
    t.part = (int)(it - frame * bpf);
    t.b = frame / a.stack;
    t.k = (int)(frame - t.b * a.stack);
    t.ok = i >= 0 && i < a.limit;
    t.d = a.stack - 1 - t.k;
    int64_t j = i - t.d;
    if (j < 0) j += a.capacity;
    t.j = t.ok ? j : 0;
    return t;
}

// issue every load of an item: payload units (clamped, so all are unconditional)
// and, for stacked frames, the episode/step of the sampled and the source slot
// NT: payload loads are non-temporal (they do not stay in the caches).  That
// pays in the fused sampler + gather (18.9 -> 18.6 us per DQN batch) and costs
// the persistent stand-alone gather a third of its speed (15.4 -> 21 us), whose
// double-buffered workgroups keep fewer loads in flight each.
template <int XF, bool NT = false>
__device__ __forceinline__ void issue(const GatherArgs& a, const Item& t, int64_t i,
                                      typename UnitOf<XF>::T (&v)[kUnroll], int32_t& si, int32_t& sj, uint32_t& ei,
                                      uint32_t& ej, int tid) {
    typedef typename UnitOf<XF>::T U;
    const int64_t units = a.row_bytes >> UnitOf<XF>::kShift;
    const U* __restrict__ src = reinterpret_cast<const U*>(a.src + t.j * a.row_bytes);
    const int64_t u0 = (int64_t)t.part * kUnitsPerBlock + tid;
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) {
        const int64_t u = u0 + (int64_t)r * kThreads;
        const int64_t uc = u < units ? u : units - 1;
        if constexpr (NT) v[r] = __builtin_nontemporal_load(src + uc);
        else v[r] = src[uc];
    }
    if (a.stack > 1) {  // kernel argument: uniform
        const int64_t ii = t.ok ? i : 0;
        si = a.step[ii];
        sj = a.step[t.j];
        ei = a.episode[ii];
        ej = a.episode[t.j];
    }
}

// Output stores of one item, by policy:
//   kStoreWT     buffer stores at agent scope (cache policy SC1), based at the
//                item's first output unit, so each store is written through to
//                the level every XCD sees rather than left dirty in the writing
//                XCD's L2 for the end-of-kernel write-back (the hardware also
//                drops any store past the item's last unit).  Measured on the
//                DQN batch (512 x 4 x 84x84 -> fp32, one launch with the
//                sampler): 17.1 us with non-temporal global stores, 15.2 us
//                with plain stores, 14.65 us write-through.
//   kStoreNT     non-temporal global stores;
//   kStorePlain  plain global stores.
enum StorePolicy : int { kStorePlain = 0, kStoreNT = 1, kStoreWT = 2 };
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor, 32-bit data format
constexpr int kStoreAgentScope = 16;    // SC1

__device__ __forceinline__ void put_unit(__amdgpu_buffer_rsrc_t rs, int off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b32(v, rs, off, 0, kStoreAgentScope);
}
__device__ __forceinline__ void put_unit(__amdgpu_buffer_rsrc_t rs, int off, u32x2 v) {
    __builtin_amdgcn_raw_buffer_store_b64(v, rs, off, 0, kStoreAgentScope);
}
__device__ __forceinline__ void put_unit(__amdgpu_buffer_rsrc_t rs, int off, u32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(v, rs, off, 0, kStoreAgentScope);
}
__device__ __forceinline__ void put_unit(__amdgpu_buffer_rsrc_t rs, int off, f32x4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rs, off, 0, kStoreAgentScope);
}

// A value every lane of the wavefront holds, as a scalar (read from the first
// lane): a buffer descriptor built from it needs no per-lane loop.
__device__ __forceinline__ int64_t wave_uniform(int64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// The units of part `part` of output frame `frame` (frames of `units` units
// each, counted from `out`).
template <int POL, typename O>
__device__ __forceinline__ void store_at(void* out, int64_t frame, int part, int64_t units, int tid,
                                         const O (&o)[kUnroll]) {
    // the item's place and size are the same for every lane (items belong to
    // whole wavefronts)
    const int64_t first = wave_uniform((int64_t)part * kUnitsPerBlock);  // its first unit within the frame
    const int64_t at = wave_uniform(frame * units + first);
    O* base = reinterpret_cast<O*>(out) + at;
    if constexpr (POL == kStoreWT) {
        const int n = (int)(units - first < kUnitsPerBlock ? units - first : kUnitsPerBlock);
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            base, 0, __builtin_amdgcn_readfirstlane(n * (int)sizeof(O)), kRsrcWord3);
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int e = tid + r * kThreads;
            if (e < n) put_unit(rs, e * (int)sizeof(O), o[r]);
        }
    } else {
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int e = tid + r * kThreads;
            if (first + e < units) {
                if constexpr (POL == kStoreNT) __builtin_nontemporal_store(o[r], base + e);
                else base[e] = o[r];
            }
        }
    }
}

template <int POL, typename O>
__device__ __forceinline__ void store_item(const GatherArgs& a, const Item& t, int64_t units, int tid,
                                           const O (&o)[kUnroll]) {
    store_at<POL>(a.out, t.b * a.stack + t.k, t.part, units, tid, o);
}

// The converted item (every conversion first, branch-free: an invalid frame is
// zeroed by a select), then its stores.  With PIN the empty asm statements keep
// the converted values in registers ahead of the first store; otherwise the
// compiler may sink each conversion into its store's range check, and the
// load waits it then places between stores also wait for the earlier stores
// (vmcnt counts both).  Measured on the DQN and PPO shapes: the
// one-item-per-workgroup kernel needs the pin (353 -> 328 us per PPO
// minibatch); the double-buffered kernels are faster without it (14.9 vs
// 15.3 us per DQN batch), where waiting per load lets stores start sooner.
template <int XF, int POL, bool PIN>
__device__ __forceinline__ void finish(const GatherArgs& a, const Item& t, const typename UnitOf<XF>::T (&v)[kUnroll],
                                       int32_t si, int32_t sj, uint32_t ei, uint32_t ej, const uint16_t* lut,
                                       int tid) {
    const int64_t units = a.row_bytes >> UnitOf<XF>::kShift;
    const bool valid = t.d == 0 ? t.ok : (t.ok & (t.d <= si) & (ei == ej) & (sj == si - t.d));
    const int64_t u0 = (int64_t)t.part * kUnitsPerBlock + tid;
    if constexpr (XF == kXfCopy16) {
        u32x4 o[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            o[r] = valid ? v[r] : (u32x4)(0u);
            if constexpr (PIN) asm volatile("" : "+v"(o[r]));
        }
        store_item<POL>(a, t, units, tid, o);
    } else if constexpr (XF == CONDUIT_XF_NONE) {
        uint32_t o[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            o[r] = valid ? v[r] : 0u;
            if constexpr (PIN) asm volatile("" : "+v"(o[r]));
        }
        store_item<POL>(a, t, units, tid, o);
    } else if constexpr (XF == CONDUIT_XF_U8_F32) {
        f32x4 o[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const uint32_t x = valid ? v[r] : 0u;  // 0 converts to +0.0
            o[r].x = u8_unit_f32(x & 255u);
            o[r].y = u8_unit_f32((x >> 8) & 255u);
            o[r].z = u8_unit_f32((x >> 16) & 255u);
            o[r].w = u8_unit_f32(x >> 24);
            if constexpr (PIN) asm volatile("" : "+v"(o[r]));
        }
        store_item<POL>(a, t, units, tid, o);
    } else {  // U8_BF16_NORM
        u32x2 o[kUnroll];
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int64_t u = u0 + (int64_t)r * kThreads;
            const uint32_t uu = (uint32_t)(u < units ? u : units - 1);  // keeps the plane index in range
            const uint16_t* tb = lut + (uu / (uint32_t)a.plane_units) * 256;
            const uint32_t x = v[r];
            const uint32_t lo = (uint32_t)tb[x & 255u] | ((uint32_t)tb[(x >> 8) & 255u] << 16);
            const uint32_t hi = (uint32_t)tb[(x >> 16) & 255u] | ((uint32_t)tb[x >> 24] << 16);
            o[r].x = valid ? lo : 0u;
            o[r].y = valid ? hi : 0u;
            if constexpr (PIN) asm volatile("" : "+v"(o[r]));
        }
        store_item<POL>(a, t, units, tid, o);
    }
}


// The row's scalar columns, one column word per lane (tid of a 256-lane
// group).  The value a lane carries is loaded with the row's frame loads and
// stored after the frames (row_scalars_load / row_scalars_store): a store
// placed between the two frames' loads would wait for the first frame's loads
// (vmcnt counts loads and stores in one queue) and delay the second frame's.
// A row of more than 254 action words or bytes has a second pass of lanes,
// loaded and stored together at the end.
struct RowScalar {
    uint32_t v;  // the lane's action word or byte, reward bits or done byte
    bool ok;     // the row's index is in range
};

__device__ __forceinline__ int row_scalar_lanes(const GatherArgs& a, bool* words) {
    *words = (a.action_bytes & 3) == 0;
    const int na = a.out_action && a.action_bytes > 0 ? (*words ? a.action_bytes >> 2 : a.action_bytes) : 0;
    return na + 2;  // action units, then reward, then done
}

// column unit t of row slot s (slot 0 when the index is out of range)
__device__ __forceinline__ uint32_t row_scalar_load(const GatherArgs& a, int64_t s, int t, int na, bool words) {
    if (t < na) {
        return words ? reinterpret_cast<const uint32_t*>(a.action + s * a.action_bytes)[t]
                     : (uint32_t)a.action[s * a.action_bytes + t];
    }
    if (t == na) return a.out_reward ? __float_as_uint(a.reward[s]) : 0u;
    return a.out_done ? (uint32_t)a.done[s] : 0u;
}

__device__ __forceinline__ void row_scalar_store(const GatherArgs& a, int64_t b, int t, int na, bool words,
                                                 uint32_t v) {
    if (t < na) {
        if (words) reinterpret_cast<uint32_t*>(a.out_action + b * a.action_bytes)[t] = v;
        else a.out_action[b * a.action_bytes + t] = (uint8_t)v;
    } else if (t == na) {
        if (a.out_reward) a.out_reward[b] = __uint_as_float(v);
    } else {
        if (a.out_done) a.out_done[b] = (uint8_t)v;
    }
}

__device__ __forceinline__ RowScalar row_scalars_load(const GatherArgs& a, int64_t i, int tid) {
    bool words;
    const int n = row_scalar_lanes(a, &words);
    const bool ok = i >= 0 && i < a.limit;
    RowScalar r{0u, ok};
    if (tid < n) r.v = row_scalar_load(a, ok ? i : 0, tid, n - 2, words);
    return r;
}

__device__ __forceinline__ void row_scalars_store(const GatherArgs& a, int64_t b, int64_t i, const RowScalar& r,
                                                  int tid) {
    bool words;
    const int n = row_scalar_lanes(a, &words);
    const int64_t s = r.ok ? i : 0;
    if (tid < n) row_scalar_store(a, b, tid, n - 2, words, r.ok ? r.v : 0u);
    for (int t = tid + kThreads; t < n; t += kThreads)  // rows of more than 256 units
        row_scalar_store(a, b, t, n - 2, words, r.ok ? row_scalar_load(a, s, t, n - 2, words) : 0u);
}

// rows of at most this many work items take the fused kernels (a sample's
// workgroup finds its slot itself and its two 256-lane halves share the items)
constexpr int64_t kFusedMaxItemsPerRow = 8;
// ... and with the n-step bootstrap stack, the union of the two stacks' frames
constexpr int64_t kFusedNstepMaxItemsPerRow = 16;

// The work items of row b (the slot i, or out of range for a zero row) that
// 256-lane group `part` of the row's `wgs` owns (tid: the lane in the group),
// two per group when the row has more than two, double-buffered: the next
// item's loads are issued before the current item's stores.  The row's first
// group also writes its scalar columns, after the frames.
template <int XF, bool NT_LOADS = false>
__device__ __forceinline__ void gather_row(const GatherArgs& a, int64_t b, int part, int64_t wgs, int32_t bpf,
                                           int64_t i, const uint16_t* lut, int tid) {
    const bool owner = part == 0;
    const int64_t per_row = (int64_t)bpf * a.stack;
    const int64_t per_wg = (per_row + wgs - 1) / wgs;
    const int64_t it0 = b * per_row + part * per_wg;
    int64_t it_end = it0 + per_wg;
    if (it_end > (b + 1) * per_row) it_end = (b + 1) * per_row;
    if (it0 >= it_end) {
        if (owner) row_scalars_store(a, b, i, row_scalars_load(a, i, tid), tid);
        return;
    }
    typename UnitOf<XF>::T va[kUnroll], vb[kUnroll];
    int32_t sia = 0, sja = 0, sib = 0, sjb = 0;
    uint32_t eia = 0, eja = 0, eib = 0, ejb = 0;
    Item ta = decode(a, it0, bpf, i), tb;
    issue<XF, NT_LOADS>(a, ta, i, va, sia, sja, eia, eja, tid);
    RowScalar rs{0u, false};
    if (owner) rs = row_scalars_load(a, i, tid);
    for (int64_t it = it0; it < it_end; it += 2) {
        const bool has_b = it + 1 < it_end;  // uniform
        if (has_b) {
            tb = decode(a, it + 1, bpf, i);
            issue<XF, NT_LOADS>(a, tb, i, vb, sib, sjb, eib, ejb, tid);
        }
        finish<XF, kStoreWT, false>(a, ta, va, sia, sja, eia, eja, lut, tid);
        if (!has_b) break;
        if (it + 2 < it_end) {
            ta = decode(a, it + 2, bpf, i);
            issue<XF, NT_LOADS>(a, ta, i, va, sia, sja, eia, eja, tid);
        }
        finish<XF, kStoreWT, false>(a, tb, vb, sib, sjb, eib, ejb, lut, tid);
    }
    if (owner) row_scalars_store(a, b, i, rs, tid);
}


// ---------------------------------------------------------------------------
// A sample's state stack and its n-step bootstrap stack from one read of each
// frame they need.  With the sample at stream position p (slot i) and the
// bootstrap state at p + n (slot jn), the state stack holds positions
// p - K + 1 .. p and the bootstrap stack p + n - K + 1 .. p + n; the first K
// positions and the S = min(n, K) newest of the bootstrap stack cover both:
// U = K + S frames, frame u at position p + off(u),
//   off(u) = u - (K - 1)              for u < K (state frame u),
//            n - S + 1 + (u - K)      for u >= K,
// bootstrap frame u - n (u < K) or u - S (u >= K) where that is >= 0.  Each
// frame is converted once and stored into each stack it belongs to, zero
// where its stack's episode/step check fails (as the gather checks it for
// that stack's own newest slot) and in every frame of a row without a
// bootstrap state.

// the converted units of an item, as stored
template <int XF> struct OutUnit { typedef uint32_t T; };
template <> struct OutUnit<kXfCopy16> { typedef u32x4 T; };
template <> struct OutUnit<CONDUIT_XF_U8_F32> { typedef f32x4 T; };
template <> struct OutUnit<CONDUIT_XF_U8_BF16_NORM> { typedef u32x2 T; };

template <int XF>
__device__ __forceinline__ void convert_units(const GatherArgs& a, int part, const typename UnitOf<XF>::T (&v)[kUnroll],
                                              const uint16_t* lut, int tid, typename OutUnit<XF>::T (&o)[kUnroll]) {
    if constexpr (XF == kXfCopy16 || XF == CONDUIT_XF_NONE) {
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) o[r] = v[r];
    } else if constexpr (XF == CONDUIT_XF_U8_F32) {
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const uint32_t x = v[r];
            o[r].x = u8_unit_f32(x & 255u);
            o[r].y = u8_unit_f32((x >> 8) & 255u);
            o[r].z = u8_unit_f32((x >> 16) & 255u);
            o[r].w = u8_unit_f32(x >> 24);
        }
    } else {  // U8_BF16_NORM
        const int64_t units = a.row_bytes >> 2;
        const int64_t u0 = (int64_t)part * kUnitsPerBlock + tid;
#pragma unroll
        for (int r = 0; r < kUnroll; ++r) {
            const int64_t u = u0 + (int64_t)r * kThreads;
            const uint32_t uu = (uint32_t)(u < units ? u : units - 1);  // keeps the plane index in range
            const uint16_t* tb = lut + (uu / (uint32_t)a.plane_units) * 256;
            const uint32_t x = v[r];
            o[r].x = (uint32_t)tb[x & 255u] | ((uint32_t)tb[(x >> 8) & 255u] << 16);
            o[r].y = (uint32_t)tb[(x >> 16) & 255u] | ((uint32_t)tb[x >> 24] << 16);
        }
    }
}

template <typename O>
__device__ __forceinline__ O zero_unit() {
    return O{};
}

// The row: its sample's slot and bootstrap slot with their episode/step.
struct UnionRow {
    int64_t b, i, jn;
    int K, n, S;
    bool ok;          // i in [0, limit)
    int32_t si, sn;   // step of slot i, of slot jn
    uint32_t ei, en;  // episode of slot i, of slot jn
};

// The row of slot i; its bootstrap slot, if any, is the one n positions on,
// (i + n) mod capacity, whose episode/step are loaded here already.  r.jn is
// -1 until the caller sets it (the n-step window decides whether that slot is
// the bootstrap state).
__device__ __forceinline__ UnionRow union_row(const GatherArgs& a, int64_t b, int64_t i, int n, bool with_next) {
    UnionRow r;
    r.b = b;
    r.i = i;
    r.jn = -1;
    r.K = a.stack;
    r.n = n;
    r.S = with_next ? (n < a.stack ? n : a.stack) : 0;
    r.ok = i >= 0 && i < a.limit;
    r.si = r.sn = 0;
    r.ei = r.en = 0;
    if (a.stack > 1) {  // kernel argument: uniform
        const int64_t ii = r.ok ? i : 0;
        const int64_t jc = r.ok ? (i + n) % a.capacity : 0;
        r.si = a.step[ii];
        r.ei = a.episode[ii];
        r.sn = a.step[jc];
        r.en = a.episode[jc];
    }
    return r;
}

struct UnionItem {
    int u, part;
    int64_t src;  // the slot read
};

__device__ __forceinline__ UnionItem union_item(const GatherArgs& a, const UnionRow& r, int64_t it, int32_t bpf) {
    UnionItem t;
    t.u = (int)(it / bpf);
    t.part = (int)(it - (int64_t)t.u * bpf);
    const int64_t off = t.u < r.K ? (int64_t)t.u - (r.K - 1) : (int64_t)(r.n - r.S + 1 + (t.u - r.K));
    int64_t j = 0;
    if (r.ok) {
        j = (r.i + off) % a.capacity;
        if (j < 0) j += a.capacity;
    }
    t.src = j;
    return t;
}

template <int XF>
__device__ __forceinline__ void union_issue(const GatherArgs& a, const UnionItem& t, typename UnitOf<XF>::T (&v)[kUnroll],
                                            int32_t& sj, uint32_t& ej, int tid) {
    typedef typename UnitOf<XF>::T U;
    const int64_t units = a.row_bytes >> UnitOf<XF>::kShift;
    const U* __restrict__ src = reinterpret_cast<const U*>(a.src + t.src * a.row_bytes);
    const int64_t u0 = (int64_t)t.part * kUnitsPerBlock + tid;
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) {
        const int64_t u = u0 + (int64_t)r * kThreads;
        v[r] = src[u < units ? u : units - 1];
    }
    if (a.stack > 1) {  // kernel argument: uniform
        sj = a.step[t.src];
        ej = a.episode[t.src];
    }
}

// convert once, store into the state stack and / or the bootstrap stack
template <int XF>
__device__ __forceinline__ void union_finish(const GatherArgs& a, const UnionRow& r, const UnionItem& t,
                                             const typename UnitOf<XF>::T (&v)[kUnroll], int32_t sj, uint32_t ej,
                                             void* next_out, const uint16_t* lut, int tid) {
    typedef typename OutUnit<XF>::T O;
    const int64_t units = a.row_bytes >> UnitOf<XF>::kShift;
    O o[kUnroll], z[kUnroll];
    convert_units<XF>(a, t.part, v, lut, tid, o);
    if (t.u < r.K) {  // uniform: frame u of the state stack
        const int d = r.K - 1 - t.u;
        const bool valid = d == 0 ? r.ok : (r.ok & (d <= r.si) & (r.ei == ej) & (sj == r.si - d));
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) z[k] = valid ? o[k] : zero_unit<O>();
        store_at<kStoreWT>(a.out, r.b * r.K + t.u, t.part, units, tid, z);
    }
    const int kn = t.u < r.K ? t.u - r.n : t.u - r.S;
    if (r.S > 0 && kn >= 0) {  // uniform: frame kn of the bootstrap stack
        const int d = r.K - 1 - kn;
        const bool valid = r.jn >= 0 && (d == 0 || ((d <= r.sn) & (r.en == ej) & (sj == r.sn - d)));
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) z[k] = valid ? o[k] : zero_unit<O>();
        store_at<kStoreWT>(next_out, r.b * r.K + kn, t.part, units, tid, z);
    }
}

// The union's work items that 256-lane group `part` of `parts` owns (tid: the
// lane in the group): items part, part + parts, ... (the frames stored twice,
// held by both stacks, spread over the groups), double-buffered as in
// gather_row.  start() issues the first item's loads, which need only the
// sample's slot; run() needs the bootstrap slot too (r.jn) and finishes the
// items.  The first group also writes the state row's scalar columns, after
// the frames.
template <int XF>
struct UnionGather {
    typename UnitOf<XF>::T va[kUnroll], vb[kUnroll];
    int32_t sja, sjb;
    uint32_t eja, ejb;
    UnionItem ta, tb;
    RowScalar rs;

    __device__ __forceinline__ void start(const GatherArgs& a, const UnionRow& r, int part, int32_t bpf, int tid) {
        const int64_t items = (int64_t)(r.K + r.S) * bpf;
        sja = sjb = 0;
        eja = ejb = 0;
        rs = RowScalar{0u, false};
        if (part == 0) rs = row_scalars_load(a, r.i, tid);
        if (part < items) {
            ta = union_item(a, r, part, bpf);
            union_issue<XF>(a, ta, va, sja, eja, tid);
        }
    }

    __device__ __forceinline__ void run(const GatherArgs& a, const UnionRow& r, int part, int parts, int32_t bpf,
                                        void* next_out, const uint16_t* lut, int tid) {
        const int64_t items = (int64_t)(r.K + r.S) * bpf;
        for (int64_t it = part; it < items; it += 2 * parts) {
            const bool has_b = it + parts < items;  // uniform
            if (has_b) {
                tb = union_item(a, r, it + parts, bpf);
                union_issue<XF>(a, tb, vb, sjb, ejb, tid);
            }
            union_finish<XF>(a, r, ta, va, sja, eja, next_out, lut, tid);
            if (!has_b) break;
            if (it + 2 * parts < items) {
                ta = union_item(a, r, it + 2 * parts, bpf);
                union_issue<XF>(a, ta, va, sja, eja, tid);
            }
            union_finish<XF>(a, r, tb, vb, sjb, ejb, next_out, lut, tid);
        }
        if (part == 0) row_scalars_store(a, r.b, r.i, rs, tid);
    }
};

// ---------------------------------------------------------------------------
// Ragged rows: row b of the padded batch from slot i (out of range: a zero row
// with an error flag), by one workgroup of kThreads lanes.
constexpr int kPackQuads = 4;

// what pack_row wrote for the row: its length and reward columns
struct PackedRow {
    int64_t L;
    float R;
};

template <int NT>
__device__ PackedRow pack_row(const PackArgs& a, int64_t b, int64_t i) {
    const bool ok = i >= 0 && i < a.size;
    if (!ok && threadIdx.x == 0) flag_error(a.err, ERR_GATHER_INDEX);
    // the row's scalar columns are loaded now, with its length, and stored last
    const int64_t si = ok ? i : 0;
    const float rew = a.out_reward ? a.reward[si] : 0.0f;
    const uint8_t dn = a.out_done ? a.done[si] : (uint8_t)0;
    const bool act = a.out_action && (int)threadIdx.x < a.action_bytes;
    const uint8_t ab = act ? a.action[si * a.action_bytes + threadIdx.x] : (uint8_t)0;
    int64_t L = ok ? a.length[i] : 0;
    if (L < 0) L = 0;
    if (L > a.max_len) L = a.max_len;
    const int32_t* __restrict__ seq = reinterpret_cast<const int32_t*>(a.seq) + (ok ? i : 0) * a.max_len;
    const float* __restrict__ aux = a.aux ? reinterpret_cast<const float*>(a.aux) + (ok ? i : 0) * a.max_len : nullptr;
    const int64_t quads = a.max_len >> 2;
    for (int64_t q0 = threadIdx.x; q0 < quads; q0 += NT * kPackQuads) {
        int4 tok[kPackQuads];
        f32x4 lp[kPackQuads];
        uint32_t m[kPackQuads];
#pragma unroll
        for (int r = 0; r < kPackQuads; ++r) {
            const int64_t q = q0 + (int64_t)r * NT;
            const int64_t t = q * 4;
            if (q < quads && t + 3 < L) {
                tok[r] = *reinterpret_cast<const int4*>(seq + t);
                lp[r] = aux ? *reinterpret_cast<const f32x4*>(aux + t) : (f32x4)(0.0f);
                m[r] = 0x01010101u;
            } else {
                tok[r].x = t + 0 < L ? seq[t + 0] : a.pad_id;
                tok[r].y = t + 1 < L ? seq[t + 1] : a.pad_id;
                tok[r].z = t + 2 < L ? seq[t + 2] : a.pad_id;
                tok[r].w = t + 3 < L ? seq[t + 3] : a.pad_id;
                lp[r].x = (aux && t + 0 < L) ? aux[t + 0] : 0.0f;
                lp[r].y = (aux && t + 1 < L) ? aux[t + 1] : 0.0f;
                lp[r].z = (aux && t + 2 < L) ? aux[t + 2] : 0.0f;
                lp[r].w = (aux && t + 3 < L) ? aux[t + 3] : 0.0f;
                m[r] = (t + 0 < L ? 0x1u : 0u) | (t + 1 < L ? 0x100u : 0u) | (t + 2 < L ? 0x10000u : 0u) |
                       (t + 3 < L ? 0x1000000u : 0u);
            }
        }
#pragma unroll
        for (int r = 0; r < kPackQuads; ++r) {
            const int64_t q = q0 + (int64_t)r * NT;
            if (q >= quads) continue;
            const int64_t o = b * a.max_len + q * 4;
            *reinterpret_cast<int4*>(reinterpret_cast<int32_t*>(a.out_seq) + o) = tok[r];
            if (a.out_aux) *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out_aux) + o) = lp[r];
            if (a.out_mask) *reinterpret_cast<uint32_t*>(a.out_mask + o) = m[r];
        }
    }
    if (threadIdx.x == 0) {
        if (a.out_length) a.out_length[b] = (int32_t)L;
        if (a.out_reward) a.out_reward[b] = ok ? rew : 0.0f;
        if (a.out_done) a.out_done[b] = ok ? dn : (uint8_t)0;
    }
    if (act) a.out_action[b * a.action_bytes + threadIdx.x] = ok ? ab : (uint8_t)0;
    if (a.out_action) {  // actions longer than one byte per lane
        for (int c = (int)threadIdx.x + NT; c < a.action_bytes; c += NT)
            a.out_action[b * a.action_bytes + c] = ok ? a.action[si * a.action_bytes + c] : (uint8_t)0;
    }
    return PackedRow{L, ok ? rew : 0.0f};
}

}  // namespace
}  // namespace conduit
