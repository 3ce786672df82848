// Internal declarations shared by the HIP kernels and the host side of
// libconduit.  Not part of the public ABI (that is include/conduit.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "conduit.h"

namespace conduit {

constexpr int kWave = 64;         // CDNA wavefront width
constexpr int kFanout = 64;       // sum-tree fanout: one wavefront scans one node's children
constexpr int kFanoutLog2 = 6;
constexpr int kMaxLevels = 8;     // levels above the leaves; 64^6 > 2^31 slots

// Sticky device-side error kinds; each has its own word in pinned host memory,
// so concurrent reporters never need an atomic read-modify-write across PCIe.
enum ErrKind : int {
    ERR_UPDATE_INDEX = 0,   // priority update index outside [0, size)
    ERR_GATHER_INDEX = 1,   // gather index outside [0, size)
    ERR_EMPTY_TREE = 2,     // sample with a zero root
    ERR_SEQ_LENGTH = 3,     // ragged sequence longer than the slot / bad GAE length
    ERR_PERM_INDEX = 4,     // minibatch permutation entry outside [0, n_src)
    ERR_GAE_WAIT = 5,       // split GAE: a later segment never published (overlapping calls)
    ERR_DESCENT = 6,        // tree descent found no child (never expected)
    ERR_OFFSETS = 7,        // ragged ingest offsets decreasing or outside [0, src_elems]
    kErrKinds = 8,
};

// Small device-resident state of one buffer.
struct DeviceState {
    uint32_t max_prio;   // running maximum priority (starts at 1)
    uint32_t leaf_min;   // sampler scratch: smallest non-zero leaf of the buffer (buffer-wide IS
                         // normalisation), UINT32_MAX between calls
    uint32_t ticket;     // sampler scratch: finished blocks, 0 between calls
    uint32_t pad;
};

// The 64-ary sum tree.  Level 0 = uint32 leaves, levels 1..depth = uint64 sums;
// level l node n covers leaves [n*64^l, (n+1)*64^l).  Every level is padded with
// zeros to a multiple of 64 entries so a wavefront can always load 64 children.
struct TreeView {
    uint32_t* leaves;
    uint64_t* level[kMaxLevels + 1];  // level[1..depth]
    int64_t nodes[kMaxLevels + 1];    // nodes per level (unpadded), nodes[0] = capacity
    int32_t depth;
    int32_t alpha_num, alpha_den, frac_bits;
    // update kernel: levels with few nodes are accumulated in LDS first
    int32_t lds_offset[kMaxLevels + 1];  // -1: direct global atomics
};

__device__ __forceinline__ void flag_error(uint32_t* err, int kind) {
    // plain vector store of a non-zero word into pinned host memory
    __hip_atomic_store(err + kind, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// ---------------------------------------------------------------------------
// wavefront primitives (64 lanes)
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return __lane_id(); }

// DPP controls: shift right (lane i reads lane i - n) and left (lane i reads
// lane i + n) within a row of 16 lanes, and broadcast of lane 15 (31) of a row
// into the next row (rows 1 and 3; rows 2 and 3)
constexpr int kDppRowShr = 0x110, kDppRowShl = 0x100, kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

// x moved by one DPP control; lanes with no source, or in rows the row mask
// leaves out, read `id`
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x, uint32_t id) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)x, CTRL, ROWS, 0xf, false);
}

// Reduction of a 32-bit value over the whole wavefront (every lane active) with
// DPP moves instead of LDS permutes: after the row shifts and the two row
// broadcasts lane 63 holds the combination of all 64 lanes, returned to every
// lane.  `id` is the identity of `op`.
template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t x, uint32_t id, Op op) {
    x = op(x, dpp_u32<kDppRowShr + 1, 0xf>(x, id));
    x = op(x, dpp_u32<kDppRowShr + 2, 0xf>(x, id));
    x = op(x, dpp_u32<kDppRowShr + 4, 0xf>(x, id));
    x = op(x, dpp_u32<kDppRowShr + 8, 0xf>(x, id));
    x = op(x, dpp_u32<kDppRowBcast15, 0xa>(x, id));
    x = op(x, dpp_u32<kDppRowBcast31, 0xc>(x, id));
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
    return wave_reduce_u32(x, 0xffffffffu, [](uint32_t p, uint32_t q) { return q < p ? q : p; });
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    return wave_reduce_u32(x, 0u, [](uint32_t p, uint32_t q) { return q > p ? q : p; });
}

// value of a 64-bit register in a wave-uniform lane
__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// lanes of a 64-bit register moved by one DPP control (lanes with no source, or
// outside the row/bank masks, read 0)
template <int CTRL, int ROWS, int BANKS>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, ROWS, BANKS, true);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), CTRL, ROWS, BANKS, true);
    return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum across the wavefront with DPP moves (no LDS traffic):
// Hillis-Steele shifts by 1, 2, 4 and 8 lanes inside each row of 16, then the
// last lane of row 0 is broadcast into row 1 and of row 2 into row 3
// (row_bcast:15), and lane 31 into rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ uint64_t wave_inclusive_scan_u64(uint64_t x) {
    x += dpp_u64<kDppRowShr + 1, 0xf, 0xf>(x);
    x += dpp_u64<kDppRowShr + 2, 0xf, 0xf>(x);
    x += dpp_u64<kDppRowShr + 4, 0xf, 0xf>(x);
    x += dpp_u64<kDppRowShr + 8, 0xf, 0xf>(x);
    x += dpp_u64<kDppRowBcast15, 0xa, 0xf>(x);
    x += dpp_u64<kDppRowBcast31, 0xc, 0xf>(x);
    return x;
}

// ---------------------------------------------------------------------------
// exact leaf quantiser  L(p) = floor(2^F p^(a/b))
// ---------------------------------------------------------------------------
// q = L(p) is the unique integer with q^b <= 2^(bF) p^a < (q+1)^b.
//
// Fast path: x = exp2(F + (a/b) log2 p) in fp64.  With the device log2/exp2
// within a few ulp, the absolute error of x is below x * 2^-45 <= 2^-13 (x is
// below 2^32), so whenever the fractional part of x lies in [2^-12, 1 - 2^-12]
// floor(x) is the exact answer.  Otherwise x is within 2^-12 of an integer n
// (about 0.05% of inputs, and every perfect power), the true value lies in
// (n - 1, n + 1), and one exact 288-bit comparison settles it: L(p) = n if
// n^b <= 2^(bF) p^a, else n - 1 (b <= 8, so both sides fit 288 bits).  All limb
// indices are compile-time constants, so the big integers live in registers.
struct Big288 {
    uint32_t w[9];
};

__device__ __forceinline__ void big_one(Big288& x) {
#pragma unroll
    for (int i = 0; i < 9; ++i) x.w[i] = 0;
    x.w[0] = 1;
}

__device__ __forceinline__ void big_mul32(Big288& x, uint32_t m) {
    uint64_t carry = 0;
#pragma unroll
    for (int i = 0; i < 9; ++i) {
        const uint64_t t = (uint64_t)x.w[i] * m + carry;
        x.w[i] = (uint32_t)t;
        carry = t >> 32;
    }
}

// x <<= bits (bits < 256): a multiply by 2^(bits mod 32), then whole-word moves
__device__ __forceinline__ void big_shl(Big288& x, int bits) {
    big_mul32(x, 1u << (bits & 31));
    const int words = bits >> 5;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        if (s < words) {
#pragma unroll
            for (int i = 8; i > 0; --i) x.w[i] = x.w[i - 1];
            x.w[0] = 0;
        }
    }
}

// -1, 0, 1 as x <, ==, > y
__device__ __forceinline__ int big_cmp(const Big288& x, const Big288& y) {
    int r = 0;
#pragma unroll
    for (int i = 0; i < 9; ++i) {  // least significant first; higher words override
        if (x.w[i] != y.w[i]) r = x.w[i] < y.w[i] ? -1 : 1;
    }
    return r;
}

__device__ __forceinline__ void big_pow(Big288& x, uint32_t base, int e) {
    big_one(x);
    for (int i = 0; i < e; ++i) big_mul32(x, base);
}

// the settlement for x within 2^-12 of the integer n (1 <= n <= 2^32)
__device__ __noinline__ uint32_t quantise_leaf_exact(uint32_t p, int a, int b, int F, uint64_t n) {
    if (n > 0xffffffffull) return 0xffffffffu;  // L(p) < 2^32 <= n
    Big288 rhs, lhs;
    big_pow(rhs, p, a);
    big_shl(rhs, b * F);
    big_pow(lhs, (uint32_t)n, b);
    return big_cmp(lhs, rhs) <= 0 ? (uint32_t)n : (uint32_t)(n - 1);
}

__device__ __forceinline__ uint32_t quantise_leaf(uint32_t p, int a, int b, int F) {
    if (p == 0u) return 0u;
    if (a == 0) return 1u << F;
    if (a == b) return p;  // F = 0
    const double x = exp2((double)F + ((double)a / (double)b) * log2((double)p));
    const double fl = floor(x);
    const double fr = x - fl;
    if (fr >= 0x1p-12 && fr <= 1.0 - 0x1p-12) return fl >= 4294967295.0 ? 0xffffffffu : (uint32_t)fl;
    return quantise_leaf_exact(p, a, b, F, (uint64_t)fl + (fr > 0.5 ? 1u : 0u));
}

// ---------------------------------------------------------------------------
// importance-sampling weights of a sampled batch
// ---------------------------------------------------------------------------
// The sampler parks each sample's leaf q_k in the weight array; one whole
// workgroup of NT lanes then overwrites it in place with
// w_k = (q_min / q_k)^beta, q_min the smallest non-zero parked leaf, in fp64
// (0 where nothing was sampled).  Each lane rewrites only the entries it read.
struct WeightsArgs {
    float* w;        // parked leaves in, weights out; NULL: no weights
    int64_t batch;
    double beta;
    uint32_t* leaf_min = nullptr;  // non-NULL: normalise by this buffer-wide minimum leaf
                                   // (folded in by the sampler) and reset it afterwards
};

// COHERENT: the leaves were parked by other workgroups of the same launch with
// agent-scope atomic stores, and are read back with agent-scope atomic loads.
template <int NT, bool COHERENT = false>
__device__ void is_weights_block(const WeightsArgs& a) {
    __shared__ uint32_t wave_min[NT / kWave];
    __shared__ uint32_t qmin_s;
    uint32_t* q_park = reinterpret_cast<uint32_t*>(a.w);
    auto parked = [&](int64_t k) -> uint32_t {
        if constexpr (COHERENT) return __hip_atomic_load(q_park + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else return q_park[k];
    };
    if (a.leaf_min) {  // buffer-wide: the samplers' fold of every stored leaf
        if (threadIdx.x == 0) {
            if constexpr (COHERENT) qmin_s = __hip_atomic_load(a.leaf_min, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            else qmin_s = *a.leaf_min;
            __hip_atomic_store(a.leaf_min, 0xffffffffu, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    } else {  // the batch's smallest sampled leaf
        uint32_t m = 0xffffffffu;
        for (int64_t k = threadIdx.x; k < a.batch; k += NT) {
            const uint32_t q = parked(k);
            if (q) m = q < m ? q : m;
        }
        m = wave_min_u32(m);
        if (lane_id() == 0) wave_min[threadIdx.x / kWave] = m;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t r = wave_min[0];
            for (int i = 1; i < NT / kWave; ++i) r = wave_min[i] < r ? wave_min[i] : r;
            qmin_s = r;
        }
    }
    __syncthreads();
    const double qmin = (double)qmin_s;
    for (int64_t k = threadIdx.x; k < a.batch; k += NT) {  // the same k per lane as above
        const uint32_t q = parked(k);
        a.w[k] = q ? (float)pow(qmin / (double)q, a.beta) : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// kernel launch entry points (host functions defined next to each kernel)
// ---------------------------------------------------------------------------
struct IngestArgs {
    // destination ring
    uint8_t* obs;
    uint8_t* aux;
    uint8_t* action;
    float* reward;
    uint8_t* done;
    uint32_t* episode;
    int32_t* step;
    int32_t* length;
    int64_t capacity;
    int64_t row_bytes;
    int64_t max_len;         // ragged: elements per slot
    int32_t elem_bytes;      // ragged: 4
    int32_t aux_elem_bytes;  // ragged: 0 or 4
    int32_t action_bytes;
    int32_t prioritized;
    // source
    const uint8_t* src_obs;
    const int64_t* src_offsets;
    int64_t src_elems;       // ragged: elements the source obs (and aux) hold
    const uint8_t* src_aux;
    const uint8_t* src_action;
    const float* src_reward;
    const uint8_t* src_done;
    const uint32_t* src_episode;
    const int32_t* src_step;
    const uint32_t* src_prio;
    int64_t n;
    int64_t head;
    TreeView tree;
    DeviceState* state;
    int64_t total;           // stream position of row 0 (transitions ingested before)
    int32_t derive;          // kDeriveEpisode | kDeriveStep: columns the caller left NULL,
                             // derived from done and written into the ring before the ingest
    uint32_t* err;
};

constexpr int32_t kDeriveEpisode = 1, kDeriveStep = 2;
hipError_t launch_ingest(const IngestArgs& a, hipStream_t s);
// the derived episode / step columns of an ingest (a.derive != 0), written into
// the ring at the rows' slots; enqueue before the ingest itself
hipError_t launch_derive_meta(const IngestArgs& a, hipStream_t s);

struct UpdateArgs {
    TreeView tree;
    const int64_t* idx;
    const uint32_t* prio;
    int64_t n;
    int64_t size;
    DeviceState* state;
    uint32_t* err;
};

hipError_t launch_update(const UpdateArgs& a, hipStream_t s);
// every tree level recomputed from the leaves, level 1 first
hipError_t launch_tree_rebuild(const TreeView& t, hipStream_t s);
// the update, then a dense ingest, in one launch (k_update_ingest.hip)
hipError_t launch_update_ingest(const UpdateArgs& u, const IngestArgs& a, hipStream_t s);

struct SampleArgs {
    TreeView tree;
    const uint64_t* uniforms;
    int64_t* idx_out;
    float* w_out;
    int64_t batch;
    double beta;
    DeviceState* state;
    uint32_t* err;
    // buffer-wide IS normalisation: the sampler workgroups fold the smallest
    // non-zero leaf of leaves4[0, n_leaves4) (uint32 x 4) into *leaf_min
    uint32_t* leaf_min = nullptr;
    const uint32_t* leaves = nullptr;
    int64_t n_leaves4 = 0;
};

// The smallest non-zero leaf of workgroup wg's share of the buffer's leaves
// (wgs workgroups split them), folded into *a.leaf_min with one agent-scope
// atomic per workgroup.  Every thread of the workgroup takes part.
template <int NT>
__device__ void fold_leaf_min(const SampleArgs& a, int64_t wg, int64_t wgs) {
    __shared__ uint32_t wmin[NT / kWave];
    const int64_t per = (a.n_leaves4 + wgs - 1) / wgs;
    const int64_t lo = wg * per;
    const int64_t hi = lo + per < a.n_leaves4 ? lo + per : a.n_leaves4;
    const uint4* v = reinterpret_cast<const uint4*>(a.leaves);
    uint32_t m = 0xffffffffu;
    auto fold = [&](uint32_t q) { m = (q != 0u && q < m) ? q : m; };
    for (int64_t i = lo + threadIdx.x; i < hi; i += NT) {
        const uint4 q = v[i];
        fold(q.x);
        fold(q.y);
        fold(q.z);
        fold(q.w);
    }
    m = wave_min_u32(m);
    if (lane_id() == 0) wmin[threadIdx.x / kWave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = wmin[0];
        for (int i = 1; i < NT / kWave; ++i) r = wmin[i] < r ? wmin[i] : r;
        if (r != 0xffffffffu)
            (void)__hip_atomic_fetch_min(a.leaf_min, r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// sampler, then the weights kernel (if w_out is set)
hipError_t launch_sample(const SampleArgs& a, hipStream_t s);
// sampler only: leaves parked in w_out for a later weights block
hipError_t launch_descend(const SampleArgs& a, hipStream_t s);

constexpr int kMaxCols = 8;

struct GatherArgs {
    const int64_t* idx;     // sample indices (or a permutation)
    int64_t n;              // rows to produce
    int64_t limit;          // valid index range [0, limit)
    int32_t stack;          // K
    int64_t capacity;       // ring size for (i - d) mod capacity
    const uint8_t* src;     // [*, row_bytes]
    int64_t row_bytes;
    const uint32_t* episode;  // frame-stack metadata (NULL if stack == 1)
    const int32_t* step;
    void* out;
    int32_t xform;          // conduit_xform_kind
    int32_t plane_units;    // U8_BF16_NORM: 4-byte units per plane
    float mean[4];
    float stdv[4];
    // scalar columns taken from the newest slot
    const uint8_t* action;
    uint8_t* out_action;
    int32_t action_bytes;
    const float* reward;
    float* out_reward;
    const uint8_t* done;
    uint8_t* out_done;
    // extra float columns (minibatch gather)
    int32_t ncols;
    const float* cols[kMaxCols];
    float* cols_out[kMaxCols];
    uint32_t* err;
    int32_t err_kind;       // flag raised for an index outside [0, limit); < 0: none
    // the IS weights of the batch the indices were sampled as (one extra
    // workgroup of the launch); weights.w NULL: none
    WeightsArgs weights;
};

// record `msg` as the calling thread's last error and return `s`
conduit_status report_error(conduit_status s, const char* msg);

// what the host code outside api.hip needs to know of a buffer's layout
struct BufferGeometry {
    int64_t row_bytes;
    int32_t frame_stack;
    int32_t action_bytes;
    bool ragged;
    bool prioritized;
    int64_t capacity;
    int64_t head;              // next slot ingestion writes (host-known)
    const uint8_t* obs;        // device [capacity, row_bytes]
};
BufferGeometry buffer_geometry(const conduit_buffer* b);

// compute units of the current device (cached per device)
int device_cus();
// whether a gather moves its rows in 16-byte units (no transform, 16-byte
// aligned source, output and row size)
bool copy16(const GatherArgs& a);

hipError_t launch_gather(const GatherArgs& a, hipStream_t s);

// Fused sampler + gather for dense buffers with short rows (returns
// hipErrorNotSupported, launching nothing, for shapes it does not take): the
// sampler's arguments and the gather's, whose idx is the sampler's idx_out.
hipError_t launch_sample_gather(const SampleArgs& sa, const GatherArgs& ga, hipStream_t s);

struct PackArgs {
    const int64_t* idx;
    int64_t n;
    int64_t size;
    const uint8_t* seq;       // [capacity, max_len] 4-byte elements
    const uint8_t* aux;       // [capacity, max_len] 4-byte elements or NULL
    const int32_t* length;
    const float* reward;
    int64_t max_len;
    int32_t pad_id;
    void* out_seq;
    uint8_t* out_mask;
    void* out_aux;
    int32_t* out_length;
    float* out_reward;
    const uint8_t* action;
    uint8_t* out_action;
    int32_t action_bytes;
    const uint8_t* done;
    uint8_t* out_done;
    uint32_t* err;
    WeightsArgs weights;  // as for GatherArgs
};

hipError_t launch_pack(const PackArgs& a, hipStream_t s);

// time-major GAE addresses a slab of the rollout with 32-bit offsets
constexpr int64_t kGaeMaxEnvs = 1ll << 19;

struct GaeArgs {
    const float* reward;
    const float* value;
    const uint8_t* done;
    const float* bootstrap;
    int64_t T, E;
    double gamma, lambda;
    float* adv;
    float* ret;
    const uint8_t* truncated;   // NULL: no truncation bootstrap
    const float* final_value;   // read where truncated (and not done)
    uint32_t* err;              // sticky error words
};

hipError_t launch_gae(const GaeArgs& a, hipStream_t s);

// The allocation-free GAE call keeps its sticky error words in the current
// GPU's look-back table (k_gae.hip): their device address (set-up on first
// use), and a synchronous read / clear of them.
hipError_t gae_noalloc_err_words(uint32_t** err);
hipError_t gae_noalloc_read_errors(uint32_t* host_words);
hipError_t gae_noalloc_clear_errors();

// n-step return targets of sampled slots (k_nstep.hip)
struct NstepArgs {
    const int64_t* idx;
    int64_t batch;
    int32_t n;
    double gamma;
    int64_t capacity, size, total;  // ring state at enqueue time
    const float* reward;
    const uint8_t* done;
    const uint32_t* episode;
    int64_t* next_idx;
    float* ret;
    float* discount;
    uint8_t* valid;
    uint32_t* err;
};

hipError_t launch_nstep(const NstepArgs& a, hipStream_t s);
// the targets and the bootstrap stacks of rows of a few work items in one
// launch (ga.idx unused: each sample's slot comes from its window);
// hipErrorNotSupported for other shapes
hipError_t launch_nstep_gather(const NstepArgs& na, const GatherArgs& ga, hipStream_t s);
// sample + gather + n-step targets (+ the bootstrap stacks into next_out if not
// NULL) in one launch, for dense rows whose state and bootstrap stacks need at
// most 16 work items (na.idx unused: slots come from the descent);
// hipErrorNotSupported for other shapes
hipError_t launch_sample_gather_nstep(const SampleArgs& sa, const GatherArgs& ga, const NstepArgs& na,
                                      void* next_out, hipStream_t s);

struct GaePackedArgs {
    const float* last_reward;
    const int32_t* length;
    const float* value;
    int64_t B, Lmax;
    double gamma, lambda;
    float* adv;
    float* ret;
    uint32_t* err;
};

hipError_t launch_gae_packed(const GaePackedArgs& a, hipStream_t s);
// sample + pack in one launch (ragged buffers), and with ga the GAE of every
// packed row in the same launch; hipErrorNotSupported if the batch and the
// other arguments disagree
hipError_t launch_sample_pack(const SampleArgs& sa, const PackArgs& pa, const GaePackedArgs* ga, hipStream_t s);

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s);
hipError_t launch_fill_u64(uint64_t* p, uint64_t v, int64_t n, hipStream_t s);

}  // namespace conduit
