// Fused sampler + gather for dense buffers whose rows are a few work items
// (the frame-stack DQN shape), and fused sampler + token packing for ragged
// buffers (k_sample_pack, at the end): one launch delivers indices,
// importance weights and the learner batch (proportional prioritised replay,
// Schaul et al.; the paper's off-policy delivery samples and then materialises
// the batch, Sec. 2.2).
//
// Two kinds of 512-lane workgroup share the grid:
//   * gather workgroups (the head of the grid, one per sample): wavefront 0
//     runs tree_descend (descend.h) for the sample -- a few KB of tree reads
//     -- so the frame loads never wait for another workgroup or for the index
//     to make a round trip through memory; then the two 256-lane halves split
//     the row's work items (two each for a stack of four frames), and the
//     first half writes the scalar columns.
//   * sampler workgroups (the tail of the grid, eight samples each, one per
//     wavefront) run the same descent, write the indices and error flags, and
//     park each sampled leaf in the weight array.
// The DQN batch's 512 gather and 64 sampler workgroups are all resident at
// once (the kernel's registers allow seven wavefronts per SIMD).  One
// workgroup per sample rather than one per pair of frames halves the
// redundant descents and lets the whole row start as soon as its one descent
// ends (17.8 against 18.7 us per DQN batch).
//
// Importance weights need the smallest sampled leaf of the whole batch (or,
// normalised buffer-wide, of the whole buffer: then each sampler workgroup
// also folds the minimum of its share of the leaves into the device state
// with one agent-scope atomic).  Each sampler workgroup parks its leaves with
// agent-scope atomic stores, waits until they are acknowledged (visible
// device-wide), and takes a ticket with one agent-scope atomic add on the
// buffer's device state.  The workgroup that
// draws the last ticket reads every leaf back with agent-scope atomic loads,
// writes the weights (is_weights_block) and resets the ticket for the next
// call.  No workgroup waits for another, no release fence (which would write
// back the L2 under the frame stores) is needed, and the ticket latency stays
// off the frame workgroups.
#include "descend.h"
#include "gae_packed_dev.h"
#include "gather_dev.h"
#include "nstep_dev.h"

namespace conduit {

namespace {

constexpr int kWg = 2 * kThreads;  // two 256-lane halves
constexpr int kSamplesPerSamplerWg = kWg / kWave;

// A sampler workgroup of NT lanes: NT / 64 samples, one per wavefront.
template <int NT, int PRE, int DEPTH>
__device__ void sampler_wg(const SampleArgs& sa, const DivB& dv, int64_t wg) {
    constexpr int64_t kPer = NT / kWave;
    __shared__ uint32_t s_last;
    const int64_t k = wg * kPer + threadIdx.x / kWave;
    if (k < sa.batch) {  // wave-uniform
        const Descent d = tree_descend<PRE, DEPTH>(sa.tree, sa.uniforms, k, dv);
        if (lane_id() == 0) {
            sa.idx_out[k] = d.slot;
            if (d.slot < 0 && k == 0) flag_error(sa.err, ERR_EMPTY_TREE);
            if (d.lost) flag_error(sa.err, ERR_DESCENT);
            if (sa.w_out)
                __hip_atomic_store(reinterpret_cast<uint32_t*>(sa.w_out) + k, d.leaf, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (!sa.w_out) return;  // kernel argument: uniform
    // buffer-wide normalisation: this workgroup's share of the leaf minimum,
    // folded in before the ticket like the parked leaves
    if (sa.leaf_min) fold_leaf_min<NT>(sa, wg, (sa.batch + kPer - 1) / kPer);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);  // this wavefront's parked leaves are acknowledged
    __syncthreads();                // ... and every wavefront's
    if (threadIdx.x == 0) {
        const uint32_t tickets = (uint32_t)((sa.batch + kPer - 1) / kPer);
        const uint32_t t = __hip_atomic_fetch_add(&sa.state->ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = t == tickets - 1;
    }
    __syncthreads();
    if (s_last) {  // every leaf of the batch is parked and visible
        is_weights_block<NT, true>(WeightsArgs{sa.w_out, sa.batch, sa.beta, sa.leaf_min});
        if (threadIdx.x == 0) __hip_atomic_store(&sa.state->ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <int XF, int PRE, int DEPTH>
__global__ __launch_bounds__(kWg) void k_sample_gather(SampleArgs sa, GatherArgs a, DivB dv, int32_t bpf,
                                                       int32_t sampler_wgs) {
    __shared__ uint16_t lut[(XF == CONDUIT_XF_U8_BF16_NORM) ? 4 * 256 : 1];
    __shared__ int64_t s_slot;
    const int64_t gather_wgs = (int64_t)gridDim.x - sampler_wgs;
    if ((int64_t)blockIdx.x >= gather_wgs) {
        sampler_wg<kWg, PRE, DEPTH>(sa, dv, (int64_t)blockIdx.x - gather_wgs);
        return;
    }
    const int64_t b = blockIdx.x;
    if (threadIdx.x < kWave) {
        const Descent d = tree_descend<PRE, DEPTH>(sa.tree, sa.uniforms, b, dv);
        if (threadIdx.x == 0) s_slot = d.slot;
    } else if constexpr (XF == CONDUIT_XF_U8_BF16_NORM) {
        build_lut(a, lut, kWave, kWg - kWave);
    }
    __syncthreads();
    // half h of the workgroup takes the row's items as part h of 2 (uniform in
    // each wavefront: read from the first lane, so that the item's output base
    // stays a scalar)
    const int half = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kThreads));
    gather_row<XF, true>(a, b, half, 2, bpf, s_slot, lut, (int)(threadIdx.x % kThreads));
}

template <int XF>
struct FusedLaunch {
    const SampleArgs& sa;
    const GatherArgs& ga;
    DivB dv;
    int64_t bpf;
    hipStream_t s;
    template <int PRE, int DEPTH>
    hipError_t operator()() const {
        const int64_t sampler_wgs = (sa.batch + kSamplesPerSamplerWg - 1) / kSamplesPerSamplerWg;
        const dim3 grid((unsigned)(sampler_wgs + sa.batch)), block(kWg);
        hipLaunchKernelGGL((k_sample_gather<XF, PRE, DEPTH>), grid, block, 0, s, sa, ga, dv, (int32_t)bpf,
                           (int32_t)sampler_wgs);
        return hipGetLastError();
    }
};

template <int XF>
hipError_t launch_xf(const SampleArgs& sa, const GatherArgs& ga, hipStream_t s, int64_t bpf) {
    return with_descent_shape(sa.tree, descend_prefetch(sa.tree),
                              FusedLaunch<XF>{sa, ga, make_divb((uint64_t)sa.batch), bpf, s});
}

// The fused sampler + gather with n-step targets: each gather workgroup's
// first wavefront descends for its sample and issues the loads of the
// sample's n-step window from the slot it found; once every wavefront knows
// the slot, the two halves issue the loads of their first frames of the union
// of the state stack and the bootstrap stack (UnionGather) while the first
// wavefront evaluates the window (lane 0 writes the targets), and after a
// second barrier, with the bootstrap slot known, they convert and store every
// frame once into the stacks it belongs to.  Sampler workgroups as in
// k_sample_gather.
constexpr int kNstepWgsPerSample = 1;  // 512-lane workgroups per sample (2: 34.8 against 31.0 us per DQN batch, n = 3; past one residency round)

template <int XF, int PRE, int DEPTH>
__global__ __launch_bounds__(kWg) void k_sample_gather_nstep(SampleArgs sa, GatherArgs a, NstepArgs na,
                                                             void* next_out, DivB dv, int32_t bpf,
                                                             int32_t sampler_wgs) {
    __shared__ uint16_t lut[(XF == CONDUIT_XF_U8_BF16_NORM) ? 4 * 256 : 1];
    __shared__ int64_t s_slot, s_next;
    const int64_t gather_wgs = (int64_t)gridDim.x - sampler_wgs;
    if ((int64_t)blockIdx.x >= gather_wgs) {
        sampler_wg<kWg, PRE, DEPTH>(sa, dv, (int64_t)blockIdx.x - gather_wgs);
        return;
    }
    const int64_t b = blockIdx.x / kNstepWgsPerSample;
    const int sub = (int)(blockIdx.x % kNstepWgsPerSample);
    WindowLoads win;
    if (threadIdx.x < kWave) {
        const Descent d = tree_descend<PRE, DEPTH>(sa.tree, sa.uniforms, b, dv);
        const int64_t slot = __builtin_amdgcn_readfirstlane((uint32_t)d.slot) |
                             ((int64_t)__builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)d.slot >> 32)) << 32);
        win = nstep_window_load(na, slot);  // in flight across the barrier
        if (threadIdx.x == 0) s_slot = slot;
    } else if constexpr (XF == CONDUIT_XF_U8_BF16_NORM) {
        build_lut(a, lut, kWave, kWg - kWave);
    }
    __syncthreads();  // the slot is known
    UnionRow r = union_row(a, b, s_slot, na.n, next_out != nullptr);
    const int half = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kThreads));
    const int part = sub * 2 + half, tid = (int)(threadIdx.x % kThreads);
    UnionGather<XF> g;
    g.start(a, r, part, bpf, tid);  // the first frames' loads, while the window is evaluated
    if (threadIdx.x < kWave) {
        const int64_t next = nstep_window_finish(na, b, win, sub == 0);
        if (threadIdx.x == 0) s_next = next;
    }
    __syncthreads();  // the bootstrap slot is known
    r.jn = r.S > 0 ? s_next : -1;
    g.run(a, r, part, 2 * kNstepWgsPerSample, bpf, next_out, lut, tid);
}

template <int XF>
struct FusedNstepLaunch {
    const SampleArgs& sa;
    const GatherArgs& ga;
    const NstepArgs& na;
    void* next_out;
    DivB dv;
    int64_t bpf;
    hipStream_t s;
    template <int PRE, int DEPTH>
    hipError_t operator()() const {
        const int64_t sampler_wgs = (sa.batch + kSamplesPerSamplerWg - 1) / kSamplesPerSamplerWg;
        const dim3 grid((unsigned)(sampler_wgs + sa.batch * kNstepWgsPerSample)), block(kWg);
        hipLaunchKernelGGL((k_sample_gather_nstep<XF, PRE, DEPTH>), grid, block, 0, s, sa, ga, na, next_out, dv,
                           (int32_t)bpf, (int32_t)sampler_wgs);
        return hipGetLastError();
    }
};

template <int XF>
hipError_t launch_nstep_xf(const SampleArgs& sa, const GatherArgs& ga, const NstepArgs& na, void* next_out,
                           hipStream_t s, int64_t bpf) {
    return with_descent_shape(sa.tree, descend_prefetch(sa.tree),
                              FusedNstepLaunch<XF>{sa, ga, na, next_out, make_divb((uint64_t)sa.batch), bpf, s});
}

// Sampler + token packing in one launch (ragged buffers): one pack workgroup
// per sample at the head of the grid, whose first wavefront descends for the
// sample before the workgroup packs the row (pack_row), and sampler workgroups
// of the same width (one sample per wavefront) at the tail for the indices and
// the importance weights, as in k_sample_gather.
//
// With GAE, each pack workgroup then runs the GAE of its packed row from the
// length and reward it has just written (gae_packed_row), as
// conduit_gae_packed would over the packed batch.
//
// Widths, measured on [256, 4096] token batches: the pack alone takes 256
// lanes (7.4 us; 7.8-8.3 us with 512), the pack + GAE 512 lanes (10.3 us
// against 12.1 us with 256: the row's recursion is 8 steps per lane instead
// of 16).
template <bool GAE>
constexpr int pack_wg() { return GAE ? 512 : kThreads; }

template <int PRE, int DEPTH, bool GAE>
__global__ __launch_bounds__(pack_wg<GAE>()) void k_sample_pack(SampleArgs sa, PackArgs pa, GaePackedArgs ga,
                                                                DivB dv, int32_t sampler_wgs) {
    constexpr int NT = pack_wg<GAE>();
    __shared__ int64_t s_slot;
    const int64_t pack_wgs = (int64_t)gridDim.x - sampler_wgs;
    if ((int64_t)blockIdx.x >= pack_wgs) {
        sampler_wg<NT, PRE, DEPTH>(sa, dv, (int64_t)blockIdx.x - pack_wgs);
        return;
    }
    const int64_t b = blockIdx.x;
    if (threadIdx.x < kWave) {
        const Descent d = tree_descend<PRE, DEPTH>(sa.tree, sa.uniforms, b, dv);
        if (threadIdx.x == 0) s_slot = d.slot;
    }
    __syncthreads();
    const PackedRow row = pack_row<NT>(pa, b, s_slot);
    if constexpr (GAE) gae_packed_row<NT>(ga, b, row.L, (double)row.R);
}

struct PackLaunch {
    const SampleArgs& sa;
    const PackArgs& pa;
    const GaePackedArgs* ga;  // NULL: no GAE
    DivB dv;
    hipStream_t s;
    template <bool GAE, int PRE, int DEPTH>
    hipError_t launch() const {
        constexpr int NT = pack_wg<GAE>();
        const int64_t sampler_wgs = (sa.batch + NT / kWave - 1) / (NT / kWave);
        const dim3 grid((unsigned)(sampler_wgs + sa.batch)), block(NT);
        hipLaunchKernelGGL((k_sample_pack<PRE, DEPTH, GAE>), grid, block, 0, s, sa, pa, ga ? *ga : GaePackedArgs{},
                           dv, (int32_t)sampler_wgs);
        return hipGetLastError();
    }
    template <int PRE, int DEPTH>
    hipError_t operator()() const {
        return ga ? launch<true, PRE, DEPTH>() : launch<false, PRE, DEPTH>();
    }
};

}  // namespace

hipError_t launch_sample_gather(const SampleArgs& sa, const GatherArgs& ga, hipStream_t s) {
    const bool c16 = copy16(ga);
    const int64_t units = ga.row_bytes >> (c16 ? 4 : 2);
    const int64_t bpf = ga.out && units > 0 ? (units + kUnitsPerBlock - 1) / kUnitsPerBlock : 0;
    const int64_t per_row = bpf * ga.stack;
    if (sa.batch <= 0 || ga.ncols != 0 || per_row > kFusedMaxItemsPerRow) return hipErrorNotSupported;
    if (c16) return launch_xf<kXfCopy16>(sa, ga, s, bpf);
    switch (ga.xform) {
        case CONDUIT_XF_NONE: return launch_xf<CONDUIT_XF_NONE>(sa, ga, s, bpf);
        case CONDUIT_XF_U8_F32: return launch_xf<CONDUIT_XF_U8_F32>(sa, ga, s, bpf);
        case CONDUIT_XF_U8_BF16_NORM: return launch_xf<CONDUIT_XF_U8_BF16_NORM>(sa, ga, s, bpf);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_sample_gather_nstep(const SampleArgs& sa, const GatherArgs& ga, const NstepArgs& na,
                                      void* next_out, hipStream_t s) {
    const bool c16 = copy16(ga);
    const int64_t units = ga.row_bytes >> (c16 ? 4 : 2);
    const int64_t bpf = ga.out && units > 0 ? (units + kUnitsPerBlock - 1) / kUnitsPerBlock : 0;
    const int64_t frames = ga.stack + (next_out ? (na.n < ga.stack ? na.n : ga.stack) : 0);
    if (sa.batch <= 0 || na.batch != sa.batch || ga.ncols != 0 || bpf < 1 ||
        bpf * frames > kFusedNstepMaxItemsPerRow)
        return hipErrorNotSupported;
    if (c16) return launch_nstep_xf<kXfCopy16>(sa, ga, na, next_out, s, bpf);
    switch (ga.xform) {
        case CONDUIT_XF_NONE: return launch_nstep_xf<CONDUIT_XF_NONE>(sa, ga, na, next_out, s, bpf);
        case CONDUIT_XF_U8_F32: return launch_nstep_xf<CONDUIT_XF_U8_F32>(sa, ga, na, next_out, s, bpf);
        case CONDUIT_XF_U8_BF16_NORM: return launch_nstep_xf<CONDUIT_XF_U8_BF16_NORM>(sa, ga, na, next_out, s, bpf);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_sample_pack(const SampleArgs& sa, const PackArgs& pa, const GaePackedArgs* ga, hipStream_t s) {
    if (sa.batch <= 0 || pa.n != sa.batch || (ga && ga->B != sa.batch)) return hipErrorNotSupported;
    return with_descent_shape(sa.tree, descend_prefetch(sa.tree),
                              PackLaunch{sa, pa, ga, make_divb((uint64_t)sa.batch), s});
}

}  // namespace conduit
