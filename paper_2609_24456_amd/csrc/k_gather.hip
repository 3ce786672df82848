// Gather / transform: materialise the learner batch (off-policy delivery
// builds it from the drawn transitions and changes its layout, paper Sec. 2.2;
// concat/stack, reshape, batching and padding/packing are the processing
// operators it lists).  The same kernels
// serve the on-policy minibatch shuffle-gather (K = 1, rows of a rollout).
//
// Two shapes over the work items of gather_dev.h: four persistent workgroups
// per compute unit walking the items double-buffered (k_gather_pipe, outputs up
// to 128 MB), or one item per workgroup (k_gather_rows, larger outputs).
// Scalar columns (action, reward, done, extra float columns) are produced by
// workgroups at the head of the grid, one lane per output row, so that their
// dependent loads (index, then the columns) start with the first dispatched
// workgroups and finish under the frame traffic.  When the indices were just
// sampled, one more workgroup there computes the batch's importance weights
// (is_weights_block).
#include "gather_dev.h"

namespace conduit {

namespace {

// an index outside [0, limit): the row is zero-filled; err_kind < 0 (indices
// produced by the library, where -1 stands for "no row") raises no flag
__device__ __forceinline__ void flag_index(const GatherArgs& a) {
    if (a.err_kind >= 0) flag_error(a.err, a.err_kind);
}

// outputs up to this size use the persistent pipelined kernel
constexpr int64_t kPipeMaxOutBytes = 128ll << 20;

// Blocks [0, tail): scalar columns, then the weights block (if any).
__device__ __forceinline__ bool tail_block(const GatherArgs& a, int64_t tail) {
    const int64_t blk = blockIdx.x;
    if (blk >= tail) return false;
    if (a.weights.w && blk == tail - 1) is_weights_block<kThreads>(a.weights);
    else gather_scalars(a, blk);
    return true;
}

// One work item per workgroup, all of the grid's loads before its stores: the
// shape for large outputs, where many resident workgroups keep the most bytes
// in flight.

template <int XF>
__global__ __launch_bounds__(kThreads) void k_gather_rows(GatherArgs a, int32_t bpf, int32_t tail) {
    __shared__ uint16_t lut[(XF == CONDUIT_XF_U8_BF16_NORM) ? 4 * 256 : 1];
    if (tail_block(a, tail)) return;
    const int64_t it = (int64_t)blockIdx.x - tail;
    if constexpr (XF == CONDUIT_XF_U8_BF16_NORM) {
        build_lut(a, lut);
        __syncthreads();
    }
    const int64_t i = a.idx[it / ((int64_t)bpf * a.stack)];
    const Item t = decode(a, it, bpf, i);
    if (!t.ok && threadIdx.x == 0 && t.part == 0 && t.k == a.stack - 1) flag_index(a);
    typename UnitOf<XF>::T v[kUnroll];
    int32_t si = 0, sj = 0;
    uint32_t ei = 0, ej = 0;
    issue<XF>(a, t, i, v, si, sj, ei, ej, threadIdx.x);
    finish<XF, kStoreNT, true>(a, t, v, si, sj, ei, ej, lut, threadIdx.x);
}

// Persistent workgroups walk the items with a stride of the grid.  Two register
// sets alternate: the loads of the next item are issued before the stores of
// the current one, so reads of one item overlap the writes of the previous one
// instead of the whole GPU reading first and writing afterwards.  The sample
// index of the item after next is fetched one step ahead as well.
template <int XF>
__global__ __launch_bounds__(kThreads) void k_gather_pipe(GatherArgs a, int32_t bpf, int64_t n_items, int32_t frame_grid,
                                                          int32_t tail) {
    __shared__ uint16_t lut[(XF == CONDUIT_XF_U8_BF16_NORM) ? 4 * 256 : 1];
    if (tail_block(a, tail)) return;
    if constexpr (XF == CONDUIT_XF_U8_BF16_NORM) {
        build_lut(a, lut);
        __syncthreads();
    }
    const int64_t G = frame_grid;
    const int64_t per_row = (int64_t)bpf * a.stack;
    auto clampi = [&](int64_t x) { return x < n_items ? x : n_items - 1; };
    int64_t it = (int64_t)blockIdx.x - tail;
    const int64_t i0 = a.idx[it / per_row];
    int64_t itn = it + G;
    int64_t i1 = a.idx[clampi(itn) / per_row];
    typename UnitOf<XF>::T va[kUnroll], vb[kUnroll];
    int32_t sia = 0, sja = 0, sib = 0, sjb = 0;
    uint32_t eia = 0, eja = 0, eib = 0, ejb = 0;
    Item ta = decode(a, it, bpf, i0), tb;
    if (!ta.ok && threadIdx.x == 0 && ta.part == 0 && ta.k == a.stack - 1) flag_index(a);
    issue<XF>(a, ta, i0, va, sia, sja, eia, eja, threadIdx.x);
    while (true) {
        tb = decode(a, clampi(itn), bpf, i1);
        issue<XF>(a, tb, i1, vb, sib, sjb, eib, ejb, threadIdx.x);
        int64_t itnn = itn + G;
        int64_t i2 = a.idx[clampi(itnn) / per_row];
        finish<XF, kStoreWT, false>(a, ta, va, sia, sja, eia, eja, lut, threadIdx.x);
        if (itn >= n_items) break;
        if (!tb.ok && threadIdx.x == 0 && tb.part == 0 && tb.k == a.stack - 1) flag_index(a);
        itn = itnn;
        i1 = i2;
        ta = decode(a, clampi(itn), bpf, i1);
        issue<XF>(a, ta, i1, va, sia, sja, eia, eja, threadIdx.x);
        itnn = itn + G;
        i2 = a.idx[clampi(itnn) / per_row];
        finish<XF, kStoreWT, false>(a, tb, vb, sib, sjb, eib, ejb, lut, threadIdx.x);
        if (itn >= n_items) break;
        if (!ta.ok && threadIdx.x == 0 && ta.part == 0 && ta.k == a.stack - 1) flag_index(a);
        itn = itnn;
        i1 = i2;
    }
}

// ragged token packing: one workgroup per sample; each lane handles up to 4
// quads (16 elements) per pass, all loads issued before the stores
__global__ __launch_bounds__(kThreads) void k_pack(PackArgs a) {
    const int64_t b = blockIdx.x;
    if (b >= a.n) {  // the weights workgroup
        is_weights_block<kThreads>(a.weights);
        return;
    }
    pack_row<kThreads>(a, b, a.idx[b]);
}

}  // namespace

int device_cus() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cached[dev]) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
        cached[dev] = cus;
    }
    return cached[dev];
}

// Stores: the persistent kernel writes through at agent scope (outputs of at
// most 128 MB: no dirty L2 lines left for the end-of-kernel write-back; the
// DQN gather 15.2 -> 14.9 us), the one-item-per-workgroup kernel writes
// non-temporal (larger outputs stream: PPO minibatch 325 us against 342 us
// written through and 344 us with plain stores; large bf16 86 against 93 and
// 94 us).
template <int XF>
hipError_t launch_gather_xf(const GatherArgs& a, hipStream_t s, int64_t tail_blocks) {
    const int64_t units = a.row_bytes >> UnitOf<XF>::kShift;
    const int64_t bpf = a.out && units > 0 ? (units + kUnitsPerBlock - 1) / kUnitsPerBlock : 0;
    const int64_t n_items = a.n * a.stack * bpf;
    if (n_items + tail_blocks == 0) return hipSuccess;
    const int64_t out_bytes = a.n * a.stack * a.row_bytes *
                              (XF == CONDUIT_XF_U8_F32 ? 4 : XF == CONDUIT_XF_U8_BF16_NORM ? 2 : 1);
    if (out_bytes <= kPipeMaxOutBytes) {
        // small batches: persistent pipelined workgroups
        const int64_t frame_grid = n_items < 4LL * device_cus() ? n_items : 4LL * device_cus();
        hipLaunchKernelGGL((k_gather_pipe<XF>), dim3((unsigned)(frame_grid + tail_blocks)), dim3(kThreads), 0,
                           s, a, (int32_t)bpf, n_items, (int32_t)frame_grid, (int32_t)tail_blocks);
    } else {
        // large batches: one workgroup per item
        hipLaunchKernelGGL((k_gather_rows<XF>), dim3((unsigned)(n_items + tail_blocks)), dim3(kThreads), 0, s,
                           a, (int32_t)bpf, (int32_t)tail_blocks);
    }
    return hipGetLastError();
}

bool copy16(const GatherArgs& a) {
    return a.xform == CONDUIT_XF_NONE &&
           ((reinterpret_cast<uintptr_t>(a.src) | reinterpret_cast<uintptr_t>(a.out) | (uintptr_t)a.row_bytes) & 15) == 0;
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    const bool scalars = a.out_action || a.out_reward || a.out_done || a.ncols > 0;
    // scalar-column workgroups and the weights workgroup, at the head of the grid
    const int64_t tail_blocks = (scalars ? (a.n + kThreads - 1) / kThreads : 0) + (a.weights.w ? 1 : 0);
    if (copy16(a)) return launch_gather_xf<kXfCopy16>(a, s, tail_blocks);
    switch (a.xform) {
        case CONDUIT_XF_NONE: return launch_gather_xf<CONDUIT_XF_NONE>(a, s, tail_blocks);
        case CONDUIT_XF_U8_F32: return launch_gather_xf<CONDUIT_XF_U8_F32>(a, s, tail_blocks);
        case CONDUIT_XF_U8_BF16_NORM: return launch_gather_xf<CONDUIT_XF_U8_BF16_NORM>(a, s, tail_blocks);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_pack, dim3((unsigned)(a.n + (a.weights.w ? 1 : 0))), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
