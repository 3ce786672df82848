// Gather / transform: materialise the learner batch (off-policy delivery
// "materializes the selected transitions, and performs batch/layout
// transformations", paper Sec. 2.2; concat/stack, reshape, batching and
// padding/packing are the processing operators it lists).  The same kernel
// serves the on-policy minibatch shuffle-gather (K = 1, rows of a rollout).
//
// Work decomposition: a work item is (sample, frame, part) of up to 1792 units
// of 4 source bytes; a workgroup of 256 lanes moves 7 units per lane, 256 lanes
// apart, so each load instruction of a wavefront reads 256 contiguous bytes and
// each store writes a contiguous run (1 KiB for fp32 output).  Four persistent
// workgroups per compute unit walk the items, double-buffered (see k_gather).
// Frame-stack validity needs the episode/step of two slots; those loads are
// unconditional and issued with the payload loads (which depend only on the
// sample index), so the metadata round trip overlaps the payload fetch.
//
// Transforms are exact:
//   U8_F32:  q0 = x * r (r = fp32(1/255)), e = fma(-q0, 255, x), fma(e, r, q0)
//            equals the correctly rounded x/255 for every x in 0..255 (checked
//            exhaustively against exact rational rounding);
//   U8_BF16_NORM: a per-workgroup LDS table of 256 entries per plane, each
//            computed with IEEE single division/subtraction and bf16
//            round-to-nearest-even.
// Scalar columns (action, reward, done, extra float columns) are produced by
// workgroups at the head of the grid, one lane per output row, so that their
// dependent loads (index, then the columns) start with the first dispatched
// workgroups and finish under the frame traffic.  When the indices were just
// sampled, one more workgroup there computes the batch's importance weights
// (is_weights_block), so sampling and delivery take two launches in all.
#include "common.h"

namespace conduit {

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 7;  // 1792 units per item: one 84x84 frame per item
constexpr int kUnitsPerBlock = kThreads * kUnroll;
// outputs up to this size use the persistent pipelined kernel
constexpr int64_t kPipeMaxOutBytes = 128ll << 20;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

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

__device__ void gather_scalars(const GatherArgs& a, int64_t block) {
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

// One work item = (row b, frame k, part) = up to kUnitsPerBlock 4-byte units.
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
__device__ __forceinline__ void issue(const GatherArgs& a, const Item& t, int64_t i, uint32_t (&v)[kUnroll],
                                      int32_t& si, int32_t& sj, uint32_t& ei, uint32_t& ej) {
    const int64_t units = a.row_bytes >> 2;
    const uint32_t* __restrict__ src = reinterpret_cast<const uint32_t*>(a.src + t.j * a.row_bytes);
    const int64_t u0 = (int64_t)t.part * kUnitsPerBlock + threadIdx.x;
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) {
        const int64_t u = u0 + (int64_t)r * kThreads;
        v[r] = src[u < units ? u : units - 1];
    }
    if (a.stack > 1) {  // kernel argument: uniform
        const int64_t ii = t.ok ? i : 0;
        si = a.step[ii];
        sj = a.step[t.j];
        ei = a.episode[ii];
        ej = a.episode[t.j];
    }
}

template <int XF, bool NT>
__device__ __forceinline__ void finish(const GatherArgs& a, const Item& t, const uint32_t (&v)[kUnroll], int32_t si,
                                       int32_t sj, uint32_t ei, uint32_t ej, const uint16_t* lut) {
    const int64_t units = a.row_bytes >> 2;
    const bool valid = t.d == 0 ? t.ok : (t.ok & (t.d <= si) & (ei == ej) & (sj == si - t.d));
    const int64_t u0 = (int64_t)t.part * kUnitsPerBlock + threadIdx.x;
    const int64_t out_unit0 = (t.b * a.stack + t.k) * units;
#pragma unroll
    for (int r = 0; r < kUnroll; ++r) {
        const int64_t u = u0 + (int64_t)r * kThreads;
        if (u >= units) continue;
        const uint32_t x = v[r];
        if constexpr (XF == CONDUIT_XF_NONE) {
            uint32_t* p = reinterpret_cast<uint32_t*>(a.out) + out_unit0 + u;
            if constexpr (NT) __builtin_nontemporal_store(valid ? x : 0u, p); else *p = valid ? x : 0u;
        } else if constexpr (XF == CONDUIT_XF_U8_F32) {
            f32x4 o;
            if (valid) {
                o.x = u8_unit_f32(x & 255u);
                o.y = u8_unit_f32((x >> 8) & 255u);
                o.z = u8_unit_f32((x >> 16) & 255u);
                o.w = u8_unit_f32(x >> 24);
            } else {
                o = (f32x4)(0.0f);
            }
            f32x4* p = reinterpret_cast<f32x4*>(a.out) + out_unit0 + u;
            if constexpr (NT) __builtin_nontemporal_store(o, p); else *p = o;
        } else {  // U8_BF16_NORM
            u32x2 o;
            if (valid) {
                const int c = (int)(u / a.plane_units);
                const uint16_t* tb = lut + c * 256;
                o.x = (uint32_t)tb[x & 255u] | ((uint32_t)tb[(x >> 8) & 255u] << 16);
                o.y = (uint32_t)tb[(x >> 16) & 255u] | ((uint32_t)tb[x >> 24] << 16);
            } else {
                o = (u32x2)(0u);
            }
            u32x2* p = reinterpret_cast<u32x2*>(a.out) + out_unit0 + u;
            if constexpr (NT) __builtin_nontemporal_store(o, p); else *p = o;
        }
    }
}

// One work item per workgroup, all of the grid's loads before its stores: the
// shape for large outputs, where many resident workgroups keep the most bytes
// in flight.
// Blocks [0, tail): scalar columns, then the weights block (if any).
__device__ __forceinline__ bool tail_block(const GatherArgs& a, int64_t tail) {
    const int64_t blk = blockIdx.x;
    if (blk >= tail) return false;
    if (a.weights.w && blk == tail - 1) is_weights_block<kThreads>(a.weights);
    else gather_scalars(a, blk);
    return true;
}

template <int XF, bool NT>
__global__ __launch_bounds__(kThreads) void k_gather_rows(GatherArgs a, int32_t bpf, int64_t n_items, int32_t tail) {
    __shared__ uint16_t lut[(XF == CONDUIT_XF_U8_BF16_NORM) ? 4 * 256 : 1];
    if (tail_block(a, tail)) return;
    const int64_t it = (int64_t)blockIdx.x - tail;
    if constexpr (XF == CONDUIT_XF_U8_BF16_NORM) {
        build_lut(a, lut);
        __syncthreads();
    }
    const int64_t i = a.idx[it / ((int64_t)bpf * a.stack)];
    const Item t = decode(a, it, bpf, i);
    if (!t.ok && threadIdx.x == 0 && t.part == 0 && t.k == a.stack - 1) flag_error(a.err, a.err_kind);
    uint32_t v[kUnroll];
    int32_t si = 0, sj = 0;
    uint32_t ei = 0, ej = 0;
    issue(a, t, i, v, si, sj, ei, ej);
    finish<XF, NT>(a, t, v, si, sj, ei, ej, lut);
}

// Persistent workgroups walk the items with a stride of the grid.  Two register
// sets alternate: the loads of the next item are issued before the stores of
// the current one, so reads of one item overlap the writes of the previous one
// instead of the whole GPU reading first and writing afterwards.  The sample
// index of the item after next is fetched one step ahead as well.
template <int XF, bool NT>
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
    uint32_t va[kUnroll], vb[kUnroll];
    int32_t sia = 0, sja = 0, sib = 0, sjb = 0;
    uint32_t eia = 0, eja = 0, eib = 0, ejb = 0;
    Item ta = decode(a, it, bpf, i0), tb;
    if (!ta.ok && threadIdx.x == 0 && ta.part == 0 && ta.k == a.stack - 1) flag_error(a.err, a.err_kind);
    issue(a, ta, i0, va, sia, sja, eia, eja);
    while (true) {
        tb = decode(a, clampi(itn), bpf, i1);
        issue(a, tb, i1, vb, sib, sjb, eib, ejb);
        int64_t itnn = itn + G;
        int64_t i2 = a.idx[clampi(itnn) / per_row];
        finish<XF, NT>(a, ta, va, sia, sja, eia, eja, lut);
        if (itn >= n_items) break;
        if (!tb.ok && threadIdx.x == 0 && tb.part == 0 && tb.k == a.stack - 1) flag_error(a.err, a.err_kind);
        itn = itnn;
        i1 = i2;
        ta = decode(a, clampi(itn), bpf, i1);
        issue(a, ta, i1, va, sia, sja, eia, eja);
        itnn = itn + G;
        i2 = a.idx[clampi(itnn) / per_row];
        finish<XF, NT>(a, tb, vb, sib, sjb, eib, ejb, lut);
        if (itn >= n_items) break;
        if (!ta.ok && threadIdx.x == 0 && ta.part == 0 && ta.k == a.stack - 1) flag_error(a.err, a.err_kind);
        itn = itnn;
        i1 = i2;
    }
}

// ragged token packing: one workgroup per sample; each lane handles up to 4
// quads (16 elements) per pass, all loads issued before the stores
constexpr int kPackQuads = 4;

__global__ __launch_bounds__(kThreads) void k_pack(PackArgs a) {
    const int64_t b = blockIdx.x;
    if (b >= a.n) {  // the weights workgroup
        is_weights_block<kThreads>(a.weights);
        return;
    }
    const int64_t i = a.idx[b];
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
    for (int64_t q0 = threadIdx.x; q0 < quads; q0 += kThreads * kPackQuads) {
        int4 tok[kPackQuads];
        f32x4 lp[kPackQuads];
        uint32_t m[kPackQuads];
#pragma unroll
        for (int r = 0; r < kPackQuads; ++r) {
            const int64_t q = q0 + (int64_t)r * kThreads;
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
            const int64_t q = q0 + (int64_t)r * kThreads;
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
        for (int c = (int)threadIdx.x + kThreads; c < a.action_bytes; c += kThreads)
            a.out_action[b * a.action_bytes + c] = ok ? a.action[si * a.action_bytes + c] : (uint8_t)0;
    }
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

// Both shapes write the learner batch with non-temporal stores: measured in the
// full ingest/sample/gather/update loop they leave the caches to the next
// kernels and beat plain stores, even when the batch would fit the 256 MB
// Infinity Cache.
template <int XF>
void launch_gather_xf(const GatherArgs& a, hipStream_t s, int64_t bpf, int64_t n_items, int64_t tail_blocks) {
    const int64_t out_bytes = n_items * kUnitsPerBlock * 4 * (XF == CONDUIT_XF_U8_F32 ? 4 : XF == CONDUIT_XF_U8_BF16_NORM ? 2 : 1);
    if (out_bytes <= kPipeMaxOutBytes) {
        // small batches: persistent pipelined workgroups
        const int64_t frame_grid = n_items < 4LL * device_cus() ? n_items : 4LL * device_cus();
        hipLaunchKernelGGL((k_gather_pipe<XF, true>), dim3((unsigned)(frame_grid + tail_blocks)), dim3(kThreads), 0,
                           s, a, (int32_t)bpf, n_items, (int32_t)frame_grid, (int32_t)tail_blocks);
    } else {
        // large batches: one workgroup per item
        hipLaunchKernelGGL((k_gather_rows<XF, true>), dim3((unsigned)(n_items + tail_blocks)), dim3(kThreads), 0, s,
                           a, (int32_t)bpf, n_items, (int32_t)tail_blocks);
    }
}

hipError_t launch_gather(const GatherArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    const int64_t units = a.row_bytes >> 2;
    const int64_t bpf = a.out && units > 0 ? (units + kUnitsPerBlock - 1) / kUnitsPerBlock : 0;
    const int64_t n_items = a.n * a.stack * bpf;
    const bool scalars = a.out_action || a.out_reward || a.out_done || a.ncols > 0;
    // scalar-column workgroups and the weights workgroup, at the head of the grid
    const int64_t tail_blocks = (scalars ? (a.n + kThreads - 1) / kThreads : 0) + (a.weights.w ? 1 : 0);
    if (n_items + tail_blocks == 0) return hipSuccess;
    switch (a.xform) {
        case CONDUIT_XF_NONE: launch_gather_xf<CONDUIT_XF_NONE>(a, s, bpf, n_items, tail_blocks); break;
        case CONDUIT_XF_U8_F32: launch_gather_xf<CONDUIT_XF_U8_F32>(a, s, bpf, n_items, tail_blocks); break;
        case CONDUIT_XF_U8_BF16_NORM: launch_gather_xf<CONDUIT_XF_U8_BF16_NORM>(a, s, bpf, n_items, tail_blocks); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
    if (a.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_pack, dim3((unsigned)(a.n + (a.weights.w ? 1 : 0))), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
