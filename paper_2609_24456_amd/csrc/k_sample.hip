// Stratified inverse-CDF sampling over the 64-ary integer sum tree, with
// importance weights (off-policy delivery "samples from a persistent replay
// dataset", paper Sec. 2.2; proportional prioritised replay, Schaul et al.).
//
// One wavefront per sample.  Stratum k's target
//     t_k = floor((k*Q + floor(u_k*Q / 2^64)) / B)
// is evaluated without 128-bit division by splitting Q and the high product
// word into quotient and remainder by B (all terms fit in 64 bits because
// k < B <= 2^20).  The descent visits depth levels; at each, the 64 lanes load
// the 64 children of the current node (one coalesced 512-byte load), take an
// inclusive wavefront prefix sum, and the first lane whose prefix exceeds the
// target (ballot + find-first-set) names the child; its exclusive prefix is
// subtracted from the target.  This is exactly "first slot whose inclusive
// prefix sum exceeds t" with half-open intervals, so zero leaves are never hit.
//
// Importance weights need the smallest sampled leaf of the whole batch.  Each
// workgroup folds its minimum into a device word with atomicMin; the last
// workgroup to finish (ticket counter, agent-scope fences) computes every
// weight (q_min / q_i)^beta in fp64 and resets the two scratch words for the
// next call, so a sample costs one launch.
#include "common.h"

namespace conduit {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;

__global__ __launch_bounds__(kThreads) void k_sample(SampleArgs a) {
    __shared__ uint32_t wave_min[kWaves];
    __shared__ int is_last;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int64_t k = (int64_t)blockIdx.x * kWaves + w;
    const TreeView& tr = a.tree;
    const uint64_t Q = tr.level[tr.depth][0];

    if (Q == 0ull) {  // nothing can be sampled (uniform across the grid)
        if (k < a.batch && lane == 0) {
            a.idx_out[k] = -1;
            if (a.w_out) a.w_out[k] = 0.0f;
        }
        if (blockIdx.x == 0 && threadIdx.x == 0) flag_error(a.err, ERR_EMPTY_TREE);
        return;
    }

    uint32_t q_sel = 0xffffffffu;
    if (k < a.batch) {
        const uint64_t B = (uint64_t)a.batch;
        const uint64_t u = a.uniforms[k];
        const uint64_t h = __umul64hi(u, Q);
        const uint64_t kk = (uint64_t)k;
        uint64_t t = kk * (Q / B) + h / B + (kk * (Q % B) + h % B) / B;
        uint64_t node = 0;
        bool lost = false;
        for (int l = tr.depth; l >= 1; --l) {
            const uint64_t child = node * kFanout + (uint64_t)lane;
            const uint64_t v = l == 1 ? (uint64_t)tr.leaves[child] : tr.level[l - 1][child];
            const uint64_t incl = wave_inclusive_scan_u64(v);
            const uint64_t mask = __ballot(incl > t);
            int sel = 63;
            if (mask) sel = __ffsll((unsigned long long)mask) - 1; else lost = true;
            const uint64_t excl = __shfl(incl - v, sel, kWave);
            t -= excl;
            node = node * kFanout + (uint64_t)sel;
            if (l == 1) q_sel = (uint32_t)__shfl(v, sel, kWave);
        }
        if (lane == 0) {
            a.idx_out[k] = (int64_t)node;
            if (lost) flag_error(a.err, ERR_DESCENT);
        }
    }
    if (a.w_out == nullptr) return;  // kernel argument: uniform

    const uint32_t m = wave_min_u32(q_sel);
    if (lane == 0) wave_min[w] = m;
    __threadfence();  // publish idx_out before the ticket
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t bm = wave_min[0];
        for (int i = 1; i < kWaves; ++i) bm = wave_min[i] < bm ? wave_min[i] : bm;
        atomicMin(&a.state->qmin, bm);
        __threadfence();
        const uint32_t ticket = atomicAdd(&a.state->ticket, 1u);
        is_last = ticket == gridDim.x - 1;
    }
    __syncthreads();
    if (!is_last) return;
    __threadfence();
    const uint32_t qmin = __hip_atomic_load(&a.state->qmin, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int64_t j = threadIdx.x; j < a.batch; j += kThreads) {
        const int64_t i = __hip_atomic_load(a.idx_out + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t q = tr.leaves[i];
        a.w_out[j] = (float)pow((double)qmin / (double)q, a.beta);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_store(&a.state->qmin, 0xffffffffu, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&a.state->ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
    const int64_t blocks = (a.batch + kWaves - 1) / kWaves;
    hipLaunchKernelGGL(k_sample, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
