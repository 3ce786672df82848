// Stratified inverse-CDF sampling over the 64-ary integer sum tree, with
// importance weights (off-policy delivery "samples from a persistent replay
// dataset", paper Sec. 2.2; proportional prioritised replay, Schaul et al.).
//
// k_sample: one wavefront per sample.  Stratum k's target
//     t_k = floor((k*Q + floor(u_k*Q / 2^64)) / B)
// is evaluated without 128-bit division by splitting Q and the high product
// word into quotient and remainder by B (all terms fit in 64 bits because
// k < B <= 2^20).  The descent visits depth levels; at each, the 64 lanes load
// the 64 children of the current node (one coalesced load), take an inclusive
// wavefront prefix sum, and the first lane whose prefix exceeds the target
// (ballot + find-first-set) names the child; its exclusive prefix is subtracted
// from the target.  This is exactly "first slot whose inclusive prefix sum
// exceeds t" with half-open intervals, so zero leaves are never hit.  The total
// Q, the uniform and the root's 64 children do not depend on each other, so the
// first three loads are issued together: depth dependent loads per sample.
//
// k_is_weights: the weights need the smallest sampled leaf of the batch.  Each
// sample's wavefront parks its leaf in the output weight slot; one workgroup
// then reduces the minimum in LDS and overwrites every slot with
// (q_min / q_i)^beta computed in fp64.  A second launch is cheaper than a
// grid-wide hand-off inside k_sample, whose agent-scope fences would write back
// the L2.
#include "common.h"

namespace conduit {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;

__global__ __launch_bounds__(kThreads) void k_sample(SampleArgs a) {
    const int lane = lane_id();
    const int64_t k = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (k >= a.batch) return;  // wave-uniform
    const TreeView& tr = a.tree;
    const int top = tr.depth;
    const uint64_t Q = tr.level[top][0];
    const uint64_t u = a.uniforms[k];
    uint64_t v = top == 1 ? (uint64_t)tr.leaves[lane] : tr.level[top - 1][lane];
    uint32_t* q_park = reinterpret_cast<uint32_t*>(a.w_out);  // sampled leaf, read by k_is_weights
    if (Q == 0ull) {  // nothing can be sampled (uniform across the grid)
        if (lane == 0) {
            a.idx_out[k] = -1;
            if (q_park) q_park[k] = 0u;
            if (k == 0) flag_error(a.err, ERR_EMPTY_TREE);
        }
        return;
    }
    const uint64_t B = (uint64_t)a.batch;
    const uint64_t h = __umul64hi(u, Q);
    const uint64_t kk = (uint64_t)k;
    uint64_t t = kk * (Q / B) + h / B + (kk * (Q % B) + h % B) / B;
    uint64_t node = 0;
    uint32_t q_sel = 0;
    bool lost = false;
    for (int l = top; l >= 1; --l) {
        if (l != top) {
            const uint64_t child = node * kFanout + (uint64_t)lane;
            v = l == 1 ? (uint64_t)tr.leaves[child] : tr.level[l - 1][child];
        }
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
        if (q_park) q_park[k] = q_sel;
        if (lost) flag_error(a.err, ERR_DESCENT);
    }
}

constexpr int kWThreads = 1024;

__global__ __launch_bounds__(kWThreads) void k_is_weights(SampleArgs a) {
    __shared__ uint32_t wave_min[kWThreads / kWave];
    __shared__ uint32_t qmin_s;
    // k_sample parked each sampled leaf in the weight array (0: nothing sampled)
    const uint32_t* q_park = reinterpret_cast<const uint32_t*>(a.w_out);
    uint32_t m = 0xffffffffu;
    for (int64_t k = threadIdx.x; k < a.batch; k += kWThreads) {
        const uint32_t q = q_park[k];
        if (q) m = q < m ? q : m;
    }
    m = wave_min_u32(m);
    if (lane_id() == 0) wave_min[threadIdx.x / kWave] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = wave_min[0];
        for (int i = 1; i < kWThreads / kWave; ++i) r = wave_min[i] < r ? wave_min[i] : r;
        qmin_s = r;
    }
    __syncthreads();
    const double qmin = (double)qmin_s;
    for (int64_t k = threadIdx.x; k < a.batch; k += kWThreads) {  // same k per lane as above
        const uint32_t q = q_park[k];
        a.w_out[k] = q ? (float)pow(qmin / (double)q, a.beta) : 0.0f;
    }
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
    const int64_t blocks = (a.batch + kWaves - 1) / kWaves;
    hipLaunchKernelGGL(k_sample, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.w_out == nullptr) return e;
    hipLaunchKernelGGL(k_is_weights, dim3(1), dim3(kWThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace conduit
