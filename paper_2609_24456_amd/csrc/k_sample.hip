// Stratified inverse-CDF sampling over the 64-ary integer sum tree, with
// importance weights (off-policy delivery "samples from a persistent replay
// dataset", paper Sec. 2.2; proportional prioritised replay, Schaul et al.).
//
// k_sample: one wavefront per sample runs tree_descend (common.h): the exact
// stratified target, then one coalesced 64-child load, wavefront prefix scan and
// ballot per tree level.
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
    const int64_t k = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (k >= a.batch) return;  // wave-uniform
    const Descent d = tree_descend(a.tree, a.uniforms, k, a.batch);
    if (lane_id() == 0) {
        a.idx_out[k] = d.slot;
        // the sampled leaf is parked in the weight slot for k_is_weights
        if (a.w_out) reinterpret_cast<uint32_t*>(a.w_out)[k] = d.leaf;
        if (d.slot < 0 && k == 0) flag_error(a.err, ERR_EMPTY_TREE);
        if (d.lost) flag_error(a.err, ERR_DESCENT);
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

hipError_t launch_is_weights(const SampleArgs& a, hipStream_t s) {
    if (a.w_out == nullptr) return hipSuccess;
    hipLaunchKernelGGL(k_is_weights, dim3(1), dim3(kWThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
    const int64_t blocks = (a.batch + kWaves - 1) / kWaves;
    hipLaunchKernelGGL(k_sample, dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_is_weights(a, s);
}

}  // namespace conduit
