// Stratified inverse-CDF sampling over the 64-ary integer sum tree, with
// importance weights (off-policy delivery draws from the replay dataset, paper
// Sec. 2.2; proportional prioritised replay, Schaul et al.).
//
// k_sample: one wavefront per sample runs tree_descend (descend.h): the exact
// stratified target, then one coalesced 64-child load, wavefront prefix scan
// and ballot per tree level.
//
// k_is_weights: the weights need the smallest sampled leaf of the batch.  Each
// sample's wavefront parks its leaf in the output weight slot; one workgroup
// then reduces the minimum in LDS and overwrites every slot with
// (q_min / q_i)^beta computed in fp64 (is_weights_block).  The sample + gather
// call instead computes the weights inside its one launch (k_sample_gather.hip),
// or, for shapes that kernel does not take, in one extra workgroup of the
// gather launch.
#include "descend.h"

namespace conduit {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * kWave;

template <int PRE, int DEPTH>
__global__ __launch_bounds__(kThreads) void k_sample(SampleArgs a, DivB dv) {
    const int64_t k = (int64_t)blockIdx.x * kWaves + threadIdx.x / kWave;
    if (k < a.batch) {  // wave-uniform
        const Descent d = tree_descend<PRE, DEPTH>(a.tree, a.uniforms, k, dv);
        if (lane_id() == 0) {
            a.idx_out[k] = d.slot;
            // the sampled leaf is parked in the weight slot for the weights block
            if (a.w_out) reinterpret_cast<uint32_t*>(a.w_out)[k] = d.leaf;
            if (d.slot < 0 && k == 0) flag_error(a.err, ERR_EMPTY_TREE);
            if (d.lost) flag_error(a.err, ERR_DESCENT);
        }
    }
    // buffer-wide normalisation: this workgroup's share of the leaf minimum
    if (a.leaf_min) fold_leaf_min<kThreads>(a, blockIdx.x, gridDim.x);
}

constexpr int kWThreads = 1024;

__global__ __launch_bounds__(kWThreads) void k_is_weights(WeightsArgs a) { is_weights_block<kWThreads>(a); }

// the sampler grid for a tree of PRE prefetched groups and depth DEPTH
struct DescendLaunch {
    const SampleArgs& a;
    DivB dv;
    hipStream_t s;
    template <int PRE, int DEPTH>
    hipError_t operator()() const {
        const int64_t blocks = (a.batch + kWaves - 1) / kWaves;
        hipLaunchKernelGGL((k_sample<PRE, DEPTH>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a, dv);
        return hipGetLastError();
    }
};

}  // namespace

hipError_t launch_descend(const SampleArgs& a, hipStream_t s) {
    return with_descent_shape(a.tree, descend_prefetch(a.tree), DescendLaunch{a, make_divb((uint64_t)a.batch), s});
}

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
    hipError_t e = launch_descend(a, s);
    if (e != hipSuccess || a.w_out == nullptr) return e;
    hipLaunchKernelGGL(k_is_weights, dim3(1), dim3(kWThreads), 0, s, WeightsArgs{a.w_out, a.batch, a.beta, a.leaf_min});
    return hipGetLastError();
}

}  // namespace conduit
