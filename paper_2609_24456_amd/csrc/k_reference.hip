// Measurement reference for the u8 -> fp32 gathers: dst[i] = src[i] / 255 over
// contiguous memory.  It moves the gathers' byte mix (one byte read, four
// written per element) with none of their work: no index, no scattered rows,
// no frame stacking.  Every wavefront takes 1,024-byte chunks; in round k lane
// j converts the 32-bit word k * 64 + j of its chunk, so each load instruction
// covers 256 contiguous bytes and each (non-temporal) store 1 KB.  Its rate at
// a gather's size is the practical ceiling that gather's fraction of the HBM
// peak is compared with.
#include "common.h"

namespace conduit {

typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kRefThreads = 256;
constexpr int kRefWords = 4;  // words per lane per chunk: 4 x 64 x 4 B = 1,024 B

__device__ __forceinline__ f32x4 expand_word(uint32_t w) {
    f32x4 f;
    f.x = (float)(w & 255u) / 255.0f;
    f.y = (float)((w >> 8) & 255u) / 255.0f;
    f.z = (float)((w >> 16) & 255u) / 255.0f;
    f.w = (float)(w >> 24) / 255.0f;
    return f;
}

__global__ __launch_bounds__(kRefThreads) void k_expand_reference(const uint32_t* __restrict__ src,
                                                                  f32x4* __restrict__ dst, int64_t chunks,
                                                                  int64_t words) {
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kRefThreads / kWave);
    for (int64_t c = (int64_t)blockIdx.x * (kRefThreads / kWave) + threadIdx.x / kWave; c < chunks; c += waves) {
        uint32_t w[kRefWords];
#pragma unroll
        for (int k = 0; k < kRefWords; ++k) w[k] = __builtin_nontemporal_load(src + c * 256 + k * kWave + lane);
#pragma unroll
        for (int k = 0; k < kRefWords; ++k)
            __builtin_nontemporal_store(expand_word(w[k]), dst + c * 256 + k * kWave + lane);
    }
    // the words after the last whole chunk (fewer than 256): workgroup 0
    if (blockIdx.x == 0)
        for (int64_t i = chunks * 256 + threadIdx.x; i < words; i += kRefThreads) dst[i] = expand_word(src[i]);
}

}  // namespace

hipError_t launch_expand_reference(const uint8_t* src, float* dst, int64_t n, hipStream_t s) {
    const int64_t words = n / 4, chunks = words / 256;
    if (words == 0) return hipSuccess;
    const int64_t want = (chunks + kRefThreads / kWave - 1) / (kRefThreads / kWave);
    const int64_t cap = 32LL * device_cus();
    const int64_t grid = want < 1 ? 1 : want < cap ? want : cap;
    hipLaunchKernelGGL(k_expand_reference, dim3((unsigned)grid), dim3(kRefThreads), 0, s,
                       reinterpret_cast<const uint32_t*>(src), reinterpret_cast<f32x4*>(dst), chunks, words);
    return hipGetLastError();
}

}  // namespace conduit

using namespace conduit;

extern "C" conduit_status conduit_expand_reference(const uint8_t* src, float* dst, int64_t n, void* stream) {
    if (n < 0 || n % 4 != 0) return report_error(CONDUIT_EINVAL, "n must be a non-negative multiple of 4");
    if (n == 0) return CONDUIT_OK;
    if (!src || !dst) return report_error(CONDUIT_EINVAL, "NULL source or destination");
    if ((reinterpret_cast<uintptr_t>(src) & 3) || (reinterpret_cast<uintptr_t>(dst) & 15))
        return report_error(CONDUIT_EINVAL, "src must be 4-byte and dst 16-byte aligned");
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
    if (s0 < d0 + (uintptr_t)n * 4 && d0 < s0 + (uintptr_t)n)
        return report_error(CONDUIT_EINVAL, "source and destination overlap");
    const hipError_t e = launch_expand_reference(src, dst, n, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(e));
    return CONDUIT_OK;
}
