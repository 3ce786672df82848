// Generalised advantage estimation (on-policy ingestion "computing
// returns/advantages", paper Sec. 2.2; GAE as used by PPO, Schulman et al.).
//
// The recursion A_t = delta_t + a_t A_{t+1}, a_t = gamma*lambda*(1 - d_t), is
// affine in A_{t+1}, so a chunk of consecutive steps composes into one map
// A_start = P * A_end + S.  Each kernel runs three phases inside one workgroup:
//   1. every lane folds its chunk of steps into (P, S) (reverse order);
//   2. a Hillis-Steele suffix scan over the chunks in LDS composes the maps, so
//      chunk c learns A at its end, A_{t1(c)} = A_start(c + 1);
//   3. every lane replays its chunk from that carry and writes A_t and
//      R_t = A_t + V_t.
// All arithmetic is fp64; outputs are rounded to fp32 once.
//
// Time-major rollouts [T, E] (k_gae): a workgroup owns 16 environments x 64
// chunks (lanes run fastest over environments, so every load instruction of a
// wavefront reads four 64-byte runs).  Padded sequences [B, Lmax]
// (k_gae_packed): one workgroup per sequence, 256 chunks along t.
#include "common.h"

namespace conduit {

namespace {

constexpr int kEnvs = 16;
constexpr int kChunks = 64;
constexpr int kTmThreads = kEnvs * kChunks;  // 1024

__global__ __launch_bounds__(kTmThreads) void k_gae(GaeArgs a, int64_t chunk_len) {
    __shared__ double sP[kChunks][kEnvs];
    __shared__ double sS[kChunks][kEnvs];
    const int el = threadIdx.x % kEnvs;
    const int c = threadIdx.x / kEnvs;
    const int64_t e = (int64_t)blockIdx.x * kEnvs + el;
    const bool active = e < a.E;
    const int64_t E = a.E;
    const int64_t t0 = (int64_t)c * chunk_len;
    const int64_t t1 = t0 + chunk_len < a.T ? t0 + chunk_len : a.T;
    const double gl = a.gamma * a.lambda;

    double v_end = 0.0;  // V_{t1}
    if (active && t0 < t1) {
        if (t1 == a.T) v_end = a.bootstrap ? (double)a.bootstrap[e] : 0.0;
        else v_end = a.value ? (double)a.value[t1 * E + e] : 0.0;
    }
    double P = 1.0, S = 0.0;
    if (active) {
        double v_next = v_end;
        for (int64_t t = t1 - 1; t >= t0; --t) {
            const int64_t at = t * E + e;
            const double v = a.value ? (double)a.value[at] : 0.0;
            const double live = a.done[at] ? 0.0 : 1.0;
            const double delta = (double)a.reward[at] + a.gamma * live * v_next - v;
            const double m = gl * live;
            S = delta + m * S;
            P = m * P;
            v_next = v;
        }
    }
    sP[c][el] = P;
    sS[c][el] = S;
    __syncthreads();
    for (int off = 1; off < kChunks; off <<= 1) {
        const bool has = c + off < kChunks;
        double p2 = 1.0, s2 = 0.0;
        if (has) {
            p2 = sP[c + off][el];
            s2 = sS[c + off][el];
        }
        __syncthreads();
        if (has) {
            S = S + P * s2;
            P = P * p2;
            sP[c][el] = P;
            sS[c][el] = S;
        }
        __syncthreads();
    }
    const double carry = c + 1 < kChunks ? sS[c + 1][el] : 0.0;
    if (!active) return;
    double A = carry;
    double v_next = v_end;
    for (int64_t t = t1 - 1; t >= t0; --t) {
        const int64_t at = t * E + e;
        const double v = a.value ? (double)a.value[at] : 0.0;
        const double live = a.done[at] ? 0.0 : 1.0;
        const double delta = (double)a.reward[at] + a.gamma * live * v_next - v;
        A = delta + gl * live * A;
        a.adv[at] = (float)A;
        a.ret[at] = (float)(A + v);
        v_next = v;
    }
}

constexpr int kPkThreads = 256;

__global__ __launch_bounds__(kPkThreads) void k_gae_packed(GaePackedArgs a, int64_t chunk_len) {
    __shared__ double sP[kPkThreads];
    __shared__ double sS[kPkThreads];
    const int c = threadIdx.x;
    const int64_t b = blockIdx.x;
    int64_t L = a.length[b];
    if (L < 0 || L > a.Lmax) {
        if (c == 0) flag_error(a.err, ERR_SEQ_LENGTH);
        L = L < 0 ? 0 : a.Lmax;
    }
    const int64_t t0 = (int64_t)c * chunk_len;
    const int64_t t1 = t0 + chunk_len < a.Lmax ? t0 + chunk_len : a.Lmax;
    const int64_t u1 = t1 < L ? t1 : L;  // live part of the chunk: [t0, u1)
    const float* val = a.value ? a.value + b * a.Lmax : nullptr;
    const double R = (double)a.last_reward[b];
    const double gl = a.gamma * a.lambda;
    const double v_end = (val && u1 < L && u1 > t0) ? (double)val[u1] : 0.0;

    double P = 1.0, S = 0.0;
    {
        double v_next = v_end;
        for (int64_t t = u1 - 1; t >= t0; --t) {
            const double v = val ? (double)val[t] : 0.0;
            const bool last = t == L - 1;
            const double live = last ? 0.0 : 1.0;
            const double delta = (last ? R : 0.0) + a.gamma * live * v_next - v;
            const double m = gl * live;
            S = delta + m * S;
            P = m * P;
            v_next = v;
        }
    }
    sP[c] = P;
    sS[c] = S;
    __syncthreads();
    for (int off = 1; off < kPkThreads; off <<= 1) {
        const bool has = c + off < kPkThreads;
        double p2 = 1.0, s2 = 0.0;
        if (has) {
            p2 = sP[c + off];
            s2 = sS[c + off];
        }
        __syncthreads();
        if (has) {
            S = S + P * s2;
            P = P * p2;
            sP[c] = P;
            sS[c] = S;
        }
        __syncthreads();
    }
    const double carry = c + 1 < kPkThreads ? sS[c + 1] : 0.0;
    float* adv = a.adv + b * a.Lmax;
    float* ret = a.ret + b * a.Lmax;
    for (int64_t t = t1 - 1; t >= u1 && t >= t0; --t) {
        adv[t] = 0.0f;
        ret[t] = 0.0f;
    }
    double A = carry;
    double v_next = v_end;
    for (int64_t t = u1 - 1; t >= t0; --t) {
        const double v = val ? (double)val[t] : 0.0;
        const bool last = t == L - 1;
        const double live = last ? 0.0 : 1.0;
        const double delta = (last ? R : 0.0) + a.gamma * live * v_next - v;
        A = delta + gl * live * A;
        adv[t] = (float)A;
        ret[t] = (float)(A + v);
        v_next = v;
    }
}

__global__ void k_fill_u32(uint32_t* p, uint32_t v, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_fill_u64(uint64_t* p, uint64_t v, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

}  // namespace

hipError_t launch_gae(const GaeArgs& a, hipStream_t s) {
    if (a.T <= 0 || a.E <= 0) return hipSuccess;
    const int64_t chunk_len = (a.T + kChunks - 1) / kChunks;
    const int64_t blocks = (a.E + kEnvs - 1) / kEnvs;
    hipLaunchKernelGGL(k_gae, dim3((unsigned)blocks), dim3(kTmThreads), 0, s, a, chunk_len);
    return hipGetLastError();
}

hipError_t launch_gae_packed(const GaePackedArgs& a, hipStream_t s) {
    if (a.B <= 0 || a.Lmax <= 0) return hipSuccess;
    const int64_t chunk_len = (a.Lmax + kPkThreads - 1) / kPkThreads;
    hipLaunchKernelGGL(k_gae_packed, dim3((unsigned)a.B), dim3(kPkThreads), 0, s, a, chunk_len);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)blocks), dim3(256), 0, s, p, v, n);
    return hipGetLastError();
}

hipError_t launch_fill_u64(uint64_t* p, uint64_t v, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_fill_u64, dim3((unsigned)blocks), dim3(256), 0, s, p, v, n);
    return hipGetLastError();
}

}  // namespace conduit
