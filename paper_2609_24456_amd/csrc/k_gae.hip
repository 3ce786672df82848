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
// Time-major rollouts [T, E] (k_gae): a workgroup owns 8 environments x 64
// chunks of 16 steps (lanes run fastest over environments, so every load
// instruction of a wavefront reads eight 32-byte runs).  Padded sequences
// [B, Lmax] (k_gae_packed): one workgroup per sequence, 256 chunks along t.
#include "common.h"

namespace conduit {

namespace {

constexpr int kEnvs = 8;                      // environments per workgroup (32-byte runs)
constexpr int kChunks = 64;                   // chunks per environment and super-chunk
constexpr int kChunkLen = 16;                 // steps per chunk, held in registers
constexpr int kSuper = kChunks * kChunkLen;   // 1024 steps per pass
constexpr int kTmThreads = kEnvs * kChunks;   // 512: leaves 256 VGPRs per lane
static_assert(kGaeMaxEnvs * kSuper * 4 <= (1ll << 32), "byte offsets of a slab fit 32 bits");

// One step of the recursion: delta_t and the coefficient a_t of A_{t+1}.
// With TRUNC, a truncated step also ends the recursion and, unless it also
// terminated, bootstraps from the value of its true next observation.
template <bool TRUNC>
__device__ __forceinline__ void gae_step(double r, double v, double v_next, uint8_t d, uint8_t tr, float fv,
                                         double gamma, double gl, double* delta, double* m) {
    if constexpr (TRUNC) {
        const double live = (d | tr) ? 0.0 : 1.0;
        const double boot = (tr && !d) ? (double)fv : 0.0;
        *delta = r + gamma * (live * v_next + boot) - v;
        *m = gl * live;
    } else {
        const double live = d ? 0.0 : 1.0;
        *delta = r + gamma * live * v_next - v;
        *m = gl * live;
    }
}

// Time-major GAE.  A workgroup owns 8 environments and walks the rollout in
// super-chunks of 1024 steps from the end; the carry (A at the start of the
// later super-chunk) is kept per environment in LDS.  Within a super-chunk every
// lane loads its 16 steps (reward, value, done) at once into registers, folds
// them into (P, S), joins the suffix scan and replays from registers.
template <bool TRUNC>
__global__ __launch_bounds__(kTmThreads) void k_gae(GaeArgs a) {
    __shared__ double sP[kChunks][kEnvs];
    __shared__ double sS[kChunks][kEnvs];
    __shared__ double carry_s[kEnvs];
    const int el = threadIdx.x % kEnvs;
    const int c = threadIdx.x / kEnvs;
    const int64_t E = a.E, T = a.T;
    const int64_t e_raw = (int64_t)blockIdx.x * kEnvs + el;
    const bool active = e_raw < E;
    const int64_t e = active ? e_raw : E - 1;  // inactive lanes read a valid column
    const double gl = a.gamma * a.lambda;
    if (c == 0) carry_s[el] = 0.0;
    const int64_t supers = (T + kSuper - 1) / kSuper;
    for (int64_t sc = supers - 1; sc >= 0; --sc) {
        // uniform base of this super-chunk + 32-bit lane offsets (kSuper * E * 4 <= 2^32)
        const int64_t sbase = sc * kSuper * E;
        const float* __restrict__ rb = a.reward + sbase;
        const float* __restrict__ vb = a.value ? a.value + sbase : nullptr;
        const uint8_t* __restrict__ db = a.done + sbase;
        const int64_t t0 = sc * kSuper + (int64_t)c * kChunkLen;
        const int last_local = (int)(T - 1 - sc * kSuper);  // >= 0
        const uint32_t e32 = (uint32_t)e, E32 = (uint32_t)E;
        float r[kChunkLen], v[kChunkLen];
        uint8_t d[kChunkLen];
        uint8_t tr[TRUNC ? kChunkLen : 1];
        float fv[TRUNC ? kChunkLen : 1];
#pragma unroll
        for (int k = 0; k < kChunkLen; ++k) {
            const int lt = c * kChunkLen + k < last_local ? c * kChunkLen + k : last_local;
            const uint32_t off = (uint32_t)lt * E32 + e32;
            r[k] = rb[off];
            v[k] = vb ? vb[off] : 0.0f;
            d[k] = db[off];
            if constexpr (TRUNC) {
                tr[k] = a.truncated[sbase + off];
                fv[k] = a.final_value[sbase + off];
            }
        }
        const int64_t t1 = t0 + kChunkLen;  // first step after this chunk
        double v_end;
        if (t1 >= T) v_end = a.bootstrap ? (double)a.bootstrap[e] : 0.0;
        else v_end = a.value ? (double)a.value[t1 * E + e] : 0.0;
        // fold the chunk into A_start = P * A_end + S
        double P = 1.0, S = 0.0, v_next = v_end;
#pragma unroll
        for (int k = kChunkLen - 1; k >= 0; --k) {
            if (t0 + k < T) {
                double delta, m;
                gae_step<TRUNC>((double)r[k], (double)v[k], v_next, d[k], TRUNC ? tr[TRUNC ? k : 0] : 0,
                                TRUNC ? fv[TRUNC ? k : 0] : 0.0f, a.gamma, gl, &delta, &m);
                S = delta + m * S;
                P = m * P;
                v_next = (double)v[k];
            }
        }
        __syncthreads();  // carry_s of the previous pass is final; sP/sS free
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
        const double cin = carry_s[el];
        // A at the end of this chunk = suffix map of the chunks after it applied to the carry
        const double A_end = c + 1 < kChunks ? sP[c + 1][el] * cin + sS[c + 1][el] : cin;
        double A = A_end;
        v_next = v_end;
        float* __restrict__ ab = a.adv + sbase;
        float* __restrict__ qb = a.ret + sbase;
#pragma unroll
        for (int k = kChunkLen - 1; k >= 0; --k) {
            if (t0 + k < T) {
                double delta, m;
                gae_step<TRUNC>((double)r[k], (double)v[k], v_next, d[k], TRUNC ? tr[TRUNC ? k : 0] : 0,
                                TRUNC ? fv[TRUNC ? k : 0] : 0.0f, a.gamma, gl, &delta, &m);
                A = delta + m * A;
                if (active) {
                    const uint32_t off = (uint32_t)(c * kChunkLen + k) * E32 + e32;
                    ab[off] = (float)A;
                    qb[off] = (float)(A + (double)v[k]);
                }
                v_next = (double)v[k];
            }
        }
        __syncthreads();  // every lane has read carry_s
        if (c == 0) carry_s[el] = sP[0][el] * cin + sS[0][el];
    }
}

constexpr int kPkThreads = 256;
constexpr int kPkChunk = 16;                      // elements per lane and segment
constexpr int kPkSeg = kPkThreads * kPkChunk;     // 4096 elements per pass
constexpr int kPkPad = kPkSeg + kPkSeg / 16 + 1;  // padded LDS row

// padded LDS index: one spare word every 16, so lanes reading their own
// contiguous chunk of 16 hit distinct banks
__device__ __forceinline__ int lpad(int t) { return t + (t >> 4); }

// GAE over right-padded sequences, one workgroup per sequence, walked in
// segments of 4096 elements from the end with a carry.  Values are staged into
// LDS with coalesced loads, each lane owns a contiguous chunk of 16 for the scan,
// and advantages/returns are staged back and written coalesced.
__global__ __launch_bounds__(kPkThreads) void k_gae_packed(GaePackedArgs a) {
    __shared__ float sV[kPkPad];
    __shared__ float sA[kPkPad];
    __shared__ float sR[kPkPad];
    __shared__ double sP[kPkThreads];
    __shared__ double sS[kPkThreads];
    const int c = threadIdx.x;
    const int64_t b = blockIdx.x;
    const int64_t Lmax = a.Lmax;
    int64_t L = a.length[b];
    if (L < 0 || L > Lmax) {
        if (c == 0) flag_error(a.err, ERR_SEQ_LENGTH);
        L = L < 0 ? 0 : Lmax;
    }
    const float* val = a.value ? a.value + b * Lmax : nullptr;
    float* adv = a.adv + b * Lmax;
    float* ret = a.ret + b * Lmax;
    const double R = (double)a.last_reward[b];
    const double gl = a.gamma * a.lambda;
    double carry = 0.0;    // A at the start of the later segment
    double v_after = 0.0;  // V at the start of the later segment
    const int64_t segs = (Lmax + kPkSeg - 1) / kPkSeg;
    for (int64_t sg = segs - 1; sg >= 0; --sg) {
        const int64_t base = sg * kPkSeg;
        const int seg_len = (int)(Lmax - base < kPkSeg ? Lmax - base : kPkSeg);
        for (int t = c; t < seg_len; t += kPkThreads) sV[lpad(t)] = val ? val[base + t] : 0.0f;
        __syncthreads();
        // this lane's chunk [t0, t1) of the segment, live part [t0, u1)
        const int t0 = c * kPkChunk;
        const int t1 = t0 + kPkChunk < seg_len ? t0 + kPkChunk : seg_len;
        const int64_t live_end = L - base;
        const int u1 = (int)(t1 < live_end ? t1 : (live_end > t0 ? live_end : t0));
        double v_end = 0.0;  // V after the chunk's live part, when the sequence continues
        if (base + u1 < L && u1 > t0) v_end = u1 < seg_len ? (double)sV[lpad(u1)] : v_after;
        double P = 1.0, S = 0.0;
        {
            double v_next = v_end;
#pragma unroll
            for (int k = kPkChunk - 1; k >= 0; --k) {
                const int t = t0 + k;
                if (t < u1) {
                    const double v = (double)sV[lpad(t)];
                    const bool last = base + t == L - 1;
                    const double live = last ? 0.0 : 1.0;
                    const double delta = (last ? R : 0.0) + a.gamma * live * v_next - v;
                    const double m = gl * live;
                    S = delta + m * S;
                    P = m * P;
                    v_next = v;
                }
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
        double A = c + 1 < kPkThreads ? sP[c + 1] * carry + sS[c + 1] : carry;
        {
            double v_next = v_end;
#pragma unroll
            for (int k = kPkChunk - 1; k >= 0; --k) {
                const int t = t0 + k;
                if (t < t1) {
                    if (t < u1) {
                        const double v = (double)sV[lpad(t)];
                        const bool last = base + t == L - 1;
                        const double live = last ? 0.0 : 1.0;
                        const double delta = (last ? R : 0.0) + a.gamma * live * v_next - v;
                        A = delta + gl * live * A;
                        sA[lpad(t)] = (float)A;
                        sR[lpad(t)] = (float)(A + v);
                        v_next = v;
                    } else {
                        sA[lpad(t)] = 0.0f;
                        sR[lpad(t)] = 0.0f;
                    }
                }
            }
        }
        __syncthreads();
        for (int t = c; t < seg_len; t += kPkThreads) {
            adv[base + t] = sA[lpad(t)];
            ret[base + t] = sR[lpad(t)];
        }
        carry = sP[0] * carry + sS[0];
        v_after = (double)sV[lpad(0)];
        __syncthreads();  // LDS is rewritten by the next segment
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
    if (a.E > kGaeMaxEnvs) return hipErrorInvalidValue;  // the ABI rejects this first
    const int64_t blocks = (a.E + kEnvs - 1) / kEnvs;
    if (a.truncated)
        hipLaunchKernelGGL(k_gae<true>, dim3((unsigned)blocks), dim3(kTmThreads), 0, s, a);
    else
        hipLaunchKernelGGL(k_gae<false>, dim3((unsigned)blocks), dim3(kTmThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_gae_packed(const GaePackedArgs& a, hipStream_t s) {
    if (a.B <= 0 || a.Lmax <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_gae_packed, dim3((unsigned)a.B), dim3(kPkThreads), 0, s, a);
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
