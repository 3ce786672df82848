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
// Time-major rollouts [T, E]: a workgroup owns 8 environments and walks the
// rollout in passes of 2048 steps.  k_gae_v4 (E a multiple of 4, aligned rows)
// gives each lane 4 environments as 16-byte vectors and 16 steps, 128 chunks
// per pass; k_gae (any E) gives each lane one environment and 32 steps, 64
// chunks per pass, lanes fastest over environments so every load instruction of
// a wavefront reads eight 32-byte runs.  Padded sequences
// [B, Lmax] (k_gae_packed): one workgroup per sequence, 256 chunks along t.
#include "common.h"

namespace conduit {

namespace {

constexpr int kEnvs = 8;                      // environments per workgroup (32-byte runs)
constexpr int kChunks = 64;                   // chunks per environment and super-chunk
constexpr int kChunkLen = 32;                 // steps per chunk, held in registers
constexpr int kSuper = kChunks * kChunkLen;   // 2048 steps per pass: a PPO rollout in one
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
// super-chunks of 2048 steps from the end; the carry (A at the start of the
// later super-chunk) is kept per environment in LDS.  Within a super-chunk every
// lane loads its 32 steps (reward, value, done) at once into registers, folds
// them into (P, S), joins the suffix scan and replays from registers.  The scan
// ping-pongs between two LDS buffers, so each of its rounds needs one barrier.
template <bool TRUNC>
__global__ __launch_bounds__(kTmThreads) void k_gae(GaeArgs a) {
    __shared__ double sP[2][kChunks][kEnvs];
    __shared__ double sS[2][kChunks][kEnvs];
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
        // step k of the lane: row `row` (uniform, elements from the slab) plus
        // the lane's offset `lo` from that row
        auto load_step = [&](int k, int64_t row, uint32_t lo) {
            r[k] = (rb + row)[lo];
            v[k] = vb ? (vb + row)[lo] : 0.0f;
            d[k] = (db + row)[lo];
            if constexpr (TRUNC) {
                tr[TRUNC ? k : 0] = (a.truncated + sbase + row)[lo];
                fv[TRUNC ? k : 0] = (a.final_value + sbase + row)[lo];
            }
        };
        if (sc * kSuper + kSuper <= T) {
            // a full super-chunk: step k of every lane lies k rows below the
            // lane's first step, so one lane offset serves all of its loads and
            // the rows advance in scalar registers
            const uint32_t lo = (uint32_t)(c * kChunkLen) * E32 + e32;
#pragma unroll
            for (int k = 0; k < kChunkLen; ++k) load_step(k, (int64_t)k * E, lo);
        } else {
            // the last, partial one: steps past the end re-read the last row
#pragma unroll
            for (int k = 0; k < kChunkLen; ++k) {
                const int lt = c * kChunkLen + k < last_local ? c * kChunkLen + k : last_local;
                load_step(k, 0, (uint32_t)lt * E32 + e32);
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
        int cur = 0;
        sP[cur][c][el] = P;
        sS[cur][c][el] = S;
        __syncthreads();
        // round r reads the buffer written in round r - 1 and writes the other
        // one, whose readers all passed the barrier that ended round r - 1
        for (int off = 1; off < kChunks; off <<= 1) {
            if (c + off < kChunks) {
                const double p2 = sP[cur][c + off][el];
                const double s2 = sS[cur][c + off][el];
                S = S + P * s2;
                P = P * p2;
            }
            sP[cur ^ 1][c][el] = P;
            sS[cur ^ 1][c][el] = S;
            cur ^= 1;
            __syncthreads();
        }
        const double cin = carry_s[el];
        // A at the end of this chunk = suffix map of the chunks after it applied to the carry
        const double A_end = c + 1 < kChunks ? sP[cur][c + 1][el] * cin + sS[cur][c + 1][el] : cin;
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
                    const uint32_t lo = (uint32_t)(c * kChunkLen) * E32 + e32;
                    (ab + (int64_t)k * E)[lo] = (float)A;
                    (qb + (int64_t)k * E)[lo] = (float)(A + (double)v[k]);
                }
                v_next = (double)v[k];
            }
        }
        __syncthreads();  // every lane has read carry_s
        if (c == 0) carry_s[el] = sP[cur][0][el] * cin + sS[cur][0][el];
    }
}

// Time-major GAE, four environments per lane: the same three phases, with every
// load and store a 16-byte vector of 4 consecutive environments (a lane pair
// covers a 32-byte run of a row) and four independent recursions per lane.
// Compared with one environment per lane this issues a quarter of the memory
// instructions, which bound the one-environment kernel on the few compute units
// a rollout of a few hundred environments occupies.  Needs E a multiple of 4,
// 16-byte aligned float rows and 4-byte aligned flag rows (checked by the
// launcher).
#ifndef CONDUIT_GAE_VEC_CHUNK
#define CONDUIT_GAE_VEC_CHUNK 16
#endif
constexpr int kGaeVecChunk = CONDUIT_GAE_VEC_CHUNK;  // steps per chunk
constexpr int kV = 4;                  // environments per lane
constexpr int kEnvsV = 8;              // environments per workgroup (32-byte runs)
constexpr int kQuads = kEnvsV / kV;    // lanes per row
constexpr int kSuperV = 2048;          // steps per pass
typedef float f32x4 __attribute__((ext_vector_type(4)));
static_assert(kGaeMaxEnvs * kSuperV * 4 <= (1ll << 32), "byte offsets of a slab fit 32 bits");

template <bool TRUNC, int L>
__global__ __launch_bounds__(kQuads * (kSuperV / L)) void k_gae_v4(GaeArgs a) {
    constexpr int kCh = kSuperV / L;  // chunks per pass
    __shared__ double sP[2][kCh][kEnvsV];
    __shared__ double sS[2][kCh][kEnvsV];
    __shared__ double carry_s[kEnvsV];
    const int q = threadIdx.x % kQuads;
    const int c = threadIdx.x / kQuads;
    const int64_t E = a.E, T = a.T;
    // workgroups are dealt round-robin to the 8 XCDs: the ones on one XCD take
    // consecutive environment groups, so the 4 groups that share each 128-byte
    // line of a row are read through the same L2
    const int64_t nb = gridDim.x;
    const int64_t group = nb % 8 == 0 ? (int64_t)(blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8 : (int64_t)blockIdx.x;
    const int64_t e_raw = group * kEnvsV + q * kV;
    const bool active = e_raw < E;                // E % 4 == 0: a quad is wholly in or out
    const int64_t e0 = active ? e_raw : E - kV;  // inactive lanes read a valid quad
    const double gl = a.gamma * a.lambda;
    if (c == 0) {
#pragma unroll
        for (int j = 0; j < kV; ++j) carry_s[q * kV + j] = 0.0;
    }
    const int64_t supers = (T + kSuperV - 1) / kSuperV;
    for (int64_t sc = supers - 1; sc >= 0; --sc) {
        const int64_t row0 = sc * kSuperV;
        const int last_local = (int)(T - 1 - row0);  // >= 0
        const bool full = row0 + kSuperV <= T;       // uniform
        // lane offset of the lane's first step from the row of step k (elements)
        const uint32_t lo = (uint32_t)(c * L) * (uint32_t)E + (uint32_t)e0;
        f32x4 r[L], v[L];
        uint32_t d[L];
        uint32_t tr[TRUNC ? L : 1];
        f32x4 fv[TRUNC ? L : 1];
#pragma unroll
        for (int k = 0; k < L; ++k) {
            // full pass: uniform row base + one lane offset; partial pass: steps
            // past the end re-read the last row
            const int64_t row = full ? row0 + k : row0 + (c * L + k < last_local ? c * L + k : last_local);
            const int64_t base = row * E;
            const uint32_t off = full ? lo : (uint32_t)e0;
            const int64_t rb = full ? (row0 + k) * E : base;
            r[k] = *reinterpret_cast<const f32x4*>(a.reward + rb + off);
            v[k] = a.value ? *reinterpret_cast<const f32x4*>(a.value + rb + off) : (f32x4)(0.0f);
            d[k] = *reinterpret_cast<const uint32_t*>(a.done + rb + off);
            if constexpr (TRUNC) {
                tr[TRUNC ? k : 0] = *reinterpret_cast<const uint32_t*>(a.truncated + rb + off);
                fv[TRUNC ? k : 0] = *reinterpret_cast<const f32x4*>(a.final_value + rb + off);
            }
        }
        const int64_t t1 = row0 + (int64_t)c * L + L;  // first step after this chunk
        f32x4 ve;
        if (t1 >= T) ve = a.bootstrap ? *reinterpret_cast<const f32x4*>(a.bootstrap + e0) : (f32x4)(0.0f);
        else ve = a.value ? *reinterpret_cast<const f32x4*>(a.value + t1 * E + e0) : (f32x4)(0.0f);
        // fold the chunk into A_start = P * A_end + S, four environments at once
        double P[kV], S[kV], vn[kV];
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            P[j] = 1.0;
            S[j] = 0.0;
            vn[j] = (double)ve[j];
        }
#pragma unroll
        for (int k = L - 1; k >= 0; --k) {
            if (c * L + k <= last_local) {
#pragma unroll
                for (int j = 0; j < kV; ++j) {
                    double delta, m;
                    gae_step<TRUNC>((double)r[k][j], (double)v[k][j], vn[j], (uint8_t)(d[k] >> (8 * j)),
                                    TRUNC ? (uint8_t)(tr[TRUNC ? k : 0] >> (8 * j)) : 0,
                                    TRUNC ? fv[TRUNC ? k : 0][j] : 0.0f, a.gamma, gl, &delta, &m);
                    S[j] = delta + m * S[j];
                    P[j] = m * P[j];
                    vn[j] = (double)v[k][j];
                }
            }
        }
        __syncthreads();  // carry_s of the previous pass is final; sP/sS free
        int cur = 0;
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            sP[cur][c][q * kV + j] = P[j];
            sS[cur][c][q * kV + j] = S[j];
        }
        __syncthreads();
        // suffix scan over the chunks, ping-pong buffers: one barrier per round
        for (int off = 1; off < kCh; off <<= 1) {
            if (c + off < kCh) {
#pragma unroll
                for (int j = 0; j < kV; ++j) {
                    const double p2 = sP[cur][c + off][q * kV + j];
                    const double s2 = sS[cur][c + off][q * kV + j];
                    S[j] = S[j] + P[j] * s2;
                    P[j] = P[j] * p2;
                }
            }
#pragma unroll
            for (int j = 0; j < kV; ++j) {
                sP[cur ^ 1][c][q * kV + j] = P[j];
                sS[cur ^ 1][c][q * kV + j] = S[j];
            }
            cur ^= 1;
            __syncthreads();
        }
        double cin[kV], A[kV];
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            cin[j] = carry_s[q * kV + j];
            A[j] = c + 1 < kCh ? sP[cur][c + 1][q * kV + j] * cin[j] + sS[cur][c + 1][q * kV + j] : cin[j];
            vn[j] = (double)ve[j];
        }
#pragma unroll
        for (int k = L - 1; k >= 0; --k) {
            if (c * L + k <= last_local) {
                f32x4 ao, ro;
#pragma unroll
                for (int j = 0; j < kV; ++j) {
                    double delta, m;
                    gae_step<TRUNC>((double)r[k][j], (double)v[k][j], vn[j], (uint8_t)(d[k] >> (8 * j)),
                                    TRUNC ? (uint8_t)(tr[TRUNC ? k : 0] >> (8 * j)) : 0,
                                    TRUNC ? fv[TRUNC ? k : 0][j] : 0.0f, a.gamma, gl, &delta, &m);
                    A[j] = delta + m * A[j];
                    ao[j] = (float)A[j];
                    ro[j] = (float)(A[j] + (double)v[k][j]);
                    vn[j] = (double)v[k][j];
                }
                if (active) {
                    const int64_t rb = full ? (row0 + k) * E : (row0 + c * L + k) * E;
                    const uint32_t off = full ? lo : (uint32_t)e0;
                    *reinterpret_cast<f32x4*>(a.adv + rb + off) = ao;
                    *reinterpret_cast<f32x4*>(a.ret + rb + off) = ro;
                }
            }
        }
        __syncthreads();  // every lane has read carry_s
        if (c == 0) {
#pragma unroll
            for (int j = 0; j < kV; ++j)
                carry_s[q * kV + j] = sP[cur][0][q * kV + j] * cin[j] + sS[cur][0][q * kV + j];
        }
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
    __shared__ double sP[2][kPkThreads];
    __shared__ double sS[2][kPkThreads];
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
    // 16-byte vectors for the value loads and the output stores when the rows
    // allow them (uniform)
    auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    const bool vec_in = val && al16(val);
    const bool vec_out = al16(adv) && al16(ret);
    const double R = (double)a.last_reward[b];
    const double gl = a.gamma * a.lambda;
    double carry = 0.0;    // A at the start of the later segment
    double v_after = 0.0;  // V at the start of the later segment
    const int64_t segs = (Lmax + kPkSeg - 1) / kPkSeg;
    for (int64_t sg = segs - 1; sg >= 0; --sg) {
        const int64_t base = sg * kPkSeg;
        const int seg_len = (int)(Lmax - base < kPkSeg ? Lmax - base : kPkSeg);
        if (vec_in) {
            // every lane's 4 vectors are loaded before the first LDS write
            constexpr int kVecs = kPkSeg / (4 * kPkThreads);
            f32x4 q[kVecs];
#pragma unroll
            for (int j = 0; j < kVecs; ++j) {
                const int t = (j * kPkThreads + c) * 4;
                if (t + 3 < seg_len) {
                    q[j] = *reinterpret_cast<const f32x4*>(val + base + t);
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) q[j][i] = t + i < seg_len ? val[base + t + i] : 0.0f;
                }
            }
#pragma unroll
            for (int j = 0; j < kVecs; ++j) {
                const int t = (j * kPkThreads + c) * 4;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (t + i < seg_len) sV[lpad(t + i)] = q[j][i];
            }
        } else {
            for (int t = c; t < seg_len; t += kPkThreads) sV[lpad(t)] = val ? val[base + t] : 0.0f;
        }
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
        // suffix scan over the lanes' chunks, ping-pong buffers: round r reads
        // what round r - 1 wrote and writes the other buffer, one barrier each
        int cur = 0;
        sP[cur][c] = P;
        sS[cur][c] = S;
        __syncthreads();
        for (int off = 1; off < kPkThreads; off <<= 1) {
            if (c + off < kPkThreads) {
                const double p2 = sP[cur][c + off];
                const double s2 = sS[cur][c + off];
                S = S + P * s2;
                P = P * p2;
            }
            sP[cur ^ 1][c] = P;
            sS[cur ^ 1][c] = S;
            cur ^= 1;
            __syncthreads();
        }
        double A = c + 1 < kPkThreads ? sP[cur][c + 1] * carry + sS[cur][c + 1] : carry;
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
        if (vec_out) {
            constexpr int kVecs = kPkSeg / (4 * kPkThreads);
#pragma unroll
            for (int j = 0; j < kVecs; ++j) {
                const int t = (j * kPkThreads + c) * 4;
                if (t + 3 < seg_len) {
                    f32x4 oa, orr;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        oa[i] = sA[lpad(t + i)];
                        orr[i] = sR[lpad(t + i)];
                    }
                    *reinterpret_cast<f32x4*>(adv + base + t) = oa;
                    *reinterpret_cast<f32x4*>(ret + base + t) = orr;
                } else {
                    for (int i = 0; i < 4 && t + i < seg_len; ++i) {
                        adv[base + t + i] = sA[lpad(t + i)];
                        ret[base + t + i] = sR[lpad(t + i)];
                    }
                }
            }
        } else {
            for (int t = c; t < seg_len; t += kPkThreads) {
                adv[base + t] = sA[lpad(t)];
                ret[base + t] = sR[lpad(t)];
            }
        }
        carry = sP[cur][0] * carry + sS[cur][0];
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
    auto al = [](const void* p, uintptr_t m) { return (reinterpret_cast<uintptr_t>(p) & (m - 1)) == 0; };
    const bool vec = a.E % kV == 0 && al(a.reward, 16) && al(a.value, 16) && al(a.bootstrap, 16) &&
                     al(a.adv, 16) && al(a.ret, 16) && al(a.done, 4) && al(a.truncated, 4) &&
                     al(a.final_value, 16);
    if (vec) {
        const int64_t vblocks = (a.E + kEnvsV - 1) / kEnvsV;
        constexpr int L = kGaeVecChunk;
        const dim3 block(kQuads * (kSuperV / L));
        if (a.truncated)
            hipLaunchKernelGGL((k_gae_v4<true, L>), dim3((unsigned)vblocks), block, 0, s, a);
        else
            hipLaunchKernelGGL((k_gae_v4<false, L>), dim3((unsigned)vblocks), block, 0, s, a);
        return hipGetLastError();
    }
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
