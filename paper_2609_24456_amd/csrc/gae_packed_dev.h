// Generalised advantage estimation over packed (right-padded) sequences, one
// workgroup per sequence: shared by the packed GAE kernel (512 lanes) and the
// fused sampler + packing + GAE kernel (its pack workgroup as it is).
#pragma once
#include "common.h"

namespace conduit {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kRsrcRaw32 = 0x00020000;  // raw buffer descriptor, 32-bit data format
constexpr int kAgentScopeStore = 16;    // cache policy SC1: written through at agent scope

// Lanes of the stand-alone packed GAE kernel.  A sequence of 4,096 elements
// as 512 lanes x 8 (against 256 x 16): [256, 4096] 6.9 -> 5.5 us, [1024, 4096]
// 13.2 -> 11.8 us, [256, 1024] 6.0 -> 4.7 us; 1,024 lanes x 4 gains at 256
// rows (5.9 us) but loses at 1,024 (18.7 us).
constexpr int kPkThreads = 512;
constexpr int kPkSeg = 4096;                      // elements per pass
constexpr int kPkPad = kPkSeg + kPkSeg / 16 + 1;  // padded LDS row

// padded LDS index: one spare word every 16, so lanes reading their own
// contiguous chunk of up to 16 hit distinct banks
__device__ __forceinline__ int lpad(int t) { return t + (t >> 4); }

// GAE over right-padded sequences, one workgroup per sequence, walked in
// segments of 4096 elements from the end with a carry.  Values are staged into
// LDS with coalesced loads, each lane owns a contiguous chunk of 16 for the scan,
// and advantages/returns are staged back and written coalesced.
// A double moved by one DPP control; lanes with no source keep `id`.
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64(double x, double id) {
    const uint64_t b = (uint64_t)__double_as_longlong(x), o = (uint64_t)__double_as_longlong(id);
    const uint32_t lo =
        (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)o, (int)(uint32_t)b, CTRL, ROWS, 0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(o >> 32), (int)(uint32_t)(b >> 32),
                                                              CTRL, ROWS, 0xf, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// One step of a wavefront prefix scan of affine maps whose lanes run backwards
// in time: the source lane (lower) covers later steps than this one.
template <int CTRL, int ROWS>
__device__ __forceinline__ void later_scan_step(double& P, double& S) {
    const double p2 = dpp_f64<CTRL, ROWS>(P, 1.0);
    const double s2 = dpp_f64<CTRL, ROWS>(S, 0.0);
    S = S + P * s2;
    P = P * p2;
}

constexpr int kDppWaveShr1 = 0x138;  // lane i reads lane i - 1 across the whole wavefront

// g^e (e >= 0) by binary exponentiation in fp64
__device__ __forceinline__ double pow_int(double g, int64_t e) {
    double r = 1.0;
    for (; e; e >>= 1, g *= g)
        if (e & 1) r *= g;
    return r;
}

// A packed row without values (V = 0): the only non-zero TD residual is the
// last live element's reward R, so A_t = R (gamma lambda)^(L-1-t) for t < L,
// 0 beyond, and R_t = A_t.  Each lane takes 16-byte vectors of the row: the
// vector's last live element from the closed form, the ones before it by the
// recursion's own step A_t = gamma lambda A_{t+1}.  No element waits for
// another lane: no scan, no barrier, no LDS.
template <int NT>
__device__ void gae_packed_row_novalue(const GaePackedArgs& a, int64_t b, int64_t L, double R) {
    const int64_t Lmax = a.Lmax;
    float* adv = a.adv + b * Lmax;
    float* ret = a.ret + b * Lmax;
    const double gl = a.gamma * a.lambda;
    // the values of elements [t, t + 4): o[i] for t + i
    auto quad = [&](int64_t t, f32x4& o) {
        const int64_t hi = (t + 3 < L - 1 ? t + 3 : L - 1);  // last live element of the quad
        double A = hi >= t ? R * pow_int(gl, L - 1 - hi) : 0.0;
#pragma unroll
        for (int i = 3; i >= 0; --i) {
            if (t + i > hi) {
                o[i] = 0.0f;
            } else {
                if (t + i < hi) A = gl * A;
                o[i] = (float)A;
            }
        }
    };
    const bool vec = ((reinterpret_cast<uintptr_t>(adv) | reinterpret_cast<uintptr_t>(ret)) & 15) == 0 &&
                     (Lmax & 3) == 0 && Lmax * 4 <= 0x7fffffffll;  // uniform
    if (vec) {
        const int nb = __builtin_amdgcn_readfirstlane((int)(Lmax * 4));
        const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(adv, 0, nb, kRsrcRaw32);
        const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(ret, 0, nb, kRsrcRaw32);
        for (int64_t t = (int64_t)threadIdx.x * 4; t < Lmax; t += (int64_t)NT * 4) {
            f32x4 o;
            quad(t, o);
            // write-through at agent scope, as the scanned path stores its rows
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o), ra, (int)(t * 4), 0, kAgentScopeStore);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, o), rr, (int)(t * 4), 0, kAgentScopeStore);
        }
    } else {
        for (int64_t t = (int64_t)threadIdx.x * 4; t < Lmax; t += (int64_t)NT * 4) {
            f32x4 o;
            quad(t, o);
            for (int i = 0; i < 4 && t + i < Lmax; ++i) {
                adv[t + i] = o[i];
                ret[t + i] = o[i];
            }
        }
    }
}

// GAE of packed row b, of L live elements (0 <= L <= Lmax) with reward R on
// the last one, by one workgroup of NT lanes (each lane a chunk of 4096 / NT
// consecutive elements per pass).
template <int NT>
__device__ void gae_packed_row(const GaePackedArgs& a, int64_t b, int64_t L, double R) {
    if (!a.value) {  // kernel argument: uniform
        gae_packed_row_novalue<NT>(a, b, L, R);
        return;
    }
    static_assert(NT % kWave == 0 && kPkSeg % (4 * NT) == 0 && kPkSeg / NT <= 16, "lanes per sequence");
    constexpr int kPkChunk = kPkSeg / NT;  // elements per lane and pass
    __shared__ float sV[kPkPad];
    __shared__ float sA[kPkPad];
    __shared__ float sR[kPkPad];
    __shared__ double sWP[NT / kWave];
    __shared__ double sWS[NT / kWave];
    const int tid = threadIdx.x;
    // chunks run backwards inside a wavefront (lane 0 holds its last chunk), so
    // the suffix composition over the chunks is a prefix scan over the lanes
    const int wv = tid / kWave, lane = tid % kWave;
    const int c = wv * kWave + (kWave - 1 - lane);
    const int64_t Lmax = a.Lmax;
    const float* val = a.value ? a.value + b * Lmax : nullptr;
    float* adv = a.adv + b * Lmax;
    float* ret = a.ret + b * Lmax;
    // 16-byte vectors for the value loads and the output stores when the rows
    // allow them (uniform)
    auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    const bool vec_in = val && al16(val);
    const bool vec_out = al16(adv) && al16(ret);
    const double gl = a.gamma * a.lambda;
    double carry = 0.0;    // A at the start of the later segment
    double v_after = 0.0;  // V at the start of the later segment
    const int64_t segs = (Lmax + kPkSeg - 1) / kPkSeg;
    for (int64_t sg = segs - 1; sg >= 0; --sg) {
        const int64_t base = sg * kPkSeg;
        const int seg_len = (int)(Lmax - base < kPkSeg ? Lmax - base : kPkSeg);
        if (vec_in) {
            // every lane's 4 vectors are loaded before the first LDS write
            constexpr int kVecs = kPkSeg / (4 * NT);
            f32x4 q[kVecs];
#pragma unroll
            for (int j = 0; j < kVecs; ++j) {
                const int t = (j * NT + tid) * 4;
                if (t + 3 < seg_len) {
                    q[j] = *reinterpret_cast<const f32x4*>(val + base + t);
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) q[j][i] = t + i < seg_len ? val[base + t + i] : 0.0f;
                }
            }
#pragma unroll
            for (int j = 0; j < kVecs; ++j) {
                const int t = (j * NT + tid) * 4;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (t + i < seg_len) sV[lpad(t + i)] = q[j][i];
            }
        } else {
            for (int t = tid; t < seg_len; t += NT) sV[lpad(t)] = val ? val[base + t] : 0.0f;
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
        // suffix composition over the chunks: a DPP prefix scan inside each
        // wavefront (shifts by 1, 2, 4, 8 in a row, then the row broadcasts),
        // the wavefront totals through LDS, one barrier
        double iP = P, iS = S;  // chunks c .. the wavefront's last
        later_scan_step<kDppRowShr + 1, 0xf>(iP, iS);
        later_scan_step<kDppRowShr + 2, 0xf>(iP, iS);
        later_scan_step<kDppRowShr + 4, 0xf>(iP, iS);
        later_scan_step<kDppRowShr + 8, 0xf>(iP, iS);
        later_scan_step<kDppRowBcast15, 0xa>(iP, iS);
        later_scan_step<kDppRowBcast31, 0xc>(iP, iS);
        const double eP = dpp_f64<kDppWaveShr1, 0xf>(iP, 1.0);  // chunks c + 1 .. the last
        const double eS = dpp_f64<kDppWaveShr1, 0xf>(iS, 0.0);
        if (lane == kWave - 1) {
            sWP[wv] = iP;
            sWS[wv] = iS;
        }
        __syncthreads();
        double lP = 1.0, lS = 0.0;  // the later wavefronts' chunks
        double tP = 1.0, tS = 0.0;  // the whole segment
#pragma unroll
        for (int w = NT / kWave - 1; w >= 0; --w) {
            tS = sWS[w] + sWP[w] * tS;
            tP = sWP[w] * tP;
            if (w == wv + 1) {
                lP = tP;
                lS = tS;
            }
        }
        double A = eP * (lP * carry + lS) + eS;  // A at the end of this chunk
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
            constexpr int kVecs = kPkSeg / (4 * NT);
            // write-through buffer stores at agent scope over this segment (the
            // rows leave no dirty lines for the end-of-kernel write-back: 7.95
            // -> 7.26 us for [256, 4096], the tokens iteration 22.7 -> 22.0 us)
            const int nb = __builtin_amdgcn_readfirstlane(seg_len * 4);
            const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(adv + base, 0, nb, kRsrcRaw32);
            const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(ret + base, 0, nb, kRsrcRaw32);
#pragma unroll
            for (int j = 0; j < kVecs; ++j) {
                const int t = (j * NT + tid) * 4;
                if (t + 3 < seg_len) {
                    f32x4 oa, orr;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        oa[i] = sA[lpad(t + i)];
                        orr[i] = sR[lpad(t + i)];
                    }
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, oa), ra, t * 4, 0, kAgentScopeStore);
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, orr), rr, t * 4, 0, kAgentScopeStore);
                } else {
                    for (int i = 0; i < 4 && t + i < seg_len; ++i) {
                        adv[base + t + i] = sA[lpad(t + i)];
                        ret[base + t + i] = sR[lpad(t + i)];
                    }
                }
            }
        } else {
            for (int t = tid; t < seg_len; t += NT) {
                adv[base + t] = sA[lpad(t)];
                ret[base + t] = sR[lpad(t)];
            }
        }
        carry = tP * carry + tS;
        v_after = (double)sV[lpad(0)];
        __syncthreads();  // LDS is rewritten by the next segment
    }
}

}  // namespace
}  // namespace conduit
