// Generalised advantage estimation (on-policy ingestion derives returns and
// advantages, paper Sec. 2.2; GAE as used by PPO, Schulman et al.).
//
// The recursion A_t = delta_t + a_t A_{t+1}, a_t = gamma*lambda*(1 - d_t), is
// affine in A_{t+1}, so a chunk of consecutive steps composes into one map
// A_start = P * A_end + S, and so does any run of chunks.  Every kernel
//   1. folds each lane's chunk of steps into (P, S) (reverse order);
//   2. composes the chunks' maps with a suffix scan, so chunk c learns A at its
//      end, A_{t1(c)} = A_start(c + 1);
//   3. replays each chunk from that carry and writes A_t and R_t = A_t + V_t.
// All arithmetic is fp64; outputs are rounded to fp32 once.  plan_gae picks
// the kernels of a time-major call:
//   * tiles of 32 environments x 32 chunks: a rollout of at most 64 steps is
//     one tile per workgroup (k_gae_look with one segment); a longer one is
//     split along T into segments whose maps are joined by a decoupled
//     look-back in one launch (k_gae_look), or, beyond its table, by three
//     launches (k_gae_seg_*).  With E a multiple of 4 and aligned rows a lane
//     moves its 4 environments as 16-byte vectors, otherwise one by one (any
//     E, any alignment: the V4 template parameter);
//   * wide rollouts beyond the table: a workgroup owns 8 environments and
//     walks the rollout in passes of 2048 steps: k_gae_v4 gives each lane 4
//     environments as 16-byte vectors and 16 steps (128 chunks per pass); k_gae
//     (any E, any alignment) one environment and 32 steps (64 chunks per
//     pass), lanes fastest over environments so every load instruction reads
//     eight 32-byte runs.
// Padded sequences [B, Lmax] (k_gae_packed): one workgroup per sequence, 512
// chunks along t, scanned with DPP inside each wavefront.
#include <atomic>

#include <mutex>

#include "common.h"
#include "gae_plan.h"
#include "gae_packed_dev.h"

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

#ifndef CONDUIT_GAE_SPLIT_MAX_ENVS
#define CONDUIT_GAE_SPLIT_MAX_ENVS 4096
#endif
#ifndef CONDUIT_GAE_SPLIT_MIN_TILES
#define CONDUIT_GAE_SPLIT_MIN_TILES 256
#endif
constexpr int64_t kGaeSplitMaxEnvs = CONDUIT_GAE_SPLIT_MAX_ENVS;    // three-launch split below this many envs
constexpr int64_t kGaeSplitMinTiles = CONDUIT_GAE_SPLIT_MIN_TILES;  // one tile per compute unit before shorter chunks
constexpr int64_t kGaeSplitManyTiles = 1024;                         // from here on, chunks of 4 steps

// ---------------------------------------------------------------------------
// Time-major GAE split along T.  With few environments the kernels above run
// on E / 8 workgroups, each walking all T steps of its 8 columns, and every
// compute unit pulls whole 128-byte lines for 32-byte runs.  The split path
// cuts [T, E] into tiles of 32 environments (one 128-byte line of every float
// row) by Ts = 32 L steps, so every compute unit of the GPU takes a share, and
// joins the segments with the same affine composition as the chunks:
//   1. k_gae_seg_fold: tile (g, s >= 1) folds its segment into (P, S) per
//      environment, A_{row0(s)} = P A_{row0(s+1)} + S, and parks the pair as
//      four 32-bit words in rows row0(s-1) .. row0(s-1)+3 of ret (segment s-1
//      is a full segment; segment 0's map is never needed);
//   2. k_gae_seg_carry: per group of 32 environments, a suffix scan over the
//      parked maps gives A at the start of every segment s >= 1, i.e. the carry
//      of segment s-1, written as two words into rows row0(s-1), row0(s-1)+1 of
//      adv (A_T = 0 seeds it);
//   3. k_gae_seg_replay: tile (g, s) folds its chunks again, scans them, takes
//      its carry (0 for the last segment) and replays, writing adv and ret.
// Launches are ordered by the stream, each launch reads what the one before
// wrote, and a tile overwrites the parked words of its own segment only after
// every lane of the tile has read its carry, so no launch needs anything but
// the caller's arrays.
constexpr int kSegQuads = 8;                         // environment quads per tile
constexpr int kSegEnvs = kSegQuads * kV;             // 32 environments: one line per row
constexpr int kSegChunks = 32;                       // chunk lanes per tile
constexpr int kSegThreads = kSegQuads * kSegChunks;  // 256
constexpr int kSegWaves = kSegThreads / kWave;       // 4
constexpr int kChunksPerWave = kWave / kSegQuads;    // 8

// Affine maps of four environments: A_start = P * A_end + S.
struct Map4 {
    double P[kV], S[kV];
};

__device__ __forceinline__ Map4 map_identity() {
    Map4 m;
#pragma unroll
    for (int j = 0; j < kV; ++j) {
        m.P[j] = 1.0;
        m.S[j] = 0.0;
    }
    return m;
}

// f then g in time (f covers the earlier steps): A_start(f) = P_f (P_g A + S_g) + S_f
__device__ __forceinline__ Map4 map_compose(const Map4& f, const Map4& g) {
    Map4 r;
#pragma unroll
    for (int j = 0; j < kV; ++j) {
        r.S[j] = f.S[j] + f.P[j] * g.S[j];
        r.P[j] = f.P[j] * g.P[j];
    }
    return r;
}

// Lane layout of a tile: wavefront w holds chunks 8w .. 8w + 7 of all 8 quads,
// lane = quad * 8 + chunk % 8.  A quad's chunks of one wavefront are 8
// neighbouring lanes (a DPP row holds two quads), and every load instruction
// still reads 8 rows of 8 quads: 8 whole 128-byte lines.
__device__ __forceinline__ void seg_lane(int* q, int* c) {
    const int lane = (int)threadIdx.x % kWave;
    *q = lane / kChunksPerWave;
    *c = (int)(threadIdx.x / kWave) * kChunksPerWave + lane % kChunksPerWave;
}

// the maps of the lane N places up in the same DPP row (register moves only)
template <int N>
__device__ __forceinline__ Map4 map_from_lane_up(const Map4& m) {
    Map4 r;
#pragma unroll
    for (int j = 0; j < kV; ++j) {
        r.P[j] = __longlong_as_double(
            (long long)dpp_u64<kDppRowShl + N, 0xf, 0xf>((uint64_t)__double_as_longlong(m.P[j])));
        r.S[j] = __longlong_as_double(
            (long long)dpp_u64<kDppRowShl + N, 0xf, 0xf>((uint64_t)__double_as_longlong(m.S[j])));
    }
    return r;
}

// Suffix composition over the 32 chunks of a tile (lanes as in seg_lane).
// Returns, for chunk c, incl = map(c) o ... o map(31) and excl = map(c + 1) o
// ... o map(31) (the identity for chunk 31).  Hillis-Steele over the 8 lanes of
// a quad with DPP row shifts, one exchange of the wavefront totals through LDS
// and one barrier.
__device__ __forceinline__ void tile_suffix(const Map4& own, int c, int q, Map4* incl, Map4* excl) {
    __shared__ double sWP[kSegWaves][kSegQuads][kV];
    __shared__ double sWS[kSegWaves][kSegQuads][kV];
    const int cw = c % kChunksPerWave;
    Map4 in = own;
    {
        const Map4 nx = map_from_lane_up<1>(in);
        if (cw + 1 < kChunksPerWave) in = map_compose(in, nx);
    }
    {
        const Map4 nx = map_from_lane_up<2>(in);
        if (cw + 2 < kChunksPerWave) in = map_compose(in, nx);
    }
    {
        const Map4 nx = map_from_lane_up<4>(in);
        if (cw + 4 < kChunksPerWave) in = map_compose(in, nx);
    }
    Map4 ex = map_from_lane_up<1>(in);
    if (cw == kChunksPerWave - 1) ex = map_identity();
    const int w = c / kChunksPerWave;
    if (cw == 0) {
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            sWP[w][q][j] = in.P[j];
            sWS[w][q][j] = in.S[j];
        }
    }
    __syncthreads();
    Map4 later = map_identity();  // wavefronts w + 1 .. 3, in time order
#pragma unroll
    for (int v = kSegWaves - 1; v > 0; --v) {
        if (v > w) {
            Map4 t;
#pragma unroll
            for (int j = 0; j < kV; ++j) {
                t.P[j] = sWP[v][q][j];
                t.S[j] = sWS[v][q][j];
            }
            later = map_compose(t, later);
        }
    }
    *incl = map_compose(in, later);
    *excl = map_compose(ex, later);
}

// Tile coordinates: workgroups are dealt round-robin to the 8 XCDs; the ones on
// one XCD take consecutive tiles, i.e. neighbouring environment groups of one
// segment, which share the lines of the done rows.
__device__ __forceinline__ int64_t tile_of_block() {
    const int64_t nb = gridDim.x;
    return nb % 8 == 0 ? (int64_t)(blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8 : (int64_t)blockIdx.x;
}

// 16-byte vectors at 4-byte aligned addresses
typedef float f32x4u __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x4u __attribute__((ext_vector_type(4), aligned(4)));

// element j of the result is element min(j + sh, 3) of x (sh in 0..3)
__device__ __forceinline__ f32x4 shift_down(const f32x4& x, int sh) {
    f32x4 y;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int i = j + sh;
        y[j] = i <= 1 ? (i == 0 ? x[0] : x[1]) : (i == 2 ? x[2] : x[3]);
    }
    return y;
}

// four consecutive bytes at any address, byte k in bits 8k .. 8k + 7
__device__ __forceinline__ uint32_t bytes4(const uint8_t* p) {
    return (uint32_t)p[0] | (uint32_t)p[1] << 8 | (uint32_t)p[2] << 16 | (uint32_t)p[3] << 24;
}

// Loads and folds one lane's chunk: L steps from row t0 of the quad at column
// e0 (steps at or past T are skipped; their loads re-read row T - 1).  V4: the
// quad's four environments are one 16-byte aligned vector of every float row
// (E % 4 == 0, aligned rows; an inactive quad passes e0 = E - 4).  Otherwise
// (any E, any alignment; e0 is the quad's first column) every quad loads 16
// bytes per float row at 4-byte alignment, a quad reaching past E the row's
// last four columns, shifted down into place; with E < 4 each environment is
// loaded on its own.
template <bool TRUNC, int L, bool V4>
struct SegChunk {
    f32x4 r[L], v[L];
    uint32_t d[L];
    uint32_t tr[TRUNC ? L : 1];
    f32x4 fv[TRUNC ? L : 1];
    f32x4 ve;

    // c: the lane's chunk in the tile.  The value after the chunk's last step
    // (ve) is the next chunk's first value, which the next lane of the DPP row
    // loads anyway; the lane loads it itself only in a wavefront's last chunk
    // (c % 8 == 7) and past the rollout's end (the bootstrap).
    __device__ __forceinline__ void load(const GaeArgs& a, int64_t t0, int64_t e0, int c) {
        const int64_t E = a.E, T = a.T;
        const bool own = c % kChunksPerWave == kChunksPerWave - 1 || t0 + L >= T;
        ve = (f32x4)(0.0f);
        if constexpr (V4) {
#pragma unroll
            for (int k = 0; k < L; ++k) {
                const int64_t t = t0 + k < T ? t0 + k : T - 1;
                const int64_t o = t * E + e0;
                r[k] = *reinterpret_cast<const f32x4*>(a.reward + o);
                v[k] = a.value ? *reinterpret_cast<const f32x4*>(a.value + o) : (f32x4)(0.0f);
                d[k] = *reinterpret_cast<const uint32_t*>(a.done + o);
                if constexpr (TRUNC) {
                    tr[TRUNC ? k : 0] = *reinterpret_cast<const uint32_t*>(a.truncated + o);
                    fv[TRUNC ? k : 0] = *reinterpret_cast<const f32x4*>(a.final_value + o);
                }
            }
            const int64_t t1 = t0 + L;
            if (own) {
                if (t1 >= T) ve = a.bootstrap ? *reinterpret_cast<const f32x4*>(a.bootstrap + e0) : (f32x4)(0.0f);
                else ve = a.value ? *reinterpret_cast<const f32x4*>(a.value + t1 * E + e0) : (f32x4)(0.0f);
            }
        } else if (E >= kV) {
            // 16 bytes per float row at a 4-byte aligned address (dword
            // alignment is all a multi-dword load needs).  A quad reaching past
            // E loads the row's last four columns instead and shifts them down
            // (environment j of the quad is loaded column eb + j + sh; columns
            // past E take column E - 1), so every lane runs the same loads.
            const int64_t eb = e0 + kV <= E ? e0 : E - kV;
            const int sh = (int)(e0 - eb < kV ? e0 - eb : kV - 1);
#pragma unroll
            for (int k = 0; k < L; ++k) {
                const int64_t t = t0 + k < T ? t0 + k : T - 1;
                const int64_t o = t * E + eb;
                r[k] = *reinterpret_cast<const f32x4u*>(a.reward + o);
                v[k] = a.value ? *reinterpret_cast<const f32x4u*>(a.value + o) : (f32x4)(0.0f);
                d[k] = bytes4(a.done + o);
                if constexpr (TRUNC) {
                    tr[TRUNC ? k : 0] = bytes4(a.truncated + o);
                    fv[TRUNC ? k : 0] = *reinterpret_cast<const f32x4u*>(a.final_value + o);
                }
            }
            const int64_t t1 = t0 + L;
            if (own) {
                if (t1 >= T) ve = a.bootstrap ? *reinterpret_cast<const f32x4u*>(a.bootstrap + eb) : (f32x4)(0.0f);
                else ve = a.value ? *reinterpret_cast<const f32x4u*>(a.value + t1 * E + eb) : (f32x4)(0.0f);
            }
            if (sh) {
#pragma unroll
                for (int k = 0; k < L; ++k) {
                    r[k] = shift_down(r[k], sh);
                    v[k] = shift_down(v[k], sh);
                    d[k] >>= 8 * sh;
                    if constexpr (TRUNC) {
                        tr[TRUNC ? k : 0] >>= 8 * sh;
                        fv[TRUNC ? k : 0] = shift_down(fv[TRUNC ? k : 0], sh);
                    }
                }
                ve = shift_down(ve, sh);
            }
        } else {
            // fewer than four environments: each on its own, columns past E
            // re-reading column E - 1
            int64_t ec[kV];
#pragma unroll
            for (int j = 0; j < kV; ++j) ec[j] = e0 + j < E ? e0 + j : E - 1;
#pragma unroll
            for (int k = 0; k < L; ++k) {
                const int64_t t = t0 + k < T ? t0 + k : T - 1;
                const int64_t row = t * E;
                d[k] = 0u;
                if constexpr (TRUNC) tr[TRUNC ? k : 0] = 0u;
#pragma unroll
                for (int j = 0; j < kV; ++j) {
                    const int64_t o = row + ec[j];
                    r[k][j] = a.reward[o];
                    v[k][j] = a.value ? a.value[o] : 0.0f;
                    d[k] |= (uint32_t)a.done[o] << (8 * j);
                    if constexpr (TRUNC) {
                        tr[TRUNC ? k : 0] |= (uint32_t)a.truncated[o] << (8 * j);
                        fv[TRUNC ? k : 0][j] = a.final_value[o];
                    }
                }
            }
            const int64_t t1 = t0 + L;
            if (own) {
#pragma unroll
                for (int j = 0; j < kV; ++j) {
                    if (t1 >= T) ve[j] = a.bootstrap ? a.bootstrap[ec[j]] : 0.0f;
                    else ve[j] = a.value ? a.value[t1 * E + ec[j]] : 0.0f;
                }
            }
        }
        // the other lanes: the next lane's first value (row_shl:1 moves lane
        // i + 1 into lane i; every lane runs it, the loads above are in place)
        f32x4 up;
#pragma unroll
        for (int j = 0; j < kV; ++j)
            up[j] = __uint_as_float((uint32_t)__builtin_amdgcn_update_dpp(0, (int)__float_as_uint(v[0][j]),
                                                                          kDppRowShl + 1, 0xf, 0xf, true));
        if (!own) ve = up;
    }

    __device__ __forceinline__ void step(const GaeArgs& a, double gl, int k, int j, double vn, double* delta,
                                         double* m) const {
        gae_step<TRUNC>((double)r[k][j], (double)v[k][j], vn, (uint8_t)(d[k] >> (8 * j)),
                        TRUNC ? (uint8_t)(tr[TRUNC ? k : 0] >> (8 * j)) : 0, TRUNC ? fv[TRUNC ? k : 0][j] : 0.0f,
                        a.gamma, gl, delta, m);
    }

    // A_start = P A_end + S over the chunk's live steps
    __device__ __forceinline__ Map4 fold(const GaeArgs& a, double gl, int64_t t0) const {
        Map4 m = map_identity();
        double vn[kV];
#pragma unroll
        for (int j = 0; j < kV; ++j) vn[j] = (double)ve[j];
#pragma unroll
        for (int k = L - 1; k >= 0; --k) {
            if (t0 + k < a.T) {
#pragma unroll
                for (int j = 0; j < kV; ++j) {
                    double delta, mk;
                    step(a, gl, k, j, vn[j], &delta, &mk);
                    m.S[j] = delta + mk * m.S[j];
                    m.P[j] = mk * m.P[j];
                    vn[j] = (double)v[k][j];
                }
            }
        }
        return m;
    }
};

// The 32-bit words of a double, low word first.
__device__ __forceinline__ uint32_t dlo(double x) { return (uint32_t)__double_as_longlong(x); }
__device__ __forceinline__ uint32_t dhi(double x) { return (uint32_t)((uint64_t)__double_as_longlong(x) >> 32); }
__device__ __forceinline__ double dword2(uint32_t lo, uint32_t hi) {
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// One row of a tile's quad in a float array [T, E] (or its 32-bit words).  V4:
// one 16-byte aligned access at column e0 (stores only for active quads).
// Otherwise a quad inside [0, E) takes one 16-byte access at 4-byte alignment,
// and the quad reaching past E one access per environment: stores skip columns
// at or past E, loads re-read column E - 1 there.
template <bool V4>
__device__ __forceinline__ void put_quad(float* p, int64_t row, int64_t E, int64_t e0, bool active, const f32x4& x) {
    if constexpr (V4) {
        if (active) *reinterpret_cast<f32x4*>(p + row * E + e0) = x;
    } else if (e0 + kV <= E) {
        *reinterpret_cast<f32x4u*>(p + row * E + e0) = x;
    } else {
#pragma unroll
        for (int j = 0; j < kV; ++j)
            if (e0 + j < E) p[row * E + e0 + j] = x[j];
    }
}

template <bool V4>
__device__ __forceinline__ void put_words(float* p, int64_t row, int64_t E, int64_t e0, bool active, const u32x4& w) {
    if constexpr (V4) {
        if (active) *reinterpret_cast<u32x4*>(p + row * E + e0) = w;
    } else if (e0 + kV <= E) {
        *reinterpret_cast<u32x4u*>(p + row * E + e0) = w;
    } else {
#pragma unroll
        for (int j = 0; j < kV; ++j)
            if (e0 + j < E) reinterpret_cast<uint32_t*>(p)[row * E + e0 + j] = w[j];
    }
}

template <bool V4>
__device__ __forceinline__ u32x4 get_words(const float* p, int64_t row, int64_t E, int64_t e0) {
    if constexpr (V4) {
        return *reinterpret_cast<const u32x4*>(p + row * E + e0);
    } else if (e0 + kV <= E) {
        return *reinterpret_cast<const u32x4u*>(p + row * E + e0);
    } else {
        u32x4 w;
#pragma unroll
        for (int j = 0; j < kV; ++j) w[j] = reinterpret_cast<const uint32_t*>(p)[row * E + (e0 + j < E ? e0 + j : E - 1)];
        return w;
    }
}

// A tile quad's first column: V4 passes an inactive quad E - 4 (every access
// stays inside the row); the per-environment accesses clamp or skip on their own.
template <bool V4>
__device__ __forceinline__ int64_t quad_base(int64_t e_raw, int64_t E) {
    return V4 ? (e_raw < E ? e_raw : E - kV) : e_raw;
}

template <bool TRUNC, int L, bool V4>
__global__ __launch_bounds__(kSegThreads) void k_gae_seg_fold(GaeArgs a, int32_t groups) {
    constexpr int64_t Ts = (int64_t)kSegChunks * L;
    int q, c;
    seg_lane(&q, &c);
    const int64_t tile = tile_of_block();
    const int64_t g = tile % groups, s = 1 + tile / groups;
    const int64_t E = a.E;
    const int64_t e_raw = g * kSegEnvs + q * kV;
    const bool active = e_raw < E;
    const int64_t e0 = quad_base<V4>(e_raw, E);
    const int64_t t0 = s * Ts + (int64_t)c * L;
    SegChunk<TRUNC, L, V4> ch;
    ch.load(a, t0, e0, c);
    const Map4 own = ch.fold(a, a.gamma * a.lambda, t0);
    Map4 incl, excl;
    tile_suffix(own, c, q, &incl, &excl);
    if (c == 0 && active) {  // the segment's map, parked in rows row0(s - 1) + 0..3
        u32x4 w0, w1, w2, w3;
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            w0[j] = dlo(incl.P[j]);
            w1[j] = dhi(incl.P[j]);
            w2[j] = dlo(incl.S[j]);
            w3[j] = dhi(incl.S[j]);
        }
        const int64_t r0 = (s - 1) * Ts;
        put_words<V4>(a.ret, r0, E, e0, true, w0);
        put_words<V4>(a.ret, r0 + 1, E, e0, true, w1);
        put_words<V4>(a.ret, r0 + 2, E, e0, true, w2);
        put_words<V4>(a.ret, r0 + 3, E, e0, true, w3);
    }
}

// One workgroup per group of 32 environments; lanes as in seg_lane, chunk = segment, 32
// segments per pass, passes from the end with the carried A.
template <bool V4>
__global__ __launch_bounds__(kSegThreads) void k_gae_seg_carry(float* adv, const float* ret, int64_t E, int64_t Ts,
                                                              int64_t S) {
    __shared__ double s_carry[kSegQuads][kV];
    int q, c;
    seg_lane(&q, &c);
    const int64_t g = blockIdx.x;
    const int64_t e_raw = g * kSegEnvs + q * kV;
    const bool active = e_raw < E;
    const int64_t e0 = quad_base<V4>(e_raw, E);
    double carry[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) carry[j] = 0.0;  // A_T = 0
    // segments 1 .. S-1 in passes of 32 from the end: pass p covers
    // hi - 31 .. hi, chunk c takes segment hi - 31 + c (chunks below 1 idle)
    for (int64_t hi = S - 1; hi >= 1; hi -= kSegChunks) {
        const int64_t seg = hi - (kSegChunks - 1) + c;
        const bool live = seg >= 1;
        const int64_t sr = live ? seg : hi;  // idle lanes read a valid map
        const int64_t r0 = (sr - 1) * Ts;
        const u32x4 w0 = get_words<V4>(ret, r0, E, e0), w1 = get_words<V4>(ret, r0 + 1, E, e0);
        const u32x4 w2 = get_words<V4>(ret, r0 + 2, E, e0), w3 = get_words<V4>(ret, r0 + 3, E, e0);
        Map4 own;
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            own.P[j] = live ? dword2(w0[j], w1[j]) : 1.0;
            own.S[j] = live ? dword2(w2[j], w3[j]) : 0.0;
        }
        Map4 incl, excl;
        tile_suffix(own, c, q, &incl, &excl);
        double A[kV];
#pragma unroll
        for (int j = 0; j < kV; ++j) A[j] = incl.P[j] * carry[j] + incl.S[j];  // A at row0(seg)
        if (live && active) {
            u32x4 lo, hw;
#pragma unroll
            for (int j = 0; j < kV; ++j) {
                lo[j] = dlo(A[j]);
                hw[j] = dhi(A[j]);
            }
            put_words<V4>(adv, (seg - 1) * Ts, E, e0, true, lo);
            put_words<V4>(adv, (seg - 1) * Ts + 1, E, e0, true, hw);
        }
        if (hi - kSegChunks < 1) break;  // uniform
        // the next pass starts from A at row0(hi - 31), held by chunk c = 0
        if (c == 0) {
#pragma unroll
            for (int j = 0; j < kV; ++j) s_carry[q][j] = A[j];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kV; ++j) carry[j] = s_carry[q][j];
        __syncthreads();  // s_carry and the scan's LDS are rewritten by the next pass
    }
}

template <bool TRUNC, int L, bool V4>
__global__ __launch_bounds__(kSegThreads) void k_gae_seg_replay(GaeArgs a, int32_t groups, int64_t S) {
    constexpr int64_t Ts = (int64_t)kSegChunks * L;
    int q, c;
    seg_lane(&q, &c);
    const int64_t tile = tile_of_block();
    const int64_t g = tile % groups, s = tile / groups;
    const int64_t E = a.E, T = a.T;
    const int64_t e_raw = g * kSegEnvs + q * kV;
    const bool active = e_raw < E;
    const int64_t e0 = quad_base<V4>(e_raw, E);
    const int64_t row0 = s * Ts;
    const int64_t t0 = row0 + (int64_t)c * L;
    // the carry first: rows row0, row0 + 1 of adv are rewritten below
    u32x4 clo = (u32x4)(0u), chi = (u32x4)(0u);
    if (s + 1 < S) {
        clo = get_words<V4>(a.adv, row0, E, e0);
        chi = get_words<V4>(a.adv, row0 + 1, E, e0);
    }
    SegChunk<TRUNC, L, V4> ch;
    ch.load(a, t0, e0, c);
    const double gl = a.gamma * a.lambda;
    const Map4 own = ch.fold(a, gl, t0);
    double cin[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) cin[j] = dword2(clo[j], chi[j]);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // every load of this lane has returned
    Map4 incl, excl;
    tile_suffix(own, c, q, &incl, &excl);  // its barrier orders the carry reads before the stores
    double A[kV], vn[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) {
        A[j] = excl.P[j] * cin[j] + excl.S[j];  // A at the end of this chunk
        vn[j] = (double)ch.ve[j];
    }
#pragma unroll
    for (int k = L - 1; k >= 0; --k) {
        if (t0 + k < T) {
            f32x4 ao, ro;
#pragma unroll
            for (int j = 0; j < kV; ++j) {
                double delta, m;
                ch.step(a, gl, k, j, vn[j], &delta, &m);
                A[j] = delta + m * A[j];
                ao[j] = (float)A[j];
                ro[j] = (float)(A[j] + (double)ch.v[k][j]);
                vn[j] = (double)ch.v[k][j];
            }
            put_quad<V4>(a.adv, t0 + k, E, e0, active, ao);
            put_quad<V4>(a.ret, t0 + k, E, e0, active, ro);
        }
    }
}

// ---------------------------------------------------------------------------
// Time-major GAE split along T in one launch (decoupled look-back).  The tiles
// are those of the three-launch path, dealt in block order with the later
// segments first: a workgroup only ever waits for workgroups with smaller
// block indices, which the dispatcher has started before it, and those publish
// their segment's map without waiting for anyone.  A tile
//   1. folds its chunks and scans them (as k_gae_seg_replay);
//   2. publishes its segment's map (P, S), or, for the last segment, A at its
//      first step (A_T = 0), and raises its flag;
//   3. looks back over the later segments of its environment group in windows
//      of 32 (one per chunk lane): it waits for every flag of the window, takes
//      A where a segment has published it (the constant map P = 0, S = A) and
//      (P, S) otherwise, composes the window, and stops at the first window
//      that holds a published A or reaches the end of the rollout;
//   4. publishes A at its own first step when the rollout is longer than one
//      window (so that look-backs of earlier tiles stop early), then replays its
//      chunks from the carry.
// A rollout of one segment (at most 64 steps) skips steps 2 to 4: each tile
// folds, scans and replays its 32 environments alone.
// Maps and flags live in a small per-GPU table (static device memory, no
// allocation).  A flag holds the call's epoch next to its state, and every
// call takes a new epoch on the host, so nothing an earlier call left in the
// table is ever taken for this call's; a call enqueued under stream capture,
// whose epoch its graph replays repeat, first clears the flags with a
// one-workgroup kernel.  Calls that overlap on one GPU share the table and
// race; a wait that outlasts its bound gives up, flags ERR_GAE_WAIT and lets
// the kernel finish.  Every published value is written with agent-scope atomic
// stores and acknowledged before the flag is raised; readers use agent-scope
// atomic loads.
constexpr int kLookSpin = 1 << 15;  // polls of one flag before a wait gives up (tens of ms)
constexpr uint64_t kFlagMap = 1, kFlagA = 2;

// The per-GPU look-back table, plus the sticky error words of the
// allocation-free call (conduit_gae_noalloc).
struct LookTable {
    uint64_t flag[kLookMaxTiles];              // epoch << 2 | state
    uint64_t map[kLookMaxTiles][2][kSegEnvs];  // P, S of the segment (fp64 bits)
    uint64_t a[kLookMaxTiles][kSegEnvs];       // A at the segment's first step
    uint32_t err[kErrKinds];
};

// Its storage: static device memory, zero when the code object loads, never
// allocated, held by each GPU until the process ends (3.2 MB).  In host code
// the name below is only a host-side stand-in: every host use goes through the
// device address hipGetSymbolAddress returns for the current GPU (gae_table).
static __device__ __align__(256) uint8_t scratch[sizeof(LookTable)];

__global__ __launch_bounds__(kSegThreads) void k_gae_look_clear(LookTable* tab, int32_t tiles) {
    for (int i = threadIdx.x; i < tiles; i += kSegThreads)
        __hip_atomic_store(&tab->flag[i], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void put_f64(uint64_t* p, double x) {
    __hip_atomic_store(p, (uint64_t)__double_as_longlong(x), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double get_f64(uint64_t* p) {
    return __longlong_as_double((long long)__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

template <bool TRUNC, int L, bool V4>
__global__ __launch_bounds__(kSegThreads) void k_gae_look(GaeArgs a, LookTable* tab, int32_t groups, int32_t S,
                                                           uint64_t epoch) {
    constexpr int64_t Ts = (int64_t)kSegChunks * L;
    __shared__ double s_cin[kSegQuads][kV];
    int q, c;
    seg_lane(&q, &c);
    const int64_t s = S - 1 - (int64_t)(blockIdx.x / (uint32_t)groups);  // later segments first
    const int64_t g = blockIdx.x % (uint32_t)groups;
    const int64_t me = s * groups + g;  // table row of this tile
    const int64_t E = a.E, T = a.T;
    const int64_t e_raw = g * kSegEnvs + q * kV;
    const bool active = e_raw < E;
    const int64_t e0 = quad_base<V4>(e_raw, E);
    const int64_t t0 = s * Ts + (int64_t)c * L;
    const double gl = a.gamma * a.lambda;
    SegChunk<TRUNC, L, V4> ch;
    ch.load(a, t0, e0, c);
    const Map4 own = ch.fold(a, gl, t0);
    Map4 incl, excl;
    tile_suffix(own, c, q, &incl, &excl);  // incl of chunk 0: the segment's map
    const bool last = s == S - 1;
    if (c == 0 && S > 1) {  // lanes 0..7 of wavefront 0, one per quad; one segment publishes nothing
#pragma unroll
        for (int j = 0; j < kV; ++j) {
            if (last) {
                put_f64(&tab->a[me][q * kV + j], incl.S[j]);
            } else {
                put_f64(&tab->map[me][0][q * kV + j], incl.P[j]);
                put_f64(&tab->map[me][1][q * kV + j], incl.S[j]);
            }
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // acknowledged device-wide
        if (q == 0)
            __hip_atomic_store(&tab->flag[me], epoch << 2 | (last ? kFlagA : kFlagMap), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
    if (!last) {  // uniform
        Map4 acc = map_identity();  // the windows so far, in time order (chunk-0 lanes)
        for (int64_t w0 = s + 1;; w0 += kSegChunks) {
            const int64_t sj = w0 + c;
            Map4 m = map_identity();
            int stop = 0;
            if (sj < S) {
                const int64_t j = sj * groups + g;
                uint64_t f = 0;
                for (int it = 0; it < kLookSpin; ++it) {
                    const uint64_t w = __hip_atomic_load(&tab->flag[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    // the 8 quads of a segment take quad 0's reading (lane
                    // chunk % 8), so they agree on where their chains end
                    f = (uint64_t)__shfl((int)((w >> 2) == epoch ? (w & 3) : 0), (int)(threadIdx.x % kChunksPerWave),
                                         kWave);
                    if (f) break;
                    __builtin_amdgcn_s_sleep(2);
                }
                if (f == kFlagMap) {
#pragma unroll
                    for (int jj = 0; jj < kV; ++jj) {
                        m.P[jj] = get_f64(&tab->map[j][0][q * kV + jj]);
                        m.S[jj] = get_f64(&tab->map[j][1][q * kV + jj]);
                    }
                } else {
                    // A published (or the wait gave up: flagged, A taken as 0)
#pragma unroll
                    for (int jj = 0; jj < kV; ++jj) {
                        m.P[jj] = 0.0;
                        m.S[jj] = f == kFlagA ? get_f64(&tab->a[j][q * kV + jj]) : 0.0;
                    }
                    if (f != kFlagA && q == 0) flag_error(a.err, ERR_GAE_WAIT);
                    stop = 1;
                }
            } else {
                stop = 1;  // past the last step: A_T = 0
            }
            __syncthreads();  // the scan's LDS is free again
            Map4 wi, we;
            tile_suffix(m, c, q, &wi, &we);
            acc = map_compose(acc, wi);
            if (__syncthreads_or(stop)) break;
        }
        // A at the end of this segment is acc applied to 0 (a constant map ends
        // every window chain); A at its first step goes to the table when some
        // look-back window does not reach the end of the rollout
        if (c == 0) {
#pragma unroll
            for (int j = 0; j < kV; ++j) s_cin[q][j] = acc.S[j];
            if (S > kSegChunks + 1) {
#pragma unroll
                for (int j = 0; j < kV; ++j) put_f64(&tab->a[me][q * kV + j], incl.P[j] * acc.S[j] + incl.S[j]);
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                if (q == 0)
                    __hip_atomic_store(&tab->flag[me], epoch << 2 | kFlagA, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    } else if (c == 0) {
#pragma unroll
        for (int j = 0; j < kV; ++j) s_cin[q][j] = 0.0;  // A_T = 0
    }
    __syncthreads();
    // A and R leave through write-through buffer stores at agent scope (no
    // dirty lines for the end-of-kernel write-back: 8.9 -> 8.7 us on
    // [2048, 256]) where the byte offsets fit a buffer store
    const bool wt = T * E * 4 <= 0x7fffffffll;  // uniform
    const int nrec = wt ? (int)(T * E * 4) : 0;
    const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc(a.adv, 0, nrec, kRsrcRaw32);
    const __amdgpu_buffer_rsrc_t rsr = __builtin_amdgcn_make_buffer_rsrc(a.ret, 0, nrec, kRsrcRaw32);
    double A[kV], vn[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) {
        A[j] = excl.P[j] * s_cin[q][j] + excl.S[j];  // A at the end of this chunk
        vn[j] = (double)ch.ve[j];
    }
#pragma unroll
    for (int k = L - 1; k >= 0; --k) {
        if (t0 + k < T) {
            f32x4 ao, ro;
#pragma unroll
            for (int j = 0; j < kV; ++j) {
                double delta, m;
                ch.step(a, gl, k, j, vn[j], &delta, &m);
                A[j] = delta + m * A[j];
                ao[j] = (float)A[j];
                ro[j] = (float)(A[j] + (double)ch.v[k][j]);
                vn[j] = (double)ch.v[k][j];
            }
            if (V4 && wt) {
                if (active) {
                    const int off = (int)(((t0 + k) * E + e0) * 4);
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, ao), rsa, off, 0, kAgentScopeStore);
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, ro), rsr, off, 0, kAgentScopeStore);
                }
            } else {
                put_quad<V4>(a.adv, t0 + k, E, e0, active, ao);
                put_quad<V4>(a.ret, t0 + k, E, e0, active, ro);
            }
        }
    }
}

__global__ __launch_bounds__(kPkThreads) void k_gae_packed(GaePackedArgs a) {
    const int64_t b = blockIdx.x;
    int64_t L = a.length[b];
    if (L < 0 || L > a.Lmax) {
        if (threadIdx.x == 0) flag_error(a.err, ERR_SEQ_LENGTH);
        L = L < 0 ? 0 : a.Lmax;
    }
    gae_packed_row<kPkThreads>(a, b, L, (double)a.last_reward[b]);
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

template <bool TRUNC, int L, bool V4>
hipError_t launch_gae_split_t(const GaeArgs& a, int64_t groups, hipStream_t s) {
    constexpr int64_t Ts = (int64_t)kSegChunks * L;
    const int64_t S = (a.T + Ts - 1) / Ts;
    const dim3 block(kSegThreads);
    hipLaunchKernelGGL((k_gae_seg_fold<TRUNC, L, V4>), dim3((unsigned)(groups * (S - 1))), block, 0, s, a,
                       (int32_t)groups);
    hipLaunchKernelGGL(k_gae_seg_carry<V4>, dim3((unsigned)groups), block, 0, s, a.adv, a.ret, a.E, Ts, S);
    hipLaunchKernelGGL((k_gae_seg_replay<TRUNC, L, V4>), dim3((unsigned)(groups * S)), block, 0, s, a,
                       (int32_t)groups, S);
    return hipGetLastError();
}

template <bool TRUNC, bool V4>
hipError_t launch_gae_split_l(const GaeArgs& a, int64_t groups, int L, hipStream_t s) {
    switch (L) {
        case 8: return launch_gae_split_t<TRUNC, 8, V4>(a, groups, s);
        case 4: return launch_gae_split_t<TRUNC, 4, V4>(a, groups, s);
        default: return launch_gae_split_t<TRUNC, 2, V4>(a, groups, s);
    }
}

hipError_t launch_gae_split(const GaeArgs& a, int64_t groups, int L, bool v4, hipStream_t s) {
    if (v4)
        return a.truncated ? launch_gae_split_l<true, true>(a, groups, L, s)
                           : launch_gae_split_l<false, true>(a, groups, L, s);
    return a.truncated ? launch_gae_split_l<true, false>(a, groups, L, s)
                       : launch_gae_split_l<false, false>(a, groups, L, s);
}

template <bool TRUNC, bool V4>
hipError_t launch_gae_look_l(const GaeArgs& a, LookTable* tab, int32_t groups, int32_t S, int L, uint64_t ep,
                             hipStream_t s) {
    const dim3 grid((unsigned)(groups * S)), block(kSegThreads);
    switch (L) {
        case 8: hipLaunchKernelGGL((k_gae_look<TRUNC, 8, V4>), grid, block, 0, s, a, tab, groups, S, ep); break;
        case 4: hipLaunchKernelGGL((k_gae_look<TRUNC, 4, V4>), grid, block, 0, s, a, tab, groups, S, ep); break;
        default: hipLaunchKernelGGL((k_gae_look<TRUNC, 2, V4>), grid, block, 0, s, a, tab, groups, S, ep); break;
    }
    return hipGetLastError();
}

std::atomic<uint64_t> g_look_epoch{0};  // epochs of the look-back table, 1, 2, ... (62 bits)

// Device address of the current GPU's table, found once per GPU (with that GPU
// current) and kept for the process.
constexpr int kMaxGpus = 64;
static std::mutex g_table_mu;
static LookTable* g_table[kMaxGpus] = {};

static hipError_t gae_table(LookTable** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxGpus) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_table_mu);
    if (!g_table[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_table[dev] = static_cast<LookTable*>(p);
    }
    *out = g_table[dev];
    return hipSuccess;
}

hipError_t launch_gae_look(const GaeArgs& a, int32_t groups, int32_t S, int L, bool v4, hipStream_t s) {
    // one segment (the short path) uses no table; split rollouts at most the
    // table's tiles (the plan never asks for more)
    if (S > 1 && (int64_t)groups * S > kLookMaxTiles) return hipErrorInvalidValue;
    LookTable* tab = nullptr;
    hipError_t e = gae_table(&tab);
    if (e != hipSuccess) return e;
    const uint64_t ep = (g_look_epoch.fetch_add(1) + 1) & ((1ull << 62) - 1);
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    e = hipStreamIsCapturing(s, &cap);
    if (e != hipSuccess) return e;
    if (S > 1 && cap != hipStreamCaptureStatusNone) {  // replays repeat the epoch: clear the flags first
        hipLaunchKernelGGL(k_gae_look_clear, dim3(1), dim3(kSegThreads), 0, s, tab, groups * S);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (v4)
        return a.truncated ? launch_gae_look_l<true, true>(a, tab, groups, S, L, ep, s)
                           : launch_gae_look_l<false, true>(a, tab, groups, S, L, ep, s);
    return a.truncated ? launch_gae_look_l<true, false>(a, tab, groups, S, L, ep, s)
                       : launch_gae_look_l<false, false>(a, tab, groups, S, L, ep, s);
}

hipError_t gae_noalloc_err_words(uint32_t** err) {
    LookTable* tab = nullptr;
    hipError_t e = gae_table(&tab);
    if (e == hipSuccess) *err = tab->err;
    return e;
}

hipError_t gae_noalloc_read_errors(uint32_t* host_words) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    LookTable* tab = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_table_mu);
        tab = dev >= 0 && dev < kMaxGpus ? g_table[dev] : nullptr;
    }
    if (!tab) {  // no allocation-free call on this GPU yet: nothing flagged
        for (int k = 0; k < kErrKinds; ++k) host_words[k] = 0;
        return hipSuccess;
    }
    return hipMemcpy(host_words, tab->err, sizeof(uint32_t) * kErrKinds, hipMemcpyDeviceToHost);
}

hipError_t gae_noalloc_clear_errors() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    LookTable* tab = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_table_mu);
        tab = dev >= 0 && dev < kMaxGpus ? g_table[dev] : nullptr;
    }
    if (!tab) return hipSuccess;
    const uint32_t zero[kErrKinds] = {};
    return hipMemcpy(tab->err, zero, sizeof(zero), hipMemcpyHostToDevice);
}

GaePlan plan_gae(int64_t T, int64_t E, bool vec) {
    GaePlan p{vec ? GAE_ONE_PASS_V4 : GAE_ONE_PASS, 0, 0, 0};
    if (T <= 0 || E <= 0) return p;
    // split along T: the longest chunk that still gives every compute unit a
    // tile, at least two segments; chunks of 4 steps where that still gives
    // 1,024 to 4,096 tiles (a tile of 8-step chunks holds 288 registers per
    // lane, one workgroup per compute unit, too few in flight for large
    // rollouts)
    const int64_t groups = (E + kSegEnvs - 1) / kSegEnvs;
    // a rollout of at most 64 steps is one segment of 2-step chunks: no table
    // and no waiting, so any number of tiles
    if (T <= (int64_t)kSegChunks * 2) return GaePlan{GAE_SHORT, 2, groups, 1};
    auto segs_of = [&](int L) { return (T + (int64_t)kSegChunks * L - 1) / ((int64_t)kSegChunks * L); };
    int L = 0;
    for (int cand : {8, 4, 2}) {
        if (segs_of(cand) >= 2 && (groups * segs_of(cand) >= kGaeSplitMinTiles || cand == 2)) {
            L = cand;
            break;
        }
    }
    if (L == 8 && groups * segs_of(4) >= kGaeSplitManyTiles && groups * segs_of(4) <= kLookMaxTiles) L = 4;
    if (!L) return p;
    const int64_t segs = segs_of(L);
    if (groups * segs <= kLookMaxTiles) return GaePlan{GAE_LOOK_BACK, L, groups, segs};
    // beyond the table: three launches for narrow rollouts; wide ones keep one
    // workgroup per 8 environments, which already fills the GPU
    if (E < kGaeSplitMaxEnvs) return GaePlan{GAE_THREE_LAUNCHES, L, groups, segs};
    return p;
}

hipError_t launch_gae(const GaeArgs& a, hipStream_t s) {
    if (a.T <= 0 || a.E <= 0) return hipSuccess;
    if (a.E > kGaeMaxEnvs) return hipErrorInvalidValue;  // the ABI rejects this first
    auto al = [](const void* p, uintptr_t m) { return (reinterpret_cast<uintptr_t>(p) & (m - 1)) == 0; };
    const bool vec = a.E % kV == 0 && al(a.reward, 16) && al(a.value, 16) && al(a.bootstrap, 16) &&
                     al(a.adv, 16) && al(a.ret, 16) && al(a.done, 4) && al(a.truncated, 4) &&
                     al(a.final_value, 16);
    const GaePlan p = plan_gae(a.T, a.E, vec);
    switch (p.path) {
        case GAE_SHORT:
        case GAE_LOOK_BACK: return launch_gae_look(a, (int32_t)p.groups, (int32_t)p.segments, p.chunk, vec, s);
        case GAE_THREE_LAUNCHES: return launch_gae_split(a, p.groups, p.chunk, vec, s);
        case GAE_ONE_PASS_V4: {
            const int64_t vblocks = (a.E + kEnvsV - 1) / kEnvsV;
            constexpr int L = kGaeVecChunk;
            const dim3 block(kQuads * (kSuperV / L));
            if (a.truncated)
                hipLaunchKernelGGL((k_gae_v4<true, L>), dim3((unsigned)vblocks), block, 0, s, a);
            else
                hipLaunchKernelGGL((k_gae_v4<false, L>), dim3((unsigned)vblocks), block, 0, s, a);
            return hipGetLastError();
        }
        default: {
            const int64_t blocks = (a.E + kEnvs - 1) / kEnvs;
            if (a.truncated)
                hipLaunchKernelGGL(k_gae<true>, dim3((unsigned)blocks), dim3(kTmThreads), 0, s, a);
            else
                hipLaunchKernelGGL(k_gae<false>, dim3((unsigned)blocks), dim3(kTmThreads), 0, s, a);
            return hipGetLastError();
        }
    }
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
