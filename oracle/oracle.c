/*
 * Reference oracle for the experience path.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU implementation of what the experience path
 * computes.  Only the test suite, the smoke check and the benchmark's CPU-baseline
 * leg may load it.  The product library never links, calls or includes it, and the
 * two share no code (no headers, helpers, tables or constants).
 *
 * What is computed, and where it comes from:
 *   - The paper (Sec. 2.2, the responsibilities of the experience path) names the operations:
 *     off-policy ingestion adds transitions to a long-lived replay store and keeps
 *     the per-slot bookkeeping that sampling and eviction need; off-policy
 *     delivery draws from it, builds the batch and changes its layout; on-policy
 *     ingestion derives returns and advantages; on-policy delivery partitions
 *     a rollout into shuffled minibatches; processing operators include
 *     concat/stack, reshape, sampling, shuffling, batching and padding/packing of
 *     variable-length sequences.  Tuples carry episode IDs (Sec. 2.1).
 *   - App. C, Invariant 2: replay priorities are updated by algorithm callbacks.
 *   - The mathematics is the one of the works the paper cites for these
 *     operations: proportional prioritised replay (Schaul et al.), truncated
 *     generalised advantage estimation as used by PPO (Schulman et al.) and the
 *     4-frame observation stack of DQN (Mnih et al.).
 *   - Points the paper leaves open are fixed by the readings listed in the design
 *     notes (leaf quantiser, stratified targets, batch-max IS normalisation,
 *     frame-stack validity, done/bootstrap alignment, token padding).
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fused multiply-add, so every
 * float/double operation below is one IEEE operation with round-to-nearest-even).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

/* ------------------------------------------------------------------------- */
/* Exact leaf quantiser  L(p) = floor(2^F * p^(a/b))                          */
/* ------------------------------------------------------------------------- */
/*
 * Proportional prioritisation uses p^alpha.  To make sampled indices exactly
 * reproducible the leaf stored for priority p (an unsigned 32-bit integer) is the
 * integer  floor(2^F * p^(a/b))  with alpha = a/b rational, b <= 8, and
 * F = min(31, floor(32 (b - a) / b)) fractional bits, which keeps every leaf below
 * 2^32.  It is the unique q with  q^b <= 2^(bF) * p^a < (q+1)^b; this oracle finds
 * it by bisection over [0, 2^32) with exact multi-word integer comparisons.
 */

#define ORC_WORDS 6 /* 384 bits; the largest operand is below 2^256 */

typedef struct { uint64_t w[ORC_WORDS]; } orc_big;

static void big_from(orc_big* x, uint64_t v) {
    memset(x, 0, sizeof(*x));
    x->w[0] = v;
}

static void big_mul_u64(orc_big* x, uint64_t m) {
    u128 carry = 0;
    for (int i = 0; i < ORC_WORDS; ++i) {
        u128 t = (u128)x->w[i] * m + carry;
        x->w[i] = (uint64_t)t;
        carry = t >> 64;
    }
}

static void big_shift_left(orc_big* x, int bits) {
    while (bits >= 64) {
        for (int i = ORC_WORDS - 1; i > 0; --i) x->w[i] = x->w[i - 1];
        x->w[0] = 0;
        bits -= 64;
    }
    if (bits > 0) {
        for (int i = ORC_WORDS - 1; i > 0; --i)
            x->w[i] = (x->w[i] << bits) | (x->w[i - 1] >> (64 - bits));
        x->w[0] <<= bits;
    }
}

static int big_cmp(const orc_big* x, const orc_big* y) {
    for (int i = ORC_WORDS - 1; i >= 0; --i) {
        if (x->w[i] < y->w[i]) return -1;
        if (x->w[i] > y->w[i]) return 1;
    }
    return 0;
}

int32_t orc_frac_bits(int32_t a, int32_t b) {
    int32_t f = (32 * (b - a)) / b;
    return f > 31 ? 31 : f;
}

uint32_t orc_leaf(uint32_t p, int32_t a, int32_t b) {
    if (p == 0) return 0;
    int32_t F = orc_frac_bits(a, b);
    orc_big rhs; /* 2^(bF) * p^a */
    big_from(&rhs, 1);
    for (int32_t i = 0; i < a; ++i) big_mul_u64(&rhs, p);
    big_shift_left(&rhs, b * F);
    uint64_t lo = 0, hi = (uint64_t)1 << 32; /* lo^b <= rhs < hi^b */
    while (hi - lo > 1) {
        uint64_t mid = lo + (hi - lo) / 2;
        orc_big lhs;
        big_from(&lhs, 1);
        for (int32_t i = 0; i < b; ++i) big_mul_u64(&lhs, mid);
        if (big_cmp(&lhs, &rhs) <= 0) lo = mid; else hi = mid;
    }
    return (uint32_t)lo;
}

/* L(p) for n priorities (a loop over orc_leaf) */
void orc_leaf_many(const uint32_t* p, int64_t n, int32_t a, int32_t b, uint32_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = orc_leaf(p[i], a, b);
}

/* ------------------------------------------------------------------------- */
/* Replay dataset                                                             */
/* ------------------------------------------------------------------------- */
/* Every array is owned by the caller; the struct only points at it. */
typedef struct {
    /* configuration */
    int64_t capacity;        /* slots */
    int64_t row_bytes;       /* bytes of one stored observation (ragged: max_len * elem_bytes) */
    int64_t elem_bytes;      /* ragged: bytes per sequence element, else 0 */
    int64_t aux_elem_bytes;  /* ragged: bytes per auxiliary element, else 0 */
    int64_t act_bytes;       /* bytes of one action */
    int32_t alpha_num, alpha_den;
    double beta;
    int32_t frame_stack;     /* K >= 1 observations per sample */
    int32_t ragged;          /* observations are variable-length sequences */
    int32_t single_stream;   /* 1: episode/step left NULL are derived from done */
    int64_t tree_leaves;     /* power of two >= capacity */
    /* storage */
    uint8_t* obs;            /* capacity*row_bytes, or NULL: observations not kept */
    uint8_t* aux;            /* ragged: capacity*max_len*aux_elem_bytes, or NULL */
    uint8_t* action;         /* capacity*act_bytes */
    float* reward;           /* capacity */
    uint8_t* done;           /* capacity */
    uint32_t* episode;       /* capacity */
    int32_t* step;           /* capacity */
    int64_t* position;       /* stream position held by a slot, -1 if never written */
    int32_t* length;         /* ragged: elements of the stored sequence */
    uint32_t* leaf;          /* capacity: quantised priority */
    uint64_t* tree;          /* 2*tree_leaves: binary sum tree, node 1 is the root */
    /* running state */
    int64_t head, size, total;
    uint32_t max_prio;
} orc_replay;

void orc_reset(orc_replay* r) {
    r->head = r->size = r->total = 0;
    r->max_prio = 1; /* new transitions get the largest priority seen so far (Schaul et al.) */
    for (int64_t s = 0; s < r->capacity; ++s) {
        r->position[s] = -1;
        r->leaf[s] = 0;
        r->episode[s] = 0;
        r->step[s] = 0;
        if (r->length) r->length[s] = 0;
    }
    memset(r->tree, 0, sizeof(uint64_t) * 2 * (size_t)r->tree_leaves);
}

/* textbook binary sum tree: set one leaf, then recompute every ancestor */
static void tree_set(orc_replay* r, int64_t slot, uint32_t q) {
    r->leaf[slot] = q;
    int64_t node = r->tree_leaves + slot;
    r->tree[node] = q;
    for (node /= 2; node >= 1; node /= 2) r->tree[node] = r->tree[2 * node] + r->tree[2 * node + 1];
}

uint64_t orc_total_priority(const orc_replay* r) { return r->tree[1]; }

/*
 * Insert n transitions at slots (head + j) mod capacity, overwriting the oldest
 * ones once the ring is full (eviction).  episode/step NULL: with
 * single_stream, derived from done as one stream (tuples carry an episode ID,
 * Sec. 2.1; the reading for callers that give none): a transition continues
 * its predecessor's episode one step on, unless the predecessor was done, when
 * it starts the next episode at step 0; the first transition ever is episode
 * 0, step 0.  Without single_stream they are stored as 0.
 * prio NULL: every new transition gets the running maximum priority.
 * Ragged datasets take concatenated sequences: row j spans elements
 * [offsets[j], offsets[j+1]) of obs and aux.
 * Returns 0, or -1 (and changes nothing) on invalid arguments.
 */
int32_t orc_ingest(orc_replay* r, int64_t n, const uint8_t* obs, const int64_t* offsets,
                   const uint8_t* aux, const uint8_t* action, const float* reward,
                   const uint8_t* done, const uint32_t* episode, const int32_t* step,
                   const uint32_t* prio) {
    if (n < 0 || n > r->capacity) return -1;
    int64_t max_len = r->ragged ? r->row_bytes / r->elem_bytes : 0;
    if (r->ragged && n > 0) {
        if (!offsets) return -1;
        for (int64_t j = 0; j < n; ++j) {
            int64_t len = offsets[j + 1] - offsets[j];
            if (len < 0 || len > max_len) return -1;
        }
    }
    uint32_t fill_prio = r->max_prio;
    for (int64_t j = 0; j < n; ++j) {
        int64_t s = (r->head + j) % r->capacity;
        if (r->obs && obs) {
            if (r->ragged) {
                int64_t len = offsets[j + 1] - offsets[j];
                memcpy(r->obs + s * r->row_bytes, obs + offsets[j] * r->elem_bytes,
                       (size_t)(len * r->elem_bytes));
                if (r->aux && aux)
                    memcpy(r->aux + s * max_len * r->aux_elem_bytes, aux + offsets[j] * r->aux_elem_bytes,
                           (size_t)(len * r->aux_elem_bytes));
            } else {
                memcpy(r->obs + s * r->row_bytes, obs + j * r->row_bytes, (size_t)r->row_bytes);
            }
        }
        if (r->ragged) r->length[s] = (int32_t)(offsets[j + 1] - offsets[j]);
        if (action) memcpy(r->action + s * r->act_bytes, action + j * r->act_bytes, (size_t)r->act_bytes);
        /* the predecessor (stream position total + j - 1) sits in the slot before s */
        uint32_t ep_d = 0;
        int32_t st_d = 0;
        if (r->total + j > 0) {
            int64_t ps = (s + r->capacity - 1) % r->capacity;
            ep_d = r->episode[ps] + (r->done[ps] ? 1u : 0u);
            st_d = r->done[ps] ? 0 : r->step[ps] + 1;
        }
        r->reward[s] = reward ? reward[j] : 0.0f;
        r->done[s] = done ? done[j] : 0;
        r->episode[s] = episode ? episode[j] : r->single_stream ? ep_d : 0;
        r->step[s] = step ? step[j] : r->single_stream ? st_d : 0;
        r->position[s] = r->total + j;
        uint32_t p = prio ? prio[j] : fill_prio;
        tree_set(r, s, orc_leaf(p, r->alpha_num, r->alpha_den));
        if (prio && p > r->max_prio) r->max_prio = p;
    }
    r->head = (r->head + n) % r->capacity;
    r->size = r->size + n < r->capacity ? r->size + n : r->capacity;
    r->total += n;
    return 0;
}

/*
 * Priority callback: apply (idx[k], prio[k]) in array order, so the last
 * occurrence of a repeated index wins.  Indices outside [0, size) are skipped.
 * Returns the number of skipped entries.
 */
int64_t orc_update(orc_replay* r, int64_t n, const int64_t* idx, const uint32_t* prio) {
    int64_t bad = 0;
    for (int64_t k = 0; k < n; ++k) {
        if (idx[k] < 0 || idx[k] >= r->size) { ++bad; continue; }
        tree_set(r, idx[k], orc_leaf(prio[k], r->alpha_num, r->alpha_den));
        if (prio[k] > r->max_prio) r->max_prio = prio[k];
    }
    return bad;
}

/*
 * Stratified proportional sampling.  The total mass Q (the root) is cut into B
 * equal strata; stratum k draws the integer target
 *     t_k = floor((k + u_k / 2^64) * Q / B) = floor((k*Q + floor(u_k*Q / 2^64)) / B)
 * (the two forms agree by the nested-floor identity) from a host-supplied 64-bit
 * uniform u_k, and the sampled slot is the first one whose inclusive prefix sum of
 * leaves exceeds t_k (half-open intervals: zero leaves are never chosen).
 * Importance weights follow Schaul et al.: w_i = (N * P(i))^-beta with
 * P(i) = q_i / Q and N the number of stored transitions, divided by the largest
 * weight in the batch, or (buffer_norm) the largest weight any stored
 * transition could receive: that of the smallest non-zero leaf in the buffer
 * (zero leaves are never sampled).  Returns 0, or -1 if nothing can be sampled.
 */
int32_t orc_sample(const orc_replay* r, int64_t B, const uint64_t* uniforms, int64_t* idx_out,
                   float* w_out, int32_t buffer_norm) {
    uint64_t Q = r->tree[1];
    if (r->size == 0 || Q == 0 || B <= 0) return -1;
    double* w = (double*)malloc(sizeof(double) * (size_t)B);
    double wmax = 0.0;
    if (buffer_norm) {
        uint32_t qmin = 0;
        for (int64_t i = 0; i < r->capacity; ++i)
            if (r->leaf[i] != 0 && (qmin == 0 || r->leaf[i] < qmin)) qmin = r->leaf[i];
        wmax = pow((double)r->size * ((double)qmin / (double)Q), -r->beta);
    }
    for (int64_t k = 0; k < B; ++k) {
        u128 h = ((u128)uniforms[k] * Q) >> 64;
        uint64_t t = (uint64_t)(((u128)k * Q + h) / (u128)B);
        int64_t node = 1;
        while (node < r->tree_leaves) {
            uint64_t left = r->tree[2 * node];
            if (t < left) {
                node = 2 * node;
            } else {
                t -= left;
                node = 2 * node + 1;
            }
        }
        int64_t slot = node - r->tree_leaves;
        idx_out[k] = slot;
        double P = (double)r->leaf[slot] / (double)Q;
        w[k] = pow((double)r->size * P, -r->beta);
        if (!buffer_norm && w[k] > wmax) wmax = w[k];
    }
    for (int64_t k = 0; k < B; ++k) w_out[k] = (float)(w[k] / wmax);
    free(w);
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Observation transforms                                                     */
/* ------------------------------------------------------------------------- */
enum { ORC_XF_NONE = 0, ORC_XF_U8_F32 = 1, ORC_XF_U8_BF16_NORM = 2 };

/* round an IEEE single to bfloat16, to nearest, ties to even */
static uint16_t to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof(u));
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t keep = u >> 16;
    uint32_t rest = u & 0xffffu;
    if (rest > 0x8000u || (rest == 0x8000u && (keep & 1u))) keep += 1;
    return (uint16_t)keep;
}

/* u8 pixel -> float in [0,1]: the single nearest to x/255 (one IEEE division) */
float orc_u8_to_f32(uint8_t x) { return (float)x / 255.0f; }

/* u8 pixel -> bfloat16 of ((x/255) - mean) / std, every step one IEEE op */
uint16_t orc_u8_to_bf16(uint8_t x, float mean, float std) {
    float v = (float)x / 255.0f;
    float centred = v - mean;
    return to_bf16(centred / std);
}

/* write one observation of row_bytes bytes to out (element j of the output) */
static void emit_row(const uint8_t* src, int64_t row_bytes, int32_t xform, const float* mean,
                     const float* std, int32_t channels, uint8_t* out) {
    if (xform == ORC_XF_NONE) {
        if (src) memcpy(out, src, (size_t)row_bytes); else memset(out, 0, (size_t)row_bytes);
    } else if (xform == ORC_XF_U8_F32) {
        float* o = (float*)out;
        for (int64_t i = 0; i < row_bytes; ++i) o[i] = src ? orc_u8_to_f32(src[i]) : 0.0f;
    } else {
        uint16_t* o = (uint16_t*)out;
        int64_t plane = row_bytes / channels;
        for (int64_t i = 0; i < row_bytes; ++i) {
            int64_t c = i / plane;
            o[i] = src ? orc_u8_to_bf16(src[i], mean[c], std[c]) : 0;
        }
    }
}

static int64_t out_elem_bytes(int32_t xform) {
    return xform == ORC_XF_U8_F32 ? 4 : (xform == ORC_XF_U8_BF16_NORM ? 2 : 1);
}

/*
 * Materialise a learner batch for sampled slots idx[0..B).  Observations are laid
 * out [B, K, row] (K = frame_stack, oldest frame first).  Frame k of sample b is
 * the observation d = K-1-k steps earlier in the same episode: it is taken from
 * slot j = (i - d) mod capacity when that slot has been written and holds
 * (episode[i], step[i] - d); otherwise that frame is all zeros (the stack does not
 * reach across an episode start, an overwritten slot or an unwritten one).
 * Scalar columns (action, reward, done) come from slot i.  Any output may be NULL.
 * Returns 0, or -1 if an index is outside [0, size).
 */
int32_t orc_gather(const orc_replay* r, int64_t B, const int64_t* idx, int32_t xform,
                   const float* mean, const float* std, int32_t channels, uint8_t* out_obs,
                   uint8_t* out_action, float* out_reward, uint8_t* out_done) {
    int64_t K = r->frame_stack;
    int64_t C = r->capacity;
    int64_t out_row = r->row_bytes * out_elem_bytes(xform);
    for (int64_t b = 0; b < B; ++b) {
        int64_t i = idx[b];
        if (i < 0 || i >= r->size) return -1;
        if (out_obs && r->obs) {
            for (int64_t k = 0; k < K; ++k) {
                int64_t d = K - 1 - k;
                int64_t j = ((i - d) % C + C) % C;
                int valid = d == 0 || (r->position[j] >= 0 && r->episode[j] == r->episode[i] &&
                                       (int64_t)r->step[j] == (int64_t)r->step[i] - d);
                const uint8_t* src = valid ? r->obs + j * r->row_bytes : NULL;
                emit_row(src, r->row_bytes, xform, mean, std, channels,
                         out_obs + (b * K + k) * out_row);
            }
        }
        if (out_action) memcpy(out_action + b * r->act_bytes, r->action + i * r->act_bytes, (size_t)r->act_bytes);
        if (out_reward) out_reward[b] = r->reward[i];
        if (out_done) out_done[b] = r->done[i];
    }
    return 0;
}

/*
 * Pack sampled variable-length sequences into right-padded [B, max_len] arrays:
 * elements [0, L) copied, positions >= L hold pad_id (sequence) and zero bytes
 * (auxiliary); mask[b][t] = 1 iff t < L.  Returns 0, or -1 on a bad index.
 */
int32_t orc_pack(const orc_replay* r, int64_t B, const int64_t* idx, int32_t pad_id,
                 uint8_t* out_seq, uint8_t* out_mask, uint8_t* out_aux, int32_t* out_length,
                 float* out_reward) {
    int64_t max_len = r->row_bytes / r->elem_bytes;
    for (int64_t b = 0; b < B; ++b) {
        int64_t i = idx[b];
        if (i < 0 || i >= r->size) return -1;
        int64_t len = r->length[i];
        for (int64_t t = 0; t < max_len; ++t) {
            uint8_t* dst = out_seq + (b * max_len + t) * r->elem_bytes;
            if (t < len) {
                memcpy(dst, r->obs + i * r->row_bytes + t * r->elem_bytes, (size_t)r->elem_bytes);
            } else {
                /* pad id in the element's width (little-endian) */
                int64_t v = pad_id;
                memcpy(dst, &v, (size_t)r->elem_bytes);
            }
            if (out_mask) out_mask[b * max_len + t] = t < len ? 1 : 0;
            if (out_aux) {
                uint8_t* a = out_aux + (b * max_len + t) * r->aux_elem_bytes;
                if (t < len)
                    memcpy(a, r->aux + (i * max_len + t) * r->aux_elem_bytes, (size_t)r->aux_elem_bytes);
                else
                    memset(a, 0, (size_t)r->aux_elem_bytes);
            }
        }
        if (out_length) out_length[b] = (int32_t)len;
        if (out_reward) out_reward[b] = r->reward[i];
    }
    return 0;
}

/*
 * Minibatch shuffle-gather: row m of the output is source row perm[m], passed
 * through the observation transform.  Returns 0, or -1 on an index outside
 * [0, n_src).
 */
int32_t orc_rows(const uint8_t* src, int64_t row_bytes, int64_t n_src, const int64_t* perm, int64_t n,
                 int32_t xform, const float* mean, const float* std, int32_t channels, uint8_t* out) {
    int64_t out_row = row_bytes * out_elem_bytes(xform);
    for (int64_t m = 0; m < n; ++m) {
        if (perm[m] < 0 || perm[m] >= n_src) return -1;
        emit_row(src + perm[m] * row_bytes, row_bytes, xform, mean, std, channels, out + m * out_row);
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Generalised advantage estimation (Schulman et al.), fp64 inside            */
/* ------------------------------------------------------------------------- */
/*
 * Time-major rollout [T, E].  done[t,e] = 1 means transition t ended its episode,
 * so nothing is bootstrapped through it.  The value after the last step is
 * bootstrap[e] (NULL: 0).  values NULL means V = 0.
 *   delta_t = r_t + gamma * (1 - d_t) * V_{t+1} - V_t
 *   A_t     = delta_t + gamma * lambda * (1 - d_t) * A_{t+1},   A_T = 0
 *   R_t     = A_t + V_t
 */
void orc_gae(int64_t T, int64_t E, const float* reward, const float* value, const uint8_t* done,
             const float* bootstrap, double gamma, double lambda, float* adv, float* ret) {
    for (int64_t e = 0; e < E; ++e) {
        double a_next = 0.0;
        double v_next = bootstrap ? (double)bootstrap[e] : 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            int64_t at = t * E + e;
            double v = value ? (double)value[at] : 0.0;
            double live = done[at] ? 0.0 : 1.0;
            double delta = (double)reward[at] + gamma * live * v_next - v;
            double a = delta + gamma * lambda * live * a_next;
            adv[at] = (float)a;
            ret[at] = (float)(a + v);
            a_next = a;
            v_next = v;
        }
    }
}

/*
 * GAE with truncation bootstrap over a time-major [T, E] rollout: a step may end
 * its episode by termination (done = 1: nothing after it is worth anything) or
 * by truncation (truncated = 1, e.g. a time limit: the episode would have
 * continued).  Either end cuts the recursion; a truncated step that did not
 * also terminate bootstraps from final_value (the critic's value of the true
 * next observation, which the rollout's next row does not hold):
 *   live_t  = 1 - max(done_t, truncated_t)
 *   boot_t  = final_value_t if truncated_t and not done_t, else 0
 *   delta_t = r_t + gamma (live_t V_{t+1} + boot_t) - V_t
 *   A_t     = delta_t + gamma lambda live_t A_{t+1},   V_T = bootstrap[e]
 */
void orc_gae_trunc(int64_t T, int64_t E, const float* reward, const float* value, const uint8_t* done,
                   const uint8_t* truncated, const float* final_value, const float* bootstrap, double gamma,
                   double lambda, float* adv, float* ret) {
    for (int64_t e = 0; e < E; ++e) {
        double a_next = 0.0;
        double v_next = bootstrap ? (double)bootstrap[e] : 0.0;
        for (int64_t t = T - 1; t >= 0; --t) {
            int64_t at = t * E + e;
            double v = value ? (double)value[at] : 0.0;
            int term = done[at] != 0, trunc = truncated[at] != 0;
            double live = (term || trunc) ? 0.0 : 1.0;
            double boot = (trunc && !term) ? (double)final_value[at] : 0.0;
            double delta = (double)reward[at] + gamma * (live * v_next + boot) - v;
            double a = delta + gamma * lambda * live * a_next;
            adv[at] = (float)a;
            ret[at] = (float)(a + v);
            a_next = a;
            v_next = v;
        }
    }
}

/*
 * GAE over right-padded sequences [B, Lmax]: a sequence of length L gets its scalar
 * reward on the last element (t = L-1), which also ends the episode; all other
 * rewards are 0.  values NULL means V = 0.  Positions t >= L are written as 0.
 */
void orc_gae_packed(int64_t B, int64_t Lmax, const float* last_reward, const int32_t* length,
                    const float* value, double gamma, double lambda, float* adv, float* ret) {
    for (int64_t b = 0; b < B; ++b) {
        int64_t L = length[b];
        for (int64_t t = Lmax - 1; t >= L && t >= 0; --t) {
            adv[b * Lmax + t] = 0.0f;
            ret[b * Lmax + t] = 0.0f;
        }
        double a_next = 0.0;
        double v_next = 0.0;
        for (int64_t t = (L < Lmax ? L : Lmax) - 1; t >= 0; --t) {
            double v = value ? (double)value[b * Lmax + t] : 0.0;
            int last = t == L - 1;
            double r = last ? (double)last_reward[b] : 0.0;
            double live = last ? 0.0 : 1.0;
            double delta = r + gamma * live * v_next - v;
            double a = delta + gamma * lambda * live * a_next;
            adv[b * Lmax + t] = (float)a;
            ret[b * Lmax + t] = (float)(a + v);
            a_next = a;
            v_next = v;
        }
    }
}
