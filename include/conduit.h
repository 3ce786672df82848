/*
 * conduit.h -- C ABI of the MI355X experience-path library (libconduit.so).
 *
 * The experience path is the per-iteration work between actors and learners
 * that the Conduit paper calls experience ingestion and experience delivery
 * (Sec. 2.2, the responsibilities of the experience path; Sec. 4, the
 * experience data plane):
 *   - off-policy ingestion adds transitions to a long-lived replay store and
 *     keeps the per-slot bookkeeping that sampling and eviction need;
 *   - off-policy delivery draws from that store, builds the learner batch and
 *     changes its layout (stacking, reshaping);
 *   - on-policy ingestion derives returns and advantages over trajectories;
 *   - on-policy delivery partitions a rollout into shuffled minibatches;
 *   - replay priorities are updated through algorithm callbacks (App. C,
 *     Invariant 2), and staging never changes contents (App. C, Invariant 1).
 * The mathematics of these operations is the one of the works the paper cites
 * for them: proportional prioritised replay (Schaul et al.), generalised
 * advantage estimation as used by PPO (Schulman et al.), the DQN frame stack
 * (Mnih et al.).  Where those leave a choice open, the choice made here is
 * stated at the entry point.
 *
 * Conventions for every entry point:
 *   - Pointers documented as "device" point to HIP device memory of the GPU
 *     that is current when the call is made (e.g. torch CUDA tensors);
 *     "host" pointers point to ordinary host memory.  The caller owns every
 *     input and output buffer; the library owns only what a buffer allocates
 *     (or the arena the caller hands it, see conduit_buffer_create).
 *   - `stream` is a hipStream_t (NULL: the default stream).  Calls enqueue their
 *     kernels and return; outputs are valid in stream order.  A buffer is not
 *     thread-safe: serialise calls on one stream or order streams with events.
 *   - Every call returns a conduit_status.  Argument errors are detected on the
 *     host before anything is enqueued and leave all state unchanged.  Errors a
 *     kernel finds in device-resident arguments (an index out of range, an empty
 *     priority tree, a sequence longer than the slot) are recorded in a sticky
 *     flag: the kernel never touches memory out of bounds (the offending element
 *     is skipped or written as zeros), and the first call that starts after the
 *     kernel has finished returns CONDUIT_ESTATE until the flag is cleared.
 *     conduit_sync_check() waits for a stream and reports the flag.
 *   - conduit_last_error() returns a thread-local message for the last failure.
 *   - The delivery and on-policy calls (conduit_sample, conduit_gather_transform,
 *     conduit_sample_gather, conduit_sample_gather_nstep, conduit_sample_pack_gae,
 *     conduit_update_priorities, conduit_nstep, the GAE
 *     calls, conduit_minibatch_gather) only enqueue kernels: no allocation,
 *     memset or synchronisation, so they may be captured into a HIP graph and
 *     replayed; a replay uses the arguments and the ring state (size, total)
 *     of the capture.  The ingest calls advance the ring's host-side head when
 *     they are enqueued, so a captured ingest would replay into the same slots.
 */
#ifndef CONDUIT_H
#define CONDUIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t conduit_status;
#define CONDUIT_OK 0
#define CONDUIT_EINVAL (-1)  /* bad argument (detected on the host) */
#define CONDUIT_ENOMEM (-2)  /* device or pinned-host allocation failed */
#define CONDUIT_EEMPTY (-3)  /* sample from a buffer holding no transitions */
#define CONDUIT_EDEVICE (-4) /* a HIP runtime call failed (text in conduit_last_error) */
#define CONDUIT_ESTATE (-5)  /* a kernel flagged bad device-side input earlier */

/* Enumerations cross the ABI as int32_t (a C enum's width is the compiler's
 * choice, and a value outside an enum's range is undefined in C++): every
 * entry point checks the value and returns EINVAL for an unknown one. */

/* observation element type */
typedef int32_t conduit_dtype;
enum {
    CONDUIT_U8 = 0,
    CONDUIT_I32 = 1,
    CONDUIT_F32 = 2,
    CONDUIT_BF16 = 3,
};

typedef struct conduit_buffer conduit_buffer;

/* ---------------------------------------------------------------------------
 * Buffer options.  Fill with conduit_buffer_opts_default() and override.
 * ------------------------------------------------------------------------- */
typedef struct {
    /* 1: keep per-slot priorities and the sum tree (prioritised replay).
     * 0: no priorities (on-policy rollouts, uniform replay by caller indices). */
    int32_t prioritized;
    /* alpha = alpha_num / alpha_den, 0 <= alpha_num <= alpha_den <= 8.
     * Default 3/5 (alpha = 0.6). */
    int32_t alpha_num;
    int32_t alpha_den;
    /* importance-sampling exponent beta >= 0.  Default 0.4. */
    double beta;
    /* observations per sample returned by gather (frame stacking), 1..16.
     * Default 1. */
    int32_t frame_stack;
    /* bytes of one action (any layout; copied verbatim), 0..256.  Default 4. */
    int32_t action_bytes;
    /* 1: observations are variable-length sequences: obs_shape = {max_len},
     * obs_dtype a 4-byte type, and each slot may also hold aux_elem_bytes per
     * element (e.g. a float log-probability).  Default 0. */
    int32_t ragged;
    /* ragged: bytes of the auxiliary per-element value, 0 or 4.  Default 0. */
    int32_t aux_elem_bytes;
    /* Where the payload (the observation column, and the auxiliary column of
     * a ragged buffer) lives (Sec. 5 placement): CONDUIT_PLACE_HBM (default)
     * or CONDUIT_PLACE_HOST_PINNED -- pinned host memory that the same kernels
     * read and write across the host link.  Metadata, priorities and the tree
     * stay in HBM either way.  CONDUIT_PLACE_HOST_PAGEABLE is a candidate of
     * conduit_place only: kernels cannot address pageable memory. */
    int32_t payload_placement;
    /* Importance-weight normalisation (Schaul et al.'s w_i / max w):
     * CONDUIT_WNORM_BATCH (default) divides by the largest weight of the
     * batch; CONDUIT_WNORM_BUFFER by the largest weight any stored transition
     * could receive, that of the smallest non-zero leaf of the buffer (the
     * sampler workgroups reduce the leaves in the same launches). */
    int32_t weight_norm;
    /* 1: the buffer holds one stream of transitions, and an ingest that gives
     * no episode_id (or no step) derives them from done (see
     * conduit_transitions), with one more small launch.  0 (default): such an
     * ingest stores episode 0 and step 0 (rollouts of several environments
     * interleaved, whose ids nothing reads), and frame-stacking buffers need
     * both arrays on every ingest. */
    int32_t single_stream;
} conduit_buffer_opts;

#define CONDUIT_WNORM_BATCH 0
#define CONDUIT_WNORM_BUFFER 1

/* Experience-buffer placements on one GPU host (Sec. 5.1): the memory tier of
 * the payload.  (The paper's fourth candidate, a buffer sharded over several
 * GPUs, needs more than one GPU.) */
#define CONDUIT_PLACE_HBM 0
#define CONDUIT_PLACE_HOST_PINNED 1
#define CONDUIT_PLACE_HOST_PAGEABLE 2
#define CONDUIT_PLACEMENTS 3

void conduit_buffer_opts_default(conduit_buffer_opts* opts);

/* ---------------------------------------------------------------------------
 * Buffer lifecycle
 * ------------------------------------------------------------------------- */
/*
 * Bytes of device memory a buffer with these parameters needs (all columns,
 * the priority tree and small state, without a payload placed in host memory),
 * rounded to 256-byte alignment.  Returns 0 for invalid parameters.
 * Host-only; allocates nothing.
 */
size_t conduit_buffer_required_bytes(int64_t capacity, const int64_t* obs_shape, int32_t ndim,
                                     conduit_dtype obs_dtype, const conduit_buffer_opts* opts);

/*
 * Create the replay dataset that off-policy ingestion writes into and keeps
 * indexed (Sec. 2.2): an HBM ring
 * of `capacity` slots, each holding one observation of shape obs_shape[0..ndim)
 * and type obs_dtype (row-major), an action, a reward, a done flag, an episode
 * id and a step index, and (prioritized) a quantised priority leaf of a 64-ary
 * sum tree.
 *   capacity   1 .. 2^31-1 slots.
 *   obs_shape  host array of ndim >= 1 positive sizes.
 *   opts       host pointer or NULL (defaults).
 *   arena      NULL: the library allocates the memory (hipMalloc) and frees it in
 *              conduit_buffer_destroy.  Otherwise device memory of at least
 *              conduit_buffer_required_bytes() bytes, 256-byte aligned, owned by
 *              the caller and kept alive until destroy.  A payload placed in
 *              pinned host memory is always allocated by the library
 *              (hipHostMalloc, coherent) and freed by destroy.
 *   out        host pointer receiving the handle.
 * The buffer is bound to the device current at creation.  Slots start empty;
 * every tree node and leaf starts at 0; the running maximum priority starts at 1.
 * Errors: EINVAL (bad sizes/options, a pageable or unknown payload placement,
 * arena too small or misaligned), ENOMEM, EDEVICE.  Synchronous.
 */
conduit_status conduit_buffer_create(int64_t capacity, const int64_t* obs_shape, int32_t ndim,
                                     conduit_dtype obs_dtype, const conduit_buffer_opts* opts,
                                     void* arena, size_t arena_bytes, conduit_buffer** out);

/* Wait for the device and free what the buffer allocated.  NULL is a no-op. */
void conduit_buffer_destroy(conduit_buffer* buf);

/* ---------------------------------------------------------------------------
 * Ingestion (Sec. 2.2 off-policy ingestion; Sec. 4.1)
 * ------------------------------------------------------------------------- */
typedef struct {
    int64_t n;                   /* transitions in this call, 0 .. capacity */
    /* dense: device [n, row] observations, row = prod(obs_shape) * dtype size.
     * ragged: device concatenated elements of the n sequences. */
    const void* obs;
    const int64_t* offsets;      /* ragged: device [n+1] element offsets, non-decreasing */
    int64_t src_elems;           /* ragged: elements obs (and aux) hold; a row whose offsets
                                    decrease or leave [0, src_elems] is stored empty and
                                    flagged (CONDUIT_ESTATE later).  Ignored for dense rows. */
    const void* aux;             /* ragged, aux_elem_bytes > 0: device concatenated aux elements */
    const void* action;          /* device [n, action_bytes] or NULL (zeros) */
    const float* reward;         /* device [n] or NULL (zeros) */
    const uint8_t* done;         /* device [n] or NULL (zeros) */
    /* device [n] episode ids and step indices within the episode (>= 0).  NULL
     * in a single_stream buffer: derived from done as one stream (the
     * transitions of every ingest follow the buffer's last stored transition):
     * a transition continues its predecessor's episode one step on, unless the
     * predecessor's done ended it, when it starts the next episode id at step
     * 0; the first transition ever is episode 0, step 0.  NULL otherwise: 0
     * (not allowed when frame_stack > 1). */
    const uint32_t* episode_id;
    const int32_t* step;
    const uint32_t* prio;        /* device [n] priorities or NULL: the running maximum */
} conduit_transitions;

/*
 * Insert transitions j = 0..n-1 into slots (head + j) mod capacity, evicting the
 * oldest transitions once the ring is full.  Then head = (head + n) mod capacity,
 * size = min(size + n, capacity).  With priorities, slot j's leaf becomes
 * L(prio[j]) and the running maximum absorbs prio[j]; without them, every new
 * transition gets L(running maximum) (new transitions enter at the largest
 * priority seen so far, as in Schaul et al.).  L(p) = floor(2^F * p^alpha) computed exactly in integers,
 * F = min(31, floor(32 (1 - alpha))) (see conduit_update_priorities).  The sum
 * tree is brought up to date before any later call in stream order.
 * Ragged rows longer than max_len are flagged (CONDUIT_ESTATE later) and stored
 * truncated; rows with offsets outside [0, src_elems] are flagged and stored
 * empty.  Observation pointers must be 4-byte aligned.
 * Errors: EINVAL (n < 0 or n > capacity, missing required pointer, ragged
 * src_elems < 0), ESTATE.
 */
conduit_status conduit_ingest(conduit_buffer* buf, const conduit_transitions* t, void* stream);

/* ---------------------------------------------------------------------------
 * Priority callback (App. C, Invariant 2: priorities updated by algorithm
 * callbacks; proportional prioritisation of Schaul et al.)
 * ------------------------------------------------------------------------- */
/*
 * Set the priority of slots idx[k] to prio[k] for k = 0..n-1 (device int64 and
 * uint32 arrays).  A repeated index takes its LAST occurrence (array order), as
 * if the updates ran one after another.  The stored leaf is the exact integer
 *     L(p) = floor(2^F * p^(alpha_num/alpha_den)),  F = min(31, floor(32(1-alpha)))
 * (F = 12 for alpha = 0.6), so every leaf is below 2^32, the tree root below
 * 2^63, and the sampling probability of a slot is its leaf over the root.
 * L(0) = 0: a zero priority is never sampled.  The running maximum priority
 * absorbs every applied prio[k].  Indices outside [0, size) are skipped and
 * flagged.  Deterministic: integer tree arithmetic, no float atomics.
 * Errors: EINVAL (n < 0, NULL arrays with n > 0, buffer not prioritized), ESTATE.
 */
conduit_status conduit_update_priorities(conduit_buffer* buf, const int64_t* idx, const uint32_t* prio,
                                         int64_t n, void* stream);



/*
 * The learner's priority update for its last batch followed by the actor's
 * next transitions (App. C Invariant 2, then Sec. 2.2 off-policy ingestion):
 * exactly conduit_update_priorities(buf, idx, prio, n_update) followed by
 * conduit_ingest(buf, t), with the same arguments, effects and errors; either
 * part may be empty (n_update = 0 or t->n = 0).  A dense buffer with both
 * parts and at most 4,096 new rows takes one launch: one workgroup applies
 * the updates and then the new rows' tree leaves, while the rest of the grid
 * copies the rows and their columns (the update's latency hides behind the
 * copy).  Otherwise the two operations are launched one after the other.
 */
conduit_status conduit_update_ingest(conduit_buffer* buf, const int64_t* idx, const uint32_t* prio, int64_t n_update,
                                     const conduit_transitions* t, void* stream);
/* ---------------------------------------------------------------------------
 * Sampling (Sec. 2.2 off-policy delivery draws from the replay dataset;
 * proportional prioritised replay)
 * ------------------------------------------------------------------------- */
/*
 * Draw `batch` slots by stratified inverse-CDF sampling over the sum tree.
 * With Q the root (sum of leaves) and u_k = uniforms[k] (device uint64, caller
 * supplied, uniform on [0, 2^64)), stratum k's target is
 *     t_k = floor((k + u_k / 2^64) * Q / batch)
 * evaluated exactly in integers, and idx_out[k] is the first slot whose
 * inclusive prefix sum of leaves exceeds t_k.  is_w_out[k] is the importance
 * weight (N P(i))^-beta normalised by the largest weight in the batch, i.e.
 * (q_min / q_i)^beta with q_min the smallest sampled leaf, computed in fp64 and
 * rounded to fp32 (the largest weight is exactly 1).
 *   uniforms  device uint64 [batch]
 *   idx_out   device int64 [batch]
 *   is_w_out  device float [batch] or NULL
 * A tree whose root is 0 (all priorities 0) is flagged, and idx_out = -1,
 * is_w_out = 0 are written.
 * Errors: EINVAL (batch < 1 or > 2^20, NULL pointers, not prioritized),
 * EEMPTY (size == 0), ESTATE.
 */
conduit_status conduit_sample(conduit_buffer* buf, int64_t batch, const uint64_t* uniforms, int64_t* idx_out,
                              float* is_w_out, void* stream);

/* ---------------------------------------------------------------------------
 * Gather / transform (Sec. 2.2 off-policy delivery builds the learner batch
 * from the drawn transitions and changes its layout; the processing operators
 * it lists are concat/stack, reshape, batching and padding/packing)
 * ------------------------------------------------------------------------- */
/* transform of a gathered row */
typedef int32_t conduit_xform_kind;
enum {
    CONDUIT_XF_NONE = 0,        /* copy observation bytes unchanged */
    CONDUIT_XF_U8_F32 = 1,      /* uint8 x -> float x/255 (the float nearest to x/255) */
    CONDUIT_XF_U8_BF16_NORM = 2,/* uint8 x -> bf16(((x/255) - mean_c) / std_c), c = plane */
    CONDUIT_XF_TOKENS_PAD = 3,  /* ragged: right-pad sequences to max_len with pad_id */
};

typedef struct {
    conduit_xform_kind kind;
    int32_t channels;  /* U8_BF16_NORM: planes per observation (1..4); the row is
                          split into `channels` equal planes */
    float mean[4];     /* U8_BF16_NORM: per-plane mean */
    float std[4];      /* U8_BF16_NORM: per-plane std (non-zero) */
    int32_t pad_id;    /* TOKENS_PAD: value written past the sequence end */
} conduit_transform;

typedef struct {
    /* dense: device [n, K, row_elems] of the transform's output type (uint8 /
     * obs dtype for NONE, float for U8_F32, bf16 bits for U8_BF16_NORM), K =
     * frame_stack, oldest frame first.  ragged: [n, max_len] sequence elements. */
    void* obs;
    void* action;      /* device [n, action_bytes] or NULL */
    float* reward;     /* device [n] or NULL */
    uint8_t* done;     /* device [n] or NULL */
    uint8_t* mask;     /* ragged: device [n, max_len], 1 where t < length, or NULL */
    void* aux;         /* ragged: device [n, max_len] aux elements (0 past the end) or NULL */
    int32_t* length;   /* ragged: device [n] sequence lengths or NULL */
} conduit_learner_batch;

/*
 * Materialise the learner batch for slots idx[0..n) (device int64), typically the
 * output of conduit_sample.
 * Frame stacking (frame_stack K > 1, the DQN input of Mnih et al.): frame k of
 * sample b is the observation d = K-1-k steps before slot i = idx[b] in the same
 * episode, read from slot j = (i - d) mod capacity when that slot holds
 * (episode_id[i], step[i] - d); otherwise the frame is written as zeros (the
 * stack does not reach across an episode start, into an overwritten slot or an
 * unwritten one).
 * Pixel transforms are exact: U8_F32 writes the float nearest to x/255;
 * U8_BF16_NORM writes bf16_rne(fl(fl(fl(x/255) - mean_c) / std_c)) with every fl
 * one IEEE single operation rounded to nearest even.
 * Ragged (TOKENS_PAD): obs[b, t] = sequence element t for t < length, pad_id
 * after; aux likewise with 0; mask[b, t] = (t < length).
 * Scalar columns come from slot i.  Indices outside [0, size) are flagged and
 * their rows written as zeros.  Output pointers must be 16-byte aligned.
 * Errors: EINVAL (transform not valid for the buffer's dtype/layout, NULL
 * pointers), ESTATE.
 */
conduit_status conduit_gather_transform(conduit_buffer* buf, const int64_t* idx, int64_t n,
                                        const conduit_transform* xf, const conduit_learner_batch* out,
                                        void* stream);

/*
 * Fused delivery (Sec. 2.2: delivery samples, then materialises the batch):
 * exactly conduit_sample(buf, batch, uniforms, idx_out, is_w_out) followed by
 * conduit_gather_transform(buf, idx_out, batch, xf, out), with the same
 * outputs, arguments and errors as the two calls.  Dense buffers whose rows
 * are at most 8 gather work items of 7,168 bytes (e.g. a stack of four 84x84
 * frames), and ragged buffers, take one launch: the workgroups that gather (or
 * pack) a sample descend the tree for it themselves, and the importance
 * weights are computed inside the same launch.  Other dense buffers take two
 * launches: the sampler, then the gather launch with one extra workgroup for
 * the weights.  The call uses
 * a word of the buffer's device state between its launches' workgroups, so
 * calls on one buffer must not overlap (as for every call on a buffer).
 */
conduit_status conduit_sample_gather(conduit_buffer* buf, int64_t batch, const uint64_t* uniforms, int64_t* idx_out,
                                     float* is_w_out, const conduit_transform* xf, const conduit_learner_batch* out,
                                     void* stream);

/*
 * n-step return targets for already-sampled slots (off-policy delivery
 * materialising training-ready transitions, Sec. 2.2; the n-step Q-learning
 * target of the DQN line of work): for sample b at slot idx[b], holding stream
 * position p, the window p, p+1, ... of its episode stops after the first done
 * (a terminal) or after n transitions; then
 *   ret[b]      = sum_k gamma^k r_{p+k} over the window (fp64 sum, k ascending)
 *   discount[b] = gamma^n if the window bootstraps (no done, the state at p+n
 *                 stored), else 0
 *   next_idx[b] = the slot holding position p+n if it bootstraps, else -1
 *   valid[b]    = 0 if the window meets a position not yet stored, or another
 *                 episode without a done (every output then 0 or -1): the
 *                 learner drops such samples.
 * If next_obs is not NULL it receives, for dense buffers, the observation
 * stack of next_idx through xf (the bootstrap state, laid out as
 * conduit_gather_transform's obs output; rows of samples without bootstrap are
 * zero-filled).  idx, next_idx (int64), ret, discount (float), valid (uint8):
 * device [batch]; 1 <= n <= 63; batch <= 2^20.  The ring state used is the
 * one at enqueue time (calls on one buffer are stream-ordered).
 * Errors: EINVAL (n or batch out of range, NULL outputs, a ragged buffer with
 * next_obs, bad transform), ESTATE (an index outside [0, size), flagged).
 */
conduit_status conduit_nstep(conduit_buffer* buf, const int64_t* idx, int64_t batch, int32_t n, double gamma,
                             int64_t* next_idx, float* ret, float* discount, uint8_t* valid,
                             const conduit_transform* xf, void* next_obs, void* stream);

/*
 * Fused off-policy delivery with n-step targets (Sec. 2.2: delivery samples,
 * then materialises training-ready transitions; the n-step target as in
 * conduit_nstep): exactly conduit_sample_gather(buf, batch, uniforms, idx_out,
 * is_w_out, xf, out) followed by conduit_nstep(buf, idx_out, batch, n, gamma,
 * next_idx, ret, discount, valid, xf, next_obs), with the same outputs,
 * layouts and errors as the two calls (next_obs may be NULL: targets only).
 * Dense buffers whose state stack and bootstrap stack together need at most
 * 16 gather work items of 7,168 bytes (e.g. 84x84 frames, a stack of 4, any
 * n) take one launch: each sample's workgroup descends the tree, evaluates
 * the window from the slot it found and reads every frame of the two stacks
 * once (K + min(n, K) frames instead of 2K), storing each into the stacks it
 * belongs to.  Other buffers take the two calls.  Calls on one buffer must
 * not overlap (as for every call on a buffer).
 */
conduit_status conduit_sample_gather_nstep(conduit_buffer* buf, int64_t batch, const uint64_t* uniforms,
                                           int64_t* idx_out, float* is_w_out, const conduit_transform* xf,
                                           const conduit_learner_batch* out, int32_t n, double gamma,
                                           int64_t* next_idx, float* ret, float* discount, uint8_t* valid,
                                           void* next_obs, void* stream);

/*
 * Token delivery with advantages in one launch (Sec. 2.2: delivery samples and
 * pads sequences into a batch; on-policy-style advantage computation over the
 * packed rows, as for GRPO-shaped token workloads): exactly
 * conduit_sample_gather(buf, batch, uniforms, idx_out, is_w_out, xf, out)
 * on a ragged buffer followed by conduit_gae_packed(out->reward, out->length,
 * values, batch, max_len, gamma, lambda, adv, ret), with the same outputs,
 * layouts and errors as the two calls.  Each sample's workgroup descends the
 * tree, packs its row and runs the row's GAE from the length and reward it has
 * just written.  out->reward and out->length must not be NULL (the GAE reads
 * them); values is NULL (V = 0) or a device [batch, max_len] array.  Errors:
 * EINVAL (a dense buffer, NULL outputs, bad transform), EEMPTY, ESTATE.
 */
conduit_status conduit_sample_pack_gae(conduit_buffer* buf, int64_t batch, const uint64_t* uniforms,
                                      int64_t* idx_out, float* is_w_out, const conduit_transform* xf,
                                      const conduit_learner_batch* out, const float* values, double gamma,
                                      double lambda, float* adv, float* ret, void* stream);

/* ---------------------------------------------------------------------------
 * Returns / advantages (Sec. 2.2: on-policy ingestion derives returns and
 * advantages; GAE as used by PPO, Schulman et al.)
 * ------------------------------------------------------------------------- */
/*
 * Generalised advantage estimation over a time-major rollout of T steps and E
 * environments (element (t, e) at t*E + e, all device arrays):
 *     delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t
 *     A_t     = delta_t + gamma lambda (1 - d_t) A_{t+1},   A_T = 0
 *     ret_t   = A_t + V_t
 * d_t = 1 means transition t ended its episode (nothing is bootstrapped through
 * it); V_T = bootstrap[e].  rewards float [T,E]; values float [T,E] or NULL (0);
 * dones uint8 [T,E]; bootstrap float [E] or NULL (0); adv, ret float [T,E]
 * outputs, which must not overlap the inputs.  Arithmetic in fp64 inside, fp32
 * out.
 * A workgroup takes 32 environments of a rollout of at most 64 steps on its
 * own; longer rollouts are split along T across workgroups, in tiles of 32
 * environments (any E and any 4-byte aligned rows; 16-byte aligned rows with
 * E a multiple of 4 take aligned vector accesses, the others 16-byte accesses
 * at 4-byte alignment): up
 * to 4,096 tiles publish their segments' affine maps in a small per-GPU table
 * (static device memory, no allocation) and each composes the later ones.
 * Calls that overlap in time on one GPU share that table and race (their
 * results are undefined; later calls are unaffected): order such calls with a
 * stream or events.  With more tiles, rollouts of fewer than 4,096
 * environments run three launches that keep their intermediate maps in adv and
 * ret instead, and wider ones one workgroup per 8 environments.
 * Errors: EINVAL (T, E < 0, E > 2^19, NULL required pointers), ESTATE (also
 * when a split call found a segment that never published: overlapping calls).
 */
conduit_status conduit_gae(const float* rewards, const float* values, const uint8_t* dones,
                           const float* bootstrap, int64_t T, int64_t E, double gamma, double lambda,
                           float* adv, float* ret, void* stream);

/*
 * conduit_gae for callers that cannot allocate memory: code recorded under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, kernels and results as conduit_gae, and it calls no allocating
 * routine on any call, the first included: its scratch memory (the look-back
 * table of the split path and its own sticky error words) is the per-GPU
 * static table conduit_gae uses too, 3.2 MB of device memory that each GPU
 * holds until the process ends; its address is looked up once per GPU, on the
 * first call made with that GPU current.  Limit: a rollout whose split path
 * needs more than 4,096 tiles of the table is rejected with EINVAL (the plan
 * of conduit_gae_plan never asks for more: wider rollouts take kernels that
 * need no table).  Calls that overlap in time on one GPU, of either function,
 * share the table and race.  Device-side errors of this call are recorded in
 * the table, not in pinned host memory, and are reported by
 * conduit_sync_check(NULL, stream) and cleared by conduit_clear_error(NULL);
 * the call itself cannot see them (it never reads device memory).
 * Errors: EINVAL, EDEVICE.
 */
conduit_status conduit_gae_noalloc(const float* rewards, const float* values, const uint8_t* dones,
                                   const float* bootstrap, int64_t T, int64_t E, double gamma, double lambda,
                                   float* adv, float* ret, void* stream);

/*
 * GAE with truncation bootstrap (on-policy ingestion also finds episode
 * boundaries and handles truncation before deriving advantages, Sec. 2.2): as
 * conduit_gae, and a step may also end by truncation (a time limit: the
 * episode would have continued).  Either end cuts the recursion; a truncated
 * step that did not also terminate bootstraps from final_values, the critic's
 * value of its true next observation:
 *     live_t  = 1 - max(d_t, u_t)
 *     delta_t = r_t + gamma (live_t V_{t+1} + [u_t and not d_t] F_t) - V_t
 *     A_t     = delta_t + gamma lambda live_t A_{t+1}
 * truncated (u) uint8 [T,E] and final_values (F) float [T,E] device arrays,
 * both required (F is read only where u_t = 1 and d_t = 0); the rest as in
 * conduit_gae.  Errors: EINVAL, ESTATE.
 */
conduit_status conduit_gae_truncated(const float* rewards, const float* values, const uint8_t* dones,
                                     const uint8_t* truncated, const float* final_values, const float* bootstrap,
                                     int64_t T, int64_t E, double gamma, double lambda, float* adv, float* ret,
                                     void* stream);

/*
 * The kernels conduit_gae and conduit_gae_truncated take for a rollout of T
 * steps and E environments whose rows are all 16-byte aligned (aligned != 0)
 * or not, as chosen by the call itself: *path = 0 one workgroup per 8
 * environments walks all T steps, one environment per lane; 1 the same with
 * four environments per lane (E % 4 == 0, aligned); 2 one tile of 32
 * environments per workgroup (T <= 64); 3 split along T, one launch with a
 * look-back over the later segments' maps (up to 4,096 tiles); 4 split along
 * T in three launches.  Paths 2-4 take any E and either alignment; paths 0
 * and 1 serve only rollouts that need more than 4,096 tiles and have at least
 * 4,096 environments.  *chunk = steps per lane of a tile (2, 4 or 8; 0 for
 * paths 0 and 1).  Host only, nothing is enqueued.  Errors: EINVAL (T, E < 0,
 * NULL outputs).
 */
conduit_status conduit_gae_plan(int64_t T, int64_t E, int32_t aligned, int32_t* path, int32_t* chunk);

/*
 * GAE over B right-padded sequences of up to Lmax elements (LLM post-training
 * shape; the paper's Verl mapping puts advantage computation in ingestion,
 * App. A, the table mapping Verl's stages): sequence b of length L = lengths[b] receives the
 * scalar last_reward[b] on element L-1, which also ends it; all other rewards
 * are 0.  values: device float [B, Lmax] or NULL (0).  adv, ret: device float
 * [B, Lmax]; positions t >= L are written as 0.  fp64 inside.
 * Lengths outside [0, Lmax] are flagged and clamped.
 * Errors: EINVAL, ESTATE.
 */
conduit_status conduit_gae_packed(const float* last_reward, const int32_t* lengths, const float* values,
                                  int64_t B, int64_t Lmax, double gamma, double lambda, float* adv,
                                  float* ret, void* stream);

/* ---------------------------------------------------------------------------
 * Minibatch shuffle-gather (Sec. 2.2: on-policy delivery splits trajectories
 * into shuffled minibatches; App. C Invariant 2)
 * ------------------------------------------------------------------------- */
/*
 * out row m = transform(src row perm[m]) for m = 0..n-1, plus up to 8 scalar
 * float columns: cols_out[c][m] = cols[c][perm[m]].
 *   src       device [n_src, row_bytes] (e.g. a rollout in flat order t*E + e),
 *             4-byte aligned, row_bytes a multiple of 4
 *   perm      device int64 [n]
 *   xf        NONE, U8_F32 or U8_BF16_NORM (as in conduit_gather_transform)
 *   out       device [n, row_bytes * out_size], 16-byte aligned
 *   cols, cols_out  host arrays of ncols device float pointers (may be NULL if
 *             ncols == 0)
 * Entries of perm outside [0, n_src) are flagged and their rows zeroed.
 * Errors: EINVAL, ESTATE.
 */
conduit_status conduit_minibatch_gather(const void* src, int64_t row_bytes, int64_t n_src, const int64_t* perm,
                                        int64_t n, const conduit_transform* xf, void* out,
                                        const float* const* cols, float* const* cols_out, int32_t ncols,
                                        void* stream);

/* ---------------------------------------------------------------------------
 * State, introspection, errors
 * ------------------------------------------------------------------------- */
typedef struct {
    int64_t capacity;
    int64_t row_bytes;        /* bytes of one stored observation */
    int64_t head;             /* next slot to write */
    int64_t size;             /* stored transitions */
    int64_t total;            /* transitions ever ingested */
    int32_t tree_depth;       /* root level (leaves are level 0) */
    int64_t tree_nodes[8];    /* nodes per level 0..tree_depth (level 0 = capacity) */
    int64_t arena_bytes;
    /* the options the buffer was created with */
    int32_t obs_dtype;        /* conduit_dtype */
    int32_t prioritized;
    int32_t frame_stack;
    int32_t action_bytes;
    int32_t ragged;
    int32_t aux_elem_bytes;
    int64_t max_len;          /* ragged: elements per slot (0 for dense buffers) */
} conduit_buffer_info;

/* Host-side state and geometry of the buffer; no device synchronisation. */
conduit_status conduit_buffer_get_info(const conduit_buffer* buf, conduit_buffer_info* info);

/*
 * Ring state of the buffer (Sec. 2.2 off-policy ingestion keeps the indices
 * and metadata of the stored transitions): *size stored transitions, *head the
 * next slot to write, *total transitions ever ingested (each output may be
 * NULL).  Synchronous: waits for all work enqueued on the buffer's device
 * (hipDeviceSynchronize), so the device-side columns and tree then hold exactly
 * these transitions.  The outputs are written in every case; the return is
 * ESTATE (with the description in conduit_last_error) if a kernel flagged
 * bad device-side input since the flag was last cleared.
 * Errors: EINVAL (NULL buffer), EDEVICE, ESTATE.
 */
conduit_status conduit_buffer_stats(conduit_buffer* buf, int64_t* size, int64_t* head, uint64_t* total);

/* a column of a buffer (conduit_buffer_read, checkpoint sections) */
typedef int32_t conduit_column;
enum {
    CONDUIT_COL_OBS = 0,      /* [capacity, row_bytes] bytes */
    CONDUIT_COL_ACTION = 1,   /* [capacity, action_bytes] */
    CONDUIT_COL_REWARD = 2,   /* float [capacity] */
    CONDUIT_COL_DONE = 3,     /* uint8 [capacity] */
    CONDUIT_COL_EPISODE = 4,  /* uint32 [capacity] */
    CONDUIT_COL_STEP = 5,     /* int32 [capacity], -1 in unwritten slots */
    CONDUIT_COL_LENGTH = 6,   /* ragged: int32 [capacity] */
    CONDUIT_COL_AUX = 7,      /* ragged: [capacity, max_len * aux_elem_bytes] */
    CONDUIT_COL_LEAVES = 8,   /* uint32 [tree_nodes[0]] quantised priorities */
    CONDUIT_COL_TREE = 9,     /* uint64 [tree_nodes[level]] sums, level 1..tree_depth */
    CONDUIT_COL_MAX_PRIO = 10,/* uint32 [1] running maximum priority */
};

/*
 * Copy `nbytes` bytes starting `offset` bytes into a column (level selects the
 * tree level for CONDUIT_COL_TREE) into device memory `dst`, in stream order.
 * Errors: EINVAL (unknown column, range outside the column).
 */
conduit_status conduit_buffer_read(const conduit_buffer* buf, conduit_column col, int32_t level, int64_t offset,
                                   int64_t nbytes, void* dst, void* stream);

/* ---------------------------------------------------------------------------
 * Checkpoint / resume of a buffer.  The paper's buffers are long-lived state
 * (Sec. 2.2: the off-policy buffer keeps the stored transitions with their
 * indices and metadata, and the priority structure over them); these calls
 * turn that state into one byte image and back, so that a run can stop and
 * resume with the same buffer contents, ring position and priorities.
 *
 * Image layout (native byte order, little-endian on this platform): a
 * conduit_ckpt_header, then the sections the header lists, each starting at a
 * multiple of 256 bytes, in this order, each present only if the buffer holds
 * the column: OBS, ACTION, REWARD, DONE, EPISODE, STEP, LENGTH, AUX, LEAVES,
 * MAX_PRIO (layouts as in conduit_column; whole columns, all `capacity` slots).
 * The sum tree above the leaves is not stored: it is a function of the leaves
 * (integer sums), and restoring recomputes it exactly.
 * ------------------------------------------------------------------------- */
#define CONDUIT_CKPT_MAGIC "CNDTCKPT"
#define CONDUIT_CKPT_VERSION 1u
#define CONDUIT_CKPT_MAX_SECTIONS 10

typedef struct {
    int32_t column;    /* conduit_column */
    int32_t reserved;  /* 0 */
    int64_t offset;    /* bytes from the start of the image, a multiple of 256 */
    int64_t bytes;     /* section length in bytes */
} conduit_ckpt_section;

typedef struct {
    char magic[8];             /* CONDUIT_CKPT_MAGIC, without its terminating NUL */
    uint32_t version;          /* CONDUIT_CKPT_VERSION */
    uint32_t n_sections;
    uint64_t image_bytes;      /* whole image: header, sections and the padding between them */
    int64_t capacity;
    int64_t row_bytes;         /* observation bytes per slot */
    int64_t max_len;           /* ragged slot length in elements, 0 otherwise */
    int32_t obs_dtype;         /* conduit_dtype */
    int32_t prioritized;
    int32_t alpha_num, alpha_den;
    int32_t action_bytes;
    int32_t ragged;
    int32_t aux_elem_bytes;
    int32_t reserved;          /* 0 */
    int64_t head, size;        /* ring state: next slot to write, stored transitions */
    uint64_t total;            /* transitions ever ingested */
    conduit_ckpt_section section[CONDUIT_CKPT_MAX_SECTIONS];
} conduit_ckpt_header;

/* Size in bytes of the checkpoint image of `buf` (*bytes).  Errors: EINVAL (NULL argument). */
conduit_status conduit_buffer_checkpoint_bytes(const conduit_buffer* buf, uint64_t* bytes);

/*
 * Write the checkpoint image of `buf` to `dst` (device memory, pinned or
 * pageable host memory; `dst_bytes` its size, at least
 * conduit_buffer_checkpoint_bytes).  The copies are ordered after the work
 * already enqueued on `stream`, and the call waits for them: on return the
 * image is complete and `buf` may change again.  Work on other streams that
 * writes the buffer must be ordered before this call by the caller.
 * The caller owns `dst`.
 * Errors: EINVAL (NULL argument, dst_bytes too small), EDEVICE.
 */
conduit_status conduit_buffer_checkpoint(const conduit_buffer* buf, void* dst, uint64_t dst_bytes, void* stream);

/*
 * Replace the whole state of `buf` with the image at `src` (device or host
 * memory, `src_bytes` long), made by conduit_buffer_checkpoint from a buffer
 * of the same capacity, observation bytes and dtype, prioritisation, alpha,
 * action bytes and ragged layout (max_len, aux_elem_bytes).  Options that only
 * steer later calls (beta, weight normalisation, frame stack, payload
 * placement, single_stream) may differ: an image taken from an HBM buffer
 * restores into a host-placed one.  The columns and the ring state (head,
 * size, total) become the image's, the sum tree is recomputed from the leaves,
 * and the running maximum priority is the image's.  Ordered after the work on
 * `stream`; the call waits for its copies and kernels, so `src` may be freed
 * on return.  The header is checked (magic, version, the layout fields above,
 * the section table against this buffer's columns, a ring state reachable by
 * ingestion: size = min(total, capacity) and head = total mod capacity); the
 * column contents are taken as they are.  On an error nothing of `buf` has
 * been changed, except on EDEVICE during the copies, after which the buffer's
 * contents are undefined (restore again).
 * Errors: EINVAL (NULL argument, src_bytes too small, a header that does not
 * describe an image of this buffer), EDEVICE.
 */
conduit_status conduit_buffer_restore(conduit_buffer* buf, const void* src, uint64_t src_bytes, void* stream);

/*
 * Wait for `stream`, then report the sticky device-side error flag of `buf`
 * (NULL: the flag shared by the stand-alone calls conduit_gae,
 * conduit_gae_packed and conduit_minibatch_gather, and then the words
 * conduit_gae_noalloc keeps in the current GPU's static table).  Returns OK or ESTATE (with
 * a description in conduit_last_error), or EDEVICE.
 */
conduit_status conduit_sync_check(const conduit_buffer* buf, void* stream);

/* Clear the sticky device-side error flag of `buf` (NULL: the stand-alone flag,
 * and conduit_gae_noalloc's words on the current GPU, a synchronous copy). */
void conduit_clear_error(conduit_buffer* buf);

/* Thread-local description of the last failed call ("" if none). */
const char* conduit_last_error(void);

/* Library version string. */
const char* conduit_version(void);

/* ---------------------------------------------------------------------------
 * Placement (Sec. 5: capacity-constrained, bandwidth-aware experience data
 * placement, restricted to the tiers of one GPU host)
 * ------------------------------------------------------------------------- */
/*
 * Profiled transfer model inputs (Sec. 5.1-5.2), indexed by placement
 * CONDUIT_PLACE_*:
 *   bw_in[a][p]  effective bytes/s of the ingestion leg, actor -> buffer at p,
 *                for an actor on the CPU (a = 0, rollouts in pageable memory)
 *                or on the GPU (a = 1, rollouts in HBM);
 *   bw_out[p]    effective bytes/s of the delivery leg, buffer at p -> the
 *                learner's GPU;
 *   mem[p]       bytes available at p (free HBM; available host memory for
 *                both host tiers).
 */
typedef struct conduit_place_profile {
    double bw_in[2][CONDUIT_PLACEMENTS];
    double bw_out[CONDUIT_PLACEMENTS];
    double mem[CONDUIT_PLACEMENTS];
} conduit_place_profile;

/*
 * Measures a conduit_place_profile on the current device with microbenchmarks
 * of each leg (Sec. 5.1: effective bandwidth from microbenchmarks on the
 * deployment stack): copies of `bytes` bytes (>= 1 MiB) between HBM, pinned
 * host memory (hipHostMalloc) and pageable host memory (malloc), device-side
 * legs with hipMemcpyAsync on a private stream timed by events, host-side legs
 * (CPU actor into a host tier) with memcpy timed by the host clock, each the
 * best of `reps` (>= 1) after a warm-up; legs through pageable memory, which
 * the runtime stages on the host's time, are timed by the host clock.
 * Allocates and frees 3 x bytes of host and 2 x bytes of device memory.
 * Synchronous.
 * Errors: EINVAL (NULL out, bytes < 1 MiB, reps < 1), ENOMEM, EDEVICE.
 */
conduit_status conduit_placement_profile(int64_t bytes, int32_t reps, conduit_place_profile* out);

/*
 * Alg. 1 (bandwidth-aware placement, linear scan) over the candidates
 * candidates[0..n) (CONDUIT_PLACE_* values, scanned in that order): a
 * candidate p is feasible if capacity * sample_bytes <= mem[p]; its latency is
 *   T_transfer(p) = x / bw_in[actor_on_gpu][p] + x / bw_out[p]   (seconds)
 * with x = sample_bytes; the first feasible candidate of least T_transfer wins.
 * *choice receives its placement, or -1 if none is feasible.  t_transfer
 * (host [n] or NULL) receives each candidate's T_transfer (also for
 * infeasible ones).  Host-only.
 * Errors: EINVAL (NULL profile/candidates/choice, n < 1, an unknown
 * placement, actor_on_gpu not 0/1, capacity < 0, sample_bytes not > 0, a
 * bandwidth not > 0 for a scanned candidate).
 */
conduit_status conduit_place(const conduit_place_profile* profile, int32_t actor_on_gpu, int64_t capacity,
                             double sample_bytes, const int32_t* candidates, int32_t n, int32_t* choice,
                             double* t_transfer);

/* ---------------------------------------------------------------------------
 * Latency-aware scheduling of ingestion and delivery (Sec. 6: timing
 * `overlap` and granularity `g` of the two operators; iteration-latency model
 * of Sec. 6.2 with the hidden-latency terms of App. E; cost-based choice of
 * Eq. (sched_opt), Sec. 6.3).  Host-only, no device work.
 * ------------------------------------------------------------------------- */
/*
 * Profiled costs of one RL configuration, all in the same time unit:
 *   t_rollout, t_update    one actor rollout / one learner update;
 *   t_sync_ing, t_sync_del the synchronisation an overlapped operator adds;
 *   g_ing[n_ing], t_ing[n_ing]  candidate ingestion granularities (rollout
 *                          units per invocation; > 0, fractions allowed for
 *                          on-policy pipelining) and the wall time of one
 *                          invocation at each;
 *   g_del[n_del], t_del[n_del]  the same for delivery (training batches per
 *                          invocation);
 *   on_policy              0: off-policy batching; 1: on-policy pipelining
 *                          (every granularity in (0, 1]).
 * All arrays are host memory owned by the caller.
 */
typedef struct conduit_sched_costs {
    double t_rollout, t_update;
    double t_sync_ing, t_sync_del;
    int32_t n_ing, n_del;
    const double* g_ing;
    const double* t_ing;
    const double* g_del;
    const double* t_del;
    int32_t on_policy;
} conduit_sched_costs;

/* One execution mode and its modelled latencies. */
typedef struct conduit_sched_mode {
    int32_t overlap_ing, overlap_del;  /* 0 = sequential, 1 = overlapped */
    int32_t i_ing, i_del;              /* indices into g_ing / g_del */
    double g_ing, g_del;
    double t_ing_path, t_del_path, t_iter;
} conduit_sched_mode;

/*
 * Scores every mode -- overlap_ing, overlap_del in {0,1} and every candidate
 * granularity pair -- with
 *   Tbar(g)    = T(g) / g                                (per-unit cost)
 *   gamma(g)   = 1 if g >= 1, else 1 - g                 (off-policy)
 *   gamma(g)   = 1 - g                                   (on-policy)
 *   hide_ing   = gamma(g_ing) * min(t_rollout, Tbar_ing(g_ing))
 *   T_ing_path = t_rollout + Tbar_ing(g_ing) + overlap_ing * (t_sync_ing - hide_ing)
 * (delivery alike with t_update), T_iter = T_ing_path + T_del_path, and
 * returns the mode of least T_iter in *best.  Modes are scored in the order
 * overlap_ing, overlap_del, i_ing, i_del (each ascending, the last fastest);
 * the first of equal minima wins.  If `all` is not NULL it receives every
 * mode in that order (4 * n_ing * n_del entries, caller-owned).
 * On-policy, App. E's fractional case applies on all of (0, 1]: App. C
 * Invariant 2 allows on-policy pipelining only within an iteration, so a
 * rollout must be ingested, and a batch delivered, within its own iteration
 * and only the part of the operator that is not its last invocation can hide;
 * at g = 1 nothing does (the g >= 1 case of App. E describes off-policy
 * batching across iterations).
 * Errors: EINVAL (NULL costs/best, n_ing or n_del < 1, NULL arrays, a
 * granularity <= 0, or > 1 on-policy, a negative or non-finite time).
 */
conduit_status conduit_schedule(const conduit_sched_costs* costs, conduit_sched_mode* best,
                                conduit_sched_mode* all);

/*
 * The candidate granularities of an RL configuration (Sec. 4.1-4.3): off-policy
 * (on_policy = 0) G_ing = {1, ..., g_max_ing} and G_del = {1, ..., g_max_del},
 * the caps bounding staleness and memory; on-policy with M = minibatches
 * updates per rollout, G_ing = {1/M, 2/M, ..., 1} and G_del = {1/M} (the caps
 * are ignored).  Each set is written in ascending order into the caller's
 * host arrays (cap_ing / cap_del entries available) with its size in *n_ing /
 * *n_del.  Errors: EINVAL (NULL outputs, minibatches < 1 on-policy, a cap < 1
 * off-policy, an array too small).
 */
conduit_status conduit_sched_candidates(int32_t on_policy, int32_t minibatches, int32_t g_max_ing,
                                        int32_t g_max_del, double* g_ing, int32_t cap_ing, int32_t* n_ing,
                                        double* g_del, int32_t cap_del, int32_t* n_del);

/*
 * Synthetic compute that stands in for an actor rollout or a learner update in
 * scheduling experiments: one workgroup of 256 lanes per compute unit, each
 * lane running `work` dependent fp32 multiply-adds in registers (no memory
 * traffic, so co-running memory-bound kernels keep their bandwidth).  Duration
 * grows linearly with `work`.  Errors: EINVAL (work < 0).
 */
conduit_status conduit_standin(int64_t work, void* stream);

/*
 * Measurement reference, not a step of the path: dst[i] = src[i] / 255
 * (correctly rounded fp32) for i < n over contiguous memory, in one streaming
 * launch with coalesced 256-byte loads and 1 KB non-temporal stores.  It moves
 * the byte mix of the u8 -> fp32 gathers (one byte read, four written per
 * element; Sec. 2.2 delivery's batch/layout transformation) without their
 * indexing, so its rate at a gather's size is the practical ceiling that
 * gather's fraction of the HBM peak is read against.  src: device, n bytes,
 * 4-byte aligned; dst: device, 4n bytes, 16-byte aligned, not overlapping src.
 * Errors: EINVAL (n < 0 or not a multiple of 4, NULL or misaligned pointers,
 * overlap), EDEVICE.
 */
conduit_status conduit_expand_reference(const uint8_t* src, float* dst, int64_t n, void* stream);

/*
 * Profiles the synchronisation cost of overlap (Sec. 6.2 T_sync) between two
 * streams of one GPU, in microseconds per dependency (each >= 0):
 *   *hop_us: a dependency the waiting stream reaches before it is met --
 *            `hops` tiny kernels alternating between s1 and s2, each waiting
 *            on an event recorded after the previous one, against the same
 *            kernels on s1 alone;
 *   *dep_us: what an overlapped operator costs the stream it overlaps -- per
 *            tiny kernel on s1, one wait on an event of s2 (pending when
 *            enqueued, met when s1 reaches it) plus one event recorded for
 *            s2, against the kernels alone (both streams are held by
 *            stand-ins while the host enqueues, so the GPU's cost is
 *            measured, not the host's).
 * Synchronises both streams.  Errors: EINVAL (NULL streams or outputs, hops
 * outside [1, 1024]), EDEVICE.
 */
conduit_status conduit_sync_cost_us(void* s1, void* s2, int32_t hops, double* hop_us, double* dep_us);

/*
 * An off-policy iteration loop on one GPU with the experience path scheduled
 * on its own stream (Sec. 4.1-4.2 decoupled ingestion and delivery; Sec. 6
 * timing and granularity).  Iteration t: the actor's rollout (stand-in compute
 * of rollout_work) produces rollout unit t; ingestion runs once g_ing units
 * have accumulated (and after the last iteration's rollout); the learner's
 * update (stand-in of update_work) consumes batch t, delivered by one
 * conduit_sample_gather of g_del * batch samples per group of g_del
 * iterations; the learner's new priorities for batch t are then applied.
 *   overlap_ing = 0: ingestion runs inline on the compute stream right after
 *                    the rollout that completes its group (the actor waits);
 *                    1: it runs on the experience stream after the iteration's
 *                    priority update, during the next rollout.
 *   overlap_del = 0: delivery and the priority update run inline on the
 *                    compute stream before and after the update;
 *                    1: they run on the experience stream, the next group's
 *                    delivery issued during the learner's update (prefetch,
 *                    so it samples before this iteration's new priorities).
 * Overlap hides work only if the two streams run concurrently.  HIP serves
 * all of a process's streams from a few hardware queues, and two streams on
 * one queue run one after the other: the loop is still correct then, but an
 * overlapped mode only adds its synchronisation.  The caller picks the pair
 * (e.g. by timing stand-in work on both at once against one alone).
 * Whatever the mode, the experience operators keep one fixed program order
 * (an operator issued on the other stream than its predecessor waits for the
 * predecessor's event), so the data produced does not depend on timing
 * (Sec. 4.3).
 * Device inputs: the actor's transitions for iteration t are rows
 * [t*unit, (t+1)*unit) of the columns in `rollout` (its n is ignored);
 * uniforms of group k are the contiguous run starting at its first
 * iteration's t*batch; new_prio[t*batch ...] are batch t's priorities.
 * Outputs: idx_out / is_w_out [iters*batch]; the learner-batch columns in
 * `out` hold iters*batch rows (group k writes from row first*batch).
 * `op_log` (host, 3 int64 per entry, NULL allowed; at most 3*iters entries)
 * receives the experience operators in stream order: (0, first unit, units)
 * for an ingestion, (1, group, first iteration) for a delivery,
 * (2, iteration, 0) for a priority update; *n_ops their count.
 * *elapsed_ms: events around the whole loop on the compute stream.
 * Errors: EINVAL (granularities < 1, iters/unit/batch < 1, NULL required
 * pointers, a non-prioritised buffer), plus those of the operators.
 */
typedef struct conduit_offpolicy_loop {
    int32_t overlap_ing, g_ing, overlap_del, g_del;
    int64_t iters, unit, batch;
    int64_t rollout_work, update_work;
    conduit_transitions rollout;
    const uint64_t* uniforms;
    const uint32_t* new_prio;
    int64_t* idx_out;
    float* is_w_out;
    const conduit_transform* xf;
    conduit_learner_batch out;
} conduit_offpolicy_loop;

conduit_status conduit_run_offpolicy(conduit_buffer* buf, const conduit_offpolicy_loop* loop, void* compute_stream,
                                     void* experience_stream, double* elapsed_ms, int64_t* op_log, int64_t* n_ops);

/*
 * An on-policy iteration loop on one GPU (Sec. 4.1-4.2 decoupled ingestion and
 * delivery, on-policy case; Sec. 6 timing and granularity; PPO-shaped).  The
 * rollout unit is `steps` x `envs` transitions, time-major (row t*envs + e).
 * Iteration i: the actor's rollout runs as M = minibatches slices of
 * steps/M time steps (stand-in compute of rollout_work/M each); ingestion
 * copies the rows of ing_slices slices per invocation (g_ing = ing_slices/M;
 * the last invocation takes what remains) into `buf`; GAE over the whole
 * rollout follows the last one; delivery then gathers the M minibatches of
 * steps*envs/M rows through perm (a shuffle of the rollout) with their
 * advantages and returns, each followed by one update slice (stand-in of
 * update_work/M).
 *   overlap_ing = 0: each ingestion runs inline on the compute stream after
 *                    its slices; 1: on the experience stream as soon as its
 *                    slices are rolled out, pipelined with the next slices.
 *   overlap_del = 0: each minibatch gather runs inline before its update
 *                    slice; 1: minibatch m+1 is gathered on the experience
 *                    stream during update slice m.
 * Whatever the mode the experience operators keep one program order (the
 * ingestions of a rollout, its GAE, its minibatches), so the outputs do not
 * depend on the mode (App. C: on-policy freshness; Sec. 4.3).
 * `buf`: a dense, non-prioritised buffer of capacity steps*envs whose head is
 * at slot 0 (each iteration refills it from slot 0).  Device inputs, per
 * iteration i at offset i*steps*envs (bootstrap at i*envs): obs [rows of the
 * buffer's row size], reward float, value float or NULL, done uint8, bootstrap
 * float [envs] or NULL, perm int64 (a permutation of 0..steps*envs-1).
 * Scratch: adv, ret float [steps*envs] (the current iteration's GAE).
 * Outputs at offset i*steps*envs rows: out_obs (rows through xf: NONE,
 * U8_F32 or U8_BF16_NORM), out_adv, out_ret float.
 * `op_log` (host, 4 int64 per entry, NULL allowed; at most
 * iters*(2*minibatches+1) entries) receives the experience operators in
 * program order: (0, iteration, first slice, slices) for an ingestion,
 * (1, iteration, minibatch, 0) for a delivery, (3, iteration, 0, 0) for the
 * GAE; *n_ops their count.  *elapsed_ms: events around the loop on the
 * compute stream.
 * Errors: EINVAL (granularities or sizes out of range, steps not a multiple
 * of minibatches, NULL required pointers, a prioritised or ragged buffer, a
 * wrong capacity or head), plus those of the operators.
 */
typedef struct conduit_onpolicy_loop {
    int32_t overlap_ing, ing_slices, overlap_del, minibatches;
    int64_t iters, steps, envs;
    int64_t rollout_work, update_work;
    const void* obs;
    const float* reward;
    const float* value;
    const uint8_t* done;
    const float* bootstrap;
    double gamma, lam;  /* GAE discount and lambda */
    const int64_t* perm;
    const conduit_transform* xf;
    float* adv;
    float* ret;
    void* out_obs;
    float* out_adv;
    float* out_ret;
} conduit_onpolicy_loop;

conduit_status conduit_run_onpolicy(conduit_buffer* buf, const conduit_onpolicy_loop* loop, void* compute_stream,
                                    void* experience_stream, double* elapsed_ms, int64_t* op_log, int64_t* n_ops);

#ifdef __cplusplus
}
#endif

#endif /* CONDUIT_H */
