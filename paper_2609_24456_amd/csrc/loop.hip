// Scheduling the experience path on one GPU (paper Sec. 4.1-4.2: ingestion and
// delivery decoupled from the actor and the learner; Sec. 6: timing `overlap`
// and granularity `g`): an off-policy iteration loop whose compute runs on one
// stream.  An operator that is not overlapped runs inline on that stream, an
// overlapped one on a second stream next to the compute stage it hides behind;
// events keep every experience operator in one program order whatever the
// mode.  Plus the synthetic compute that stands in for rollout and update, and
// a probe of the cost of one cross-stream dependency.
#include <vector>

#include "common.h"

namespace conduit {

namespace {

constexpr int kStandinThreads = 256;
constexpr int32_t kMaxSyncHops = 1024;

// `work` dependent fp32 multiply-adds per lane, registers only; the empty asm
// statement consumes the result so the chain is not optimised away
__global__ __launch_bounds__(kStandinThreads) void k_standin(int64_t work) {
    float x = 1.0f + (float)threadIdx.x * 0x1p-12f;
    const float y = 0.99993896484375f;
    for (int64_t i = 0; i < work; ++i) x = __builtin_fmaf(x, y, 0x1p-20f);
    asm volatile("" ::"v"(x));
}

__global__ void k_tick() {}

hipError_t launch_standin(int64_t work, hipStream_t s) {
    if (work <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_standin, dim3((unsigned)device_cus()), dim3(kStandinThreads), 0, s, work);
    return hipGetLastError();
}

// Events that order streams of one device, created once per loop and
// destroyed with it: no timing, and a device-scope release when recorded
// (their only consumers are other streams of the same GPU).
constexpr unsigned kOrderEventFlags = hipEventDisableTiming | hipEventReleaseToDevice;

struct EventPool {
    std::vector<hipEvent_t> ev;
    size_t used = 0;
    hipError_t err = hipSuccess;
    explicit EventPool(size_t n) {
        ev.resize(n, nullptr);
        for (auto& e : ev)
            if (err == hipSuccess) err = hipEventCreateWithFlags(&e, kOrderEventFlags);
    }
    ~EventPool() {
        for (auto e : ev)
            if (e) (void)hipEventDestroy(e);
    }
    hipEvent_t mark(hipStream_t s) {
        if (used >= ev.size()) {  // sized for the loop's worst case; never expected
            if (err == hipSuccess) err = hipErrorInvalidValue;
            return ev.empty() ? nullptr : ev.back();
        }
        hipEvent_t e = ev[used++];
        if (err == hipSuccess) err = hipEventRecord(e, s);
        return e;
    }
    void wait(hipStream_t s, hipEvent_t e) {
        if (err == hipSuccess) err = hipStreamWaitEvent(s, e, 0);
    }
};

// One program order over operators issued on two streams C and E: an
// operator issued on the other stream than its predecessor waits for the
// predecessor's event.  Events are recorded only where the other stream can
// wait on them: after every operator on E, and after every operator when
// operators live on both streams (`both`).  A stream does not wait twice in a
// row for the same event.
struct OpOrder {
    EventPool& pool;
    hipStream_t C, E;
    bool both;
    hipEvent_t last_ev = nullptr;
    hipStream_t last_s = nullptr;
    hipEvent_t waited[2] = {nullptr, nullptr};
    OpOrder(EventPool& p, hipStream_t c, hipStream_t e, bool b) : pool(p), C(c), E(e), both(b) {}
    void wait(hipStream_t s, hipEvent_t e) {
        hipEvent_t& w = waited[s == C ? 0 : 1];
        if (!e || w == e) return;
        pool.wait(s, e);
        w = e;
    }
    void before(hipStream_t s) {
        if (last_ev && last_s != s) wait(s, last_ev);
    }
    hipEvent_t after(hipStream_t s) {
        last_ev = (s == E || both) ? pool.mark(s) : nullptr;
        last_s = s;
        return last_ev;
    }
};

// output bytes per input byte of a row transform usable by the loops
int xf_out_elem(const conduit_transform* xf) {
    switch (xf->kind) {
        case CONDUIT_XF_NONE: return 1;
        case CONDUIT_XF_U8_F32: return 4;
        case CONDUIT_XF_U8_BF16_NORM: return 2;
        default: return 0;
    }
}

}  // namespace

}  // namespace conduit

using namespace conduit;

extern "C" conduit_status conduit_standin(int64_t work, void* stream) {
    if (work < 0) return report_error(CONDUIT_EINVAL, "work must be >= 0");
    const hipError_t e = launch_standin(work, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(e));
    return CONDUIT_OK;
}

namespace {

// elapsed milliseconds between two timing events recorded around `body` on s
template <class F>
hipError_t timed(hipStream_t s, hipEvent_t t0, hipEvent_t t1, float* ms, F&& body) {
    hipError_t e = hipEventRecord(t0, s);
    if (e == hipSuccess) e = body();
    if (e == hipSuccess) e = hipEventRecord(t1, s);
    if (e == hipSuccess) e = hipEventSynchronize(t1);
    if (e == hipSuccess) e = hipEventElapsedTime(ms, t0, t1);
    return e;
}

hipError_t ticks(hipStream_t s, int n) {
    for (int i = 0; i < n; ++i) hipLaunchKernelGGL(k_tick, dim3(1), dim3(64), 0, s);
    return hipGetLastError();
}

}  // namespace

extern "C" conduit_status conduit_sync_cost_us(void* s1v, void* s2v, int32_t hops, double* hop_us, double* dep_us) {
    if (!s1v || !s2v || !hop_us || !dep_us || hops < 1 || hops > kMaxSyncHops)
        return report_error(CONDUIT_EINVAL, "need two streams, both outputs and 1 <= hops <= 1024");
    hipStream_t s1 = static_cast<hipStream_t>(s1v), s2 = static_cast<hipStream_t>(s2v);
    hipEvent_t t0 = nullptr, t1 = nullptr;
    hipError_t e = hipEventCreate(&t0);
    if (e == hipSuccess) e = hipEventCreate(&t1);
    EventPool pool(3 * (size_t)hops + 2);
    if (e == hipSuccess) e = pool.err;
    // (1) a dependency the waiting stream reaches before it is met: tiny
    // kernels alternating between the streams, against the same on s1 alone
    float single = 0.0f, pingpong = 0.0f;
    if (e == hipSuccess) e = timed(s1, t0, t1, &single, [&] { return ticks(s1, hops); });
    if (e == hipSuccess)
        e = timed(s1, t0, t1, &pingpong, [&] {
            hipStream_t cur = s1, other = s2;
            hipError_t r = hipSuccess;
            for (int i = 0; i < hops && r == hipSuccess; ++i) {
                r = ticks(cur, 1);
                pool.wait(other, pool.mark(cur));
                hipStream_t t = cur;
                cur = other;
                other = t;
            }
            pool.wait(s1, pool.mark(cur));
            return r == hipSuccess ? pool.err : r;
        });
    // (2) what an overlapped operator costs the stream it overlaps: one event
    // recorded for the other stream and one wait that is already met when the
    // stream reaches it, though not yet when it was enqueued (as in a loop the
    // host runs ahead of).  s1 is held by a stand-in long enough for the host
    // to enqueue everything behind it, so both runs time the GPU, not the
    // host; s2 by one a third as long, so its events complete in between.
    float rate_ms = 0.0f, plain = 0.0f, dep = 0.0f;
    constexpr int64_t kRateWork = 20000;
    if (e == hipSuccess) e = timed(s1, t0, t1, &rate_ms, [&] { return launch_standin(kRateWork, s1); });
    const double us_per_work = rate_ms > 0.0f ? (double)rate_ms * 1e3 / kRateWork : 1.0;
    const double gate_us = 3000.0 + 100.0 * hops;
    const int64_t gate = (int64_t)(gate_us / us_per_work) + 1;
    if (e == hipSuccess) e = launch_standin(gate, s1);
    if (e == hipSuccess) e = timed(s1, t0, t1, &plain, [&] { return ticks(s1, hops); });
    if (e == hipSuccess) e = launch_standin(gate, s1);
    if (e == hipSuccess) e = launch_standin(gate / 3, s2);
    std::vector<hipEvent_t> met((size_t)hops, nullptr);
    for (int i = 0; i < hops && e == hipSuccess; ++i) {
        e = ticks(s2, 1);
        met[(size_t)i] = pool.mark(s2);
    }
    if (e == hipSuccess)
        e = timed(s1, t0, t1, &dep, [&] {
            hipError_t r = hipSuccess;
            for (int i = 0; i < hops && r == hipSuccess; ++i) {
                pool.wait(s1, met[(size_t)i]);
                r = ticks(s1, 1);
                (void)pool.mark(s1);
            }
            return r == hipSuccess ? pool.err : r;
        });
    if (e == hipSuccess) e = hipStreamSynchronize(s2);
    if (t0) (void)hipEventDestroy(t0);
    if (t1) (void)hipEventDestroy(t1);
    if (e != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(e));
    const double h = ((double)pingpong - (double)single) * 1e3 / hops;
    const double d = ((double)dep - (double)plain) * 1e3 / hops;
    *hop_us = h > 0.0 ? h : 0.0;
    *dep_us = d > 0.0 ? d : 0.0;
    return CONDUIT_OK;
}

extern "C" conduit_status conduit_run_offpolicy(conduit_buffer* buf, const conduit_offpolicy_loop* lp,
                                                void* compute_stream, void* experience_stream, double* elapsed_ms,
                                                int64_t* op_log, int64_t* n_ops) {
    if (!buf || !lp || !elapsed_ms) return report_error(CONDUIT_EINVAL, "NULL buffer, loop or elapsed_ms");
    const conduit_offpolicy_loop& L = *lp;
    if (L.g_ing < 1 || L.g_del < 1) return report_error(CONDUIT_EINVAL, "granularities must be >= 1");
    if (L.iters < 1 || L.unit < 1 || L.batch < 1) return report_error(CONDUIT_EINVAL, "iters, unit, batch must be >= 1");
    if (L.rollout_work < 0 || L.update_work < 0) return report_error(CONDUIT_EINVAL, "work must be >= 0");
    if (!L.rollout.obs || !L.uniforms || !L.new_prio || !L.idx_out || !L.xf)
        return report_error(CONDUIT_EINVAL, "NULL rollout obs, uniforms, new_prio, idx_out or transform");
    const BufferGeometry G = buffer_geometry(buf);
    if (G.ragged) return report_error(CONDUIT_EINVAL, "the loop takes dense buffers");
    if (!G.prioritized) return report_error(CONDUIT_EINVAL, "the loop needs a prioritised buffer");
    const int xf_elem = xf_out_elem(L.xf);
    if (xf_elem == 0) return report_error(CONDUIT_EINVAL, "the loop's transform must be NONE, U8_F32 or U8_BF16_NORM");
    const int64_t out_row = G.frame_stack * G.row_bytes * xf_elem;
    hipStream_t C = static_cast<hipStream_t>(compute_stream);
    hipStream_t E = static_cast<hipStream_t>(experience_stream);
    const int64_t B = L.batch, U = L.unit;
    const int64_t n_groups = (L.iters + L.g_del - 1) / L.g_del;

    EventPool pool((size_t)(6 * L.iters + 8));
    hipEvent_t t_start = nullptr, t_end = nullptr;
    hipError_t he = pool.err;
    if (he == hipSuccess) he = hipEventCreate(&t_start);
    if (he == hipSuccess) he = hipEventCreate(&t_end);
    conduit_status st = CONDUIT_OK;
    int64_t logged = 0;
    auto log = [&](int64_t a, int64_t b, int64_t c) {
        if (op_log && logged < 3 * L.iters) {
            op_log[3 * logged] = a;
            op_log[3 * logged + 1] = b;
            op_log[3 * logged + 2] = c;
        }
        ++logged;
    };
    // Operators that are not overlapped run inline on the compute stream;
    // overlapped ones run on the experience stream.
    hipStream_t S_ing = L.overlap_ing ? E : C;
    hipStream_t S_del = L.overlap_del ? E : C;
    auto ingest = [&](int64_t first, int64_t n) {
        conduit_transitions tr = L.rollout;
        const int64_t r0 = first * U;
        tr.n = n * U;
        tr.obs = static_cast<const uint8_t*>(L.rollout.obs) + r0 * G.row_bytes;
        if (tr.action) tr.action = static_cast<const uint8_t*>(L.rollout.action) + r0 * G.action_bytes;
        if (tr.reward) tr.reward += r0;
        if (tr.done) tr.done += r0;
        if (tr.episode_id) tr.episode_id += r0;
        if (tr.step) tr.step += r0;
        if (tr.prio) tr.prio += r0;
        return conduit_ingest(buf, &tr, S_ing);
    };
    std::vector<char> delivered((size_t)n_groups, 0);
    std::vector<hipEvent_t> delivered_ev((size_t)n_groups, nullptr);
    auto deliver = [&](int64_t k, hipStream_t s) {
        const int64_t first = k * L.g_del;
        const int64_t n = (first + L.g_del < L.iters ? first + L.g_del : L.iters) - first;
        const int64_t r0 = first * B;
        conduit_learner_batch ob = L.out;
        if (ob.obs) ob.obs = static_cast<uint8_t*>(L.out.obs) + r0 * out_row;
        if (ob.action) ob.action = static_cast<uint8_t*>(L.out.action) + r0 * G.action_bytes;
        if (ob.reward) ob.reward += r0;
        if (ob.done) ob.done += r0;
        const conduit_status r = conduit_sample_gather(buf, n * B, L.uniforms + r0, L.idx_out + r0,
                                                       L.is_w_out ? L.is_w_out + r0 : nullptr, L.xf, &ob, s);
        log(1, k, first);
        return r;
    };

    // experience operators in one program order across the two streams
    const bool uses_E = S_ing == E || S_del == E;
    OpOrder order(pool, C, E, S_ing != S_del);
    auto before = [&](hipStream_t s) { order.before(s); };
    auto after = [&](hipStream_t s) { return order.after(s); };
    int64_t first_pending = 0;
    auto run_ingest = [&](int64_t upto) {  // the units accumulated up to iteration upto
        before(S_ing);
        st = ingest(first_pending, upto + 1 - first_pending);
        log(0, first_pending, upto + 1 - first_pending);
        after(S_ing);
        first_pending = upto + 1;
    };

    if (he == hipSuccess) he = hipEventRecord(t_start, C);
    if (uses_E) pool.wait(E, pool.mark(C));
    for (int64_t t = 0; t < L.iters && st == CONDUIT_OK && he == hipSuccess; ++t) {
        he = launch_standin(L.rollout_work, C);
        const bool ing_due = t + 1 - first_pending == L.g_ing || t == L.iters - 1;
        // inline ingestion: right after the rollout, on the compute stream
        if (!L.overlap_ing && ing_due) run_ingest(t);
        if (st != CONDUIT_OK) break;
        // delivery of the batch the learner needs now (unless prefetched)
        const int64_t k = t / L.g_del;
        if (!delivered[(size_t)k]) {
            before(S_del);
            st = deliver(k, S_del);
            delivered_ev[(size_t)k] = after(S_del);
            delivered[(size_t)k] = 1;
        }
        if (st != CONDUIT_OK) break;
        if (S_del != C) order.wait(C, delivered_ev[(size_t)k]);
        if (he == hipSuccess) he = launch_standin(L.update_work, C);
        // overlapped delivery: the next group is prepared during the update
        if (L.overlap_del && (t + 1) % L.g_del == 0 && t + 1 < L.iters) {
            const int64_t kn = (t + 1) / L.g_del;
            before(E);
            st = deliver(kn, E);
            delivered_ev[(size_t)kn] = after(E);
            delivered[(size_t)kn] = 1;
        }
        if (st != CONDUIT_OK) break;
        // the learner's new priorities, after its update
        if (S_del != C) order.wait(E, pool.mark(C));
        before(S_del);
        st = conduit_update_priorities(buf, L.idx_out + t * B, L.new_prio + t * B, B, S_del);
        log(2, t, 0);
        after(S_del);
        // overlapped ingestion: after this iteration's learner step, so it runs
        // during the next rollout (the next inline operator waits for it)
        if (st == CONDUIT_OK && L.overlap_ing && ing_due) run_ingest(t);
    }
    if (uses_E) pool.wait(C, pool.mark(E));
    if (he == hipSuccess) he = pool.err;
    if (he == hipSuccess) he = hipEventRecord(t_end, C);
    if (he == hipSuccess) he = hipEventSynchronize(t_end);
    float ms = 0.0f;
    if (he == hipSuccess) he = hipEventElapsedTime(&ms, t_start, t_end);
    if (t_start) (void)hipEventDestroy(t_start);
    if (t_end) (void)hipEventDestroy(t_end);
    if (st != CONDUIT_OK) return st;
    if (he != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(he));
    *elapsed_ms = ms;
    if (n_ops) *n_ops = logged;
    return CONDUIT_OK;
}

extern "C" conduit_status conduit_run_onpolicy(conduit_buffer* buf, const conduit_onpolicy_loop* lp,
                                               void* compute_stream, void* experience_stream, double* elapsed_ms,
                                               int64_t* op_log, int64_t* n_ops) {
    if (!buf || !lp || !elapsed_ms) return report_error(CONDUIT_EINVAL, "NULL buffer, loop or elapsed_ms");
    const conduit_onpolicy_loop& L = *lp;
    const int64_t M = L.minibatches;
    if (M < 1 || L.ing_slices < 1 || L.ing_slices > M)
        return report_error(CONDUIT_EINVAL, "need minibatches >= 1 and 1 <= ing_slices <= minibatches");
    if (L.iters < 1 || L.steps < 1 || L.envs < 1 || L.steps % M != 0)
        return report_error(CONDUIT_EINVAL, "iters, steps, envs must be >= 1 and steps a multiple of minibatches");
    if (L.rollout_work < 0 || L.update_work < 0) return report_error(CONDUIT_EINVAL, "work must be >= 0");
    if (!L.obs || !L.reward || !L.done || !L.perm || !L.xf || !L.adv || !L.ret || !L.out_obs || !L.out_adv ||
        !L.out_ret)
        return report_error(CONDUIT_EINVAL, "NULL required pointer");
    const int xf_elem = xf_out_elem(L.xf);
    if (xf_elem == 0) return report_error(CONDUIT_EINVAL, "the loop's transform must be NONE, U8_F32 or U8_BF16_NORM");
    const BufferGeometry G = buffer_geometry(buf);
    if (G.ragged || G.prioritized) return report_error(CONDUIT_EINVAL, "the loop takes a dense, non-prioritised buffer");
    const int64_t U = L.steps * L.envs;  // rows of one rollout
    if (G.capacity != U || G.head != 0)
        return report_error(CONDUIT_EINVAL, "buffer capacity must be steps*envs with its head at slot 0");
    const int64_t out_row = G.row_bytes * xf_elem;
    const int64_t slice_rows = (L.steps / M) * L.envs;
    const int64_t mb = U / M;
    hipStream_t C = static_cast<hipStream_t>(compute_stream);
    hipStream_t E = static_cast<hipStream_t>(experience_stream);
    hipStream_t S_ing = L.overlap_ing ? E : C;
    hipStream_t S_del = L.overlap_del ? E : C;
    const bool uses_E = S_ing == E || S_del == E;

    EventPool pool((size_t)(L.iters * (4 * M + 4) + 8));
    OpOrder order(pool, C, E, S_ing != S_del);
    hipEvent_t t_start = nullptr, t_end = nullptr;
    hipError_t he = pool.err;
    if (he == hipSuccess) he = hipEventCreate(&t_start);
    if (he == hipSuccess) he = hipEventCreate(&t_end);
    conduit_status st = CONDUIT_OK;
    const int64_t log_cap = L.iters * (2 * M + 1);
    int64_t logged = 0;
    auto log = [&](int64_t a, int64_t b, int64_t c, int64_t d) {
        if (op_log && logged < log_cap) {
            int64_t* e = op_log + 4 * logged;
            e[0] = a;
            e[1] = b;
            e[2] = c;
            e[3] = d;
        }
        ++logged;
    };
    // ingestion of rollout i's slices [first, first + n): rows copied into
    // the buffer from slot first * slice_rows on
    auto ingest = [&](int64_t i, int64_t first, int64_t n) {
        conduit_transitions tr{};
        const int64_t r0 = i * U + first * slice_rows;
        tr.n = n * slice_rows;
        tr.obs = static_cast<const uint8_t*>(L.obs) + r0 * G.row_bytes;
        tr.reward = L.reward + r0;
        tr.done = L.done + r0;
        return conduit_ingest(buf, &tr, S_ing);
    };
    // delivery of rollout i's minibatch m: rows perm[m*mb ...] with their
    // advantages and returns
    const float* cols[2] = {L.adv, L.ret};
    auto deliver = [&](int64_t i, int64_t m, hipStream_t s) {
        const int64_t o = i * U + m * mb;
        float* cols_out[2] = {L.out_adv + o, L.out_ret + o};
        return conduit_minibatch_gather(G.obs, G.row_bytes, U, L.perm + i * U + m * mb, mb, L.xf,
                                        static_cast<uint8_t*>(L.out_obs) + o * out_row, cols, cols_out, 2, s);
    };
    std::vector<hipEvent_t> delivered((size_t)M, nullptr);

    if (he == hipSuccess) he = hipEventRecord(t_start, C);
    if (uses_E) pool.wait(E, pool.mark(C));
    for (int64_t i = 0; i < L.iters && st == CONDUIT_OK && he == hipSuccess; ++i) {
        // rollout slices, each ingestion issued once its slices are rolled out
        int64_t first = 0;
        for (int64_t sl = 0; sl < M && st == CONDUIT_OK && he == hipSuccess; ++sl) {
            he = launch_standin(L.rollout_work / M, C);
            if (sl + 1 - first == L.ing_slices || sl == M - 1) {
                if (S_ing != C) order.wait(E, pool.mark(C));
                order.before(S_ing);
                st = ingest(i, first, sl + 1 - first);
                log(0, i, first, sl + 1 - first);
                order.after(S_ing);
                first = sl + 1;
            }
        }
        if (st != CONDUIT_OK || he != hipSuccess) break;
        // GAE over the whole rollout ends the ingestion path
        order.before(S_ing);
        st = conduit_gae(L.reward + i * U, L.value ? L.value + i * U : nullptr, L.done + i * U,
                         L.bootstrap ? L.bootstrap + i * L.envs : nullptr, L.steps, L.envs, L.gamma, L.lam,
                         L.adv, L.ret, S_ing);
        log(3, i, 0, 0);
        order.after(S_ing);
        if (st != CONDUIT_OK) break;
        // minibatches, each before its update slice
        if (S_del == E) {
            order.before(E);
            st = deliver(i, 0, E);
            log(1, i, 0, 0);
            delivered[0] = order.after(E);
        }
        for (int64_t m = 0; m < M && st == CONDUIT_OK && he == hipSuccess; ++m) {
            if (S_del == C) {
                order.before(C);
                st = deliver(i, m, C);
                log(1, i, m, 0);
                order.after(C);
            } else {
                order.wait(C, delivered[(size_t)m]);
                if (m + 1 < M) {  // prepared during this update slice
                    order.before(E);
                    st = deliver(i, m + 1, E);
                    log(1, i, m + 1, 0);
                    delivered[(size_t)m + 1] = order.after(E);
                }
            }
            if (st == CONDUIT_OK) he = launch_standin(L.update_work / M, C);
        }
    }
    if (uses_E) pool.wait(C, pool.mark(E));
    if (he == hipSuccess) he = pool.err;
    if (he == hipSuccess) he = hipEventRecord(t_end, C);
    if (he == hipSuccess) he = hipEventSynchronize(t_end);
    float ms = 0.0f;
    if (he == hipSuccess) he = hipEventElapsedTime(&ms, t_start, t_end);
    if (t_start) (void)hipEventDestroy(t_start);
    if (t_end) (void)hipEventDestroy(t_end);
    if (st != CONDUIT_OK) return st;
    if (he != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(he));
    *elapsed_ms = ms;
    if (n_ops) *n_ops = logged;
    return CONDUIT_OK;
}
