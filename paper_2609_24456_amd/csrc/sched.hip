// Cost-based choice of ingestion/delivery timing and granularity (Sec. 6):
// the iteration-latency model of Sec. 6.2 with the hidden-latency terms of
// App. E, minimised over the finite mode set of Eq. (sched_opt).  Host code.
#include <cmath>

#include "common.h"

namespace conduit {

namespace {

// gamma(g) of App. E: an overlapped off-policy batch (g >= 1) can hide its whole
// per-unit cost; a pipelined fraction only the part not yet exposed.  On-policy
// every granularity is a fraction of the current iteration's work (g <= 1):
// App. C Invariant 2 allows pipelining only within the iteration, so the
// fractional case holds up to g = 1, whose single invocation hides nothing.
double overlappable(double g, bool on_policy) { return !on_policy && g >= 1.0 ? 1.0 : 1.0 - g; }

// exposed latency of one path: neighbour stage (rollout or update) plus the
// operator's per-unit cost, plus, when overlapped, synchronisation minus the
// hidden part
double path_latency(double t_neighbour, double g, double t_op, double t_sync, int overlap, bool on_policy) {
    const double per_unit = t_op / g;
    const double hide = overlappable(g, on_policy) * std::fmin(t_neighbour, per_unit);
    return t_neighbour + per_unit + (overlap ? t_sync - hide : 0.0);
}

bool good_time(double t) { return std::isfinite(t) && t >= 0.0; }

}  // namespace

}  // namespace conduit

using namespace conduit;

extern "C" conduit_status conduit_schedule(const conduit_sched_costs* c, conduit_sched_mode* best,
                                           conduit_sched_mode* all) {
    if (!c || !best) return report_error(CONDUIT_EINVAL, "NULL costs or best");
    if (c->n_ing < 1 || c->n_del < 1) return report_error(CONDUIT_EINVAL, "need at least one granularity per operator");
    if (!c->g_ing || !c->t_ing || !c->g_del || !c->t_del) return report_error(CONDUIT_EINVAL, "NULL granularity/cost array");
    if (!good_time(c->t_rollout) || !good_time(c->t_update) || !good_time(c->t_sync_ing) || !good_time(c->t_sync_del))
        return report_error(CONDUIT_EINVAL, "times must be finite and >= 0");
    const bool on = c->on_policy != 0;
    const double g_top = on ? 1.0 : INFINITY;
    for (int i = 0; i < c->n_ing; ++i)
        if (!(c->g_ing[i] > 0.0) || !(c->g_ing[i] <= g_top) || !std::isfinite(c->g_ing[i]) || !good_time(c->t_ing[i]))
            return report_error(CONDUIT_EINVAL,
                                "ingestion granularities must be > 0 (<= 1 on-policy) and costs finite and >= 0");
    for (int i = 0; i < c->n_del; ++i)
        if (!(c->g_del[i] > 0.0) || !(c->g_del[i] <= g_top) || !std::isfinite(c->g_del[i]) || !good_time(c->t_del[i]))
            return report_error(CONDUIT_EINVAL,
                                "delivery granularities must be > 0 (<= 1 on-policy) and costs finite and >= 0");
    bool have = false;
    int64_t k = 0;
    for (int oi = 0; oi < 2; ++oi)
        for (int od = 0; od < 2; ++od)
            for (int ii = 0; ii < c->n_ing; ++ii)
                for (int id = 0; id < c->n_del; ++id, ++k) {
                    conduit_sched_mode m;
                    m.overlap_ing = oi;
                    m.overlap_del = od;
                    m.i_ing = ii;
                    m.i_del = id;
                    m.g_ing = c->g_ing[ii];
                    m.g_del = c->g_del[id];
                    m.t_ing_path = path_latency(c->t_rollout, m.g_ing, c->t_ing[ii], c->t_sync_ing, oi, on);
                    m.t_del_path = path_latency(c->t_update, m.g_del, c->t_del[id], c->t_sync_del, od, on);
                    m.t_iter = m.t_ing_path + m.t_del_path;
                    if (all) all[k] = m;
                    if (!have || m.t_iter < best->t_iter) {
                        *best = m;
                        have = true;
                    }
                }
    return CONDUIT_OK;
}

extern "C" conduit_status conduit_sched_candidates(int32_t on_policy, int32_t minibatches, int32_t g_max_ing,
                                                   int32_t g_max_del, double* g_ing, int32_t cap_ing, int32_t* n_ing,
                                                   double* g_del, int32_t cap_del, int32_t* n_del) {
    if (!g_ing || !n_ing || !g_del || !n_del) return report_error(CONDUIT_EINVAL, "NULL output");
    if (on_policy) {
        // Sec. 4.1: ingestion pipelines at minibatch granularity, j/M of a
        // rollout per invocation; Sec. 4.2: delivery feeds one minibatch
        if (minibatches < 1) return report_error(CONDUIT_EINVAL, "on-policy needs minibatches >= 1");
        if (cap_ing < minibatches || cap_del < 1) return report_error(CONDUIT_EINVAL, "output arrays too small");
        for (int j = 1; j <= minibatches; ++j) g_ing[j - 1] = (double)j / (double)minibatches;
        g_del[0] = 1.0 / (double)minibatches;
        *n_ing = minibatches;
        *n_del = 1;
        return CONDUIT_OK;
    }
    // off-policy batching of 1..g_max units per invocation
    if (g_max_ing < 1 || g_max_del < 1) return report_error(CONDUIT_EINVAL, "off-policy caps must be >= 1");
    if (cap_ing < g_max_ing || cap_del < g_max_del) return report_error(CONDUIT_EINVAL, "output arrays too small");
    for (int g = 1; g <= g_max_ing; ++g) g_ing[g - 1] = g;
    for (int g = 1; g <= g_max_del; ++g) g_del[g - 1] = g;
    *n_ing = g_max_ing;
    *n_del = g_max_del;
    return CONDUIT_OK;
}
