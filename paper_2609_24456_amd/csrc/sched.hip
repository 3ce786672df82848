// Cost-based choice of ingestion/delivery timing and granularity (Sec. 6):
// the iteration-latency model of Sec. 6.2 with the hidden-latency terms of
// App. E, minimised over the finite mode set of Eq. (sched_opt).  Host code.
#include <cmath>

#include "common.h"

namespace conduit {

namespace {

// gamma(g) of App. E: an overlapped off-policy batch (g >= 1) can hide its whole
// per-unit cost; a pipelined on-policy fraction only the part not yet exposed
double overlappable(double g) { return g >= 1.0 ? 1.0 : 1.0 - g; }

// exposed latency of one path: neighbour stage (rollout or update) plus the
// operator's per-unit cost, plus, when overlapped, synchronisation minus the
// hidden part
double path_latency(double t_neighbour, double g, double t_op, double t_sync, int overlap) {
    const double per_unit = t_op / g;
    const double hide = overlappable(g) * std::fmin(t_neighbour, per_unit);
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
    for (int i = 0; i < c->n_ing; ++i)
        if (!(c->g_ing[i] > 0.0) || !std::isfinite(c->g_ing[i]) || !good_time(c->t_ing[i]))
            return report_error(CONDUIT_EINVAL, "ingestion granularities must be > 0 and costs finite and >= 0");
    for (int i = 0; i < c->n_del; ++i)
        if (!(c->g_del[i] > 0.0) || !std::isfinite(c->g_del[i]) || !good_time(c->t_del[i]))
            return report_error(CONDUIT_EINVAL, "delivery granularities must be > 0 and costs finite and >= 0");
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
                    m.t_ing_path = path_latency(c->t_rollout, m.g_ing, c->t_ing[ii], c->t_sync_ing, oi);
                    m.t_del_path = path_latency(c->t_update, m.g_del, c->t_del[id], c->t_sync_del, od);
                    m.t_iter = m.t_ing_path + m.t_del_path;
                    if (all) all[k] = m;
                    if (!have || m.t_iter < best->t_iter) {
                        *best = m;
                        have = true;
                    }
                }
    return CONDUIT_OK;
}
