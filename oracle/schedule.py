"""Reference oracle for the scheduling cost model -- TEST INFRASTRUCTURE ONLY.

Plain Python (fp64) statement of the paper's iteration-latency model and its
cost-based choice of execution mode, written from the text:

* Sec. 6.2 (Iteration-Latency Model): an iteration is the exposed ingestion
  path plus the exposed delivery path; an operator invocation that processes
  g units costs T(g), i.e. T(g)/g per unit; overlapping an operator with its
  neighbouring compute stage (rollout for ingestion, update for delivery) adds
  a synchronisation cost and hides part of the operator.
* App. E (Iteration-Latency Model Details): the hidden part is
  gamma(g) * min(neighbour stage, per-unit cost), gamma(g) = 1 for g >= 1 and
  1 - g for 0 < g < 1.
* Sec. 6.3, Eq. (sched_opt): choose both overlap flags and both granularities
  to minimise the iteration latency over the finite candidate set.

Only ``tests/`` may import this module.  It shares no code with the library.
"""
import itertools


def gamma(g, on_policy=False):
    """App. E: the overlappable fraction of the per-unit cost.  Off-policy
    batches (g >= 1) can hide all of it, fractions only 1 - g.  Reading: on
    policy every g is a fraction of the current iteration (g <= 1; App. C
    Invariant 2 allows pipelining only within the iteration), so the
    fractional case is taken up to g = 1."""
    if g >= 1 and not on_policy:
        return 1.0
    return 1.0 - g


def path(t_neighbour, g, t_op, t_sync, overlap, on_policy=False):
    """Sec. 6.2: exposed latency of one path (ingestion or delivery)."""
    per_unit = t_op / g
    exposed = t_neighbour + per_unit
    if overlap:
        hide = gamma(g, on_policy) * min(t_neighbour, per_unit)  # App. E
        exposed += t_sync - hide
    return exposed


def candidates(on_policy, minibatches=1, g_max_ing=1, g_max_del=1):
    """Sec. 4.1-4.3: the feasible granularity sets of an RL configuration.
    Off-policy batching: {1..g_max} for each operator.  On-policy with M
    minibatch updates per rollout: ingestion {1/M, 2/M, ..., 1}, delivery
    {1/M}."""
    if on_policy:
        M = minibatches
        return [j / M for j in range(1, M + 1)], [1 / M]
    return list(range(1, g_max_ing + 1)), list(range(1, g_max_del + 1))


def modes(t_rollout, t_update, g_ing, t_ing, g_del, t_del, t_sync_ing, t_sync_del, on_policy=False):
    """Every candidate of Eq. (sched_opt) with its modelled latencies, in the
    order overlap_ing, overlap_del, ingestion candidate, delivery candidate."""
    out = []
    for oi, od, ii, idl in itertools.product((0, 1), (0, 1), range(len(g_ing)), range(len(g_del))):
        ti = path(t_rollout, g_ing[ii], t_ing[ii], t_sync_ing, oi, on_policy)
        td = path(t_update, g_del[idl], t_del[idl], t_sync_del, od, on_policy)
        out.append({"overlap_ing": oi, "overlap_del": od, "i_ing": ii, "i_del": idl,
                    "g_ing": g_ing[ii], "g_del": g_del[idl],
                    "t_ing_path": ti, "t_del_path": td, "t_iter": ti + td})
    return out


def best(*args, on_policy=False):
    """Eq. (sched_opt): the first candidate of least iteration latency."""
    ms = modes(*args, on_policy=on_policy)
    return min(range(len(ms)), key=lambda k: (ms[k]["t_iter"], k)), ms
