"""Scheduling cost model (Sec. 6.2, App. E, Eq. sched_opt): the oracle pinned by
closed-form cases the text fixes, and the library's conduit_schedule against the
oracle on random cost sets.  Host-only: no GPU needed."""
import ctypes as C
import math

import numpy as np
import pytest

from oracle import schedule as osch
from paper_2609_24456_amd import conduit as cd


# ----------------------------------------------------------------------------
# pins of the oracle
# ----------------------------------------------------------------------------
def test_sequential_mode_is_stage_plus_amortised_cost():
    # no overlap: nothing is hidden and no synchronisation is paid; an
    # invocation of g units costing a + b g is a/g + b per unit
    a, b = 30.0, 2.0
    gs = [1, 2, 4, 8]
    ts = [a + b * g for g in gs]
    ms = osch.modes(100.0, 200.0, gs, ts, [1], [50.0], 1e9, 1e9)
    seq = [m for m in ms if m["overlap_ing"] == 0 and m["overlap_del"] == 0]
    for m in seq:
        assert m["t_iter"] == pytest.approx(100.0 + a / m["g_ing"] + b + 200.0 + 50.0)
    # larger g amortises the fixed cost: the largest g is the best sequential one
    assert min(seq, key=lambda m: m["t_iter"])["g_ing"] == 8


def test_overlap_hides_an_operator_shorter_than_its_stage():
    # zero synchronisation, per-unit cost below the neighbouring stage: fully hidden
    ms = osch.modes(100.0, 200.0, [1, 2], [60.0, 80.0], [1, 4], [150.0, 400.0], 0.0, 0.0)
    for m in ms:
        if m["overlap_ing"]:
            assert m["t_ing_path"] == pytest.approx(100.0)
        if m["overlap_del"]:
            assert m["t_del_path"] == pytest.approx(200.0)


def test_overlap_of_a_longer_operator_exposes_it_plus_sync():
    # per-unit cost above the stage: the stage is what gets hidden
    ms = osch.modes(10.0, 20.0, [1], [70.0], [1], [90.0], 3.0, 4.0)
    m = next(m for m in ms if m["overlap_ing"] and m["overlap_del"])
    assert m["t_ing_path"] == pytest.approx(70.0 + 3.0)
    assert m["t_del_path"] == pytest.approx(90.0 + 4.0)


@pytest.mark.parametrize("M", [2, 4, 8])
def test_fractional_pipelining_hides_only_the_unexposed_fraction(M):
    # on-policy g = 1/M: T(g) is the cost of one mini-batch slice, so the per-unit
    # cost is M T(1/M); overlap hides (1 - 1/M) of min(stage, per-unit cost)
    g = 1.0 / M
    slice_cost = 5.0
    ms = osch.modes(100.0, 1.0, [g], [slice_cost], [1], [0.0], 0.0, 0.0)
    ov = next(m for m in ms if m["overlap_ing"] == 1 and m["overlap_del"] == 0)
    per_unit = M * slice_cost
    assert ov["t_ing_path"] == pytest.approx(100.0 + per_unit - (1 - g) * min(100.0, per_unit))
    assert ov["t_ing_path"] == pytest.approx(100.0 + per_unit / M)  # here per_unit < stage


def test_expensive_synchronisation_turns_overlap_off():
    k, ms = osch.best(100.0, 200.0, [1], [50.0], [1], [50.0], 1000.0, 1000.0)
    assert ms[k]["overlap_ing"] == 0 and ms[k]["overlap_del"] == 0
    k, ms = osch.best(100.0, 200.0, [1], [50.0], [1], [50.0], 1.0, 1.0)
    assert ms[k]["overlap_ing"] == 1 and ms[k]["overlap_del"] == 1


def test_superlinear_invocation_cost_gives_an_interior_granularity():
    # the paper's large-transition case: beyond some g, managing the chunk costs
    # more than the amortisation saves, so the optimum moves back to a middle g
    gs = [1, 2, 4, 8, 16]
    ts = [40.0 + 5.0 * g + 1.2 * g * g for g in gs]  # per unit 40/g + 5 + 1.2 g, least at g ~ 5.8
    k, ms = osch.best(500.0, 500.0, gs, ts, [1], [10.0], 1e9, 1e9)
    assert ms[k]["g_ing"] in (4, 8) and ms[k]["g_ing"] not in (1, 16)
    per = [t / g for g, t in zip(gs, ts)]
    assert ms[k]["g_ing"] == gs[int(np.argmin(per))]


def test_mode_count_order_and_ties():
    ms = osch.modes(1.0, 1.0, [1, 2, 3], [0.0, 0.0, 0.0], [1, 2], [0.0, 0.0], 0.0, 0.0)
    assert len(ms) == 4 * 3 * 2
    assert [(m["overlap_ing"], m["overlap_del"], m["i_ing"], m["i_del"]) for m in ms[:7]] == \
        [(0, 0, 0, 0), (0, 0, 0, 1), (0, 0, 1, 0), (0, 0, 1, 1), (0, 0, 2, 0), (0, 0, 2, 1), (0, 1, 0, 0)]
    k, _ = osch.best(1.0, 1.0, [1, 2, 3], [0.0, 0.0, 0.0], [1, 2], [0.0, 0.0], 0.0, 0.0)
    assert k == 0  # every mode costs 2.0: the first wins


def test_on_policy_whole_rollout_overlap_hides_nothing():
    # on-policy the g = 1 ingestion is the iteration's last invocation (App. C
    # Invariant 2: pipelining only within the iteration), so overlap only adds
    # the synchronisation (off-policy the same g hides fully).  This states the
    # model's reading; what pins it is the measurement on the executor,
    # test_onpolicy_whole_rollout_ingestion_overlaps_nothing_on_the_executor
    # (GPU), and the limit below.
    on = osch.modes(100.0, 200.0, [1.0], [40.0], [1.0], [30.0], 3.0, 4.0, on_policy=True)
    off = osch.modes(100.0, 200.0, [1.0], [40.0], [1.0], [30.0], 3.0, 4.0)
    seq_on = next(m for m in on if m["overlap_ing"] == 0 and m["overlap_del"] == 0)
    ov_on = next(m for m in on if m["overlap_ing"] == 1 and m["overlap_del"] == 1)
    assert ov_on["t_ing_path"] == pytest.approx(seq_on["t_ing_path"] + 3.0)
    assert ov_on["t_del_path"] == pytest.approx(seq_on["t_del_path"] + 4.0)
    ov_off = next(m for m in off if m["overlap_ing"] == 1 and m["overlap_del"] == 1)
    assert ov_off["t_ing_path"] == pytest.approx(100.0 + 3.0)


def test_on_policy_whole_rollout_is_the_limit_of_the_fractional_case():
    # App. E's fractional case hides (1 - g) min(stage, per-unit cost); the
    # on-policy value at g = 1 is the limit of that expression as g -> 1 from
    # below, computed here from the formula the paper prints for 0 < g < 1
    t_roll, t_ing1, sync = 100.0, 40.0, 3.0
    at_one = osch.modes(t_roll, 200.0, [1.0], [t_ing1], [1.0], [30.0], sync, 4.0, on_policy=True)
    ov = next(m for m in at_one if m["overlap_ing"] == 1 and m["overlap_del"] == 0)
    for k in (10, 20, 40):
        g = 1.0 - 2.0 ** -k
        per_unit = t_ing1 / 1.0  # T(g) / g with T(g) = g * T(1): the per-unit cost of a linear operator
        limit = t_roll + per_unit + sync - (1.0 - g) * min(t_roll, per_unit)
        assert ov["t_ing_path"] == pytest.approx(limit, abs=t_roll * 2.0 ** -k * 2)


@pytest.mark.parametrize("M", [2, 4, 8])
def test_on_policy_fraction_matches_off_policy_below_one(M):
    # below g = 1 the two regimes share App. E's fractional case
    gs = [j / M for j in range(1, M)]
    ts = [5.0 * j for j in range(1, M)]
    on = osch.modes(100.0, 150.0, gs, ts, [1 / M], [7.0], 2.0, 2.0, on_policy=True)
    off = osch.modes(100.0, 150.0, gs, ts, [1 / M], [7.0], 2.0, 2.0)
    for a, b in zip(on, off):
        assert a["t_iter"] == pytest.approx(b["t_iter"])


def test_candidate_sets():
    assert osch.candidates(False, g_max_ing=4, g_max_del=3) == ([1, 2, 3, 4], [1, 2, 3])
    gi, gd = osch.candidates(True, minibatches=4)
    assert gi == [0.25, 0.5, 0.75, 1.0] and gd == [0.25]
    for on, kw in [(False, dict(g_max_ing=8, g_max_del=2)), (True, dict(minibatches=32)), (True, dict(minibatches=1))]:
        lg = cd.conduit_sched_candidates(on, **kw)
        og = osch.candidates(on, **kw)
        assert [list(x) for x in lg] == [list(map(float, x)) for x in og]


def test_candidate_and_on_policy_errors():
    L = cd.lib()
    buf = (C.c_double * 4)()
    n1, n2 = C.c_int32(), C.c_int32()
    assert L.conduit_sched_candidates(1, 0, 1, 1, buf, 4, C.byref(n1), buf, 4, C.byref(n2)) == cd.EINVAL
    assert L.conduit_sched_candidates(1, 5, 1, 1, buf, 4, C.byref(n1), buf, 4, C.byref(n2)) == cd.EINVAL
    assert L.conduit_sched_candidates(0, 1, 0, 1, buf, 4, C.byref(n1), buf, 4, C.byref(n2)) == cd.EINVAL
    assert L.conduit_sched_candidates(0, 1, 5, 1, buf, 4, C.byref(n1), buf, 4, C.byref(n2)) == cd.EINVAL
    assert L.conduit_sched_candidates(0, 1, 1, 1, None, 4, C.byref(n1), buf, 4, C.byref(n2)) == cd.EINVAL
    with pytest.raises(cd.ConduitError) as e:
        cd.conduit_schedule(1.0, 1.0, [2.0], [1.0], [0.5], [1.0], on_policy=True)  # g > 1 on-policy
    assert e.value.status == cd.EINVAL


# ----------------------------------------------------------------------------
# the library against the oracle
# ----------------------------------------------------------------------------
def _random_case(rng):
    n_i, n_d = int(rng.integers(1, 6)), int(rng.integers(1, 6))
    frac = rng.random() < 0.3
    g_i = sorted(set(rng.choice([0.125, 0.25, 0.5, 1, 2, 3, 4, 8, 16], n_i).tolist())) if frac else \
        sorted(set(rng.integers(1, 17, n_i).tolist()))
    g_d = sorted(set(rng.integers(1, 9, n_d).tolist()))
    t_i = (rng.random(len(g_i)) * 400).tolist()
    t_d = (rng.random(len(g_d)) * 400).tolist()
    return (float(rng.random() * 500), float(rng.random() * 500), g_i, t_i, g_d, t_d,
            float(rng.random() * 50), float(rng.random() * 50))


def _random_on_policy_case(rng):
    M = int(rng.integers(1, 17))
    g_i, g_d = osch.candidates(True, minibatches=M)
    t_i = (rng.random(len(g_i)) * 400).tolist()
    t_d = (rng.random(len(g_d)) * 400).tolist()
    return (float(rng.random() * 500), float(rng.random() * 500), g_i, t_i, g_d, t_d,
            float(rng.random() * 50), float(rng.random() * 50))


@pytest.mark.parametrize("on_policy", [False, True])
def test_library_matches_oracle_on_random_cost_sets(on_policy):
    rng = np.random.default_rng(17 + on_policy)
    for _ in range(2000):
        case = _random_on_policy_case(rng) if on_policy else _random_case(rng)
        k, oms = osch.best(*case, on_policy=on_policy)
        best, lms = cd.conduit_schedule(*case, on_policy=on_policy)
        assert len(lms) == len(oms)
        for lm, om in zip(lms, oms):
            for f in ("overlap_ing", "overlap_del", "i_ing", "i_del"):
                assert lm[f] == om[f]
            for f in ("t_ing_path", "t_del_path", "t_iter"):
                assert lm[f] == pytest.approx(om[f], rel=1e-12, abs=1e-9)
        ob = oms[k]
        assert (best["overlap_ing"], best["overlap_del"], best["i_ing"], best["i_del"]) == \
            (ob["overlap_ing"], ob["overlap_del"], ob["i_ing"], ob["i_del"])


@pytest.mark.parametrize("bad", [
    dict(g_ing=[], t_ing=[]), dict(g_ing=[0.0], t_ing=[1.0]), dict(g_ing=[-1.0], t_ing=[1.0]),
    dict(t_ing=[-1.0]), dict(t_ing=[math.nan]), dict(t_rollout=math.inf), dict(t_sync_del=-0.5)])
def test_schedule_rejects_bad_costs(bad):
    args = dict(t_rollout=1.0, t_update=1.0, g_ing=[1.0], t_ing=[1.0], g_del=[1.0], t_del=[1.0],
                t_sync_ing=0.0, t_sync_del=0.0)
    args.update(bad)
    with pytest.raises(cd.ConduitError) as e:
        cd.conduit_schedule(**args)
    assert e.value.status == cd.EINVAL


def test_loop_entry_points_reject_bad_arguments_on_the_host():
    # argument checks return before any device call, so they run without a GPU
    L = cd.lib()
    dummy = C.c_void_p(1)
    hop, dep = C.c_double(), C.c_double()
    assert L.conduit_standin(-1, None) == cd.EINVAL
    for hops in (0, 1025):
        assert L.conduit_sync_cost_us(dummy, dummy, hops, C.byref(hop), C.byref(dep)) == cd.EINVAL
    assert L.conduit_sync_cost_us(None, dummy, 8, C.byref(hop), C.byref(dep)) == cd.EINVAL
    assert L.conduit_sync_cost_us(dummy, dummy, 8, None, C.byref(dep)) == cd.EINVAL
    ms = C.c_double()
    lp = cd.OffpolicyLoop()
    assert L.conduit_run_offpolicy(None, C.byref(lp), None, None, C.byref(ms), None, None) == cd.EINVAL
    op = cd.OnpolicyLoop()
    assert L.conduit_run_onpolicy(None, C.byref(op), None, None, C.byref(ms), None, None) == cd.EINVAL
