"""Placement (Sec. 5): the oracle of Alg. 1 pinned by cases the text fixes, and
the library's conduit_place against it.  Host-only."""
import ctypes as C

import numpy as np
import pytest

from oracle import placement as opl
from paper_2609_24456_amd import conduit as cd


def _profile(bw_in_cpu, bw_in_gpu, bw_out, mem):
    p = cd.PlaceProfile()
    for i in range(3):
        p.bw_in[0][i], p.bw_in[1][i], p.bw_out[i], p.mem[i] = bw_in_cpu[i], bw_in_gpu[i], bw_out[i], mem[i]
    return p


# ----------------------------------------------------------------------------
# pins of the oracle
# ----------------------------------------------------------------------------
def test_transfer_is_two_legs():
    # 8 KB over 4 GB/s in and 2 GB/s out: 2 us + 4 us
    assert opl.transfer(8e3, 4e9, 2e9) == pytest.approx(6e-6)


def test_fastest_feasible_wins_and_infeasible_is_skipped():
    bw_in = {0: 1e12, 1: 5e10, 2: 1e10}
    bw_out = {0: 1e12, 1: 5e10, 2: 2e10}
    # everything fits: the fastest tier
    assert opl.scan([0, 1, 2], 100, 1e3, bw_in, bw_out, {0: 1e9, 1: 1e9, 2: 1e9})[0] == 0
    # the fast tier is too small: the next fastest that holds C_buf * x
    assert opl.scan([0, 1, 2], 100, 1e3, bw_in, bw_out, {0: 99e3, 1: 1e9, 2: 1e9})[0] == 1
    # capacity exactly equal to the memory is feasible (<=)
    assert opl.scan([0, 1, 2], 100, 1e3, bw_in, bw_out, {0: 100e3, 1: 0, 2: 0})[0] == 0
    # nothing fits
    assert opl.scan([0, 1, 2], 100, 1e3, bw_in, bw_out, {0: 0, 1: 0, 2: 0})[0] is None


def test_scan_order_breaks_ties_and_restricts_candidates():
    bw = {0: 1e9, 1: 1e9, 2: 1e9}
    mem = {0: 1e9, 1: 1e9, 2: 1e9}
    assert opl.scan([2, 1, 0], 1, 1.0, bw, bw, mem)[0] == 2  # equal latency: the first scanned
    assert opl.scan([1], 1, 1.0, {0: 1e12, 1: 1.0, 2: 1.0}, bw, mem)[0] == 1  # user-restricted candidates


def test_larger_samples_move_the_buffer_off_the_gpu():
    # the growth case of Sec. 5.3: as x grows past Mem(HBM) / C_buf the choice
    # moves to the fastest host tier that still holds the buffer
    bw_in = {0: 3e12, 1: 5e10, 2: 1e10}
    bw_out = {0: 3e12, 1: 5e10, 2: 2e10}
    mem = {0: 288e9, 1: 1.5e12, 2: 1.5e12}
    choices = [opl.scan([0, 1, 2], 10**6, x, bw_in, bw_out, mem)[0] for x in (1e4, 2.88e5, 2.89e5, 1.5e6, 1.6e6)]
    assert choices == [0, 0, 1, 1, None]


# ----------------------------------------------------------------------------
# the library against the oracle
# ----------------------------------------------------------------------------
def test_library_matches_oracle_on_random_profiles():
    rng = np.random.default_rng(29)
    for _ in range(3000):
        bw_cpu = 10 ** rng.uniform(9, 12.5, 3)
        bw_gpu = 10 ** rng.uniform(9, 12.5, 3)
        bw_out = 10 ** rng.uniform(9, 12.5, 3)
        if rng.random() < 0.2:  # force ties
            bw_gpu[:] = bw_gpu[0]
            bw_out[:] = bw_out[0]
        mem = 10 ** rng.uniform(8, 12, 3)
        actor = int(rng.integers(0, 2))
        cap = int(rng.integers(0, 10**7))
        x = float(10 ** rng.uniform(1, 6))
        cand = list(rng.permutation(3)[: rng.integers(1, 4)])
        prof = _profile(bw_cpu, bw_gpu, bw_out, mem)
        got, t = cd.conduit_place(prof, actor, cap, x, cand)
        bw_in = bw_gpu if actor else bw_cpu
        want, t_o = opl.scan(cand, cap, x, dict(enumerate(bw_in)), dict(enumerate(bw_out)), dict(enumerate(mem)))
        assert got == (-1 if want is None else want)
        assert np.allclose(t, t_o, rtol=1e-15, atol=0)


def test_place_rejects_bad_arguments():
    prof = _profile([1e9] * 3, [1e9] * 3, [1e9] * 3, [1e9] * 3)
    L = cd.lib()
    ch = C.c_int32()
    cand = (C.c_int32 * 3)(0, 1, 2)
    bad = (C.c_int32 * 1)(3)
    assert L.conduit_place(C.byref(prof), 0, 1, 1.0, cand, 0, C.byref(ch), None) == cd.EINVAL
    assert L.conduit_place(C.byref(prof), 2, 1, 1.0, cand, 3, C.byref(ch), None) == cd.EINVAL
    assert L.conduit_place(C.byref(prof), 0, -1, 1.0, cand, 3, C.byref(ch), None) == cd.EINVAL
    assert L.conduit_place(C.byref(prof), 0, 1, 0.0, cand, 3, C.byref(ch), None) == cd.EINVAL
    assert L.conduit_place(C.byref(prof), 0, 1, 1.0, bad, 1, C.byref(ch), None) == cd.EINVAL
    zero = _profile([0.0] * 3, [1e9] * 3, [1e9] * 3, [1e9] * 3)
    assert L.conduit_place(C.byref(zero), 0, 1, 1.0, cand, 3, C.byref(ch), None) == cd.EINVAL
    assert L.conduit_placement_profile(1 << 19, 1, C.byref(cd.PlaceProfile())) == cd.EINVAL


def test_pageable_payload_is_rejected_and_host_payload_needs_no_device_arena():
    o = cd.default_opts(payload_placement=cd.PLACE_HOST_PAGEABLE)
    assert cd.lib().conduit_buffer_required_bytes(1000, (ctypes_shape := (C.c_int64 * 1)(64)), 1, 0, C.byref(o)) == 0
    hbm = cd.default_opts()
    pin = cd.default_opts(payload_placement=cd.PLACE_HOST_PINNED)
    b_hbm = cd.lib().conduit_buffer_required_bytes(1000, ctypes_shape, 1, 0, C.byref(hbm))
    b_pin = cd.lib().conduit_buffer_required_bytes(1000, ctypes_shape, 1, 0, C.byref(pin))
    assert b_hbm - b_pin == 1000 * 64  # the observation column left the device arena
