"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point include/conduit.h declares, and rejects invalid arguments
before touching the device."""
import ctypes as C
import os
import re

import pytest

from paper_2609_24456_amd import conduit as cd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "conduit.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(conduit_[a-z_]+)\s*\(", text)))


# the calls the experience path's boundary is stated in: buffer lifecycle,
# ingestion, the priority callback, sampling, gather/transform, the two GAE
# forms, the minibatch shuffle-gather, the ring-state query and the error text
BOUNDARY = ["conduit_buffer_create", "conduit_buffer_required_bytes", "conduit_buffer_destroy", "conduit_ingest",
            "conduit_update_priorities", "conduit_sample", "conduit_gather_transform", "conduit_gae",
            "conduit_gae_packed", "conduit_minibatch_gather", "conduit_buffer_stats", "conduit_last_error"]


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in BOUNDARY:
        assert required in names, required


def test_library_exports_the_boundary():
    L = cd.lib()
    for name in BOUNDARY:
        assert hasattr(L, name), name


def test_library_exports_every_declared_symbol():
    L = cd.lib()
    for name in _declared_functions():
        assert hasattr(L, name), name
    assert set(_declared_functions()) == set(cd.SIGNATURES)


def test_version_and_defaults():
    assert "gfx950" in cd.conduit_version()
    o = cd.default_opts()
    assert (o.prioritized, o.alpha_num, o.alpha_den, o.beta, o.frame_stack, o.action_bytes, o.ragged) == \
        (1, 3, 5, 0.4, 1, 4, 0)


def _shape(*dims):
    return (C.c_int64 * len(dims))(*dims)


def test_required_bytes_layout():
    o = cd.default_opts(frame_stack=4)
    n = cd.lib().conduit_buffer_required_bytes(1_000_000, _shape(84, 84), 2, cd.U8, C.byref(o))
    # observations dominate: 1M x 7056 B, plus scalar columns, leaves and tree
    assert 1_000_000 * 7056 < n < 1_000_000 * 7056 + 40 * 1_000_000
    assert cd.lib().conduit_buffer_required_bytes(0, _shape(84, 84), 2, cd.U8, None) == 0
    assert cd.lib().conduit_buffer_required_bytes(10, _shape(3), 1, cd.U8, None) == 0  # 3-byte rows


@pytest.mark.parametrize("cap,shape,dtype,kw,msg", [
    (0, (4,), cd.U8, {}, "capacity"),
    (1 << 31, (4,), cd.U8, {}, "capacity"),
    (10, (3,), cd.U8, {}, "multiple of 4"),
    (10, (4,), 9, {}, "dtype"),
    (10, (4,), cd.U8, {"alpha_den": 9}, "alpha"),
    (10, (4,), cd.U8, {"alpha_num": 6}, "alpha"),
    (10, (4,), cd.U8, {"beta": -1.0}, "beta"),
    (10, (4,), cd.U8, {"frame_stack": 0}, "frame_stack"),
    (2, (4,), cd.U8, {"frame_stack": 4}, "frame_stack"),
    (10, (4,), cd.U8, {"action_bytes": 300}, "action_bytes"),
    (10, (6,), cd.I32, {"ragged": 1}, "multiple of 4"),
    (10, (8,), cd.U8, {"ragged": 1}, "ragged"),
    (10, (8,), cd.U8, {"aux_elem_bytes": 4}, "ragged"),
])
def test_create_rejects_bad_arguments(cap, shape, dtype, kw, msg):
    o = cd.default_opts(**kw)
    out = C.c_void_p()
    st = cd.lib().conduit_buffer_create(cap, _shape(*shape), len(shape), dtype, C.byref(o), None, 0, C.byref(out))
    assert st == cd.EINVAL
    assert msg in cd.last_error()
    assert out.value is None


def test_null_arguments_rejected():
    L = cd.lib()
    assert L.conduit_buffer_create(10, _shape(4), 1, cd.U8, None, None, 0, None) == cd.EINVAL
    assert L.conduit_ingest(None, None, None) == cd.EINVAL
    assert L.conduit_update_priorities(None, None, None, 1, None) == cd.EINVAL
    assert L.conduit_sample(None, 1, None, None, None, None) == cd.EINVAL
    assert L.conduit_gather_transform(None, None, 1, None, None, None) == cd.EINVAL
    assert L.conduit_buffer_get_info(None, None) == cd.EINVAL
    assert L.conduit_buffer_read(None, 0, 0, 0, 0, None, None) == cd.EINVAL
    assert L.conduit_buffer_stats(None, None, None, None) == cd.EINVAL
    assert L.conduit_buffer_checkpoint_bytes(None, None) == cd.EINVAL
    assert L.conduit_buffer_checkpoint(None, None, 0, None) == cd.EINVAL
    assert L.conduit_buffer_restore(None, None, 0, None) == cd.EINVAL
    L.conduit_buffer_destroy(None)  # no-op


def test_standalone_calls_validate_on_host():
    L = cd.lib()
    P = C.c_void_p(16)  # never dereferenced: validation fails first
    assert L.conduit_gae(None, None, None, None, 4, 4, 0.99, 0.95, None, None, None) == cd.EINVAL
    assert L.conduit_gae(P, None, P, None, -1, 4, 0.99, 0.95, P, P, None) == cd.EINVAL
    assert L.conduit_gae(P, None, P, None, 4, 4, float("nan"), 0.95, P, P, None) == cd.EINVAL
    assert L.conduit_gae(None, None, None, None, 0, 4, 0.99, 0.95, None, None, None) == cd.OK  # empty
    # [4, 4] rollouts: 64-byte float arrays, 16-byte flag arrays; outputs that
    # overlap each other or an input by one element are refused
    R, D, A, B, F, U = (C.c_void_p(k << 20) for k in range(1, 7))
    at = lambda p, off: C.c_void_p(p.value + off)  # noqa: E731
    assert L.conduit_gae(R, None, D, None, 4, 4, 0.99, 0.95, A, at(A, 60), None) == cd.EINVAL
    assert L.conduit_gae(R, None, D, None, 4, 4, 0.99, 0.95, at(R, 60), B, None) == cd.EINVAL
    assert L.conduit_gae(R, None, D, None, 4, 4, 0.99, 0.95, A, at(D, 15), None) == cd.EINVAL
    assert L.conduit_gae(R, A, D, None, 4, 4, 0.99, 0.95, at(A, -60), B, None) == cd.EINVAL
    assert "overlap" in cd.last_error()
    assert L.conduit_gae_truncated(R, None, D, U, F, None, 4, 4, 0.99, 0.95, at(F, 48), B, None) == cd.EINVAL
    assert L.conduit_gae_truncated(R, None, D, U, F, None, 4, 4, 0.99, 0.95, A, at(U, 15), None) == cd.EINVAL
    assert L.conduit_gae_packed(None, None, None, 2, 8, 1.0, 0.95, None, None, None) == cd.EINVAL
    assert L.conduit_gae_packed(None, None, None, 0, 8, 1.0, 0.95, None, None, None) == cd.OK
    xf = cd.transform(cd.XF_NONE)
    assert L.conduit_minibatch_gather(P, 4, 1, None, 1, C.byref(xf), P, None, None, 0, None) == cd.EINVAL
    assert L.conduit_minibatch_gather(P, 6, 1, P, 1, C.byref(xf), P, None, None, 0, None) == cd.EINVAL
    assert L.conduit_minibatch_gather(P, 4, 1, P, 1, C.byref(xf), P, None, None, 9, None) == cd.EINVAL
    tok = cd.transform(cd.XF_TOKENS_PAD)
    assert L.conduit_minibatch_gather(P, 4, 1, P, 1, C.byref(tok), P, None, None, 0, None) == cd.EINVAL
    bad = cd.transform(cd.XF_U8_BF16_NORM, (0.5, 0.5, 0.5), (0.2, 0.0, 0.2))
    assert L.conduit_minibatch_gather(P, 12, 1, P, 1, C.byref(bad), P, None, None, 0, None) == cd.EINVAL
    assert L.conduit_minibatch_gather(None, 4, 1, None, 0, C.byref(xf), None, None, None, 0, None) == cd.OK


def test_struct_layouts_match_header(tmp_path):
    """The ctypes mirrors have the sizes and field offsets the C compiler gives
    the header's structs."""
    import subprocess
    structs = {"conduit_buffer_opts": cd.BufferOpts, "conduit_transitions": cd.Transitions,
               "conduit_transform": cd.Transform, "conduit_learner_batch": cd.LearnerBatch,
               "conduit_buffer_info": cd.BufferInfo, "conduit_sched_costs": cd.SchedCosts,
               "conduit_sched_mode": cd.SchedMode, "conduit_offpolicy_loop": cd.OffpolicyLoop,
               "conduit_onpolicy_loop": cd.OnpolicyLoop, "conduit_place_profile": cd.PlaceProfile,
               "conduit_ckpt_section": cd.CkptSection, "conduit_ckpt_header": cd.CkptHeader}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "conduit.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} %zu\\n", sizeof({cname}));')
        for field, _ in py._fields_:
            lines.append(f'printf("{cname}.{field} %zu\\n", offsetof({cname}, {field}));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                 check=True).stdout.splitlines())
    for cname, py in structs.items():
        assert int(got[cname]) == C.sizeof(py), cname
        for field, _ in py._fields_:
            assert int(got[f"{cname}.{field}"]) == getattr(py, field).offset, (cname, field)


# (T, E, aligned) -> (path, chunk) that conduit_gae_plan reports (the GPU tests
# run these shapes and assert the same plan)
GAE_PLANS = [
    ((2048, 256, True), ("look", 2)),       # the PPO rollout: 8 groups x 32 segments
    ((2048, 1024, True), ("look", 8)),      # 256 tiles of 8-step chunks
    ((2048, 4096, True), ("look", 4)),      # 8-step chunks would give 1,152 tiles
    ((4097, 4100, True), ("look", 8)),      # 4-step chunks would need 4,257 tiles
    ((40000, 4, True), ("look", 4)),
    ((65, 4, True), ("look", 2)),           # two segments
    ((64, 4, True), ("short", 2)),          # one segment
    ((1, 4, True), ("short", 2)),
    ((33, 131072, True), ("short", 2)),     # any number of tiles
    ((1048576, 4, True), ("look", 8)),      # 4,096 tiles: the table's size
    ((1100000, 4, True), ("split", 8)),     # 4,297 tiles, fewer than 4,096 envs
    ((65, 131072, True), ("one_v4", 0)),    # 8,192 tiles, 4,096 envs or more
    ((2049, 65536, True), ("one_v4", 0)),
    ((2048, 256, False), ("look", 2)),      # rows off a 16-byte boundary: per-element tiles
    ((2048, 255, True), ("look", 2)),       # E not a multiple of 4: per-element tiles
    ((64, 4099, True), ("short", 2)),
    ((1100000, 3, True), ("split", 8)),     # 4,297 tiles of one partial group
    ((65, 131071, True), ("one", 0)),       # 8,192 tiles, 4,096 envs or more, E % 4 != 0
    ((65, 131072, False), ("one", 0)),
    ((0, 4, True), ("one_v4", 0)),          # empty rollouts enqueue nothing
]


@pytest.mark.parametrize("shape,plan", GAE_PLANS)
def test_gae_plan_on_the_host(shape, plan):
    T, E, aligned = shape
    assert cd.gae_plan(T, E, aligned) == plan


def test_gae_plan_validates():
    L = cd.lib()
    x = C.c_int32()
    assert L.conduit_gae_plan(-1, 4, 1, C.byref(x), C.byref(x)) == cd.EINVAL
    assert L.conduit_gae_plan(4, 4, 1, None, C.byref(x)) == cd.EINVAL


def test_single_stream_option():
    o = cd.default_opts()
    assert o.single_stream == 0
    shape = (C.c_int64 * 1)(8)
    o.single_stream = 2
    assert cd.lib().conduit_buffer_required_bytes(16, shape, 1, cd.F32, C.byref(o)) == 0
    o.single_stream = 1
    assert cd.lib().conduit_buffer_required_bytes(16, shape, 1, cd.F32, C.byref(o)) > 0


def test_expand_reference_validates_on_host():
    L = cd.lib()
    P, Q = C.c_void_p(1 << 20), C.c_void_p(16 << 20)  # never dereferenced: validation fails first
    assert L.conduit_expand_reference(None, None, 0, None) == cd.OK  # empty
    assert L.conduit_expand_reference(P, Q, -4, None) == cd.EINVAL
    assert L.conduit_expand_reference(P, Q, 6, None) == cd.EINVAL
    assert L.conduit_expand_reference(None, Q, 8, None) == cd.EINVAL
    assert L.conduit_expand_reference(P, C.c_void_p(Q.value + 4), 8, None) == cd.EINVAL  # dst not 16-byte aligned
    assert L.conduit_expand_reference(C.c_void_p(P.value + 2), Q, 8, None) == cd.EINVAL  # src not 4-byte aligned
    assert L.conduit_expand_reference(P, C.c_void_p(P.value + 16), 64, None) == cd.EINVAL
    assert "overlap" in cd.last_error()
