"""Host-only calls of libconduit, run against its AddressSanitizer +
UndefinedBehaviorSanitizer build (test_host_sanitizer.py builds it and runs
this file in a child process with the sanitizer runtime preloaded).

Only code that needs no GPU runs here: argument validation of every entry
point (pointers are never dereferenced: validation fails first), buffer
layouts, the GAE plan, the scheduling cost model and the placement algorithm.
No torch: the ABI declarations are loaded from abi.py by path.
Usage: python host_sanitizer_checks.py <library path>
"""
import ctypes as C
import importlib.util
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
spec = importlib.util.spec_from_file_location("abi", os.path.join(ROOT, "paper_2609_24456_amd", "abi.py"))
abi = importlib.util.module_from_spec(spec)
spec.loader.exec_module(abi)
L = abi.load(sys.argv[1])


def shape(*dims):
    return (C.c_int64 * len(dims))(*dims)


def opts(**kw):
    o = abi.BufferOpts()
    L.conduit_buffer_opts_default(C.byref(o))
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def expect(st, want, what):
    if st != want:
        raise SystemExit(f"{what}: status {st}, expected {want} ({L.conduit_last_error().decode()})")


assert b"gfx950" in L.conduit_version()

# layouts, valid and invalid
for cap, dims, dt, kw in [(1_000_000, (84, 84), abi.U8, dict(frame_stack=4)), (16384, (8,), abi.F32, {}),
                          (65536, (4096,), abi.I32, dict(ragged=1, aux_elem_bytes=4, action_bytes=0)),
                          (200_000, (3, 224, 224), abi.U8, dict(action_bytes=24)), (1, (4,), abi.U8, {}),
                          ((1 << 31) - 1, (4,), abi.U8, {}), (1000, (64,), abi.U8, dict(payload_placement=1)),
                          (1000, (64,), abi.U8, dict(prioritized=0)), (0, (4,), abi.U8, {}), (10, (3,), abi.U8, {}),
                          (10, (4,), 9, {}), (10, (4,), abi.U8, dict(alpha_den=9)),
                          (2, (4,), abi.U8, dict(frame_stack=4)), (10, (6,), abi.I32, dict(ragged=1)),
                          (1000, (64,), abi.U8, dict(payload_placement=2))]:
    o = opts(**kw)
    L.conduit_buffer_required_bytes(cap, shape(*dims), len(dims), dt, C.byref(o))
    L.conduit_buffer_required_bytes(cap, shape(*dims), len(dims), dt, None)
out = C.c_void_p()
for cap, dims, dt, kw in [(0, (4,), abi.U8, {}), (10, (3,), abi.U8, {}), (10, (4,), abi.U8, dict(beta=-1.0)),
                          (10, (4,), abi.U8, dict(action_bytes=300)), (10, (8,), abi.U8, dict(aux_elem_bytes=4)),
                          (10, (4,), abi.U8, dict(single_stream=2)), (10, (4,), abi.U8, dict(weight_norm=7))]:
    expect(L.conduit_buffer_create(cap, shape(*dims), len(dims), dt, C.byref(opts(**kw)), None, 0, C.byref(out)),
           abi.EINVAL, f"create {cap} {dims} {kw}")
expect(L.conduit_buffer_create(10, None, 1, abi.U8, None, None, 0, C.byref(out)), abi.EINVAL, "create NULL shape")

# NULL buffers and arguments
expect(L.conduit_ingest(None, None, None), abi.EINVAL, "ingest")
expect(L.conduit_update_priorities(None, None, None, 1, None), abi.EINVAL, "update")
expect(L.conduit_sample(None, 1, None, None, None, None), abi.EINVAL, "sample")
expect(L.conduit_gather_transform(None, None, 1, None, None, None), abi.EINVAL, "gather")
expect(L.conduit_buffer_get_info(None, None), abi.EINVAL, "info")
expect(L.conduit_buffer_stats(None, None, None, None), abi.EINVAL, "stats")
expect(L.conduit_buffer_read(None, 0, 0, 0, 0, None, None), abi.EINVAL, "read")
expect(L.conduit_buffer_checkpoint_bytes(None, None), abi.EINVAL, "checkpoint bytes")
expect(L.conduit_buffer_checkpoint(None, None, 0, None), abi.EINVAL, "checkpoint")
expect(L.conduit_buffer_restore(None, None, 0, None), abi.EINVAL, "restore")
L.conduit_buffer_destroy(None)

# stand-alone calls: validation and overlap checks on fake addresses
P = C.c_void_p(16)
R, D, A, B, F, U = (C.c_void_p(k << 20) for k in range(1, 7))


def at(p, off):
    return C.c_void_p(p.value + off)


expect(L.conduit_gae(None, None, None, None, 4, 4, 0.99, 0.95, None, None, None), abi.EINVAL, "gae NULL")
expect(L.conduit_gae(P, None, P, None, -1, 4, 0.99, 0.95, P, P, None), abi.EINVAL, "gae T")
expect(L.conduit_gae(P, None, P, None, 4, 4, float("nan"), 0.95, P, P, None), abi.EINVAL, "gae gamma")
expect(L.conduit_gae(R, None, D, None, 4, 4, 0.99, 0.95, A, at(A, 60), None), abi.EINVAL, "gae overlap")
expect(L.conduit_gae_noalloc(R, None, D, None, 4, 4, 0.99, 0.95, A, at(A, 60), None), abi.EINVAL, "noalloc")
expect(L.conduit_gae_truncated(R, None, D, U, F, None, 4, 4, 0.99, 0.95, at(F, 48), B, None), abi.EINVAL, "trunc")
expect(L.conduit_gae_packed(None, None, None, 2, 8, 1.0, 0.95, None, None, None), abi.EINVAL, "packed")
xf = abi.Transform()
xf.kind = abi.XF_NONE
expect(L.conduit_minibatch_gather(P, 4, 1, None, 1, C.byref(xf), P, None, None, 0, None), abi.EINVAL, "minibatch")
expect(L.conduit_minibatch_gather(P, 4, 1, P, 1, C.byref(xf), P, None, None, 9, None), abi.EINVAL, "minibatch cols")
expect(L.conduit_expand_reference(P, at(P, 16), 64, None), abi.EINVAL, "expand overlap")
expect(L.conduit_expand_reference(P, C.c_void_p(16 << 20), 6, None), abi.EINVAL, "expand n")

# the GAE plan over shapes
path, chunk = C.c_int32(), C.c_int32()
for T in (0, 1, 63, 64, 65, 2048, 40000, 1100000):
    for E in (1, 3, 4, 255, 256, 4099, 131072):
        for aligned in (0, 1):
            expect(L.conduit_gae_plan(T, E, aligned, C.byref(path), C.byref(chunk)), abi.OK, f"plan {T} {E}")
expect(L.conduit_gae_plan(-1, 4, 1, C.byref(path), C.byref(chunk)), abi.EINVAL, "plan T < 0")

# the scheduling cost model: every mode of a few configurations, and its errors
for on_policy in (0, 1):
    for gi, gd in (([1.0], [1.0]), ([1.0, 2.0, 4.0], [1.0, 2.0]), ([0.25, 0.5, 1.0], [1.0, 8.0])):
        if on_policy and max(gi + gd) > 1.0:  # on-policy granularities are fractions of the rollout
            continue
        arr = lambda xs: (C.c_double * len(xs))(*xs)  # noqa: E731
        c = abi.SchedCosts(600.0, 800.0, 12.0, 14.0, len(gi), len(gd), arr(gi), arr([50.0 * g for g in gi]),
                           arr(gd), arr([30.0 * g for g in gd]), on_policy)
        best = abi.SchedMode()
        modes = (abi.SchedMode * (4 * len(gi) * len(gd)))()
        expect(L.conduit_schedule(C.byref(c), C.byref(best), modes), abi.OK, f"schedule {gi} {gd}")
        c.n_ing = 0
        expect(L.conduit_schedule(C.byref(c), C.byref(best), modes), abi.EINVAL, "schedule empty set")
cap = 64
gi, gd, ni, nd = (C.c_double * cap)(), (C.c_double * cap)(), C.c_int32(), C.c_int32()
for args in ((0, 1, 8, 8), (1, 32, 1, 1), (1, 4, 1, 1), (0, 1, 1, 16)):
    expect(L.conduit_sched_candidates(*args, gi, cap, C.byref(ni), gd, cap, C.byref(nd)), abi.OK, f"cand {args}")
expect(L.conduit_sched_candidates(1, 0, 1, 1, gi, cap, C.byref(ni), gd, cap, C.byref(nd)), abi.EINVAL, "cand 0")
expect(L.conduit_sched_candidates(0, 1, cap + 1, 1, gi, cap, C.byref(ni), gd, cap, C.byref(nd)), abi.EINVAL,
       "cand arrays too small")

# the placement algorithm over a synthetic bandwidth profile
prof = abi.PlaceProfile()
for i, (bi, bg, bo, m) in enumerate(((50e9, 400e9, 4000e9, 288e9), (25e9, 50e9, 50e9, 1e12), (10e9, 20e9, 20e9, 2e12))):
    prof.bw_in[0][i], prof.bw_in[1][i], prof.bw_out[i], prof.mem[i] = bi, bg, bo, m
choice, t = C.c_int32(), (C.c_double * 3)()
for actor_on_gpu in (0, 1):
    for capacity, sample in ((1_000_000, 7056.0), (200_000, 150528.0), (10 ** 7, 160000.0)):
        cand = (C.c_int32 * 3)(0, 1, 2)
        expect(L.conduit_place(C.byref(prof), actor_on_gpu, capacity, sample, cand, 3, C.byref(choice), t), abi.OK,
               f"place {capacity}")
bad = (C.c_int32 * 1)(7)
expect(L.conduit_place(C.byref(prof), 0, 1000, 64.0, bad, 1, C.byref(choice), t), abi.EINVAL, "place candidate")
print("host checks ok", flush=True)
