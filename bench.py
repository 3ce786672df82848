"""Benchmark of the experience path on one MI355X.

Headline workload (the configuration the metric is quoted on): DQN replay of
1,000,000 single 84x84 uint8 frames, frame stack 4, batch 512, proportional
prioritisation alpha 0.6 / beta 0.4.  One step = ingest 512 new frames + sample
512 + gather/transform 512 -> [512, 4, 84, 84] fp32 + priority update 512, as
two calls per step: conduit_update_ingest (the previous step's priority update
with this step's ingest) and conduit_sample_gather (sampling, IS weights and
the gather in one launch).  The same steps with a separate update call and
through separate conduit_sample / conduit_gather_transform calls are reported
beside it.  Inputs (frames of the steps, uniforms, new priorities) are resident
in HBM before the timed region.

Prints ONE JSON line on stdout, the last line and compact: the headline, the
roofline of the dominant kernel, the oracle timed on the host cores
(cpu_baseline: one pinned core, median of 5 reps, and every allowed core with
one instance each; timed in forked children before this process touches the
GPU) and a few figures of each other workload's row (DQN ingest and n-step
targets, PPO rollout ingest + GAE + minibatch gather, large-payload bf16
gather, token packing + packed GAE, tiny replay latency, the synthetic stress
transitions, the scheduling model against measured schedules, placement).
Each row's full record goes to stderr as a line 'bench.detail {...}' (and to
--detail-out).  The rows are timed GPU-paced (a stand-in kernel queued ahead
of the first event), so each brackets GPU time only.
"""
import argparse
import ctypes as C
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published
METRIC = "sampled transitions/sec + gather HBM GB/s (% of peak), DQN 1M-replay config"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-rows", action="store_true", help="only the headline DQN workload")
    p.add_argument("--only", default="", help="comma list of extra rows to run (ppo,large,tokens,tiny,stress,schedule)")
    p.add_argument("--calibrate-copy", action="store_true", help="run a plain 1 GiB device copy (counter scale)")
    p.add_argument("--sources-sha", action="store_true",
                   help="print the hash of the fused kernel's sources (for the counter summary)")
    p.add_argument("--cpu-rep-seconds", type=float, default=2.0, help="seconds per timed rep of the oracle")
    p.add_argument("--detail-out", default="", help="also append the per-row JSON records to this file")
    return p.parse_args()


# ----------------------------------------------------------------------------
# helpers
# ----------------------------------------------------------------------------
def _dev(a):
    import numpy as np
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    elif a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).cuda()


class Timer:
    """HIP events on the stream the library launches on (torch's current stream)."""

    def __init__(self):
        import torch
        self.torch = torch

    def ev(self):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        return e


_DELAY_US_PER_WORK = []


def _gpu_delay(us):
    """Enqueue about `us` microseconds of GPU work (the library's register-only
    stand-in kernel, one workgroup per compute unit) on torch's current stream."""
    import torch
    from paper_2609_24456_amd import conduit as cd
    if not _DELAY_US_PER_WORK:
        probe = 200_000
        cd.conduit_standin(probe)  # loads its code
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        cd.conduit_standin(probe)
        e1.record()
        torch.cuda.synchronize()
        _DELAY_US_PER_WORK.append(max(e0.elapsed_time(e1) * 1e3 / probe, 1e-6))
    cd.conduit_standin(int(us / _DELAY_US_PER_WORK[0]) + 1)


def _b2b_ms(calls, reps=1, warm=2):
    """Milliseconds per call of `calls` (zero-argument callables that enqueue
    on the library's stream, torch's current stream), launched back to back
    between two events, after `warm` untimed calls (a kernel's first launch
    loads its code).  The GPU is paced: a stand-in kernel queued ahead of the
    first event outlasts the host's enqueue of every timed call, so the events
    bracket GPU time only, also for calls whose kernels are shorter than their
    host-side enqueue (Python + ctypes, a few microseconds per call)."""
    import torch
    per_call_us = 15.0
    for i, f in enumerate(calls[:warm]):
        t0 = time.perf_counter()
        f()
        if i > 0:  # the first call may include loading code
            per_call_us = max(per_call_us, 1.5e6 * (time.perf_counter() - t0))
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    rc = 0
    _gpu_delay(min(per_call_us * reps * len(calls) + 500.0, 30_000.0))
    e0.record()
    for _ in range(reps):
        for f in calls:
            rc |= f()
    e1.record()
    torch.cuda.synchronize()
    assert rc == 0, "a timed call failed"
    return e0.elapsed_time(e1) / (reps * len(calls))


def _kernel_stats(durs_ms):
    import numpy as np
    d = np.asarray(durs_ms)
    return {"mean_us": float(d.mean() * 1e3), "median_us": float(np.median(d) * 1e3)}


# ----------------------------------------------------------------------------
# headline: DQN 1M replay
# ----------------------------------------------------------------------------
def bench_dqn(steps, warmup):
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd

    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    Cap, B, K, prefill, chunk = 1_000_000, 512, 4, 1_050_000, 4096
    # passes: timed headline, separate-update and unfused (each after one
    # untimed step of its own), two instrumented
    iters = warmup + 5 * steps + 2
    cfg = synth.DQN(prefill + iters * B)
    buf = cd.ReplayBuffer(Cap, (84, 84), torch.uint8, frame_stack=K, action_bytes=4)
    t0 = time.time()
    for a in range(0, prefill, chunk):
        b = min(prefill, a + chunk)
        buf.ingest(cfg.frames(a, b - a, "cuda"), action=_dev(cfg.action[a:b]), reward=_dev(cfg.reward[a:b]),
                   done=_dev(cfg.done[a:b]), episode_id=_dev(cfg.episode[a:b]), step=_dev(cfg.step[a:b]),
                   prio=_dev(cfg.prio[a:b]))
    torch.cuda.synchronize()
    prefill_s = time.time() - t0

    # prefill-style ingest throughput: 32768-frame chunks, the call's argument
    # struct prepared up front, back-to-back launches (GPU-paced)
    big = cfg.frames(0, 32768, "cuda")
    meta = [_dev(x[:32768]) for x in (cfg.action, cfg.reward, cfg.done, cfg.episode, cfg.step)]
    bigp = _dev(cfg.prio[:32768])
    tb = cd.Transitions()
    tb.n = 32768
    tb.obs = big.data_ptr()
    tb.action, tb.reward, tb.done = meta[0].data_ptr(), meta[1].data_ptr(), meta[2].data_ptr()
    tb.episode_id, tb.step, tb.prio = meta[3].data_ptr(), meta[4].data_ptr(), bigp.data_ptr()
    hb = C.c_void_p(buf.handle)
    st_b = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    ingest_big_ms = _b2b_ms([lambda: cd.lib().conduit_ingest(hb, C.byref(tb), st_b)] * 6)
    torch.cuda.synchronize()
    del big
    tm = Timer()

    # stage every step's inputs in HBM
    s0 = prefill
    frames = cfg.frames(s0, iters * B, "cuda")
    act = _dev(cfg.action[s0:s0 + iters * B])
    rew = _dev(cfg.reward[s0:s0 + iters * B])
    done = _dev(cfg.done[s0:s0 + iters * B])
    epi = _dev(cfg.episode[s0:s0 + iters * B])
    stp = _dev(cfg.step[s0:s0 + iters * B])
    u, prio = cfg.draws(iters, B)
    u_d, prio_d = _dev(u), _dev(prio)
    idx = torch.empty((iters, B), dtype=torch.int64, device="cuda")
    w = torch.empty((iters, B), dtype=torch.float32, device="cuda")
    obs_out = torch.empty((B, K, 84, 84), dtype=torch.float32, device="cuda")
    act_out = torch.empty(B, dtype=torch.int32, device="cuda")
    rew_out = torch.empty(B, dtype=torch.float32, device="cuda")
    done_out = torch.empty(B, dtype=torch.uint8, device="cuda")
    xf = cd.transform(cd.XF_U8_F32)
    lb = cd.LearnerBatch()
    lb.obs, lb.action, lb.reward, lb.done = obs_out.data_ptr(), act_out.data_ptr(), rew_out.data_ptr(), done_out.data_ptr()
    # every call's arguments prepared up front: the timed loop only enters the C ABI
    trans = []
    for i in range(iters):
        t = cd.Transitions()
        sl = slice(i * B, (i + 1) * B)
        t.n = B
        t.obs = frames[sl].data_ptr()
        t.action, t.reward, t.done = act[sl].data_ptr(), rew[sl].data_ptr(), done[sl].data_ptr()
        t.episode_id, t.step = epi[sl].data_ptr(), stp[sl].data_ptr()
        t.prio = None
        trans.append(t)
    h = C.c_void_p(buf.handle)
    ing, smp, gat, upd = L.conduit_ingest, L.conduit_sample, L.conduit_gather_transform, L.conduit_update_priorities
    sgat = L.conduit_sample_gather
    pu = [u_d[i].data_ptr() for i in range(iters)]
    pp = [prio_d[i].data_ptr() for i in range(iters)]
    pi = [idx[i].data_ptr() for i in range(iters)]
    pw = [w[i].data_ptr() for i in range(iters)]
    xfr, lbr = C.byref(xf), C.byref(lb)

    def step(i):  # ingest, fused sample + gather (+ IS weights), priority update
        r = ing(h, C.byref(trans[i]), stream)
        r |= sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
        r |= upd(h, pi[i], pp[i], B, stream)
        return r

    uing = L.conduit_update_ingest

    def step_ui(i):  # step i-1's priority update with step i's ingest (one call), fused sample + gather
        r = uing(h, pi[i - 1], pp[i - 1], B, C.byref(trans[i]), stream)
        r |= sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
        return r

    def step_unfused(i):  # the same step with separate sample and gather calls
        r = ing(h, C.byref(trans[i]), stream)
        r |= smp(h, B, pu[i], pi[i], pw[i], stream)
        r |= gat(h, pi[i], B, xfr, lbr, stream)
        r |= upd(h, pi[i], pp[i], B, stream)
        return r

    # warm-up through the timed step's own calls (every kernel loaded before
    # the clock starts); its last update is left to the first timed step
    rc = ing(h, C.byref(trans[0]), stream)
    rc |= sgat(h, B, pu[0], pi[0], pw[0], xfr, lbr, stream)
    for i in range(1, warmup):
        rc |= step_ui(i)
    assert rc == 0, cd.last_error()
    torch.cuda.synchronize()
    # timed pass: each step applies the previous step's update with its own
    # ingest, so K steps hold K ingests, K samples + gathers and K updates.  A
    # stand-in kernel queued ahead of the first event keeps the GPU busy while
    # the host enqueues the first steps, so the events bracket GPU time only
    _gpu_delay(1000.0)
    e_start = tm.ev()
    h0 = time.perf_counter()
    rc = 0
    for i in range(warmup, warmup + steps):
        rc |= step_ui(i)
    e_end = tm.ev()
    host_enqueue_s = time.perf_counter() - h0
    rc |= upd(h, pi[warmup + steps - 1], pp[warmup + steps - 1], B, stream)  # after the clock
    torch.cuda.synchronize()
    assert rc == 0, cd.last_error()
    total_ms = e_start.elapsed_time(e_end)
    # the same number of steps with the update as a call of its own
    p1 = warmup + steps
    rc |= step(p1)  # one untimed step first
    torch.cuda.synchronize()
    _gpu_delay(1000.0)
    s_start = tm.ev()
    for i in range(p1 + 1, p1 + 1 + steps):
        rc |= step(i)
    s_end = tm.ev()
    torch.cuda.synchronize()
    assert rc == 0, cd.last_error()
    separate_ms = s_start.elapsed_time(s_end)
    # and through separate sample and gather calls too
    p2 = p1 + 1 + steps
    rc |= step_unfused(p2)
    torch.cuda.synchronize()
    _gpu_delay(1000.0)
    u_start = tm.ev()
    for i in range(p2 + 1, p2 + 1 + steps):
        rc |= step_unfused(i)
    u_end = tm.ev()
    torch.cuda.synchronize()
    assert rc == 0, cd.last_error()
    unfused_ms = u_start.elapsed_time(u_end)
    # instrumented passes: an event between consecutive calls
    p3 = p2 + 1 + steps
    evs = []
    for i in range(p3, p3 + steps):
        e = [tm.ev()]
        ing(h, C.byref(trans[i]), stream)
        e.append(tm.ev())
        sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
        e.append(tm.ev())
        upd(h, pi[i], pp[i], B, stream)
        e.append(tm.ev())
        evs.append(e)
    ui_durs = []
    p4 = p3 + steps
    for i in range(p4, p4 + steps):
        e0 = tm.ev()
        uing(h, pi[i - 1], pp[i - 1], B, C.byref(trans[i]), stream)
        e1 = tm.ev()
        sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
        ui_durs.append((e0, e1))
    upd(h, pi[p4 + steps - 1], pp[p4 + steps - 1], B, stream)
    torch.cuda.synchronize()
    ui_stats = _kernel_stats([a.elapsed_time(b) for a, b in ui_durs])
    assert buf.sync_check() == cd.OK, cd.last_error()
    # kernels alone, back to back between two events on the library's stream,
    # over the timed steps' own inputs: the fused sampler + gather (the dominant
    # kernel of the step, weights included as in the step) and the stand-alone
    # gather of the same batches
    fb0 = tm.ev()
    for i in range(warmup, warmup + steps):
        sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
    fb1 = tm.ev()
    for i in range(warmup, warmup + steps):
        gat(h, pi[i], B, xfr, lbr, stream)
    gb1 = tm.ev()
    torch.cuda.synchronize()
    fused_b2b_ms = fb0.elapsed_time(fb1) / steps
    gather_b2b_ms = fb1.elapsed_time(gb1) / steps
    names = ["ingest_512", "sample_gather_512 (sampler + gather launches)", "update_512"]
    per = {n: [e[k].elapsed_time(e[k + 1]) for e in evs] for k, n in enumerate(names)}
    kern = {n: _kernel_stats(v) for n, v in per.items()}

    # algorithmic bytes of the gather of the last instrumented step: frames the
    # stack actually reads (zero-filled frames are not read), 4x-wide writes,
    # plus the index and the three scalar columns
    last = idx[warmup + steps - 1].cpu().numpy()
    ep_col = torch.empty(Cap * 4, dtype=torch.uint8, device="cuda")
    st_col = torch.empty(Cap * 4, dtype=torch.uint8, device="cuda")
    buf.read(cd.COL_EPISODE, ep_col)
    buf.read(cd.COL_STEP, st_col)
    torch.cuda.synchronize()
    ep_h = ep_col.cpu().numpy().view(np.uint32)
    st_h = st_col.cpu().numpy().view(np.int32)
    valid = 0
    for i in last:
        for d in range(K):
            j = (i - d) % Cap
            if d == 0 or (d <= st_h[i] and ep_h[j] == ep_h[i] and st_h[j] == st_h[i] - d):
                valid += 1
    row = 84 * 84
    # gather: valid source frames, the index, the episode/step of the two slots
    # each stacked frame compares, action/reward/done in and out, the output
    gather_bytes = valid * row + B * (8 + 4 + 4 + 1) + B * K * row * 4 + B * (4 + 4 + 1)
    # fused sampler + gather: no index read; per sample one descent (the total,
    # 64 children at each of depth-1 node levels and 64 leaves), the uniform,
    # and the index and weight written
    depth = buf.info().tree_depth
    descent_bytes = 8 + (depth - 1) * 64 * 8 + 64 * 4
    fused_bytes = gather_bytes - B * 8 + B * (descent_bytes + 8 + 8 + 4)
    ingest_bytes_per_frame = 2 * row + (4 + 4 + 1 + 4 + 4) * 2 + 4 + 4  # obs r+w, scalars r+w, leaf r+w
    # n-step targets (n = 3, gamma 0.99) and bootstrap stacks of the timed
    # steps' samples, back to back, and the step with them
    n_step, gam = 3, 0.99
    nxt = torch.empty(B, dtype=torch.int64, device="cuda")
    nret = torch.empty(B, dtype=torch.float32, device="cuda")
    ndisc = torch.empty(B, dtype=torch.float32, device="cuda")
    nval = torch.empty(B, dtype=torch.uint8, device="cuda")
    next_out = torch.empty((B, K, 84, 84), dtype=torch.float32, device="cuda")
    nst = L.conduit_nstep
    ns_args = (nxt.data_ptr(), nret.data_ptr(), ndisc.data_ptr(), nval.data_ptr(), xfr, next_out.data_ptr(), stream)
    ns_calls = [lambda i=i: nst(h, pi[i], B, n_step, gam, *ns_args) for i in range(warmup, warmup + steps)]
    _b2b_ms(ns_calls[:5])
    nstep_ms = _b2b_ms(ns_calls)
    boot = int(nval.sum().item())
    # delivery with n-step targets and bootstrap stacks: one call
    # (conduit_sample_gather_nstep, one launch that reads every frame of the
    # two stacks once) against conduit_sample_gather + conduit_nstep
    sgn = L.conduit_sample_gather_nstep
    one_calls = [lambda i=i: sgn(h, B, pu[i], pi[i], pw[i], xfr, lbr, n_step, gam, nxt.data_ptr(), nret.data_ptr(),
                                 ndisc.data_ptr(), nval.data_ptr(), next_out.data_ptr(), stream)
                 for i in range(warmup, warmup + steps)]
    two_calls = [lambda i=i: sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream) | nst(h, pi[i], B, n_step, gam, *ns_args)
                 for i in range(warmup, warmup + steps)]
    _b2b_ms(one_calls[:5])
    _b2b_ms(two_calls[:5])
    deliver_nstep_one_ms = _b2b_ms(one_calls)
    deliver_nstep_two_ms = _b2b_ms(two_calls)
    assert buf.sync_check() == cd.OK, cd.last_error()
    ckpt = _checkpoint_times(buf)
    buf.close()
    # references for the batch's read/write mix over B x K frames laid out
    # contiguously (no sampling, no gather): the library's streaming expand
    # (conduit_expand_reference) and torch's elementwise u8 -> fp32 scale
    ref_bytes, ref_ms, torch_ms = _expand_references(B * K * row, next_out.view(-1), steps, stream)
    return {
        "nstep3": {"us": nstep_ms * 1e3, "n": n_step, "gamma": gam, "valid_in_last_batch": boot,
                   "call": "conduit_nstep: targets plus the bootstrap frame stacks [512,4,84,84] fp32"},
        "deliver_nstep3": {"one_call_us": deliver_nstep_one_ms * 1e3, "two_calls_us": deliver_nstep_two_ms * 1e3,
                           "call": "conduit_sample_gather_nstep (sample 512, [512,4,84,84] fp32 batch, n = 3 "
                                   "targets and bootstrap stacks) against conduit_sample_gather + conduit_nstep"},
        "B": B, "steps": steps, "warmup": warmup, "total_ms": total_ms, "host_enqueue_s": host_enqueue_s,
        "gather_b2b_ms": gather_b2b_ms, "fused_b2b_ms": fused_b2b_ms, "unfused_ms": unfused_ms,
        "separate_ms": separate_ms, "update_ingest_call": ui_stats,
        "kernels": kern, "gather_bytes": gather_bytes, "fused_bytes": fused_bytes, "descent_bytes": descent_bytes,
        "valid_frames": valid, "prefill_s": prefill_s,
        "ingest_big": {"frames": 32768, "ms": ingest_big_ms,
                       "GBps": 32768 * ingest_bytes_per_frame / ingest_big_ms / 1e6},
        "ingest_bytes_per_frame": ingest_bytes_per_frame,
        "expand_reference": _expand_record(ref_bytes, ref_ms, torch_ms, "the batch's 512 x 4 frames"),
        "checkpoint": ckpt,
    }


# ----------------------------------------------------------------------------
# other rows
# ----------------------------------------------------------------------------
def _checkpoint_times(buf):
    """Wall time of a checkpoint of the whole buffer into HBM and into pinned
    host memory, and of restoring it from HBM (the copies plus the tree
    rebuild); each call waits for its own copies.  The image is restored into
    the buffer it came from, so the state does not change."""
    import torch
    from paper_2609_24456_amd import conduit as cd
    n = cd.conduit_buffer_checkpoint_bytes(buf.handle)
    out = {"image_bytes": n}
    img = torch.empty(n, dtype=torch.uint8, device="cuda")
    for name, fn in (("checkpoint_hbm", lambda: buf.checkpoint(dst=img)), ("restore_hbm", lambda: buf.restore(img))):
        fn()  # first call: page-in, code load
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        out[name] = {"ms": dt * 1e3, "GBps": n / dt / 1e9}
    del img
    host = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    buf.checkpoint(dst=host)
    t0 = time.perf_counter()
    buf.checkpoint(dst=host)
    dt = time.perf_counter() - t0
    out["checkpoint_pinned_host"] = {"ms": dt * 1e3, "GBps": n / dt / 1e9}
    del host
    assert buf.sync_check() == cd.OK, cd.last_error()
    return out


def _expand_references(n, out_f32, calls, stream):
    """(bytes, ms, torch ms) of u8 -> fp32 over n contiguous bytes into
    out_f32: conduit_expand_reference (a streaming kernel with the gathers'
    1:4 read/write mix and none of their indexing) and torch.mul(u8, 1/255)."""
    import torch
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = out_f32[:n]
    ref = lambda: L.conduit_expand_reference(src.data_ptr(), dst.data_ptr(), n, stream)  # noqa: E731
    tch = lambda: torch.mul(src, 1.0 / 255.0, out=dst) is None  # noqa: E731  (a status of 0)
    _b2b_ms([ref] * 3)
    ref_ms = _b2b_ms([ref] * calls)
    _b2b_ms([tch] * 3)
    torch_ms = _b2b_ms([tch] * calls)
    return 5 * n, ref_ms, torch_ms


def _expand_record(nbytes, ref_ms, torch_ms, what):
    return {"bytes": nbytes, "us": ref_ms * 1e3, "GBps": nbytes / ref_ms / 1e6,
            "frac": nbytes / ref_ms / 1e6 / PEAK_HBM_GBPS,
            "torch_us": torch_ms * 1e3, "torch_frac": nbytes / torch_ms / 1e6 / PEAK_HBM_GBPS,
            "what": "u8 -> fp32 /255 over " + what + " laid out contiguously (the same 1:4 read/write mix, no "
                    "indexing): conduit_expand_reference, and torch.mul(u8, 1/255, out=fp32) beside it"}


def bench_ppo(reps=3):
    """PPO rollout [2048 x 256] of 3x84x84 u8: rollout ingest (32 calls of 64
    steps), GAE over [T, E], and the 32 minibatch gathers of one epoch; each
    timed as back-to-back launches with prepared arguments."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    cfg = synth.PPO()
    T, E, row = cfg.T, cfg.E, 3 * 84 * 84
    N = T * E
    # rollout ingest into an on-policy buffer (no priorities), 64 steps per call
    buf = cd.ReplayBuffer(N, cfg.obs_shape, torch.uint8, prioritized=False, action_bytes=0)
    obs_all = cfg.obs_steps(0, T, "cuda")
    rew_d, done_d = _dev(cfg.reward.reshape(-1)), _dev(cfg.done.reshape(-1))
    structs = []
    for t0 in range(0, T, 64):
        t = cd.Transitions()
        sl = slice(t0 * E, (t0 + 64) * E)
        t.n = 64 * E
        t.obs = obs_all[t0:t0 + 64].data_ptr()
        t.reward, t.done = rew_d[sl].data_ptr(), done_d[sl].data_ptr()
        structs.append(t)
    h = C.c_void_p(buf.handle)
    torch.cuda.synchronize()
    ing_ms = _b2b_ms([lambda t=t: L.conduit_ingest(h, C.byref(t), stream) for t in structs]) * len(structs)
    del obs_all
    src = torch.empty(N * row, dtype=torch.uint8, device="cuda")
    buf.read(cd.COL_OBS, src)
    torch.cuda.synchronize()
    buf.close()
    r, v, d, b = _dev(cfg.reward), _dev(cfg.value), _dev(cfg.done), _dev(cfg.bootstrap)
    adv = torch.empty((T, E), dtype=torch.float32, device="cuda")
    ret = torch.empty((T, E), dtype=torch.float32, device="cuda")
    gae_args = (r.data_ptr(), v.data_ptr(), d.data_ptr(), b.data_ptr(), T, E, cfg.gamma, cfg.lam,
                adv.data_ptr(), ret.data_ptr(), stream)
    gae = lambda: L.conduit_gae(*gae_args)  # noqa: E731
    _b2b_ms([gae] * 3)
    gae_ms = _b2b_ms([gae] * 20)
    gae_bytes = N * (4 + 4 + 1 + 4 + 4) + E * 4
    A, R = adv.view(-1), ret.view(-1)
    mb = 16384
    perm = _dev(cfg.perm)
    out = torch.empty((mb, 3, 84, 84), dtype=torch.float32, device="cuda")
    a_out = torch.empty(mb, dtype=torch.float32, device="cuda")
    r_out = torch.empty(mb, dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_U8_F32)
    cols = (C.c_void_p * 2)(A.data_ptr(), R.data_ptr())
    cols_out = (C.c_void_p * 2)(a_out.data_ptr(), r_out.data_ptr())
    calls = [lambda m=m: L.conduit_minibatch_gather(src.data_ptr(), row, N, perm[m * mb:(m + 1) * mb].data_ptr(), mb,
                                                    C.byref(xf), out.data_ptr(), cols, cols_out, 2, stream)
             for m in range(32)]
    _b2b_ms(calls)  # first epoch: warm-up
    mb_ms = _b2b_ms(calls, reps=reps - 1 if reps > 1 else 1)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    mb_bytes = mb * (row + row * 4 + 8 + 2 * 4 + 2 * 4)
    ing_bytes = N * (2 * row + 2 * (4 + 1) + 2 * (4 + 4))
    # references for the read/write mix over the same bytes laid out
    # contiguously (no index, no scattered rows)
    ex_bytes, ex_ms, ex_torch_ms = _expand_references(mb * row, out.view(-1), 10, stream)
    return {
        "rollout_ingest": {"bytes": ing_bytes, "ms": ing_ms, "GBps": ing_bytes / ing_ms / 1e6,
                           "frac": ing_bytes / ing_ms / 1e6 / PEAK_HBM_GBPS},
        "gae_2048x256": {"bytes": gae_bytes, "us": gae_ms * 1e3, "GBps": gae_bytes / gae_ms / 1e6,
                         "frac": gae_bytes / gae_ms / 1e6 / PEAK_HBM_GBPS,
                         "kernels": "%s, %d-step chunks (conduit_gae_plan)" % cd.gae_plan(T, E)},
        "minibatch_gather_16384": {"bytes": mb_bytes, "us": mb_ms * 1e3, "GBps": mb_bytes / mb_ms / 1e6,
                                   "frac": mb_bytes / mb_ms / 1e6 / PEAK_HBM_GBPS},
        "epoch_32_minibatches_ms": mb_ms * 32,
        "expand_reference": _expand_record(ex_bytes, ex_ms, ex_torch_ms, "one minibatch's 16,384 frames"),
        "minibatch_over_expand_reference": (mb_bytes / mb_ms) / (ex_bytes / ex_ms),
        "timing": "back-to-back launches between two events, arguments prepared up front",
    }


def bench_large(iters=10):
    """Large visual replay (200,000 slots of 3x224x224 u8): sample 1,024 (with
    IS weights), gather -> normalised bf16 [1024, 3, 224, 224] with action and
    reward, update 1,024; each call type timed as back-to-back launches with
    prepared arguments, and whole iterations through the sample + gather call."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    Cap, B, row = 200_000, 1024, 3 * 224 * 224
    cfg = synth.Large(Cap)
    buf = cd.ReplayBuffer(Cap, cfg.obs_shape, torch.uint8, action_bytes=24)
    for a in range(0, Cap, 2048):
        b = min(Cap, a + 2048)
        buf.ingest(cfg.rows(a, b - a, "cuda"), action=_dev(cfg.action[a:b]), reward=_dev(cfg.reward[a:b]),
                   done=_dev(cfg.done[a:b]), prio=_dev(cfg.prio[a:b]))
    u, prio = cfg.draws(iters, B)
    u_d, p_d = _dev(u), _dev(prio)
    idx = torch.empty((iters, B), dtype=torch.int64, device="cuda")
    w = torch.empty((iters, B), dtype=torch.float32, device="cuda")
    out = torch.empty((B, 1) + cfg.obs_shape, dtype=torch.bfloat16, device="cuda")
    act = torch.empty((B, 6), dtype=torch.float32, device="cuda")
    rew = torch.empty(B, dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_U8_BF16_NORM, cfg.mean, cfg.std)
    lb = cd.LearnerBatch()
    lb.obs, lb.action, lb.reward = out.data_ptr(), act.data_ptr(), rew.data_ptr()
    h = C.c_void_p(buf.handle)
    xfr, lbr = C.byref(xf), C.byref(lb)
    pu = [u_d[i].data_ptr() for i in range(iters)]
    pp = [p_d[i].data_ptr() for i in range(iters)]
    pi = [idx[i].data_ptr() for i in range(iters)]
    pw = [w[i].data_ptr() for i in range(iters)]
    torch.cuda.synchronize()
    it_calls = []
    for i in range(iters):
        it_calls.append(lambda i=i: L.conduit_sample_gather(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream))
        it_calls.append(lambda i=i: L.conduit_update_priorities(h, pi[i], pp[i], B, stream))
    iter_ms = _b2b_ms(it_calls) * 2
    smp_ms = _b2b_ms([lambda i=i: L.conduit_sample(h, B, pu[i], pi[i], pw[i], stream) for i in range(iters)])
    gat_ms = _b2b_ms([lambda i=i: L.conduit_gather_transform(h, pi[i], B, xfr, lbr, stream) for i in range(iters)])
    upd_ms = _b2b_ms([lambda i=i: L.conduit_update_priorities(h, pi[i], pp[i], B, stream) for i in range(iters)])
    assert buf.sync_check() == cd.OK, cd.last_error()
    buf.close()
    gbytes = B * (row + 2 * row + 8 + 24 + 4 + 24 + 4)
    return {
        "gather_bf16_1024": {"bytes": gbytes, "us": gat_ms * 1e3, "GBps": gbytes / gat_ms / 1e6,
                             "frac": gbytes / gat_ms / 1e6 / PEAK_HBM_GBPS},
        "sample_1024_us": smp_ms * 1e3,
        "update_1024_us": upd_ms * 1e3,
        "iteration_us": iter_ms * 1e3,
        "timing": "back-to-back launches between two events, arguments prepared up front",
    }


def bench_tokens(iters=10):
    """Token replay (65,536 ragged sequences of up to 4,096 int32 tokens + fp32
    log-probs): per iteration sample 256 + pack to [256, 4096] with mask, log-probs
    and lengths, GAE over the packed rows, update 256; whole iterations and each
    call type timed as back-to-back launches with prepared arguments."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    Cap, Lmax, B = 65536, 4096, 256
    cfg = synth.Tokens(Cap)
    buf = cd.ReplayBuffer(Cap, (Lmax,), torch.int32, action_bytes=4, ragged=True, aux_elem_bytes=4)
    for a in range(0, Cap, 4096):
        b = min(Cap, a + 4096)
        tok, lp, off = cfg.packed(a, b - a, "cuda")
        buf.ingest(tok, offsets=off, aux=lp, action=_dev(cfg.action[a:b]), reward=_dev(cfg.reward[a:b]),
                   done=_dev(cfg.done[a:b]), prio=_dev(cfg.prio[a:b]))
        del tok, lp
    u, prio = cfg.draws(iters, B)
    u_d, p_d = _dev(u), _dev(prio)
    idx = torch.empty((iters, B), dtype=torch.int64, device="cuda")
    w = torch.empty((iters, B), dtype=torch.float32, device="cuda")
    seq = torch.empty((B, Lmax), dtype=torch.int32, device="cuda")
    mask = torch.empty((B, Lmax), dtype=torch.uint8, device="cuda")
    lp_out = torch.empty((B, Lmax), dtype=torch.float32, device="cuda")
    length = torch.empty(B, dtype=torch.int32, device="cuda")
    rew = torch.empty(B, dtype=torch.float32, device="cuda")
    adv = torch.empty((B, Lmax), dtype=torch.float32, device="cuda")
    ret = torch.empty((B, Lmax), dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_TOKENS_PAD)
    lb = cd.LearnerBatch()
    lb.obs, lb.mask, lb.aux, lb.length, lb.reward = (seq.data_ptr(), mask.data_ptr(), lp_out.data_ptr(),
                                                     length.data_ptr(), rew.data_ptr())
    h = C.c_void_p(buf.handle)
    xfr, lbr = C.byref(xf), C.byref(lb)
    pu = [u_d[i].data_ptr() for i in range(iters)]
    pp = [p_d[i].data_ptr() for i in range(iters)]
    pi = [idx[i].data_ptr() for i in range(iters)]
    pw = [w[i].data_ptr() for i in range(iters)]
    gae_args = (rew.data_ptr(), length.data_ptr(), None, B, Lmax, cfg.gamma, cfg.lam, adv.data_ptr(), ret.data_ptr(),
                stream)
    gae = lambda: L.conduit_gae_packed(*gae_args)  # noqa: E731
    torch.cuda.synchronize()
    it_calls = []
    for i in range(iters):
        it_calls.append(lambda i=i: L.conduit_sample_gather(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream))
        it_calls.append(gae)
        it_calls.append(lambda i=i: L.conduit_update_priorities(h, pi[i], pp[i], B, stream))
    iter_ms = _b2b_ms(it_calls) * 3
    # the same iterations with the packed rows' GAE inside the delivery launch
    # (conduit_sample_pack_gae)
    spg = L.conduit_sample_pack_gae
    one_calls = []
    for i in range(iters):
        one_calls.append(lambda i=i: spg(h, B, pu[i], pi[i], pw[i], xfr, lbr, None, cfg.gamma, cfg.lam,
                                         adv.data_ptr(), ret.data_ptr(), stream))
        one_calls.append(lambda i=i: L.conduit_update_priorities(h, pi[i], pp[i], B, stream))
    iter_one_ms = _b2b_ms(one_calls) * 2
    mean_len = float(length.float().mean())
    pack_ms = _b2b_ms([lambda i=i: L.conduit_gather_transform(h, pi[i], B, xfr, lbr, stream) for i in range(iters)])
    gae_ms = _b2b_ms([gae] * iters)
    # the two delivery launches alone: sampler + pack, and sampler + pack + GAE
    sp_ms = _b2b_ms([lambda i=i: L.conduit_sample_gather(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
                     for i in range(iters)])
    spg_ms = _b2b_ms([lambda i=i: spg(h, B, pu[i], pi[i], pw[i], xfr, lbr, None, cfg.gamma, cfg.lam, adv.data_ptr(),
                                      ret.data_ptr(), stream) for i in range(iters)])
    assert buf.sync_check() == cd.OK, cd.last_error()
    buf.close()
    pbytes = int(B * mean_len * 8 + B * Lmax * (4 + 1 + 4) + B * (8 + 4 + 4 + 4 + 4))
    gbytes = B * (4 + 4) + B * Lmax * 8
    return {
        "pack_256x4096": {"bytes": pbytes, "us": pack_ms * 1e3, "GBps": pbytes / pack_ms / 1e6,
                          "frac": pbytes / pack_ms / 1e6 / PEAK_HBM_GBPS},
        "gae_packed_256x4096": {"bytes": gbytes, "us": gae_ms * 1e3, "GBps": gbytes / gae_ms / 1e6,
                                "frac": gbytes / gae_ms / 1e6 / PEAK_HBM_GBPS},
        "iteration_us": iter_ms * 1e3,
        "iteration_one_launch_gae_us": iter_one_ms * 1e3,
        "sample_pack_us": sp_ms * 1e3,
        "sample_pack_gae_us": spg_ms * 1e3,
        "timing": "back-to-back launches between two events, arguments prepared up front",
    }


def bench_stress(dims=(128, 1000, 5000, 10000, 20000), iters=20):
    """The paper's synthetic stress sweep at capacity 10^6 and batch 512: for
    each transition dimension d (obs and next_obs, d fp32 each, 8d bytes per
    slot) a full buffer (up to 160 GB at d = 20,000), then iterations of
    ingest 512 + sample + gather 512 (one call, IS weights, no transform) +
    update 512, timed as back-to-back launches with prepared arguments; each
    update is applied with the next iteration's ingest in one call
    (conduit_update_ingest), the separate-call iteration reported beside."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    Cap, B = 1_000_000, 512
    res = {}
    for d in dims:
        torch.cuda.empty_cache()
        cfg = synth.Stress(d, Cap + iters * B)
        row = 8 * d
        buf = cd.ReplayBuffer(Cap, cfg.obs_shape, torch.float32, action_bytes=4)
        act_d, rew_d, done_d, prio_d = _dev(cfg.action), _dev(cfg.reward), _dev(cfg.done), _dev(cfg.prio)
        chunk = max(512, min(65536, (1 << 30) // row))
        t0 = time.time()
        for a in range(0, Cap, chunk):
            b = min(Cap, a + chunk)
            buf.ingest(cfg.rows(a, b - a, "cuda"), action=act_d[a:b], reward=rew_d[a:b], done=done_d[a:b],
                       prio=prio_d[a:b])
        torch.cuda.synchronize()
        prefill_s = time.time() - t0
        new_rows = cfg.rows(Cap, iters * B, "cuda")
        u, prio = cfg.draws(iters, B)
        u_d, p_d = _dev(u), _dev(prio)
        idx = torch.empty((iters, B), dtype=torch.int64, device="cuda")
        w = torch.empty((iters, B), dtype=torch.float32, device="cuda")
        out = torch.empty((B, 1) + cfg.obs_shape, dtype=torch.float32, device="cuda")
        act = torch.empty(B, dtype=torch.int32, device="cuda")
        rew = torch.empty(B, dtype=torch.float32, device="cuda")
        xf = cd.transform(cd.XF_NONE)
        lb = cd.LearnerBatch()
        lb.obs, lb.action, lb.reward = out.data_ptr(), act.data_ptr(), rew.data_ptr()
        structs = []
        for i in range(iters):
            t = cd.Transitions()
            sl = slice(Cap + i * B, Cap + (i + 1) * B)
            t.n = B
            t.obs = new_rows[i * B:(i + 1) * B].data_ptr()
            t.action, t.reward, t.done = act_d[sl].data_ptr(), rew_d[sl].data_ptr(), done_d[sl].data_ptr()
            t.prio = prio_d[sl].data_ptr()
            structs.append(t)
        h = C.c_void_p(buf.handle)
        xfr, lbr = C.byref(xf), C.byref(lb)
        pu = [u_d[i].data_ptr() for i in range(iters)]
        pp = [p_d[i].data_ptr() for i in range(iters)]
        pi = [idx[i].data_ptr() for i in range(iters)]
        pw = [w[i].data_ptr() for i in range(iters)]
        calls = []
        for i in range(iters):
            calls.append(lambda i=i: L.conduit_ingest(h, C.byref(structs[i]), stream))
            calls.append(lambda i=i: L.conduit_sample_gather(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream))
            calls.append(lambda i=i: L.conduit_update_priorities(h, pi[i], pp[i], B, stream))
        _b2b_ms(calls[:3])
        iter_sep_ms = _b2b_ms(calls) * 3
        # each update applied with the next iteration's ingest in one call
        calls = []
        for i in range(iters):
            if i == 0:
                calls.append(lambda: L.conduit_ingest(h, C.byref(structs[0]), stream))
            else:
                calls.append(lambda i=i: L.conduit_update_ingest(h, pi[i - 1], pp[i - 1], B, C.byref(structs[i]),
                                                                 stream))
            calls.append(lambda i=i: L.conduit_sample_gather(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream))
        calls.append(lambda: L.conduit_update_priorities(h, pi[iters - 1], pp[iters - 1], B, stream))
        iter_ms = _b2b_ms(calls) * len(calls) / iters
        ing_ms = _b2b_ms([lambda i=i: L.conduit_ingest(h, C.byref(structs[i]), stream) for i in range(iters)])
        sg_ms = _b2b_ms([lambda i=i: L.conduit_sample_gather(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
                         for i in range(iters)])
        assert buf.sync_check() == cd.OK, cd.last_error()
        buf.close()
        del new_rows, out
        # algorithmic bytes: ingest reads and writes each row and 17 B of scalars
        # plus the leaf; delivery reads and writes each sampled row and scalars
        ing_bytes = B * (2 * row + 2 * 17 + 8)
        sg_bytes = B * (2 * row + 8 + 2 * (4 + 4))
        res[f"d={d}"] = {"buffer_GB": Cap * row / 1e9, "prefill_s": prefill_s, "iteration_us": iter_ms * 1e3,
                         "sampled_per_s": B / (iter_ms / 1e3), "iteration_us_separate_update": iter_sep_ms * 1e3,
                         "ingest_512_us": ing_ms * 1e3, "ingest_GBps": ing_bytes / ing_ms / 1e6,
                         "sample_gather_512_us": sg_ms * 1e3, "sample_gather_GBps": sg_bytes / sg_ms / 1e6}
    return res


def bench_schedule(d=10000, t_stage_us=(100.0, 150.0), iters=64, gs=(1, 2, 4, 8)):
    """Latency-aware scheduling on one GPU (the paper's Sec. 6 knobs): the
    native off-policy loop (conduit_run_offpolicy) on the synthetic stress
    workload (dimension d, 10^6 slots, rollout units and learner batches of
    512) with the library's compute stand-in for the actor's rollout and the
    learner's update.  The model's inputs are profiled (stage times, one
    invocation of each operator at each granularity, one cross-stream
    dependency), conduit_schedule scores every mode, and every mode is then
    run and timed.  Reports model-predicted vs measured iteration latency per
    mode, the model's choice against the measured best, and the rank
    correlation of prediction and measurement."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    Cap, U, B = 1_000_000, 512, 512
    torch.cuda.empty_cache()
    cfg = synth.Stress(d, Cap + iters * U)
    buf = cd.ReplayBuffer(Cap, cfg.obs_shape, torch.float32, action_bytes=4)
    act_d, rew_d, done_d, prio_d = _dev(cfg.action), _dev(cfg.reward), _dev(cfg.done), _dev(cfg.prio)
    chunk = max(512, min(65536, (1 << 30) // (8 * d)))
    for a in range(0, Cap, chunk):
        b = min(Cap, a + chunk)
        buf.ingest(cfg.rows(a, b - a, "cuda"), action=act_d[a:b], reward=rew_d[a:b], done=done_d[a:b],
                   prio=prio_d[a:b])
    rows = cfg.rows(Cap, iters * U, "cuda")
    rng = np.random.default_rng(5)
    u_d = _dev(synth.uniforms(rng, iters * B))
    p_d = _dev(synth.quantise_priority(rng.lognormal(0, 1, iters * B)))
    idx = torch.empty(iters * B, dtype=torch.int64, device="cuda")
    w = torch.empty(iters * B, dtype=torch.float32, device="cuda")
    out = torch.empty((iters * B, 1) + cfg.obs_shape, dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_NONE)
    h = C.c_void_p(buf.handle)
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)

    def loop_struct(mode, work):
        lp = cd.OffpolicyLoop()
        lp.overlap_ing, lp.g_ing, lp.overlap_del, lp.g_del = mode
        lp.iters, lp.unit, lp.batch = iters, U, B
        lp.rollout_work, lp.update_work = work
        lp.rollout.obs, lp.rollout.action = rows.data_ptr(), act_d[Cap:].data_ptr()
        lp.rollout.reward, lp.rollout.done, lp.rollout.prio = (rew_d[Cap:].data_ptr(), done_d[Cap:].data_ptr(),
                                                               prio_d[Cap:].data_ptr())
        lp.uniforms, lp.new_prio = u_d.data_ptr(), p_d.data_ptr()
        lp.idx_out, lp.is_w_out = idx.data_ptr(), w.data_ptr()
        lp.xf = C.pointer(xf)
        lp.out.obs = out.data_ptr()
        return lp

    # the stand-in's time per unit of work, then the work for each stage
    base = 20000
    _b2b_ms([lambda: L.conduit_standin(base, stream)] * 5)
    us_per_work = _b2b_ms([lambda: L.conduit_standin(base, stream)] * 20) * 1e3 / base
    work = (int(t_stage_us[0] / us_per_work), int(t_stage_us[1] / us_per_work))
    t_roll = _b2b_ms([lambda: L.conduit_standin(work[0], stream)] * 20) * 1e3
    t_upd = _b2b_ms([lambda: L.conduit_standin(work[1], stream)] * 20) * 1e3
    # operator costs at each granularity: one invocation, back to back
    t_ing, t_del = [], []
    for g in gs:
        tr = cd.Transitions()
        tr.n = g * U
        tr.obs, tr.action = rows.data_ptr(), act_d[Cap:].data_ptr()
        tr.reward, tr.done, tr.prio = rew_d[Cap:].data_ptr(), done_d[Cap:].data_ptr(), prio_d[Cap:].data_ptr()
        t_ing.append(_b2b_ms([lambda tr=tr: L.conduit_ingest(h, C.byref(tr), stream)] * 10) * 1e3)
        lb = cd.LearnerBatch()
        lb.obs = out.data_ptr()

        def one(g=g, lb=lb):
            r = L.conduit_sample_gather(h, g * B, u_d.data_ptr(), idx.data_ptr(), w.data_ptr(), C.byref(xf),
                                        C.byref(lb), stream)
            for j in range(g):
                r |= L.conduit_update_priorities(h, idx[j * B:].data_ptr(), p_d[j * B:].data_ptr(), B, stream)
            return r
        t_del.append(_b2b_ms([one] * 10) * 1e3)
    comp, exp, co_run = _co_running_streams()
    t_hop, t_sync = cd.conduit_sync_cost_us(comp, exp, 200)
    best, modes = cd.conduit_schedule(t_roll, t_upd, list(gs), t_ing, list(gs), t_del, t_sync, t_sync)
    best_hop, _ = cd.conduit_schedule(t_roll, t_upd, list(gs), t_ing, list(gs), t_del, t_hop, t_hop)
    # every mode, run natively and timed
    cd.conduit_run_offpolicy(buf.handle, loop_struct((0, 1, 0, 1), work), comp, exp)  # warm-up
    measured = []
    for m in modes:
        lp = loop_struct((m["overlap_ing"], int(m["g_ing"]), m["overlap_del"], int(m["g_del"])), work)
        _head_start(comp, iters * 600.0)
        ms, _ = cd.conduit_run_offpolicy(buf.handle, lp, comp, exp)
        measured.append(ms * 1e3 / iters)
    assert buf.sync_check() == cd.OK, cd.last_error()
    buf.close()
    name = lambda m: f"ov_ing={m['overlap_ing']} g_ing={int(m['g_ing'])} ov_del={m['overlap_del']} g_del={int(m['g_del'])}"  # noqa: E731
    seq = next(i for i, m in enumerate(modes) if m["overlap_ing"] == 0 and m["overlap_del"] == 0 and
               m["g_ing"] == 1 and m["g_del"] == 1)
    out = {
        "workload": f"stress d={d}, 10^6 slots, rollout unit = batch = 512, {iters} iterations per mode; "
                    f"register-only compute stand-in (one workgroup per CU) for rollout and update",
        "profiled_us": {"t_rollout": t_roll, "t_update": t_upd, "t_sync": t_sync, "t_hop_unmet": t_hop,
                        "t_ing": dict(zip(map(str, gs), t_ing)), "t_del": dict(zip(map(str, gs), t_del))},
        "streams_co_run_us": co_run,
    }
    out.update(_schedule_report(modes, best, measured, name, seq, t_roll + t_upd))
    out["model_choice_with_unmet_hop_as_t_sync"] = name(best_hop)
    return out


def _head_start(stream, us):
    """Queue about `us` microseconds of stand-in compute on `stream` ahead of a
    native loop, so that its events time the GPU and not the host's enqueue of
    the iterations (the loop records its start event after this work)."""
    import torch
    with torch.cuda.stream(stream):
        _gpu_delay(us)


def _co_run_us(a, b, us=300.0):
    """GPU time of about `us` of stand-in work on stream `a` alone, and of the
    same work on `a` and on `b` at once (one workgroup per CU each, so two
    streams that run concurrently take about as long as one): shows whether
    the two streams of an overlapped schedule really overlap."""
    import torch
    from paper_2609_24456_amd import conduit as cd
    _gpu_delay(1.0)  # calibrates the stand-in's rate
    work = max(1, int(us / _DELAY_US_PER_WORK[0]))
    cd.conduit_standin(work, a)
    cd.conduit_standin(work, b)
    torch.cuda.synchronize()

    def run(both):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(a)
        b.wait_event(e0)
        cd.conduit_standin(work, a)
        if both:
            cd.conduit_standin(work, b)
        e1.record(b)
        a.wait_event(e1)
        e2.record(a)
        torch.cuda.synchronize()
        return e0.elapsed_time(e2) * 1e3

    return {"alone_us": min(run(False) for _ in range(3)), "both_us": min(run(True) for _ in range(3))}


def _co_running_streams(tries=8):
    """Two torch streams measured to run concurrently.  HIP serves every
    stream of a process from a few hardware queues (4 here), shared among
    all streams, torch's pool of 32 included, so two streams can land on one
    queue and run one after the other, and an overlapped schedule on them
    then hides nothing.  The first stream is kept; candidates for the second
    are drawn from the pool until one co-runs with it (both stand-ins
    together within 1.3x of one alone)."""
    import torch
    comp = torch.cuda.Stream()
    for k in range(1, tries + 1):
        exp = torch.cuda.Stream()
        co = _co_run_us(comp, exp)
        co["candidates_tried"] = k
        if co["both_us"] < 1.3 * co["alone_us"]:
            break
    return comp, exp, co


def _schedule_report(modes, best, measured, name, seq, stages):
    """Model vs measurement over every mode: the model's choice against the
    measured best, the sequential reference, exposed time, rank correlation."""
    import numpy as np
    pred = np.array([m["t_iter"] for m in modes])
    meas = np.array(measured)
    k_best = int(np.argmin(meas))
    k_model = next(i for i, m in enumerate(modes) if all(m[f] == best[f] for f in ("overlap_ing", "overlap_del",
                                                                                    "i_ing", "i_del")))
    rank = lambda v: np.argsort(np.argsort(v))  # noqa: E731
    spearman = float(np.corrcoef(rank(pred), rank(meas))[0, 1])
    return {
        "model_choice": {"mode": name(modes[k_model]), "predicted_us": float(pred[k_model]),
                         "measured_us": float(meas[k_model])},
        "measured_best": {"mode": name(modes[k_best]), "predicted_us": float(pred[k_best]),
                          "measured_us": float(meas[k_best])},
        "sequential": {"mode": name(modes[seq]), "predicted_us": float(pred[seq]), "measured_us": float(meas[seq])},
        "exposed_us": {"sequential": float(meas[seq] - stages), "model_choice": float(meas[k_model] - stages),
                       "measured_best": float(meas[k_best] - stages)},
        "model_regret": float(meas[k_model] / meas[k_best] - 1.0),
        "spearman_pred_vs_measured": spearman,
        "modes": [{"mode": name(m), "predicted_us": float(p), "measured_us": float(x)}
                  for m, p, x in zip(modes, pred, meas)],
    }


def bench_schedule_onpolicy(T=256, E=64, M=8, iters=8, t_stage_us=(600.0, 800.0)):
    """On-policy scheduling on one GPU (Sec. 6 knobs, pipelined case): the
    native on-policy loop (conduit_run_onpolicy) on a PPO-shaped rollout of
    E x T transitions of 3x84x84 u8, M minibatches gathered with the u8 -> fp32
    transform plus advantages and returns, GAE gamma 0.99 lambda 0.95.
    Candidates come from conduit_sched_candidates (ingestion j/M, delivery
    1/M); the model's inputs are profiled (stage slices, ingestion of j
    slices plus j/M of the GAE, one minibatch gather, one cross-stream
    dependency); every mode is then run and timed."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    cfg = synth.PPO(T=T, E=E)
    U, row = T * E, 3 * 84 * 84
    torch.cuda.empty_cache()
    obs = cfg.obs_steps(0, T, "cuda").reshape(1, U, row).expand(iters, U, row).contiguous()
    tile = lambda a: _dev(np.ascontiguousarray(np.broadcast_to(a.reshape(1, -1), (iters, a.size))))  # noqa: E731
    rew, val, done, boot = tile(cfg.reward), tile(cfg.value), tile(cfg.done), tile(cfg.bootstrap)
    perm = _dev(np.stack([np.random.default_rng(7 + i).permutation(U) for i in range(iters)]).astype(np.int64))
    adv = torch.empty(U, dtype=torch.float32, device="cuda")
    ret = torch.empty(U, dtype=torch.float32, device="cuda")
    out = torch.empty((iters, U, row), dtype=torch.float32, device="cuda")
    out_adv = torch.empty((iters, U), dtype=torch.float32, device="cuda")
    out_ret = torch.empty((iters, U), dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_U8_F32)
    buf = cd.ReplayBuffer(U, cfg.obs_shape, torch.uint8, prioritized=False, action_bytes=0)
    h = C.c_void_p(buf.handle)

    def loop_struct(mode, work):
        lp = cd.OnpolicyLoop()
        lp.overlap_ing, lp.ing_slices, lp.overlap_del, lp.minibatches = mode[0], mode[1], mode[2], M
        lp.iters, lp.steps, lp.envs = iters, T, E
        lp.rollout_work, lp.update_work = work
        lp.obs, lp.reward, lp.value, lp.done = obs.data_ptr(), rew.data_ptr(), val.data_ptr(), done.data_ptr()
        lp.bootstrap, lp.gamma, lp.lam, lp.perm = boot.data_ptr(), cfg.gamma, cfg.lam, perm.data_ptr()
        lp.xf = C.pointer(xf)
        lp.adv, lp.ret = adv.data_ptr(), ret.data_ptr()
        lp.out_obs, lp.out_adv, lp.out_ret = out.data_ptr(), out_adv.data_ptr(), out_ret.data_ptr()
        return lp

    # stand-ins: each stage runs as M slices
    base = 20000
    _b2b_ms([lambda: L.conduit_standin(base, stream)] * 5)
    us_per_work = _b2b_ms([lambda: L.conduit_standin(base, stream)] * 20) * 1e3 / base
    work = (int(t_stage_us[0] / us_per_work), int(t_stage_us[1] / us_per_work))
    t_roll = _b2b_ms([lambda: L.conduit_standin(work[0] // M, stream)] * (10 * M)) * 1e3 * M
    t_upd = _b2b_ms([lambda: L.conduit_standin(work[1] // M, stream)] * (10 * M)) * 1e3 * M
    g_ing, g_del = cd.conduit_sched_candidates(True, M)
    # Operator costs, each call on memory the previous calls did not touch (a
    # rollout is larger than the 256 MB last-level cache, so repeating one
    # call on the same data would time cache hits the loop never sees).
    slice_rows = U // M
    sweep = torch.empty(1 << 29, dtype=torch.uint8, device="cuda")
    gae_ms = []
    for i in range(iters):  # GAE: one call after a 512 MB sweep, timed alone
        sweep.fill_(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        assert L.conduit_gae(rew[i].data_ptr(), val[i].data_ptr(), done[i].data_ptr(), boot[i].data_ptr(), T, E,
                             cfg.gamma, cfg.lam, adv.data_ptr(), ret.data_ptr(), stream) == 0
        e1.record()
        torch.cuda.synchronize()
        gae_ms.append(e0.elapsed_time(e1))
    del sweep
    t_gae = float(np.median(gae_ms[1:])) * 1e3
    t_ing = []
    for j in range(1, M + 1):
        # M calls of j slices walk j whole rollouts of the staged rows (the
        # head returns to slot 0)
        structs = []
        for c in range(M):
            tr = cd.Transitions()
            r0 = (c * j * slice_rows) % (iters * U)
            tr.n = j * slice_rows
            tr.obs = obs.data_ptr() + r0 * row
            tr.reward, tr.done = rew.data_ptr() + 4 * r0, done.data_ptr() + r0
            structs.append(tr)
        calls = [lambda tr=tr: L.conduit_ingest(h, C.byref(tr), stream) for tr in structs]
        _b2b_ms(calls)
        t_ing.append(_b2b_ms(calls) * 1e3 + j / M * t_gae)
    assert buf.info().head == 0
    # delivery: the M minibatches of each staged rollout in turn
    mb = U // M
    cols = (C.c_void_p * 2)(adv.data_ptr(), ret.data_ptr())
    calls = []
    for i in range(iters):
        for m in range(M):
            o = i * U + m * mb
            co = (C.c_void_p * 2)(out_adv.data_ptr() + 4 * o, out_ret.data_ptr() + 4 * o)
            calls.append(lambda i=i, m=m, o=o, co=co: L.conduit_minibatch_gather(
                obs.data_ptr() + i * U * row, row, U, perm.data_ptr() + 8 * (i * U + m * mb), mb, C.byref(xf),
                out.data_ptr() + o * row * 4, cols, co, 2, stream))
    _b2b_ms(calls)
    t_del = [_b2b_ms(calls) * 1e3]
    comp, exp, co_run = _co_running_streams()
    t_hop, t_sync = cd.conduit_sync_cost_us(comp, exp, 200)
    best, modes = cd.conduit_schedule(t_roll, t_upd, g_ing, t_ing, g_del, t_del, t_sync, t_sync, on_policy=True)
    cd.conduit_run_onpolicy(buf.handle, loop_struct((0, M, 0), work), comp, exp)  # warm-up
    measured = []
    for m in modes:
        lp = loop_struct((m["overlap_ing"], round(m["g_ing"] * M), m["overlap_del"]), work)
        _head_start(comp, iters * 3000.0)
        ms, _ = cd.conduit_run_onpolicy(buf.handle, lp, comp, exp)
        measured.append(ms * 1e3 / iters)
    assert buf.sync_check() == cd.OK, cd.last_error()
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    buf.close()
    name = lambda m: f"ov_ing={m['overlap_ing']} g_ing={round(m['g_ing'] * M)}/{M} ov_del={m['overlap_del']} g_del=1/{M}"  # noqa: E731
    seq = next(i for i, m in enumerate(modes) if m["overlap_ing"] == 0 and m["overlap_del"] == 0 and
               m["g_ing"] == 1.0)
    out_d = {
        "workload": f"PPO-shaped rollout {E} envs x {T} steps of 3x84x84 u8, {M} minibatches of {mb} -> fp32 "
                    f"with advantages and returns, GAE over the rollout; {iters} iterations per mode; "
                    f"register-only compute stand-in for rollout and update, each run as {M} slices",
        "profiled_us": {"t_rollout": t_roll, "t_update": t_upd, "t_sync": t_sync, "t_hop_unmet": t_hop,
                        "t_gae": t_gae, "t_ing": {f"{j}/{M}": t for j, t in zip(range(1, M + 1), t_ing)},
                        "t_del": {f"1/{M}": t_del[0]}},
        "streams_co_run_us": co_run,
    }
    out_d.update(_schedule_report(modes, best, measured, name, seq, t_roll + t_upd))
    return out_d


def bench_placement(cap=200_000, steps=20):
    """Capacity-constrained, bandwidth-aware placement on one GPU host (Sec. 5):
    the profiled effective bandwidth of each leg and the memory of each tier
    (conduit_placement_profile), Alg. 1's choice (conduit_place) for the
    workload shapes of this repository, and a check of the model's ranking:
    the DQN step (ingest 512 frames, fused sample + frame-stack gather 512,
    priority update 512) on a buffer of `cap` frames with the frames in HBM and
    in pinned host memory, the same kernels in both."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    prof = cd.conduit_placement_profile(256 << 20, 3)
    names = cd.PLACEMENT_NAMES
    meta = 4 + 4 + 1 + 4 + 4 + 4  # action, reward, done, episode id, step, priority leaf
    shapes = {
        "dqn 1M frames 84x84 u8": (1_000_000, 84 * 84 + meta),
        "ppo rollout 2048x256 of 3x84x84 u8": (2048 * 256, 3 * 84 * 84 + 9),
        "large 200k of 3x224x224 u8": (200_000, 3 * 224 * 224 + 24 + meta),
        "tokens 64k of up to 4096 (int32 token + fp32 logprob)": (65536, 4096 * 8 + 4 + meta),
        "stress d=20000, 10^6": (1_000_000, 2 * 20000 * 4 + meta),
        "stress d=20000, 1.95x10^6": (1_950_000, 2 * 20000 * 4 + meta),
        "stress d=20000, 2x10^6": (2_000_000, 2 * 20000 * 4 + meta),
        "stress d=20000, 10^7": (10_000_000, 2 * 20000 * 4 + meta),
    }
    decisions = {}
    for wl, (c, x) in shapes.items():
        decisions[wl] = {"bytes": c * x}
        for actor, who in ((1, "gpu_actor"), (0, "cpu_actor")):
            choice, t = cd.conduit_place(prof, actor, c, x)
            decisions[wl][who] = {"choice": names[choice] if choice >= 0 else None,
                                  "t_transfer_us": {names[i]: t[i] * 1e6 for i in range(3)}}
    # the DQN step with the frames in each executable tier
    B, K = 512, 4
    cfg = synth.DQN(cap + (steps + 2) * B)
    u, prio = cfg.draws(steps + 2, B)
    u_d, prio_d = _dev(u), _dev(prio)
    frames = cfg.frames(cap, (steps + 2) * B, "cuda")
    sl = slice(cap, cap + (steps + 2) * B)
    act, rew, done = _dev(cfg.action[sl]), _dev(cfg.reward[sl]), _dev(cfg.done[sl])
    epi, stp = _dev(cfg.episode[sl]), _dev(cfg.step[sl])
    idx = torch.empty((steps + 2, B), dtype=torch.int64, device="cuda")
    w = torch.empty((steps + 2, B), dtype=torch.float32, device="cuda")
    obs_out = torch.empty((B, K, 84, 84), dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_U8_F32)
    lb = cd.LearnerBatch()
    lb.obs = obs_out.data_ptr()
    measured = {}
    for pl in (cd.PLACE_HBM, cd.PLACE_HOST_PINNED):
        buf = cd.ReplayBuffer(cap, (84, 84), torch.uint8, frame_stack=K, action_bytes=4, placement=pl)
        for a in range(0, cap, 8192):
            b = min(cap, a + 8192)
            buf.ingest(cfg.frames(a, b - a, "cuda"), action=_dev(cfg.action[a:b]), reward=_dev(cfg.reward[a:b]),
                       done=_dev(cfg.done[a:b]), episode_id=_dev(cfg.episode[a:b]), step=_dev(cfg.step[a:b]),
                       prio=_dev(cfg.prio[a:b]))
        torch.cuda.synchronize()
        h = C.c_void_p(buf.handle)
        trans = []
        for i in range(steps + 2):
            t = cd.Transitions()
            r = slice(i * B, (i + 1) * B)
            t.n, t.obs = B, frames[r].data_ptr()
            t.action, t.reward, t.done = act[r].data_ptr(), rew[r].data_ptr(), done[r].data_ptr()
            t.episode_id, t.step = epi[r].data_ptr(), stp[r].data_ptr()
            trans.append(t)
        ing = [lambda i=i: L.conduit_ingest(h, C.byref(trans[i]), stream) for i in range(steps + 2)]
        sg = [lambda i=i: L.conduit_sample_gather(h, B, u_d[i].data_ptr(), idx[i].data_ptr(), w[i].data_ptr(),
                                                  C.byref(xf), C.byref(lb), stream) for i in range(steps + 2)]
        up = [lambda i=i: L.conduit_update_priorities(h, idx[i].data_ptr(), prio_d[i].data_ptr(), B, stream)
              for i in range(steps + 2)]
        step = [lambda i=i: ing[i]() | sg[i]() | up[i]() for i in range(steps + 2)]
        step[0]()
        step[1]()
        step_ms = _b2b_ms(step[2:])
        ing_ms = _b2b_ms(ing[2:])
        sg_ms = _b2b_ms(sg[2:])
        assert buf.sync_check() == cd.OK, cd.last_error()
        buf.close()
        link_in = B * 84 * 84  # frame bytes an ingestion writes into the tier
        link_out = B * K * 84 * 84  # frame bytes a delivery reads from it
        # the transfer model's two legs for one step (Sec. 5.1, GPU actor)
        pred_us = (link_in / prof.bw_in[1][pl] + link_out / prof.bw_out[pl]) * 1e6
        measured[names[pl]] = {"step_us": step_ms * 1e3, "ingest_us": ing_ms * 1e3, "sample_gather_us": sg_ms * 1e3,
                               "ingest_tier_GBps": link_in / ing_ms / 1e6,
                               "delivery_tier_GBps": link_out / sg_ms / 1e6,
                               "model_transfer_us": pred_us}
    ranking_holds = measured["hbm"]["step_us"] < measured["host_pinned"]["step_us"]
    return {
        "profile_GBps": {"bw_in_gpu_actor": dict(zip(names, (v / 1e9 for v in prof.bw_in[1]))),
                         "bw_in_cpu_actor": dict(zip(names, (v / 1e9 for v in prof.bw_in[0]))),
                         "bw_out": dict(zip(names, (v / 1e9 for v in prof.bw_out)))},
        "mem_GB": dict(zip(names, (v / 1e9 for v in prof.mem))),
        "alg1": decisions,
        "dqn_step_by_tier": {"capacity": cap, "batch": B, **measured,
                             "model_ranking_holds": bool(ranking_holds)},
    }


def bench_tiny(iters=100):
    """Tiny replay (16,384 slots of 8 fp32): 100 x [ingest 64, sample + gather 256
    with IS weights (one launch), update 256], every call's arguments prepared
    before the timed loop.  Launch-latency bound."""
    import numpy as np
    import torch
    import synth
    from paper_2609_24456_amd import conduit as cd
    L = cd.lib()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    cfg = synth.Tiny()
    u, prio = cfg.draws()
    B, n_in = cfg.batch, cfg.ingest_n
    buf = cd.ReplayBuffer(cfg.capacity, (8,), torch.float32, action_bytes=4)
    obs, act, rew, done = _dev(cfg.obs), _dev(cfg.action), _dev(cfg.reward), _dev(cfg.done)
    epi, stp = _dev(cfg.episode), _dev(cfg.step)
    u_d, p_d = _dev(u), _dev(prio)
    idx = torch.empty((iters, B), dtype=torch.int64, device="cuda")
    w = torch.empty((iters, B), dtype=torch.float32, device="cuda")
    out = torch.empty((B, 1, 8), dtype=torch.float32, device="cuda")
    act_out = torch.empty(B, dtype=torch.int32, device="cuda")
    rew_out = torch.empty(B, dtype=torch.float32, device="cuda")
    done_out = torch.empty(B, dtype=torch.uint8, device="cuda")
    xf = cd.transform(cd.XF_NONE)
    lb = cd.LearnerBatch()
    lb.obs, lb.action, lb.reward, lb.done = out.data_ptr(), act_out.data_ptr(), rew_out.data_ptr(), done_out.data_ptr()
    structs = []
    for i in range(iters):
        t = cd.Transitions()
        sl = slice(i * n_in, (i + 1) * n_in)
        t.n = n_in
        t.obs = obs[sl].data_ptr()
        t.action, t.reward, t.done = act[sl].data_ptr(), rew[sl].data_ptr(), done[sl].data_ptr()
        t.episode_id, t.step = epi[sl].data_ptr(), stp[sl].data_ptr()
        t.prio = None
        structs.append(t)
    trans = [C.byref(t) for t in structs]
    h = C.c_void_p(buf.handle)
    xfr, lbr = C.byref(xf), C.byref(lb)
    pu = [u_d[i].data_ptr() for i in range(iters)]
    pp = [p_d[i].data_ptr() for i in range(iters)]
    pi = [idx[i].data_ptr() for i in range(iters)]
    pw = [w[i].data_ptr() for i in range(iters)]
    ing, sgat, upd = L.conduit_ingest, L.conduit_sample_gather, L.conduit_update_priorities
    uing = L.conduit_update_ingest
    tm = Timer()
    torch.cuda.synchronize()
    # separate calls: ingest, sample + gather, update
    e0 = tm.ev()
    h0 = time.perf_counter()
    rc = 0
    for i in range(iters):
        rc |= ing(h, trans[i], stream)
        rc |= sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
        rc |= upd(h, pi[i], pp[i], B, stream)
    e1 = tm.ev()
    host_s = time.perf_counter() - h0
    torch.cuda.synchronize()
    assert rc == 0, cd.last_error()
    assert buf.sync_check() == cd.OK, cd.last_error()
    buf.close()
    ms_sep = e0.elapsed_time(e1)
    # the same iterations on a fresh buffer, each update applied with the next
    # ingest in one call (the last one after the loop, inside the clock)
    buf = cd.ReplayBuffer(cfg.capacity, (8,), torch.float32, action_bytes=4)
    h = C.c_void_p(buf.handle)
    torch.cuda.synchronize()
    e0 = tm.ev()
    h0 = time.perf_counter()
    for i in range(iters):
        if i == 0:
            rc |= ing(h, trans[i], stream)
        else:
            rc |= uing(h, pi[i - 1], pp[i - 1], B, trans[i], stream)
        rc |= sgat(h, B, pu[i], pi[i], pw[i], xfr, lbr, stream)
    rc |= upd(h, pi[iters - 1], pp[iters - 1], B, stream)
    e1 = tm.ev()
    host_ui = time.perf_counter() - h0
    torch.cuda.synchronize()
    assert rc == 0, cd.last_error()
    assert buf.sync_check() == cd.OK, cd.last_error()
    buf.close()
    ms = e0.elapsed_time(e1)
    return {"iterations": iters, "us_per_iteration": ms * 1e3 / iters, "launches_per_iteration": 2,
            "calls": "conduit_update_ingest (previous update + this ingest) + conduit_sample_gather",
            "host_enqueue_us_per_iteration": host_ui * 1e6 / iters, "sampled_per_s": iters * B / (ms / 1e3),
            "separate_calls": {"us_per_iteration": ms_sep * 1e3 / iters, "launches_per_iteration": 3,
                               "host_enqueue_us_per_iteration": host_s * 1e6 / iters}}


# ----------------------------------------------------------------------------
# CPU baseline: the oracle on the host cores, timed before the GPU is touched
# ----------------------------------------------------------------------------
def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_dqn_state(n_iter_max):
    """The oracle's DQN replay at the headline's capacity: every observation
    page resident (real DRAM traffic), metadata and priorities prefilled with
    1.05M transitions, and the inputs of n_iter_max steps generated up front."""
    import numpy as np
    import oracle
    import synth
    Cap, B, K, prefill = 1_000_000, 512, 4, 1_050_000
    cfg = synth.DQN(prefill + n_iter_max * B)
    row = 84 * 84
    store = np.empty((Cap, row), np.uint8)
    tile = cfg.frames(0, 4096).reshape(4096, row).numpy()
    for a in range(0, Cap, 4096):
        b = min(Cap, a + 4096)
        store[a:b] = tile[:b - a]
    orc = oracle.Replay(Cap, (84, 84), np.uint8, act_bytes=4, frame_stack=K, obs_storage=store)
    for a in range(0, prefill, 65536):
        b = min(prefill, a + 65536)
        orc.ingest(b - a, action=cfg.action[a:b], reward=cfg.reward[a:b], done=cfg.done[a:b],
                   episode=cfg.episode[a:b], step=cfg.step[a:b], prio=cfg.prio[a:b])
    u, prio = cfg.draws(n_iter_max, B)
    frames = cfg.frames(prefill, 8 * B).reshape(8 * B, row).numpy()
    cols = {k: np.ascontiguousarray(getattr(cfg, k)[prefill:prefill + n_iter_max * B])
            for k in ("action", "reward", "done", "episode", "step")}
    return orc, frames, cols, u, prio


def _oracle_steps(state, first, n):
    """Seconds for n oracle DQN steps (ingest 512, sample 512 with IS weights,
    gather 512 -> [512,4,84,84] fp32, update 512) starting at step `first`."""
    import oracle
    orc, frames, cols, u, prio = state
    B = 512
    t0 = time.perf_counter()
    for i in range(first, first + n):
        a = i * B
        orc.ingest(B, obs=frames[(i % 8) * B:(i % 8 + 1) * B], action=cols["action"][a:a + B],
                   reward=cols["reward"][a:a + B], done=cols["done"][a:a + B], episode=cols["episode"][a:a + B],
                   step=cols["step"][a:a + B])
        idx, _w = orc.sample(u[i])
        orc.gather(idx, oracle.XF_U8_F32)
        orc.update(idx, prio[i])
    return time.perf_counter() - t0


def _in_child(core, fn):
    """Run fn() in a forked child pinned to `core`; returns its result (a
    JSON-serialisable value).  The parent has not touched the GPU."""
    r, w = os.pipe()
    pid = os.fork()
    if pid == 0:  # child: pinned, runs the oracle only, reports, exits
        os.close(r)
        code = 0
        try:
            os.sched_setaffinity(0, {core})
            msg = json.dumps({"ok": fn()})
        except BaseException as e:  # noqa: BLE001 - reported to the parent
            msg = json.dumps({"error": repr(e)})
            code = 1
        with os.fdopen(w, "w") as f:
            f.write(msg)
        os._exit(code)
    os.close(w)
    return pid, r


def _collect(pid, r):
    with os.fdopen(r) as f:
        msg = f.read()
    os.waitpid(pid, 0)
    rec = json.loads(msg) if msg else {"error": "no result"}
    if "error" in rec:
        raise RuntimeError(f"oracle worker failed: {rec['error']}")
    return rec["ok"]


def cpu_baseline(rep_seconds=2.0, reps=5, all_core_seconds=3.0, max_workers=16):
    """The oracle (single-threaded C, never tuned for speed) on the DQN step at
    the headline's capacity, timed in forked children before this process
    touches the GPU: one child pinned to one core runs a few warm-up steps and
    then `reps` reps of ~rep_seconds (the median is reported); then one independent
    oracle instance per core (up to max_workers cores, each pinned) runs
    concurrently for ~all_core_seconds, and the aggregate rate is reported
    beside it.  Data generation is outside every timed region."""
    import statistics
    B = 512
    cores = sorted(os.sched_getaffinity(0))
    probe_steps = 3  # the warm-up, which also sizes the reps
    n_iter_max = 1200
    t_setup = time.perf_counter()
    state = _oracle_dqn_state(n_iter_max)
    setup_s = time.perf_counter() - t_setup

    def single():
        warm = _oracle_steps(state, 0, probe_steps)
        n = max(3, int(rep_seconds / (warm / probe_steps)))
        n = min(n, (n_iter_max - probe_steps) // reps)
        times = []
        first = probe_steps
        for _ in range(reps):
            times.append(_oracle_steps(state, first, n))
            first += n
        return {"steps_per_rep": n, "rep_s": times}

    pid, r = _in_child(cores[0], single)
    one = _collect(pid, r)
    med = statistics.median(one["rep_s"])
    per_step_s = med / one["steps_per_rep"]
    value = B / per_step_s
    # all cores: independent instances (copy-on-write copies of one state)
    workers = cores[:max_workers]
    n_all = max(2, min(int(all_core_seconds / per_step_s), n_iter_max - 1))

    def many():
        return _oracle_steps(state, 1, n_all)

    kids = [_in_child(c, many) for c in workers]
    t_all = [_collect(p, fd) for p, fd in kids]
    value_all = len(workers) * n_all * B / max(t_all)
    del state
    import gc
    gc.collect()
    return {
        "value": value, "unit": "sampled transitions/s", "cores": 1, "kind": "oracle",
        "sample": f"median of {reps} reps x {one['steps_per_rep']} DQN steps (the same step) on the 1M-slot "
                  f"replay (1.05M prefill) after {probe_steps} warm-up steps; one-thread C oracle on core {cores[0]}",
        "rep_s": one["rep_s"], "steps_per_rep": one["steps_per_rep"],
        "all_cores": {"value": value_all, "cores": len(workers), "steps_per_worker": n_all,
                      "worker_s_max": max(t_all),
                      "how": "one independent oracle instance per core, each pinned, run concurrently"},
        "nproc": os.cpu_count(), "cores_allowed": len(cores), "cpu_model": _cpu_model(),
        "setup_s": setup_s,
    }


def calibrate_copy():
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n}), flush=True)


# the sources the fused sampler + gather is built from: a counter summary taken
# on other sources no longer describes the kernel
FUSED_KERNEL_SOURCES = ["k_sample_gather.hip", "gather_dev.h", "descend.h", "common.h"]


def kernel_sources_sha():
    hsh = hashlib.sha256()
    for name in FUSED_KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_24456_amd", "csrc", name), "rb") as f:
            hsh.update(f.read())
    return hsh.hexdigest()[:16]


def _traffic_from_profile():
    """HBM bytes per fused sampler + gather launch from the committed counter
    summary, if it was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "sample_gather_dqn_counters.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:  # the file's first block is the fused kernel's; later blocks are context
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                rec.setdefault(k.strip(), v.strip())
    if rec.get("kernel_sources_sha256_16") != kernel_sources_sha():
        return None
    return float(rec["hbm_bytes_per_launch"])


ROWS = {"tiny": lambda: bench_tiny(), "ppo": lambda: bench_ppo(), "large": lambda: bench_large(),
        "tokens": lambda: bench_tokens(), "stress": lambda: bench_stress(), "schedule": lambda: bench_schedule(),
        "schedule_onpolicy": lambda: bench_schedule_onpolicy(), "placement": lambda: bench_placement()}


def _row_summary(name, r):
    """A few figures of an extra row for the headline line (its full record
    goes to stderr and, with --detail-out, to a file)."""
    try:
        if name == "tiny":
            return {"us_per_iteration": r["us_per_iteration"], "sampled_per_s": r["sampled_per_s"]}
        if name == "ppo":
            return {"rollout_ingest_frac": r["rollout_ingest"]["frac"], "gae_us": r["gae_2048x256"]["us"],
                    "minibatch_us": r["minibatch_gather_16384"]["us"],
                    "minibatch_frac": r["minibatch_gather_16384"]["frac"],
                    "expand_reference_frac": r["expand_reference"]["frac"],
                    "torch_expand_frac": r["expand_reference"]["torch_frac"]}
        if name == "large":
            return {"gather_bf16_us": r["gather_bf16_1024"]["us"], "gather_bf16_frac": r["gather_bf16_1024"]["frac"],
                    "iteration_us": r["iteration_us"]}
        if name == "tokens":
            return {"pack_us": r["pack_256x4096"]["us"], "gae_packed_us": r["gae_packed_256x4096"]["us"],
                    "iteration_us": r["iteration_us"], "iteration_one_launch_gae_us": r["iteration_one_launch_gae_us"]}
        if name == "stress":
            return {k: round(v["iteration_us"], 2) for k, v in r.items()}
        if name in ("schedule", "schedule_onpolicy"):
            return {"model_us": r["model_choice"]["measured_us"], "best_us": r["measured_best"]["measured_us"],
                    "sequential_us": r["sequential"]["measured_us"], "spearman": r["spearman_pred_vs_measured"]}
        if name == "placement":
            t = r["dqn_step_by_tier"]
            return {"hbm_step_us": t["hbm"]["step_us"], "pinned_step_us": t["host_pinned"]["step_us"],
                    "ranking_holds": t["model_ranking_holds"]}
    except (KeyError, TypeError):
        pass
    return None


def _emit_detail(rec, path):
    """Per-row detail: one JSON line on stderr, and appended to `path`."""
    line = json.dumps(rec)
    print("bench.detail " + line, file=sys.stderr, flush=True)
    if path:
        with open(path, "a") as f:
            f.write(line + "\n")


def main():
    args = parse()
    if args.sources_sha:
        print(kernel_sources_sha())
        return
    if args.gpus != 1:
        print(f"bench.py: the experience path runs on one GPU; --gpus {args.gpus} is not supported "
              "(one process, one GPU; no collectives)", flush=True)
        sys.exit(2)
    if args.detail_out:
        os.makedirs(os.path.dirname(os.path.abspath(args.detail_out)), exist_ok=True)
        open(args.detail_out, "w").close()
    # the oracle first, in forked children, before anything touches the GPU
    cb = None
    if not args.no_cpu_baseline:
        print("bench.py: CPU baseline (oracle, before GPU initialisation) ...", file=sys.stderr, flush=True)
        cb = cpu_baseline(rep_seconds=args.cpu_rep_seconds)
        _emit_detail({"cpu_baseline": cb}, args.detail_out)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a HIP device"
    from paper_2609_24456_amd import conduit as cd
    cd.lib()
    if args.calibrate_copy:
        calibrate_copy()
        return
    print("bench.py: DQN 1M-replay step ...", file=sys.stderr, flush=True)
    d = bench_dqn(args.steps, args.warmup)
    ms_per_step = d["total_ms"] / args.steps
    value = d["B"] * args.steps / (d["total_ms"] / 1e3)
    g_ms = d["gather_b2b_ms"]
    g_gbps = d["gather_bytes"] / g_ms / 1e6
    f_ms = d["fused_b2b_ms"]
    achieved = d["fused_bytes"] / f_ms / 1e6
    _emit_detail({"dqn": d}, args.detail_out)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "sampled transitions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8->f32",
        "data": "synthetic",
        "config": {"workload": "dqn-1M-replay: 1,000,000 slots of 84x84 u8, stack 4, batch 512, PER a=0.6 b=0.4; "
                               "step = ingest 512 + sample 512 + gather -> [512,4,84,84] f32 + update 512",
                   "capacity": 1_000_000, "batch": 512, "frame_stack": 4},
        "roofline": {"bound": "hbm", "kernel": "k_sample_gather<U8_F32> (descent + IS weights + gather, one launch)",
                     "achieved": achieved, "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBPS,
                     "traffic": _traffic_from_profile(),
                     "algorithmic_bytes": d["fused_bytes"], "avg_launch_us": f_ms * 1e3,
                     "timing": "HIP events around back-to-back launches"},
        "gather_GBps": g_gbps,
        "gather_frac_of_peak": g_gbps / PEAK_HBM_GBPS,
        "gather_avg_launch_us": g_ms * 1e3,
        "expand_reference_frac": d["expand_reference"]["frac"],
        "torch_expand_frac": d["expand_reference"]["torch_frac"],
        "ms_per_step_separate_update": d["separate_ms"] / args.steps,
        "ms_per_step_unfused": d["unfused_ms"] / args.steps,
        "kernels_us_in_step": {k.split(" ")[0]: round(v["mean_us"], 3) for k, v in d["kernels"].items()},
        "rows": {"dqn_ingest_32768_frac": d["ingest_big"]["GBps"] / PEAK_HBM_GBPS,
                 "dqn_nstep3_us": d["nstep3"]["us"],
                 "dqn_deliver_nstep3_us": {"one_call": d["deliver_nstep3"]["one_call_us"],
                                           "two_calls": d["deliver_nstep3"]["two_calls_us"]},
                 "dqn_checkpoint_GBps": {k: round(v["GBps"], 1) for k, v in d["checkpoint"].items()
                                         if isinstance(v, dict)}},
    }
    if not args.no_rows:
        only = set(x for x in args.only.split(",") if x) or set(ROWS)
        for name in ("tiny", "ppo", "large", "tokens", "stress", "schedule", "schedule_onpolicy", "placement"):
            if name in only:
                print(f"bench.py: row {name} ...", file=sys.stderr, flush=True)
                r = ROWS[name]()
                _emit_detail({"row": name, "result": r}, args.detail_out)
                out["rows"][name] = _row_summary(name, r)
                torch.cuda.empty_cache()
    if cb is not None:
        out["cpu_baseline"] = {"value": cb["value"], "unit": cb["unit"], "cores": cb["cores"], "kind": cb["kind"],
                               "sample": cb["sample"], "nproc": cb["nproc"], "cpu_model": cb["cpu_model"],
                               "all_cores": {k: cb["all_cores"][k] for k in ("value", "cores")}}
        out["gpu_over_cpu"] = value / cb["value"]
        out["gpu_over_cpu_all_cores"] = value / cb["all_cores"]["value"]
    out["detail"] = "per-row records: stderr lines 'bench.detail {...}'" + (
        f" and {args.detail_out}" if args.detail_out else "")
    # the headline: the last stdout line, compact
    print(json.dumps(out, separators=(",", ":")), flush=True)


if __name__ == "__main__":
    main()
