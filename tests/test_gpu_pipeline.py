"""The native loops with the experience path on a second stream, in several
timing/granularity modes.  Off-policy (conduit_run_offpolicy): whatever the
mode the experience operators keep one program order, so every delivered
batch, weight and the final tree must equal the oracle replaying the
operations of the loop's log in that order.  On-policy (conduit_run_onpolicy):
the outputs do not depend on the mode at all; every minibatch, advantage and
return must equal the oracle's GAE and shuffle-gather of each rollout."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_gae_close, assert_weights_close, dev, host, read_col, tree_consistent

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def _loop(mode, cap=5000, d=64, U=64, B=64, iters=16, prefill=4000, work=(2000, 3000)):
    overlap_ing, g_ing, overlap_del, g_del = mode
    cfg = synth.Stress(d, prefill + iters * U)
    buf = cd.ReplayBuffer(cap, cfg.obs_shape, torch.float32, action_bytes=4)
    orc = oracle.Replay(cap, cfg.obs_shape, np.float32, act_bytes=4, keep_obs=False)
    for a in range(0, prefill, 1000):
        b = min(prefill, a + 1000)
        buf.ingest(cfg.rows(a, b - a, "cuda"), action=dev(cfg.action[a:b]), reward=dev(cfg.reward[a:b]),
                   done=dev(cfg.done[a:b]), prio=dev(cfg.prio[a:b]))
        orc.ingest(b - a, obs=None, action=cfg.action[a:b], reward=cfg.reward[a:b], done=cfg.done[a:b],
                   prio=cfg.prio[a:b])
    # the actor's rollout units, staged: unit t = stream positions prefill + [t U, (t+1) U)
    rows = cfg.rows(prefill, iters * U, "cuda")
    sl = slice(prefill, prefill + iters * U)
    act_d, rew_d, done_d, prio_d = dev(cfg.action[sl]), dev(cfg.reward[sl]), dev(cfg.done[sl]), dev(cfg.prio[sl])
    rng = np.random.default_rng(11)
    u = synth.uniforms(rng, iters * B)
    new_prio = synth.quantise_priority(rng.lognormal(0, 1, iters * B))
    u_d, p_d = dev(u), dev(new_prio)
    idx = torch.empty(iters * B, dtype=torch.int64, device="cuda")
    w = torch.empty(iters * B, dtype=torch.float32, device="cuda")
    obs = torch.empty((iters * B, 1) + cfg.obs_shape, dtype=torch.float32, device="cuda")
    rew = torch.empty(iters * B, dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_NONE)
    lp = cd.OffpolicyLoop()
    lp.overlap_ing, lp.g_ing, lp.overlap_del, lp.g_del = overlap_ing, g_ing, overlap_del, g_del
    lp.iters, lp.unit, lp.batch = iters, U, B
    lp.rollout_work, lp.update_work = work
    lp.rollout.obs, lp.rollout.action, lp.rollout.reward = rows.data_ptr(), act_d.data_ptr(), rew_d.data_ptr()
    lp.rollout.done, lp.rollout.prio = done_d.data_ptr(), prio_d.data_ptr()
    lp.uniforms, lp.new_prio = u_d.data_ptr(), p_d.data_ptr()
    lp.idx_out, lp.is_w_out = idx.data_ptr(), w.data_ptr()
    lp.xf = C.pointer(xf)
    lp.out.obs, lp.out.reward = obs.data_ptr(), rew.data_ptr()
    comp, exp = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    ms, log = cd.conduit_run_offpolicy(buf.handle, lp, comp, exp)
    assert ms > 0
    assert buf.sync_check() == cd.OK, cd.last_error()
    # the oracle replays the experience stream's operations in order
    idx_h, w_h, obs_h, rew_h = host(idx), host(w), host(obs), host(rew)
    for kind, a, b in log:
        if kind == cd.OP_INGEST:
            p0, p1 = prefill + a * U, prefill + (a + b) * U
            orc.ingest(p1 - p0, obs=None, action=cfg.action[p0:p1], reward=cfg.reward[p0:p1],
                       done=cfg.done[p0:p1], prio=cfg.prio[p0:p1])
        elif kind == cd.OP_DELIVER:
            first = b
            n = min(iters, first + g_del) - first
            r = slice(first * B, (first + n) * B)
            o_idx, o_w = orc.sample(u[r])
            assert np.array_equal(idx_h[r], o_idx), (kind, a, b)
            assert_weights_close(w_h[r], o_w)
            want = cfg.rows_at(orc.position[o_idx]).numpy()
            assert np.array_equal(obs_h[r].reshape(want.shape).view(np.uint32), want.view(np.uint32)), (kind, a, b)
            _, _, o_rew, _ = orc.gather(o_idx)
            assert np.array_equal(rew_h[r], o_rew), (kind, a, b)
        else:
            assert kind == cd.OP_PRIO
            orc.update(idx_h[a * B:(a + 1) * B], new_prio[a * B:(a + 1) * B])
    assert np.array_equal(read_col(buf, cd.COL_LEAVES, cap * 4, np.uint32), orc.leaf)
    assert tree_consistent(buf, cap) == orc.total_priority()
    buf.close()
    return log


@pytest.mark.parametrize("mode", [(0, 1, 0, 1), (1, 1, 1, 1), (1, 4, 0, 2), (0, 2, 1, 4), (1, 8, 1, 8), (0, 3, 1, 5)])
def test_offpolicy_loop_matches_oracle_in_every_mode(mode):
    print(f"offpolicy loop mode {mode}", flush=True)
    log = _loop(mode)
    kinds = [op[0] for op in log]
    assert kinds.count(cd.OP_PRIO) == 16
    assert sum(op[2] for op in log if op[0] == cd.OP_INGEST) == 16  # every rollout unit ingested once
    firsts = [op[2] for op in log if op[0] == cd.OP_DELIVER]
    assert firsts == list(range(0, 16, mode[3]))  # every iteration's batch delivered once, in order


def test_offpolicy_loop_rejects_bad_modes():
    buf = cd.ReplayBuffer(64, (4,), torch.uint8)
    lp = cd.OffpolicyLoop()
    lp.g_ing, lp.g_del, lp.iters, lp.unit, lp.batch = 0, 1, 1, 1, 1
    with pytest.raises(cd.ConduitError) as e:
        cd.conduit_run_offpolicy(buf.handle, lp, None, None)
    assert e.value.status == cd.EINVAL
    buf.close()


def test_standin_scales_with_work_and_sync_costs_are_finite():
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    times = []
    for work in (20000, 40000):
        cd.conduit_standin(work, s1)  # warm
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(s1):
            a.record()
            cd.conduit_standin(work, s1)
            b.record()
        b.synchronize()
        times.append(a.elapsed_time(b))
    assert 1.6 < times[1] / times[0] < 2.4, times
    hop, dep = cd.conduit_sync_cost_us(s1, s2, 64)
    assert 0.0 <= dep < 1000.0 and 0.0 <= hop < 1000.0, (hop, dep)


def _onpolicy(mode, iters=3, T=32, E=16, M=4, shape=(3, 8, 8), work=(4000, 4000), placement=cd.PLACE_HBM):
    overlap_ing, ing_slices, overlap_del = mode
    rng = np.random.default_rng(23)
    U = T * E
    obs = rng.integers(0, 256, (iters, U) + shape, dtype=np.uint8)
    rew = rng.standard_normal((iters, U)).astype(np.float32)
    val = rng.standard_normal((iters, U)).astype(np.float32)
    done = (rng.random((iters, U)) < 0.05).astype(np.uint8)
    boot = rng.standard_normal((iters, E)).astype(np.float32)
    perm = np.stack([rng.permutation(U) for _ in range(iters)]).astype(np.int64)
    gamma, lam = 0.99, 0.95
    buf = cd.ReplayBuffer(U, shape, torch.uint8, prioritized=False, action_bytes=0, placement=placement)
    d = {k: dev(v) for k, v in dict(obs=obs, rew=rew, val=val, done=done, boot=boot, perm=perm).items()}
    adv = torch.empty(U, dtype=torch.float32, device="cuda")
    ret = torch.empty(U, dtype=torch.float32, device="cuda")
    out = torch.empty((iters, U) + shape, dtype=torch.float32, device="cuda")
    out_adv = torch.empty((iters, U), dtype=torch.float32, device="cuda")
    out_ret = torch.empty((iters, U), dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_U8_F32)
    lp = cd.OnpolicyLoop()
    lp.overlap_ing, lp.ing_slices, lp.overlap_del, lp.minibatches = overlap_ing, ing_slices, overlap_del, M
    lp.iters, lp.steps, lp.envs = iters, T, E
    lp.rollout_work, lp.update_work = work
    lp.obs, lp.reward, lp.value, lp.done = d["obs"].data_ptr(), d["rew"].data_ptr(), d["val"].data_ptr(), \
        d["done"].data_ptr()
    lp.bootstrap, lp.gamma, lp.lam, lp.perm = d["boot"].data_ptr(), gamma, lam, d["perm"].data_ptr()
    lp.xf = C.pointer(xf)
    lp.adv, lp.ret = adv.data_ptr(), ret.data_ptr()
    lp.out_obs, lp.out_adv, lp.out_ret = out.data_ptr(), out_adv.data_ptr(), out_ret.data_ptr()
    comp, exp = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    ms, log = cd.conduit_run_onpolicy(buf.handle, lp, comp, exp)
    assert ms > 0
    assert buf.sync_check() == cd.OK, cd.last_error()
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    out_h, adv_h, ret_h = host(out), host(out_adv), host(out_ret)
    for i in range(iters):
        oa, orr = oracle.gae(rew[i].reshape(T, E), val[i].reshape(T, E), done[i].reshape(T, E), boot[i], gamma, lam)
        want = oracle.rows(obs[i], perm[i], oracle.XF_U8_F32)
        assert np.array_equal(out_h[i].view(np.uint32), want.view(np.uint32)), i
        assert_gae_close(adv_h[i], oa.reshape(-1)[perm[i]])
        assert_gae_close(ret_h[i], orr.reshape(-1)[perm[i]])
    # the rollout left in the buffer is the last iteration's
    assert np.array_equal(read_col(buf, cd.COL_OBS, obs[-1].nbytes, np.uint8), obs[-1].reshape(-1))
    buf.close()
    return log


@pytest.mark.parametrize("mode", [(0, 4, 0), (1, 1, 1), (1, 3, 0), (0, 2, 1), (1, 4, 1), (0, 1, 0)])
def test_onpolicy_loop_matches_oracle_in_every_mode(mode):
    print(f"onpolicy loop mode {mode}", flush=True)
    M, iters = 4, 3
    log = _onpolicy(mode, iters=iters, M=M)
    j = mode[1]
    want_ing = []
    first = 0
    for s in range(M):
        if s + 1 - first == j or s == M - 1:
            want_ing.append((first, s + 1 - first))
            first = s + 1
    for i in range(iters):
        ops = [op for op in log if op[1] == i]
        assert [(op[2], op[3]) for op in ops if op[0] == cd.OP_INGEST] == want_ing
        kinds = [op[0] for op in ops]
        # program order: the rollout's ingestions, its GAE, its minibatches in order
        assert kinds == [cd.OP_INGEST] * len(want_ing) + [cd.OP_GAE] + [cd.OP_DELIVER] * M
        assert [op[2] for op in ops if op[0] == cd.OP_DELIVER] == list(range(M))


def test_onpolicy_loop_with_the_rollout_in_pinned_host_memory():
    print("onpolicy loop: rollout buffer in pinned host memory, mode (1, 2, 1)", flush=True)
    _onpolicy((1, 2, 1), placement=cd.PLACE_HOST_PINNED)


def test_placement_profile_is_sane():
    prof = cd.conduit_placement_profile(64 << 20, 2)
    d = prof.as_dict()
    print("placement profile", d, flush=True)
    assert all(v > 0 for v in d["bw_in_cpu_actor"] + d["bw_in_gpu_actor"] + d["bw_out"] + d["mem"])
    # HBM to HBM is the fastest leg of all on any sane host
    assert d["bw_out"][cd.PLACE_HBM] > d["bw_out"][cd.PLACE_HOST_PINNED]
    choice, t = cd.conduit_place(prof, 1, 1000, 28224.0)
    assert choice == cd.PLACE_HBM and t[0] == min(t)


def test_onpolicy_loop_rejects_bad_configurations():
    buf = cd.ReplayBuffer(64, (4,), torch.uint8, prioritized=False, action_bytes=0)
    lp = cd.OnpolicyLoop()
    lp.overlap_ing, lp.ing_slices, lp.overlap_del, lp.minibatches = 0, 1, 0, 3
    lp.iters, lp.steps, lp.envs = 1, 8, 8  # steps not a multiple of minibatches
    with pytest.raises(cd.ConduitError) as e:
        cd.conduit_run_onpolicy(buf.handle, lp, None, None)
    assert e.value.status == cd.EINVAL
    buf.close()


def _standin_us_per_work(stream):
    L = cd.lib()
    s = C.c_void_p(stream.cuda_stream)
    L.conduit_standin(100_000, s)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        e0.record()
        L.conduit_standin(400_000, s)
        e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / 400_000


def test_onpolicy_whole_rollout_ingestion_overlaps_nothing_on_the_executor():
    """The reading that an on-policy ingestion of the whole rollout (g = 1)
    hides nothing when overlapped, measured on the executor rather than taken
    from the model.  App. C Invariant 2 lets on-policy training pipeline only
    within its own iteration: the g = 1 ingestion is one invocation that needs
    the rollout's last slice and must end before that iteration's delivery, so
    there is no rollout left to run beside it.  Taken at g >= 1, App. E would
    instead predict that overlap hides min(T_rollout, T_ing(1)).  On a rollout
    whose ingestion costs over 50 us, the overlapped mode must not come out
    faster than the inline one by half of that cost."""
    print("onpolicy: g = 1 ingestion inline vs overlapped, 64 envs x 256 steps of 3x84x84", flush=True)
    L = cd.lib()
    T, E, M, iters = 256, 64, 8, 3
    shape = (3, 84, 84)
    row = int(np.prod(shape))
    U = T * E
    rng = np.random.default_rng(31)
    obs = torch.randint(0, 256, (iters, U, row), dtype=torch.uint8, device="cuda")
    d = {k: dev(v) for k, v in dict(
        rew=rng.standard_normal((iters, U)).astype(np.float32), val=rng.standard_normal((iters, U)).astype(np.float32),
        done=(rng.random((iters, U)) < 0.01).astype(np.uint8), boot=rng.standard_normal((iters, E)).astype(np.float32),
        perm=np.stack([rng.permutation(U) for _ in range(iters)]).astype(np.int64)).items()}
    buf = cd.ReplayBuffer(U, shape, torch.uint8, prioritized=False, action_bytes=0)
    adv = torch.empty(U, dtype=torch.float32, device="cuda")
    ret = torch.empty(U, dtype=torch.float32, device="cuda")
    out = torch.empty((iters, U, row), dtype=torch.float32, device="cuda")
    out_adv = torch.empty((iters, U), dtype=torch.float32, device="cuda")
    out_ret = torch.empty((iters, U), dtype=torch.float32, device="cuda")
    xf = cd.transform(cd.XF_U8_F32)
    comp, exp = torch.cuda.Stream(), torch.cuda.Stream()
    upw = _standin_us_per_work(comp)
    work = (int(600.0 / upw), int(800.0 / upw))  # rollout 600 us, update 800 us per iteration

    def loop(overlap_ing):
        lp = cd.OnpolicyLoop()
        lp.overlap_ing, lp.ing_slices, lp.overlap_del, lp.minibatches = overlap_ing, M, 0, M
        lp.iters, lp.steps, lp.envs = iters, T, E
        lp.rollout_work, lp.update_work = work
        lp.obs, lp.reward, lp.value, lp.done = obs.data_ptr(), d["rew"].data_ptr(), d["val"].data_ptr(), \
            d["done"].data_ptr()
        lp.bootstrap, lp.gamma, lp.lam, lp.perm = d["boot"].data_ptr(), 0.99, 0.95, d["perm"].data_ptr()
        lp.xf = C.pointer(xf)
        lp.adv, lp.ret = adv.data_ptr(), ret.data_ptr()
        lp.out_obs, lp.out_adv, lp.out_ret = out.data_ptr(), out_adv.data_ptr(), out_ret.data_ptr()
        # the GPU starts behind a stand-in, so the loop's events time the GPU
        # and not the host's enqueue
        L.conduit_standin(int(iters * 3000.0 / upw), C.c_void_p(comp.cuda_stream))
        ms, log = cd.conduit_run_onpolicy(buf.handle, lp, comp, exp)
        assert [op for op in log if op[0] == cd.OP_INGEST] == [(cd.OP_INGEST, i, 0, M) for i in range(iters)]
        return ms * 1e3 / iters

    # the cost of the g = 1 ingestion: all U rows in one call, alone
    tr = cd.Transitions()
    tr.n, tr.obs = U, obs[0].data_ptr()
    tr.reward, tr.done = d["rew"][0].data_ptr(), d["done"][0].data_ptr()
    s = C.c_void_p(comp.cuda_stream)
    assert L.conduit_ingest(buf.handle, C.byref(tr), s) == 0
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(comp):
        e0.record()
        for _ in range(4):
            assert L.conduit_ingest(buf.handle, C.byref(tr), s) == 0
        e1.record()
    torch.cuda.synchronize()
    t_ing1 = e0.elapsed_time(e1) * 1e3 / 4
    assert buf.info().head == 0  # every ingest filled the ring exactly
    loop(0)  # warm-up
    inline = min(loop(0) for _ in range(2))
    overlapped = min(loop(1) for _ in range(2))
    print(f"T_ing(1) = {t_ing1:.1f} us; iteration inline {inline:.1f} us, overlapped {overlapped:.1f} us",
          flush=True)
    assert t_ing1 > 50.0
    assert overlapped - inline > -0.5 * t_ing1, (inline, overlapped, t_ing1)
    assert buf.sync_check() == cd.OK and cd.conduit_sync_check() == cd.OK, cd.last_error()
    buf.close()
