"""The native off-policy loop (conduit_run_offpolicy) with the experience path
on its own stream, in several timing/granularity modes: whatever the mode, the
experience operators run in one program order on their stream, so every
delivered batch, weight and the final tree must equal the oracle replaying the
operations of the loop's log in that order."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_weights_close, dev, host, read_col, tree_consistent

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
