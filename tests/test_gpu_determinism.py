"""Run-to-run determinism on the GPU: the same inputs through fresh buffers
give bit-identical outputs, every step.  Nothing in the path depends on the
order in which workgroups or atomics land (integer tree arithmetic,
last-writer-wins updates, integer minimum for the IS weights, fixed
composition order in the split GAE), so any difference here would be a race."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import buffer_columns, dev

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def _dqn_run(cfg, u, prio, cap, prefill, iters, B, K=4):
    buf = cd.ReplayBuffer(cap, (84, 84), torch.uint8, frame_stack=K, action_bytes=4)
    for a in range(0, prefill, 1024):
        b = min(prefill, a + 1024)
        buf.ingest(cfg.frames(a, b - a, "cuda"), action=dev(cfg.action[a:b]), reward=dev(cfg.reward[a:b]),
                   done=dev(cfg.done[a:b]), episode_id=dev(cfg.episode[a:b]), step=dev(cfg.step[a:b]),
                   prio=dev(cfg.prio[a:b]))
    xf = cd.transform(cd.XF_U8_F32)
    outs = []
    pos, pending = prefill, None
    for it in range(iters):
        cols = dict(action=dev(cfg.action[pos:pos + B]), reward=dev(cfg.reward[pos:pos + B]),
                    done=dev(cfg.done[pos:pos + B]), episode_id=dev(cfg.episode[pos:pos + B]),
                    step=dev(cfg.step[pos:pos + B]))
        if pending is None:
            buf.ingest(cfg.frames(pos, B, "cuda"), **cols)
        else:
            buf.update_ingest(pending[0], pending[1], cfg.frames(pos, B, "cuda"), **cols)
        pos += B
        obs = torch.empty((B, K, 84, 84), dtype=torch.float32, device="cuda")
        rew = torch.empty(B, dtype=torch.float32, device="cuda")
        idx, w = buf.sample_gather(dev(u[it]), xf, obs=obs, reward=rew)
        pending = (idx.clone(), dev(prio[it]))
        outs.append([t.cpu().numpy().copy() for t in (idx, w, obs, rew)])
    buf.update(pending[0], pending[1])
    assert buf.sync_check() == cd.OK, cd.last_error()
    cols = buffer_columns(buf)
    buf.close()
    return outs, cols


def test_dqn_steps_are_bit_identical_across_runs():
    print("determinism: DQN cap 4096, 6 steps of update + ingest 512, sample + gather 512, twice", flush=True)
    cap, prefill, iters, B = 4096, 5000, 6, 512
    cfg = synth.DQN(prefill + iters * B)
    u, prio = cfg.draws(iters, B)
    o1, c1 = _dqn_run(cfg, u, prio, cap, prefill, iters, B)
    o2, c2 = _dqn_run(cfg, u, prio, cap, prefill, iters, B)
    for it, (a, b) in enumerate(zip(o1, o2)):
        for x, y, name in zip(a, b, ("idx", "w", "obs", "reward")):
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), (it, name)
    assert c1.keys() == c2.keys()
    for k in c1:
        assert np.array_equal(c1[k], c2[k]), k


@pytest.mark.parametrize("T,E", [(2048, 256), (4097, 4100), (65, 131072)])
def test_gae_is_bit_identical_across_calls(T, E):
    print(f"determinism: GAE [{T}, {E}], three calls", flush=True)
    rng = np.random.default_rng(T + E)
    r = dev(rng.standard_normal((T, E)).astype(np.float32))
    v = dev(rng.standard_normal((T, E)).astype(np.float32))
    d = dev((rng.random((T, E)) < 0.01).astype(np.uint8))
    b = dev(rng.standard_normal(E).astype(np.float32))
    res = []
    for _ in range(3):
        adv, ret = torch.empty((T, E), device="cuda"), torch.empty((T, E), device="cuda")
        cd.conduit_gae(r, v, d, b, 0.99, 0.95, adv, ret)
        res.append((adv.cpu().numpy(), ret.cpu().numpy()))
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    for a, c in res[1:]:
        assert np.array_equal(a.view(np.uint32), res[0][0].view(np.uint32))
        assert np.array_equal(c.view(np.uint32), res[0][1].view(np.uint32))


def test_split_gae_over_many_calls():
    # the look-back table is reused by every call (a new epoch each time): 300
    # calls in a row, each equal bit for bit to the first
    print("determinism: GAE [2048, 256], 300 calls back to back", flush=True)
    T, E = 2048, 256
    rng = np.random.default_rng(9)
    r = dev(rng.standard_normal((T, E)).astype(np.float32))
    v = dev(rng.standard_normal((T, E)).astype(np.float32))
    d = dev((rng.random((T, E)) < 0.01).astype(np.uint8))
    b = dev(rng.standard_normal(E).astype(np.float32))
    adv0, ret0 = torch.empty((T, E), device="cuda"), torch.empty((T, E), device="cuda")
    cd.conduit_gae(r, v, d, b, 0.99, 0.95, adv0, ret0)
    adv, ret = torch.empty_like(adv0), torch.empty_like(ret0)
    bad = 0
    for _ in range(300):
        cd.conduit_gae(r, v, d, b, 0.99, 0.95, adv, ret)
        bad += int(not torch.equal(adv.view(torch.int32), adv0.view(torch.int32)))
        bad += int(not torch.equal(ret.view(torch.int32), ret0.view(torch.int32)))
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    assert bad == 0
