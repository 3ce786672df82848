"""HIP graph capture of the delivery calls: the fused sampler + gather and the
priority update only enqueue kernels (no allocation, memset or host
synchronisation), so they can be captured once and replayed.  Every replay,
with new uniforms and priorities written into the captured input buffers and
eager library work between replays, is checked against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_gae_close, assert_weights_close, dev, host

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def test_captured_sample_gather_and_update_replays():
    print("graph: capture sample_gather + update, 6 replays", flush=True)
    cfg = synth.Tiny(n=synth.Tiny.capacity + 2000)
    C, B = cfg.capacity, cfg.batch
    buf = cd.ReplayBuffer(C, (8,), torch.float32, action_bytes=4)
    orc = oracle.Replay(C, (8,), np.float32, act_bytes=4)
    n = C + 2000  # full ring, wrapped: the captured size stays valid
    for a in range(0, n, 4096):
        b = min(n, a + 4096)
        cols = dict(action=cfg.action[a:b], reward=cfg.reward[a:b], done=cfg.done[a:b], episode=cfg.episode[a:b],
                    step=cfg.step[a:b])
        buf.ingest(dev(cfg.obs[a:b]), action=dev(cols["action"]), reward=dev(cols["reward"]),
                   done=dev(cols["done"]), episode_id=dev(cols["episode"]), step=dev(cols["step"]))
        orc.ingest(b - a, obs=cfg.obs[a:b], **cols)
    u, prio = cfg.draws(iters=7)

    # captured inputs and outputs: fixed addresses, refilled between replays
    u_s = dev(u[0]).clone()
    p_s = dev(prio[0]).clone()
    idx = torch.empty(B, dtype=torch.int64, device="cuda")
    w = torch.empty(B, dtype=torch.float32, device="cuda")
    obs = torch.empty((B, 1, 8), dtype=torch.float32, device="cuda")
    act = torch.empty((B, 4), dtype=torch.uint8, device="cuda")
    rew = torch.empty(B, dtype=torch.float32, device="cuda")
    dn = torch.empty(B, dtype=torch.uint8, device="cuda")
    xf = cd.transform(cd.XF_NONE)

    def step():
        buf.sample_gather(u_s, xf, idx_out=idx, w_out=w, obs=obs, action=act, reward=rew, done=dn)
        buf.update(idx, p_s)

    # warm-up on a side stream (kernels loaded), then put the state back: the
    # oracle has not seen this step
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    o_idx0, _ = orc.sample(u[0])
    orc.update(o_idx0, prio[0])  # mirror the warm-up step in the oracle

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    assert buf.sync_check() == cd.OK, cd.last_error()

    for r in range(1, 7):
        u_s.copy_(dev(u[r]))
        p_s.copy_(dev(prio[r]))
        g.replay()
        torch.cuda.synchronize()
        o_idx, o_w = orc.sample(u[r])
        assert np.array_equal(host(idx), o_idx), r
        assert_weights_close(host(w), o_w)
        o_obs, o_act, o_rew, o_done = orc.gather(o_idx, oracle.XF_NONE)
        assert np.array_equal(host(obs).reshape(-1).view(np.uint32), o_obs.reshape(-1).view(np.uint32)), r
        assert np.array_equal(host(act).reshape(o_act.shape), o_act), r
        assert np.array_equal(host(rew), o_rew), r
        assert np.array_equal(host(dn), o_done), r
        orc.update(o_idx, prio[r])
        # eager library work between replays: an extra priority update
        extra = np.arange(r * 10, r * 10 + 5, dtype=np.int64)
        extra_p = np.full(5, 1000 + r, np.uint32)
        buf.update(dev(extra), dev(extra_p))
        orc.update(extra, extra_p)
        torch.cuda.synchronize()
    assert buf.sync_check() == cd.OK, cd.last_error()
    leaves = torch.empty(C * 4, dtype=torch.uint8, device="cuda")
    buf.read(cd.COL_LEAVES, leaves)
    assert np.array_equal(host(leaves).view(np.uint32), orc.leaf)
    buf.close()


@pytest.mark.parametrize("T,E,path", [(2048, 256, "look"), (40, 4096, "short"), (1100000, 4, "split")])
def test_captured_gae_replays(T, E, path):
    """Time-major GAE captured once and replayed with new rollouts, with eager
    GAE calls of other shapes between the replays: the one-launch split (its
    capture records the table clear before the look-back kernel), the short
    tile path and the three-launch split."""
    print(f"graph: capture gae [{T}, {E}] ({path}), 4 replays", flush=True)
    assert cd.gae_plan(T, E)[0] == path
    rng = np.random.default_rng(5)
    r_s = torch.empty((T, E), dtype=torch.float32, device="cuda")
    v_s = torch.empty((T, E), dtype=torch.float32, device="cuda")
    d_s = torch.empty((T, E), dtype=torch.uint8, device="cuda")
    b_s = torch.empty(E, dtype=torch.float32, device="cuda")
    adv = torch.empty((T, E), dtype=torch.float32, device="cuda")
    ret = torch.empty((T, E), dtype=torch.float32, device="cuda")

    def draw():
        return (rng.standard_normal((T, E)).astype(np.float32), rng.standard_normal((T, E)).astype(np.float32),
                (rng.random((T, E)) < 0.01).astype(np.uint8), rng.standard_normal(E).astype(np.float32))

    def gae():
        cd.conduit_gae(r_s, v_s, d_s, b_s, 0.99, 0.95, adv, ret)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        gae()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gae()
    torch.cuda.synchronize()
    for k in range(4):
        r, v, d, b = draw()
        for dst, src in ((r_s, r), (v_s, v), (d_s, d), (b_s, b)):
            dst.copy_(dev(src))
        adv.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        oa, orr = oracle.gae(r, v, d, b, 0.99, 0.95)
        assert_gae_close(host(adv), oa)
        assert_gae_close(host(ret), orr)
        # eager calls between replays: more tiles, then fewer
        for T2, E2 in ((3000, 1000), (300, 8)):
            r2 = rng.standard_normal((T2, E2)).astype(np.float32)
            d2 = np.zeros((T2, E2), np.uint8)
            a2 = torch.empty((T2, E2), dtype=torch.float32, device="cuda")
            x2 = torch.empty((T2, E2), dtype=torch.float32, device="cuda")
            cd.conduit_gae(dev(r2), None, dev(d2), None, 0.9, 0.8, a2, x2)
            oa2, _ = oracle.gae(r2, None, d2, None, 0.9, 0.8)
            assert_gae_close(host(a2), oa2)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
