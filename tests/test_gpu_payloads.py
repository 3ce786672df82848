"""GPU parity for the large-payload replay (3x224x224 uint8 -> normalised bf16)
and the long-context token replay (ragged sequences -> padded batch + mask +
log-probs, then per-sequence GAE), against the oracle through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_gae_close, assert_weights_close, dev, host, read_col, swap_through_checkpoint, tree_consistent

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def run_large(cap, prefill, iters, batch, chunk, check_rows, fused=False):
    cfg = synth.Large(prefill)
    u, prio = cfg.draws(iters, batch)
    shape = cfg.obs_shape
    row = int(np.prod(shape))
    buf = cd.ReplayBuffer(cap, shape, torch.uint8, action_bytes=24)
    store = np.zeros((cap, row), np.uint8)
    orc = oracle.Replay(cap, shape, np.uint8, act_bytes=24, obs_storage=store)
    for a in range(0, prefill, chunk):
        b = min(prefill, a + chunk)
        buf.ingest(cfg.rows(a, b - a, "cuda"), action=dev(cfg.action[a:b]), reward=dev(cfg.reward[a:b]),
                   done=dev(cfg.done[a:b]), prio=dev(cfg.prio[a:b]))
        orc.ingest(b - a, obs=None, action=cfg.action[a:b], reward=cfg.reward[a:b], done=cfg.done[a:b],
                   prio=cfg.prio[a:b])
    xf = cd.transform(cd.XF_U8_BF16_NORM, cfg.mean, cfg.std)
    out = torch.empty((batch, 1) + shape, dtype=torch.bfloat16, device="cuda")
    act = torch.empty((batch, 6), dtype=torch.float32, device="cuda")
    rew = torch.empty(batch, dtype=torch.float32, device="cuda")
    for it in range(iters):
        if fused:
            idx, w = buf.sample_gather(dev(u[it]), xf, obs=out, action=act, reward=rew)
        else:
            idx, w = buf.sample(dev(u[it]))
            buf.gather(idx, xf, obs=out, action=act, reward=rew)
        buf.update(idx, dev(prio[it]))
        o_idx, o_w = orc.sample(u[it])
        assert np.array_equal(host(idx), o_idx), it
        assert_weights_close(host(w), o_w)
        sel = o_idx[check_rows]
        need = np.unique(sel)
        store[need] = cfg.rows_at(orc.position[need]).reshape(len(need), -1).numpy()
        o_obs, o_act, o_rew, _ = orc.gather(sel, oracle.XF_U8_BF16_NORM, cfg.mean, cfg.std)
        g = host(out[torch.as_tensor(check_rows, device="cuda")].view(torch.int16)).view(np.uint16)
        assert np.array_equal(g, o_obs), it
        assert np.array_equal(host(act)[check_rows].view(np.uint8).reshape(len(sel), -1), o_act), it
        assert np.array_equal(host(rew)[check_rows], o_rew), it
        orc.update(o_idx, prio[it])
    assert buf.sync_check() == cd.OK, cd.last_error()
    assert np.array_equal(read_col(buf, cd.COL_LEAVES, cap * 4, np.uint32), orc.leaf)
    assert tree_consistent(buf, cap) == orc.total_priority()
    buf.close()


@pytest.mark.parametrize("fused", [False, True])
def test_large_payload_reduced(fused):
    print(f"large: cap 600, prefill 700, batch 64 -> bf16, fused={fused}", flush=True)
    run_large(cap=600, prefill=700, iters=3, batch=64, chunk=256, check_rows=np.arange(64), fused=fused)


@pytest.mark.slow
def test_large_payload_full_size():
    print("large: cap 200000 (30 GB), batch 1024 -> bf16, 2 iterations, every row", flush=True)
    run_large(cap=200_000, prefill=200_000, iters=2, batch=1024, chunk=2048, check_rows=np.arange(1024))


def run_tokens(cap, max_len, min_len, prefill, iters, batch, chunk, with_values, fused=False, placement=cd.PLACE_HBM,
               weight_norm=cd.WNORM_BATCH, with_gae=False, resume=None):
    """resume = (iteration, via, placement, tmp_dir): before that iteration the
    buffer goes through a checkpoint and a restore into a new buffer."""
    cfg = synth.Tokens(prefill, max_len=max_len, min_len=min_len)
    u, prio = cfg.draws(iters, batch)
    buf = cd.ReplayBuffer(cap, (max_len,), torch.int32, action_bytes=4, ragged=True, aux_elem_bytes=4,
                          placement=placement, weight_norm=weight_norm)
    store = np.zeros((cap, max_len * 4), np.uint8)
    aux_store = np.zeros((cap, max_len * 4), np.uint8)
    orc = oracle.Replay(cap, (max_len,), np.int32, act_bytes=4, ragged=True, aux_dtype=np.float32,
                        obs_storage=store, buffer_norm=weight_norm == cd.WNORM_BUFFER)
    orc.aux = aux_store
    orc._s.aux = aux_store.ctypes.data
    for a in range(0, prefill, chunk):
        b = min(prefill, a + chunk)
        tok, lp, off = cfg.packed(a, b - a, "cuda")
        buf.ingest(tok, offsets=off, aux=lp, action=dev(cfg.action[a:b]), reward=dev(cfg.reward[a:b]),
                   done=dev(cfg.done[a:b]), prio=dev(cfg.prio[a:b]))
        off_h = cfg.offsets[a:b + 1] - cfg.offsets[a]
        orc.ingest(b - a, obs=None, offsets=off_h, action=cfg.action[a:b], reward=cfg.reward[a:b],
                   done=cfg.done[a:b], prio=cfg.prio[a:b])
    xf = cd.transform(cd.XF_TOKENS_PAD, pad_id=0)
    seq = torch.empty((batch, max_len), dtype=torch.int32, device="cuda")
    mask = torch.empty((batch, max_len), dtype=torch.uint8, device="cuda")
    lp_out = torch.empty((batch, max_len), dtype=torch.float32, device="cuda")
    length = torch.empty(batch, dtype=torch.int32, device="cuda")
    rew = torch.empty(batch, dtype=torch.float32, device="cuda")
    adv = torch.empty((batch, max_len), dtype=torch.float32, device="cuda")
    ret = torch.empty((batch, max_len), dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(4)
    for it in range(iters):
        if resume is not None and it == resume[0]:
            buf = swap_through_checkpoint(
                buf, resume[1], lambda: cd.ReplayBuffer(cap, (max_len,), torch.int32, action_bytes=4, ragged=True,
                                                        aux_elem_bytes=4, placement=resume[2],
                                                        weight_norm=weight_norm), resume[3])
        vals = rng.standard_normal((batch, max_len)).astype(np.float32) if with_values else None
        if with_gae:  # sampler + packing + GAE of the packed rows, one launch
            adv.fill_(float("nan"))
            ret.fill_(float("nan"))
            idx, w = buf.sample_pack_gae(dev(u[it]), xf, cfg.gamma, cfg.lam, adv, ret,
                                         values=dev(vals) if vals is not None else None, obs=seq, mask=mask,
                                         aux=lp_out, length=length, reward=rew)
        else:
            if fused:  # ragged: the sampler + packing kernel, one launch
                idx, w = buf.sample_gather(dev(u[it]), xf, obs=seq, mask=mask, aux=lp_out, length=length, reward=rew)
            else:
                idx, w = buf.sample(dev(u[it]))
                buf.gather(idx, xf, obs=seq, mask=mask, aux=lp_out, length=length, reward=rew)
            cd.conduit_gae_packed(rew, length, dev(vals) if vals is not None else None, max_len, cfg.gamma, cfg.lam,
                                  adv, ret)
        buf.update(idx, dev(prio[it]))
        o_idx, o_w = orc.sample(u[it])
        assert np.array_equal(host(idx), o_idx), it
        assert_weights_close(host(w), o_w)
        need = np.unique(o_idx)
        for j, (t, l) in zip(need, cfg.sequences_at(orc.position[need])):
            store[j, :4 * len(t)] = t.view(np.uint8)
            aux_store[j, :4 * len(l)] = l.view(np.uint8)
        o_seq, o_mask, o_aux, o_len, o_rew = orc.pack(o_idx, pad_id=0)
        assert np.array_equal(host(seq), o_seq), it
        assert np.array_equal(host(mask), o_mask), it
        assert np.array_equal(host(lp_out).view(np.uint32), o_aux.view(np.uint32)), it
        assert np.array_equal(host(length), o_len), it
        assert np.array_equal(host(rew), o_rew), it
        oa, orr = oracle.gae_packed(o_rew, o_len, vals, max_len, cfg.gamma, cfg.lam)
        assert_gae_close(host(adv), oa)
        assert_gae_close(host(ret), orr)
        orc.update(o_idx, prio[it])
    assert buf.sync_check() == cd.OK, cd.last_error()
    assert tree_consistent(buf, cap) == orc.total_priority()
    lens = read_col(buf, cd.COL_LENGTH, cap * 4, np.int32)
    written = orc.position >= 0
    assert np.array_equal(lens[written], orc.length[written])
    buf.close()


@pytest.mark.parametrize("fused", [False, True])
def test_tokens_reduced(fused):
    print(f"tokens: cap 300, max_len 256, prefill 400 (wraps), batch 64, fused={fused}", flush=True)
    run_tokens(cap=300, max_len=256, min_len=8, prefill=400, iters=3, batch=64, chunk=128, with_values=True,
               fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_tokens_buffer_wide_weights(fused):
    print(f"tokens: buffer-wide IS normalisation, cap 300, fused={fused}", flush=True)
    run_tokens(cap=300, max_len=256, min_len=8, prefill=400, iters=3, batch=64, chunk=128, with_values=True,
               fused=fused, weight_norm=cd.WNORM_BUFFER)


@pytest.mark.parametrize("fused", [False, True])
def test_tokens_payload_in_pinned_host_memory(fused):
    # token and log-probability columns in pinned host memory (Sec. 5 placement)
    print(f"tokens: payload in pinned host memory, cap 300, fused={fused}", flush=True)
    run_tokens(cap=300, max_len=256, min_len=8, prefill=400, iters=3, batch=64, chunk=128, with_values=True,
               fused=fused, placement=cd.PLACE_HOST_PINNED)


@pytest.mark.parametrize("with_gae", [False, True])
def test_tokens_long_rows_segmented_gae(with_gae):
    print(f"tokens: max_len 8192 (two GAE segments), batch 16, one-launch GAE={with_gae}", flush=True)
    run_tokens(cap=40, max_len=8192, min_len=3000, prefill=50, iters=2, batch=16, chunk=25, with_values=True,
               with_gae=with_gae)


@pytest.mark.parametrize("with_values,weight_norm", [(True, cd.WNORM_BATCH), (False, cd.WNORM_BUFFER)])
def test_tokens_sample_pack_gae_one_launch(with_values, weight_norm):
    print(f"tokens: sample + pack + GAE in one launch, values={with_values}, weight_norm={weight_norm}", flush=True)
    run_tokens(cap=300, max_len=256, min_len=8, prefill=400, iters=3, batch=64, chunk=128, with_values=with_values,
               weight_norm=weight_norm, with_gae=True)
    run_tokens(cap=300, max_len=300, min_len=1, prefill=330, iters=2, batch=77, chunk=100, with_values=with_values,
               weight_norm=weight_norm, with_gae=True)


@pytest.mark.slow
@pytest.mark.parametrize("fused,with_gae", [(False, False), (True, False), (True, True)])
def test_tokens_full_size(fused, with_gae):
    print(f"tokens: cap 65536 x 4096, batch 256, 2 iterations, fused={fused}, one-launch GAE={with_gae}", flush=True)
    run_tokens(cap=65536, max_len=4096, min_len=512, prefill=65536, iters=2, batch=256, chunk=4096,
               with_values=False, fused=fused, with_gae=with_gae)


def run_stress(cap, d, prefill, iters, batch, chunk, check_rows):
    """Synthetic stress transitions (obs and next_obs, d fp32 each) through
    ingest, the one-call sample + gather and update; indices and weights against
    the oracle, gathered rows against the rows the stream holds at the sampled
    slots (no transform: the gather is the stored row)."""
    cfg = synth.Stress(d, prefill + iters * batch)
    u, prio = cfg.draws(iters, batch)
    buf = cd.ReplayBuffer(cap, cfg.obs_shape, torch.float32, action_bytes=4)
    orc = oracle.Replay(cap, cfg.obs_shape, np.float32, act_bytes=4, keep_obs=False)

    def ingest(a, b):
        buf.ingest(cfg.rows(a, b - a, "cuda"), action=dev(cfg.action[a:b]), reward=dev(cfg.reward[a:b]),
                   done=dev(cfg.done[a:b]), prio=dev(cfg.prio[a:b]))
        orc.ingest(b - a, obs=None, action=cfg.action[a:b], reward=cfg.reward[a:b], done=cfg.done[a:b],
                   prio=cfg.prio[a:b])

    for a in range(0, prefill, chunk):
        ingest(a, min(prefill, a + chunk))
    pos = prefill
    xf = cd.transform(cd.XF_NONE)
    out = torch.empty((batch, 1) + cfg.obs_shape, dtype=torch.float32, device="cuda")
    act = torch.empty(batch, dtype=torch.int32, device="cuda")
    rew = torch.empty(batch, dtype=torch.float32, device="cuda")
    for it in range(iters):
        ingest(pos, pos + batch)
        pos += batch
        idx, w = buf.sample_gather(dev(u[it]), xf, obs=out, action=act, reward=rew)
        o_idx, o_w = orc.sample(u[it])
        assert np.array_equal(host(idx), o_idx), it
        assert_weights_close(host(w), o_w)
        sel = check_rows
        want = cfg.rows_at(orc.position[o_idx[sel]]).numpy()
        got = host(out[torch.as_tensor(sel, device="cuda")]).reshape(want.shape)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), it
        _, o_act, o_rew, _ = orc.gather(o_idx)
        assert np.array_equal(host(act).view(np.uint8).reshape(batch, 4), o_act), it
        assert np.array_equal(host(rew), o_rew), it
        buf.update(idx, dev(prio[it]))
        orc.update(o_idx, prio[it])
    assert buf.sync_check() == cd.OK, cd.last_error()
    assert np.array_equal(read_col(buf, cd.COL_LEAVES, cap * 4, np.uint32), orc.leaf)
    assert tree_consistent(buf, cap) == orc.total_priority()
    buf.close()


@pytest.mark.parametrize("d", [128, 1000, 5000, 12000])
def test_stress_transitions_reduced(d):
    print(f"stress: d={d}, cap 3000, prefill 3500 (wraps), batch 512", flush=True)
    run_stress(cap=3000, d=d, prefill=3500, iters=3, batch=512, chunk=1000, check_rows=np.arange(512))


@pytest.mark.slow
def test_stress_transitions_full_size():
    print("stress: d=20000, cap 10^6 (160 GB), batch 512, 2 iterations", flush=True)
    torch.cuda.empty_cache()  # the 160 GB arena is the library's own allocation
    run_stress(cap=1_000_000, d=20000, prefill=1_000_000, iters=2, batch=512, chunk=4096,
               check_rows=np.random.default_rng(0).choice(512, 24, replace=False))
