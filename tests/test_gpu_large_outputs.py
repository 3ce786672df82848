"""Whole-output parity of the gather for learner batches larger than 128 MB.

Batches up to 128 MB go through the persistent double-buffered gather; larger
ones through the one-item-per-workgroup gather (the Large bf16 batch of 308 MB
and every PPO minibatch of 1.39 GB take it).  Each test here builds an output
over 128 MB, asserts that it is, and compares every byte against the oracle
(delivery materialises the selected transitions unchanged or exactly
transformed: Sec. 2.2, App. C Invariant 1)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_gae_close, dev, host
from test_gpu_payloads import run_large
from test_gpu_replay import run_dqn

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402

MB128 = 128 << 20


@pytest.mark.parametrize("fused", [False, True])
def test_large_bf16_batch_over_128mb(fused):
    # 901 rows of 3x224x224 -> bf16 = 271 MB; a ring of 1,100 slots after 1,500
    # ingests (wrapped); every row, action and reward compared
    print(f"large bf16: batch 901 (271 MB out), cap 1100, fused={fused}", flush=True)
    assert 901 * 3 * 224 * 224 * 2 > MB128
    run_large(cap=1100, prefill=1500, iters=2, batch=901, chunk=256, check_rows=np.arange(901), fused=fused)


def test_dqn_stacks_batch_over_128mb():
    # 1,201 stacks of 4 x 84x84 -> fp32 = 136 MB, short episodes (many zero-filled
    # frames), wrapped ring; every row compared
    print("dqn stacks: batch 1201 x 4 frames (136 MB out), short episodes", flush=True)
    assert 1201 * 4 * 84 * 84 * 4 > MB128
    run_dqn(cap=4096, prefill=5000, iters=2, batch=1201, chunk=1024, short_episodes=True)


def _src(rng, n_src, row):
    return rng.integers(0, 256, size=(n_src, row), dtype=np.uint8)


def test_minibatch_u8_f32_over_128mb_with_columns_and_bad_entries():
    # PPO-shaped rows (3x84x84 u8) -> fp32: 2,049 rows = 174 MB, plus two
    # float columns; then the same with two entries outside [0, n_src)
    print("minibatch u8->f32: 2049 rows of 21168 B (174 MB out), 2 columns, bad entries", flush=True)
    rng = np.random.default_rng(21)
    n_src, row, n = 3000, 3 * 84 * 84, 2049
    src_h = _src(rng, n_src, row)
    cols_h = [rng.standard_normal(n_src).astype(np.float32) for _ in range(2)]
    perm = rng.permutation(n_src)[:n].astype(np.int64)
    src, cols = dev(src_h), [dev(c) for c in cols_h]
    out = torch.full((n, row), -1.0, dtype=torch.float32, device="cuda")
    assert out.numel() * 4 > MB128
    c_out = [torch.full((n,), np.nan, dtype=torch.float32, device="cuda") for _ in range(2)]
    xf = cd.transform(cd.XF_U8_F32)
    cd.conduit_minibatch_gather(src, row, n_src, dev(perm), xf, out, cols=cols, cols_out=c_out)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    want = oracle.rows(src_h, perm, oracle.XF_U8_F32)
    assert np.array_equal(host(out).view(np.uint32), want.reshape(n, row).view(np.uint32))
    for g, c in zip(c_out, cols_h):
        assert np.array_equal(host(g), c[perm])
    bad = perm.copy()
    bad[0], bad[1000], bad[n - 1] = n_src, -1, n_src + 7
    out.fill_(-1.0)
    cd.conduit_minibatch_gather(src, row, n_src, dev(bad), xf, out, cols=cols, cols_out=c_out)
    assert cd.conduit_sync_check() == cd.ESTATE
    cd.conduit_clear_error()
    o = host(out).view(np.uint32)
    ok = np.ones(n, bool)
    ok[[0, 1000, n - 1]] = False
    assert np.all(o[~ok] == 0)
    assert np.array_equal(o[ok], want.reshape(n, row).view(np.uint32)[ok])
    for g, c in zip(c_out, cols_h):
        gh = host(g)
        assert np.all(gh[~ok] == 0.0) and np.array_equal(gh[ok], c[bad[ok]])


@pytest.mark.parametrize("row", [3 * 224 * 224, 21172])
def test_minibatch_copy_over_128mb(row):
    # no transform: 150,528-byte rows take the 16-byte copy, 21,172-byte rows
    # (a multiple of 4, not of 16) the 4-byte one
    n = (MB128 // row) + 37
    print(f"minibatch copy: {n} rows of {row} B ({n * row >> 20} MB out)", flush=True)
    rng = np.random.default_rng(row)
    n_src = n + 200
    src_h = _src(rng, n_src, row)
    perm = rng.integers(0, n_src, size=n).astype(np.int64)
    out = torch.zeros((n, row), dtype=torch.uint8, device="cuda")
    assert out.numel() > MB128
    cd.conduit_minibatch_gather(dev(src_h), row, n_src, dev(perm), cd.transform(cd.XF_NONE), out)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    assert np.array_equal(host(out), oracle.rows(src_h, perm).reshape(n, row))


def test_minibatch_bf16_over_128mb():
    # per-plane normalisation of 3x224x224 rows -> bf16: 900 rows = 271 MB
    print("minibatch u8->bf16 norm: 900 rows of 3x224x224 (271 MB out)", flush=True)
    rng = np.random.default_rng(9)
    row, n, n_src = 3 * 224 * 224, 900, 1000
    src_h = _src(rng, n_src, row)
    perm = rng.integers(0, n_src, size=n).astype(np.int64)
    mean, std = synth.Large.mean, synth.Large.std
    out = torch.zeros((n, row), dtype=torch.bfloat16, device="cuda")
    assert out.numel() * 2 > MB128
    cd.conduit_minibatch_gather(dev(src_h), row, n_src, dev(perm), cd.transform(cd.XF_U8_BF16_NORM, mean, std), out)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    want = oracle.rows(src_h, perm, oracle.XF_U8_BF16_NORM, mean, std).reshape(n, row)
    assert np.array_equal(host(out.view(torch.int16)).view(np.uint16), want)


@pytest.mark.slow
def test_ppo_full_size_minibatch_every_row():
    # the PPO rollout (2048 x 256 x 3x84x84 u8, 11.1 GB) and two of its 32
    # minibatches of 16,384 rows (1.39 GB each), compared row by row on the host
    # in chunks of 1,024 rows regenerated from the seeded generator
    print("ppo: full rollout, minibatches 0 and 31, every row", flush=True)
    cfg = synth.PPO()
    T, E = cfg.T, cfg.E
    row = 3 * 84 * 84
    buf = cd.ReplayBuffer(T * E, cfg.obs_shape, torch.uint8, prioritized=False, action_bytes=0)
    for t0 in range(0, T, 64):
        buf.ingest(cfg.obs_steps(t0, t0 + 64, "cuda"), reward=dev(cfg.reward[t0:t0 + 64].reshape(-1)),
                   done=dev(cfg.done[t0:t0 + 64].reshape(-1)))
    src = torch.empty(T * E * row, dtype=torch.uint8, device="cuda")
    buf.read(cd.COL_OBS, src)
    torch.cuda.synchronize()
    buf.close()
    oa, orr = oracle.gae(cfg.reward, cfg.value, cfg.done, cfg.bootstrap, cfg.gamma, cfg.lam)
    adv = torch.empty((T, E), dtype=torch.float32, device="cuda")
    ret = torch.empty((T, E), dtype=torch.float32, device="cuda")
    cd.conduit_gae(dev(cfg.reward), dev(cfg.value), dev(cfg.done), dev(cfg.bootstrap), cfg.gamma, cfg.lam, adv, ret)
    A, R = adv.view(-1), ret.view(-1)
    mb = 16384
    out = torch.empty((mb, row), dtype=torch.float32, device="cuda")
    a_out = torch.empty(mb, dtype=torch.float32, device="cuda")
    r_out = torch.empty(mb, dtype=torch.float32, device="cuda")
    for m in [0, 31]:
        rows = cfg.perm[m * mb:(m + 1) * mb]
        cd.conduit_minibatch_gather(src, row, T * E, dev(rows), cd.transform(cd.XF_U8_F32), out, cols=[A, R],
                                    cols_out=[a_out, r_out])
        assert cd.conduit_sync_check() == cd.OK, cd.last_error()
        for c0 in range(0, mb, 1024):
            sel = rows[c0:c0 + 1024]
            want = oracle.rows(cfg.obs_rows(sel).numpy().reshape(len(sel), row), np.arange(len(sel)),
                               oracle.XF_U8_F32)
            got = host(out[c0:c0 + 1024]).view(np.uint32)
            assert np.array_equal(got, want.reshape(len(sel), row).view(np.uint32)), (m, c0)
        assert_gae_close(host(a_out), oa.reshape(-1)[rows])
        assert_gae_close(host(r_out), orr.reshape(-1)[rows])
    print("ppo: every row of minibatches 0 and 31 equal", flush=True)
