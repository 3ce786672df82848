"""GPU parity of the on-policy path: rollout ingest, GAE (time-major and packed)
and the minibatch shuffle-gather, against the oracle through the C ABI.
GAE within 1e-5 max(|o|, 1); gathered bytes and u8 transforms bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_gae_close, dev, host

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def _gae_gpu(r, v, d, b, gamma, lam):
    T, E = r.shape
    adv = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
    ret = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
    cd.conduit_gae(dev(r), dev(v) if v is not None else None, dev(d), dev(b) if b is not None else None,
                   gamma, lam, adv, ret)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    return host(adv), host(ret)


@pytest.mark.parametrize("T,E,p_done,with_v,with_b", [
    (1, 1, 0.0, True, True), (2, 3, 0.5, True, False), (37, 19, 0.05, True, True), (64, 16, 0.0, False, False),
    (65, 17, 1.0, True, True), (200, 70, 0.01, True, True), (1000, 5, 0.002, True, True),
    (2500, 9, 0.003, True, True), (1024, 8, 0.0, True, False), (3073, 3, 0.01, False, True),
    # E a multiple of 4 or not: one tile per 32 environments for T <= 64, split
    # along T beyond (see SPLIT_CASES below)
    (100, 12, 0.02, True, True), (2500, 12, 0.003, True, True), (4096, 8, 0.001, True, True),
    (2049, 4, 0.01, True, False), (300, 128, 0.01, True, True), (33, 64, 0.1, False, False),
    # the most environments the ABI takes (2^19), on both kernels
    (3, 1 << 19, 0.2, True, True), (2, (1 << 19) - 1, 0.2, True, True)])
def test_gae_time_major_shapes(T, E, p_done, with_v, with_b):
    print(f"gae T={T} E={E}", flush=True)
    rng = np.random.default_rng(T * 131 + E)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32) if with_v else None
    d = (rng.random((T, E)) < p_done).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32) if with_b else None
    for gamma, lam in [(0.99, 0.95), (1.0, 1.0), (0.0, 0.5)]:
        ga, gr = _gae_gpu(r, v, d, b, gamma, lam)
        oa, orr = oracle.gae(r, v, d, b, gamma, lam)
        assert_gae_close(ga, oa)
        assert_gae_close(gr, orr)


@pytest.mark.parametrize("T,E,p_done,p_trunc", [
    (1, 1, 0.0, 1.0), (37, 19, 0.05, 0.05), (200, 70, 0.01, 0.02), (1024, 8, 0.0, 0.01), (2500, 9, 0.003, 0.002),
    (65, 17, 0.5, 0.5), (3073, 3, 0.0, 0.0), (300, 128, 0.01, 0.01), (2049, 12, 0.01, 0.01)])
def test_gae_truncated_shapes(T, E, p_done, p_trunc):
    print(f"gae truncated T={T} E={E}", flush=True)
    rng = np.random.default_rng(T * 137 + E)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < p_done).astype(np.uint8)
    tr = (rng.random((T, E)) < p_trunc).astype(np.uint8)
    fv = rng.standard_normal((T, E)).astype(np.float32)
    b = rng.standard_normal(E).astype(np.float32)
    for gamma, lam in [(0.99, 0.95), (1.0, 1.0), (0.0, 0.5)]:
        adv = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
        ret = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
        cd.conduit_gae_truncated(dev(r), dev(v), dev(d), dev(tr), dev(fv), dev(b), gamma, lam, adv, ret)
        assert cd.conduit_sync_check() == cd.OK, cd.last_error()
        oa, orr = oracle.gae(r, v, d, b, gamma, lam, truncated=tr, final_value=fv)
        assert_gae_close(host(adv), oa)
        assert_gae_close(host(ret), orr)


# Which kernels a shape takes (E a multiple of 4 with aligned rows): a rollout of
# at most 64 steps is one tile per 32 environments ("short"); a longer one is
# split along T into tiles of 32 environments by 32 L steps, L the
# longest of 8, 4, 2 that still gives 256 tiles (4 when 8 would fit but 4 gives
# 1,024 to 4,096 tiles); up to 4,096 tiles run in one launch with a look-back
# over the later segments ("look"); more run in three launches below 4,096
# environments ("split") and otherwise as one workgroup walking all T steps of
# 8 environments ("one_v4"; "one" for E not a multiple of 4 or unaligned rows).
# The tiles take any E and rows off a 16-byte boundary (SPLIT_CASES_ANY_E).
# conduit_gae_plan reports the choice; tests/test_abi_cpu.py checks it on the
# host.
SPLIT_CASES = [
    # (T, E, p_done, expected path, expected chunk length)
    (1, 4, 0.5, "short", 2),          # one step
    (16, 4100, 0.02, "short", 2),     # 129 groups, the last one 4 envs
    (64, 65536, 0.01, "short", 2),    # 2,048 tiles, every chunk full
    (33, 131072, 0.01, "short", 2),   # 4,096 tiles and beyond: no table is used
    (65, 4, 0.05, "look", 2),         # two segments, the last one a single step
    (129, 36, 0.02, "look", 2),       # a partial environment group (36 = 32 + 4)
    (2048, 256, 0.001, "look", 2),    # 32 segments of 64 steps: one look-back window
    (40000, 4, 0.0005, "look", 4),    # 313 segments: look-backs chained over windows
    (16000, 100, 0.001, "look", 4),   # 125 segments x 4 groups (last one 4 envs)
    (65573, 4, 0.0005, "look", 8),    # 257 segments of 256 steps, ragged end
    (2100, 1000, 0.003, "look", 8),   # 9 segments, 32 groups (last one 8 envs)
    (1100, 4052, 0.003, "look", 4),   # 9 segments, 127 groups (last one 20 envs)
    (3000, 4092, 0.01, "look", 4),    # 3,072 tiles
    (2100, 4096, 0.002, "look", 4),   # 4,096 environments and up split too
    (4097, 4100, 0.002, "look", 8),   # 2,193 tiles (chunks of 4 would need 4,257)
    (1048576, 4, 0.0001, "look", 8),  # 4,096 tiles: the most one launch takes
    (1100000, 4, 0.0001, "split", 8),  # 4,297 tiles: three launches, 135 carry passes
    (600000, 36, 0.0002, "split", 8),  # 4,688 tiles, a partial group
]


def _time_major_path(T, E):
    """(path, chunk length) the library picks for an aligned [T, E] rollout."""
    return cd.gae_plan(T, E, aligned=True)


@pytest.mark.parametrize("T,E,p_done,path,L", SPLIT_CASES)
def test_gae_split_along_t(T, E, p_done, path, L):
    print(f"gae split T={T} E={E} {path} L={L}", flush=True)
    assert _time_major_path(T, E) == (path, L)
    rng = np.random.default_rng(T * 7 + E)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < p_done).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32)
    for gamma, lam in [(0.99, 0.95), (1.0, 1.0)]:
        ga, gr = _gae_gpu(r, v, d, b, gamma, lam)
        oa, orr = oracle.gae(r, v, d, b, gamma, lam)
        assert_gae_close(ga, oa)
        assert_gae_close(gr, orr)
    # no values, no bootstrap, every step done: delta = r and A = r exactly
    ones = np.ones((T, E), np.uint8)
    ga, gr = _gae_gpu(r, None, ones, None, 0.99, 0.95)
    assert np.array_equal(ga, r) and np.array_equal(gr, r)


# E not a multiple of 4: the same tiles, each lane loading and storing its
# four environments one by one (columns past E skipped on store, clamped on load)
SPLIT_CASES_ANY_E = [
    # (T, E, p_done, expected path, expected chunk length)
    (1, 3, 0.5, "short", 2),           # fewer environments than a quad
    (16, 4101, 0.02, "short", 2),      # 129 groups, the last one 5 envs (a partial quad)
    (64, 131071, 0.01, "short", 2),    # 4,096 tiles
    (65, 5, 0.05, "look", 2),          # two segments, one partial quad
    (129, 37, 0.02, "look", 2),        # a partial group and a partial quad
    (2048, 255, 0.001, "look", 2),     # the PPO rollout with one environment fewer
    (40000, 6, 0.0005, "look", 4),     # chained look-back windows
    (2100, 1001, 0.003, "look", 8),
    (3000, 4091, 0.01, "look", 4),     # 3,072 tiles
    (1100000, 3, 0.0001, "split", 8),  # three launches, one partial quad
    (600000, 37, 0.0002, "split", 8),  # three launches, a partial group and quad
]


@pytest.mark.parametrize("T,E,p_done,path,L", SPLIT_CASES_ANY_E)
def test_gae_split_along_t_any_e(T, E, p_done, path, L):
    print(f"gae split any E T={T} E={E} {path} L={L}", flush=True)
    assert _time_major_path(T, E) == (path, L)
    rng = np.random.default_rng(T * 13 + E)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < p_done).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32)
    for gamma, lam in [(0.99, 0.95), (1.0, 1.0)]:
        ga, gr = _gae_gpu(r, v, d, b, gamma, lam)
        oa, orr = oracle.gae(r, v, d, b, gamma, lam)
        assert_gae_close(ga, oa)
        assert_gae_close(gr, orr)
    ga, gr = _gae_gpu(r, None, np.ones((T, E), np.uint8), None, 0.99, 0.95)
    assert np.array_equal(ga, r) and np.array_equal(gr, r)


@pytest.mark.parametrize("T,E", [(2100, 1000), (1100, 4052), (700, 36), (1100000, 4), (40, 4100), (64, 36),
                                 (2100, 1001), (700, 37), (1100000, 3), (40, 4101)])
def test_gae_truncated_split_along_t(T, E):
    print(f"gae truncated split T={T} E={E}", flush=True)
    assert _time_major_path(T, E)[0] in ("short", "look", "split")
    rng = np.random.default_rng(T * 11 + E)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < 0.004).astype(np.uint8)
    tr = (rng.random((T, E)) < 0.004).astype(np.uint8)
    fv = rng.standard_normal((T, E)).astype(np.float32)
    b = rng.standard_normal(E).astype(np.float32)
    adv = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
    ret = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
    cd.conduit_gae_truncated(dev(r), dev(v), dev(d), dev(tr), dev(fv), dev(b), 0.99, 0.95, adv, ret)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    oa, orr = oracle.gae(r, v, d, b, 0.99, 0.95, truncated=tr, final_value=fv)
    assert_gae_close(host(adv), oa)
    assert_gae_close(host(ret), orr)


@pytest.mark.parametrize("T,E,path", [(65, 131072, "one_v4"), (65, 131071, "one"), (2100, 16383, "one"),
                                      pytest.param(2049, 65536, "one_v4", marks=pytest.mark.slow)])
def test_gae_single_pass_kernel_several_passes(T, E, path):
    """Wide rollouts beyond the look-back table keep one workgroup per 8
    environments walking 2,048-step passes (two passes, the last of one step,
    in the slow case and at T = 2,100); four environments per lane where E is
    a multiple of 4, one otherwise."""
    print(f"gae single-pass T={T} E={E}", flush=True)
    assert _time_major_path(T, E)[0] == path
    rng = np.random.default_rng(T + E)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < 0.002).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32)
    ga, gr = _gae_gpu(r, v, d, b, 0.99, 0.95)
    oa, orr = oracle.gae(r, v, d, b, 0.99, 0.95)
    assert_gae_close(ga, oa)
    assert_gae_close(gr, orr)


@pytest.mark.parametrize("T,E,path", [(333, 16, "look"), (40, 16, "short"), (1100000, 4, "split"),
                                      (65, 131072, "one")])
def test_gae_misaligned_rows_take_per_element_access(T, E, path):
    """E a multiple of 4 but rows 4 bytes off a 16-byte boundary: the launcher
    must not use 16-byte vectors (tiles load and store each environment on its
    own, the wide one-pass kernel takes one environment per lane); results
    still match the oracle."""
    print(f"gae misaligned rows T={T} E={E}", flush=True)
    assert cd.gae_plan(T, E, aligned=False)[0] == path
    rng = np.random.default_rng(7)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < 0.02).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32)

    def off(a):  # the same values at an address 4 bytes past a 16-byte boundary
        flat = torch.empty(a.size + 1, dtype=torch.float32, device="cuda")
        view = flat[1:].view(a.shape)
        view.copy_(torch.from_numpy(a))
        assert view.data_ptr() % 16 == 4
        return view

    adv = torch.full((T * E + 1,), np.nan, dtype=torch.float32, device="cuda")[1:].view(T, E)
    ret = torch.full((T * E + 1,), np.nan, dtype=torch.float32, device="cuda")[1:].view(T, E)
    cd.conduit_gae(off(r), off(v), dev(d), dev(b), 0.99, 0.95, adv, ret)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()
    oa, orr = oracle.gae(r, v, d, b, 0.99, 0.95)
    assert_gae_close(host(adv), oa)
    assert_gae_close(host(ret), orr)


def test_gae_ppo_config_full_size():
    print("gae: PPO rollout 2048 x 256", flush=True)
    cfg = synth.PPO()
    ga, gr = _gae_gpu(cfg.reward, cfg.value, cfg.done, cfg.bootstrap, cfg.gamma, cfg.lam)
    oa, orr = oracle.gae(cfg.reward, cfg.value, cfg.done, cfg.bootstrap, cfg.gamma, cfg.lam)
    assert_gae_close(ga, oa)
    assert_gae_close(gr, orr)


@pytest.mark.parametrize("B,Lmax,with_v", [(1, 4, False), (5, 8, True), (33, 260, True), (256, 4096, False),
                                           (64, 4096, True), (7, 4097, True), (5, 9000, True), (3, 12288, False),
                                           # rows off a 16-byte boundary and short vector tails
                                           (9, 6, True), (6, 1001, True), (4, 4099, True),
                                           # the same without values (the closed form's scalar stores)
                                           (9, 6, False), (6, 1001, False), (4, 4099, False)])
def test_gae_packed(B, Lmax, with_v):
    print(f"gae packed B={B} Lmax={Lmax}", flush=True)
    rng = np.random.default_rng(B * 7 + Lmax)
    length = rng.integers(0, Lmax + 1, B).astype(np.int32)
    length[0] = Lmax
    if B > 2:
        length[1] = 1
        length[2] = 0
    R = rng.standard_normal(B).astype(np.float32)
    v = rng.standard_normal((B, Lmax)).astype(np.float32) if with_v else None
    # gamma lambda = 0 (the degenerate cases): only the last live element keeps a non-zero advantage without values
    for gamma, lam in [(1.0, 0.95), (0.99, 0.9), (0.0, 0.95), (0.99, 0.0)]:
        adv = torch.full((B, Lmax), np.nan, dtype=torch.float32, device="cuda")
        ret = torch.full((B, Lmax), np.nan, dtype=torch.float32, device="cuda")
        cd.conduit_gae_packed(dev(R), dev(length), dev(v) if v is not None else None, Lmax, gamma, lam, adv, ret)
        assert cd.conduit_sync_check() == cd.OK, cd.last_error()
        oa, orr = oracle.gae_packed(R, length, v, Lmax, gamma, lam)
        assert_gae_close(host(adv), oa)
        assert_gae_close(host(ret), orr)


def _ppo_rollout_buffer(cfg, steps_per_call):
    T, E = cfg.T, cfg.E
    buf = cd.ReplayBuffer(T * E, cfg.obs_shape, torch.uint8, prioritized=False, action_bytes=0)
    for t0 in range(0, T, steps_per_call):
        t1 = min(T, t0 + steps_per_call)
        buf.ingest(cfg.obs_steps(t0, t1, "cuda"), reward=dev(cfg.reward[t0:t1].reshape(-1)),
                   done=dev(cfg.done[t0:t1].reshape(-1)))
    return buf


def _obs_column_tensor(buf, n_rows, row_bytes):
    out = torch.empty(n_rows * row_bytes, dtype=torch.uint8, device="cuda")
    buf.read(cd.COL_OBS, out)
    return out


@pytest.mark.parametrize("T,E,M", [(64, 32, 4), (33, 7, 3)])
def test_ppo_minibatches_reduced(T, E, M):
    print(f"ppo minibatches T={T} E={E} M={M}", flush=True)
    cfg = synth.PPO(T=T, E=E)
    row = 3 * 84 * 84
    buf = _ppo_rollout_buffer(cfg, steps_per_call=5)
    src = _obs_column_tensor(buf, T * E, row)
    ga, gr = _gae_gpu(cfg.reward, cfg.value, cfg.done, cfg.bootstrap, cfg.gamma, cfg.lam)
    A, R = dev(ga.reshape(-1)), dev(gr.reshape(-1))
    oa, orr = oracle.gae(cfg.reward, cfg.value, cfg.done, cfg.bootstrap, cfg.gamma, cfg.lam)
    obs_host = cfg.obs_steps(0, T).numpy()
    perm = cfg.perm
    mb = (T * E) // M
    seen = []
    for m in range(M):
        rows = perm[m * mb:(m + 1) * mb]
        out = torch.empty((mb, 3, 84, 84), dtype=torch.float32, device="cuda")
        a_out = torch.empty(mb, dtype=torch.float32, device="cuda")
        r_out = torch.empty(mb, dtype=torch.float32, device="cuda")
        cd.conduit_minibatch_gather(src, row, T * E, dev(rows), cd.transform(cd.XF_U8_F32), out, cols=[A, R],
                                    cols_out=[a_out, r_out])
        assert cd.conduit_sync_check() == cd.OK, cd.last_error()
        want = oracle.rows(obs_host, rows, oracle.XF_U8_F32)
        assert np.array_equal(host(out).view(np.uint32), want.view(np.uint32))
        assert_gae_close(host(a_out), oa.reshape(-1)[rows])
        assert_gae_close(host(r_out), orr.reshape(-1)[rows])
        seen.append(rows)
    # on-policy freshness: the M minibatches cover the rollout exactly once
    assert np.array_equal(np.sort(np.concatenate(seen)), np.arange(M * mb))
    buf.close()


def test_minibatch_transforms_and_bad_perm():
    print("minibatch gather: NONE / BF16 transforms, out-of-range perm", flush=True)
    rng = np.random.default_rng(3)
    n_src, shape = 50, (3, 8, 12)
    row = int(np.prod(shape))
    src_h = rng.integers(0, 256, size=(n_src,) + shape, dtype=np.uint8)
    src = dev(src_h)
    perm = rng.integers(0, n_src, size=40)
    out = torch.empty((40,) + shape, dtype=torch.uint8, device="cuda")
    cd.conduit_minibatch_gather(src, row, n_src, dev(perm), cd.transform(cd.XF_NONE), out)
    assert np.array_equal(host(out), oracle.rows(src_h, perm))
    mean, std = (0.485, 0.456, 0.406), (0.229, 0.224, 0.225)
    outb = torch.empty((40,) + shape, dtype=torch.bfloat16, device="cuda")
    cd.conduit_minibatch_gather(src, row, n_src, dev(perm), cd.transform(cd.XF_U8_BF16_NORM, mean, std), outb)
    assert np.array_equal(host(outb.view(torch.int16)).view(np.uint16),
                          oracle.rows(src_h, perm, oracle.XF_U8_BF16_NORM, mean, std))
    assert cd.conduit_sync_check() == cd.OK
    bad = perm.copy()
    bad[5] = n_src
    bad[6] = -1
    out.fill_(9)
    cd.conduit_minibatch_gather(src, row, n_src, dev(bad), cd.transform(cd.XF_NONE), out)
    assert cd.conduit_sync_check() == cd.ESTATE
    cd.conduit_clear_error()
    o = host(out)
    assert np.all(o[5] == 0) and np.all(o[6] == 0)
    assert np.array_equal(o[7:], src_h[bad[7:]])
