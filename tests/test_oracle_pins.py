"""Pins of the reference oracle against things other than itself.

Each test checks the oracle (``oracle/``) against a closed form, an invariant, a
brute-force computation written by a different method (``oracle/brute.py``), or
a worked example under ``tests/golden/``.  CPU only.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth
from oracle import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------
# Leaf quantiser L(p) = floor(2^F p^alpha)
# ----------------------------------------------------------------------------
ALPHAS = [(3, 5), (1, 2), (7, 8), (1, 1), (0, 1), (2, 3), (1, 8), (5, 7)]


def test_leaf_exhaustive_low_range():
    # every priority up to 2^18 at the default alpha = 3/5
    for p in range(0, 1 << 18):
        assert oracle.leaf(p, 3, 5) == brute.leaf(p, 3, 5), p


@pytest.mark.parametrize("a,b", ALPHAS)
def test_leaf_random_full_range(a, b):
    rng = np.random.default_rng(7 + 13 * a + b)
    ps = list(rng.integers(0, 1 << 32, size=3000, dtype=np.uint64))
    ps += [0, 1, 2, 3, 4095, 4096, (1 << 31) - 1, 1 << 31, (1 << 32) - 2, (1 << 32) - 1]
    # perfect powers sit exactly on the boundary q^b == 2^(bF) p^a
    ps += [k ** b for k in range(1, 60) if k ** b < (1 << 32)]
    for p in ps:
        assert oracle.leaf(int(p), a, b) == brute.leaf(int(p), a, b), (a, b, p)


def test_leaf_many_matches_scalar():
    p = np.random.default_rng(2).integers(0, 1 << 32, size=500, dtype=np.uint64).astype(np.uint32)
    assert list(oracle.leaves(p, 2, 3)) == [oracle.leaf(int(x), 2, 3) for x in p]


def test_leaf_closed_forms():
    assert oracle.frac_bits(3, 5) == 12
    for p in [1, 2, 17, 1 << 20, (1 << 32) - 1]:
        assert oracle.leaf(p, 1, 1) == p  # alpha = 1: leaf = priority
        assert oracle.leaf(p, 0, 1) == 1 << 31  # alpha = 0: uniform
    for a, b in ALPHAS:
        assert oracle.leaf(0, a, b) == 0  # zero priority: never sampled
        assert oracle.leaf((1 << 32) - 1, a, b) < (1 << 32)
    # against the real-valued formula away from integer boundaries
    for p in [5, 123, 99999, 3141592653]:
        exact = 4096.0 * p ** 0.6
        assert abs(oracle.leaf(p) - exact) < 1.0


def test_leaf_monotone():
    prev = -1
    for p in range(0, 200000, 7):
        q = oracle.leaf(p)
        assert q >= prev
        prev = q


# ----------------------------------------------------------------------------
# Sum tree, sampling, importance weights
# ----------------------------------------------------------------------------
def _tree_consistent(r):
    t = r.tree.astype(object)
    tl = len(t) // 2
    for node in range(1, tl):
        assert t[node] == t[2 * node] + t[2 * node + 1]
    assert int(t[1]) == int(r.leaf.astype(np.uint64).sum())


def test_sum_tree_invariant_random_ops():
    rng = np.random.default_rng(3)
    for cap in [1, 2, 3, 5, 64, 100]:
        r = oracle.Replay(cap, (2,), np.uint8, act_bytes=4)
        for _ in range(30):
            n = int(rng.integers(0, cap + 1))
            prio = rng.integers(0, 1 << 20, size=n).astype(np.uint32) if rng.random() < 0.5 else None
            r.ingest(n, obs=np.zeros((n, 2), np.uint8), prio=prio)
            if r.size:
                m = int(rng.integers(1, 2 * cap + 2))
                r.update(rng.integers(0, r.size, size=m), rng.integers(0, 1 << 32, size=m, dtype=np.uint64))
            _tree_consistent(r)


def _filled_replay(leaves_prio, alpha=(1, 1), beta=0.4):
    n = len(leaves_prio)
    r = oracle.Replay(n, (1,), np.uint8, alpha=alpha, beta=beta)
    r.ingest(n, obs=np.zeros((n, 1), np.uint8), prio=np.asarray(leaves_prio, np.uint32))
    return r


def test_derived_episodes_hand_example():
    # a stream of 7 transitions in two ingests into a 5-slot ring, no episode
    # ids or steps given; done at positions 1, 5 and 6.  Position p continues
    # p-1's episode one step on unless p-1 was done:
    #   position: 0  1  2  3  4  5  6
    #   done:     0  1  0  0  0  1  1
    #   episode:  0  0  1  1  1  1  2
    #   step:     0  1  0  1  2  3  0
    # the ring then holds positions 5, 6, 2, 3, 4 in slots 0..4
    r = oracle.Replay(5, (1,), np.uint8, single_stream=True)
    r.ingest(3, obs=np.zeros((3, 1), np.uint8), done=np.array([0, 1, 0], np.uint8))
    r.ingest(4, obs=np.zeros((4, 1), np.uint8), done=np.array([0, 0, 1, 1], np.uint8))
    assert list(r.position) == [5, 6, 2, 3, 4]
    assert list(r.episode) == [1, 2, 1, 1, 1]
    assert list(r.step) == [3, 0, 0, 1, 2]


def test_derived_episodes_match_the_actor_bookkeeping():
    # any split of one stream into ingests, wrapping rings included, stores the
    # episode ids and steps an actor would have attached to the whole stream
    # (the generator's own bookkeeping, written independently)
    rng = np.random.default_rng(41)
    for trial in range(40):
        total = int(rng.integers(1, 400))
        cap = int(rng.integers(1, 120))
        done = (rng.random(total) < rng.choice([0.0, 0.05, 0.3, 1.0])).astype(np.uint8)
        ep, st = synth.episodes_from_done(done)
        r = oracle.Replay(cap, (1,), np.uint8, single_stream=True)
        a = 0
        while a < total:
            b = min(total, a + int(rng.integers(1, cap + 1)))
            r.ingest(b - a, obs=np.zeros((b - a, 1), np.uint8), done=done[a:b])
            a = b
        held = r.position >= 0
        assert np.array_equal(r.episode[held], ep[r.position[held]]), trial
        assert np.array_equal(r.step[held], st[r.position[held]]), trial


def test_derived_episodes_continue_given_ones():
    # ids given by one ingest, derived by the next: the stream continues from
    # the last given transition (episode 7, step 41, not done)
    r = oracle.Replay(8, (1,), np.uint8, single_stream=True)
    r.ingest(2, obs=np.zeros((2, 1), np.uint8), done=np.array([0, 0], np.uint8),
             episode=np.array([7, 7], np.uint32), step=np.array([40, 41], np.int32))
    r.ingest(3, obs=np.zeros((3, 1), np.uint8), done=np.array([1, 0, 0], np.uint8))
    assert list(r.episode[:5]) == [7, 7, 7, 8, 8]
    assert list(r.step[:5]) == [40, 41, 42, 0, 1]
    # without the single-stream option, omitted ids are stored as 0
    r = oracle.Replay(8, (1,), np.uint8)
    r.ingest(3, obs=np.zeros((3, 1), np.uint8), done=np.array([1, 0, 1], np.uint8))
    assert list(r.episode[:3]) == [0, 0, 0] and list(r.step[:3]) == [0, 0, 0]


def test_sample_matches_linear_scan():
    rng = np.random.default_rng(11)
    for trial in range(200):
        n = int(rng.integers(1, 65))
        prio = rng.integers(0, 50, size=n)
        if trial % 5 == 0:
            prio[rng.integers(0, n)] = 0
        if prio.sum() == 0:
            prio[0] = 1
        r = _filled_replay(prio)
        B = int(rng.integers(1, 300))
        u = rng.integers(0, 1 << 64, size=B, dtype=np.uint64)
        idx, _ = r.sample(u)
        Q = int(prio.sum())
        assert r.total_priority() == Q
        targets = brute.stratified_targets(Q, B, u)
        want = [brute.linear_sample(prio, t) for t in targets]
        assert list(idx) == want
        assert all(prio[i] > 0 for i in idx)


def test_sample_extreme_uniforms_and_large_total():
    # Q close to 2^52 and uniforms at both ends of the 64-bit range
    prio = np.array([(1 << 32) - 1] * 4 + [1, 0, 7], np.uint64)
    r = oracle.Replay(len(prio), (1,), np.uint8, alpha=(1, 1))
    r.ingest(len(prio), obs=np.zeros((len(prio), 1), np.uint8), prio=prio.astype(np.uint32))
    Q = int(prio.sum())
    for B in [1, 3, 1000, 1 << 20]:
        u = np.array([0, (1 << 64) - 1, 1 << 63] * (B // 3 + 1), np.uint64)[:B]
        idx, _ = r.sample(u)
        t = brute.stratified_targets(Q, B, u)
        assert max(t) < Q
        check = range(0, B, max(1, B // 997))
        assert [int(idx[k]) for k in check] == [brute.linear_sample(prio, t[k]) for k in check]


def test_sample_equal_leaves_closed_form():
    q = 5
    n = 40
    r = _filled_replay([q] * n)
    rng = np.random.default_rng(5)
    u = rng.integers(0, 1 << 64, size=333, dtype=np.uint64)
    idx, w = r.sample(u)
    t = brute.stratified_targets(q * n, 333, u)
    assert list(idx) == [tk // q for tk in t]
    assert np.all(w == 1.0)


def test_stratified_counts_within_two_of_expectation():
    rng = np.random.default_rng(17)
    prio = rng.integers(1, 1000, size=64)
    r = _filled_replay(prio)
    B = 1 << 16
    idx, _ = r.sample(rng.integers(0, 1 << 64, size=B, dtype=np.uint64))
    counts = np.bincount(idx, minlength=64)
    expect = B * prio / prio.sum()
    assert np.all(np.abs(counts - expect) < 2.0)


def test_sampling_frequencies_chi_square():
    from scipy.stats import chi2
    rng = np.random.default_rng(23)
    prio = np.round(1e4 * np.abs(rng.standard_normal(64))).astype(np.uint32) + 1
    r = _filled_replay(prio, alpha=(3, 5))
    leaves = np.array([oracle.leaf(int(p)) for p in prio], np.float64)
    counts = np.zeros(64)
    batches, B = 1 << 16, 64  # 2^22 draws
    for _ in range(batches):
        idx, _ = r.sample(rng.integers(0, 1 << 64, size=B, dtype=np.uint64))
        counts += np.bincount(idx, minlength=64)
    expect = batches * B * leaves / leaves.sum()
    stat = float(((counts - expect) ** 2 / expect).sum())
    assert stat < chi2.isf(1e-6, df=63), stat
    # leaves follow p^alpha, not p: the same counts are far from p-proportional
    wrong = batches * B * prio.astype(np.float64) / float(prio.sum())
    assert float(((counts - wrong) ** 2 / wrong).sum()) > chi2.isf(1e-6, df=63)


def test_is_weights_closed_form_and_cases():
    rng = np.random.default_rng(29)
    prio = rng.integers(1, 10 ** 6, size=50)
    for beta in [0.0, 0.4, 1.0]:
        r = _filled_replay(prio, alpha=(3, 5), beta=beta)
        idx, w = r.sample(rng.integers(0, 1 << 64, size=64, dtype=np.uint64))
        q = r.leaf.astype(np.float64)
        closed = (q[idx].min() / q[idx]) ** beta  # (N P_i)^-beta / max, N and Q cancel
        np.testing.assert_allclose(w, closed.astype(np.float32), rtol=2e-7)
        np.testing.assert_allclose(w, brute.is_weights(r.leaf, r.size, idx, beta), rtol=1e-6)
        assert w.max() == 1.0
        if beta == 0.0:
            assert np.all(w == 1.0)


def test_buffer_wide_is_weights():
    # normalised by the largest weight any stored transition could get: the
    # smallest non-zero leaf of the buffer, not of the batch
    rng = np.random.default_rng(37)
    prio = rng.integers(1, 10 ** 6, size=300)
    prio[17] = 0  # a zero priority is never sampled and never the minimum
    for beta in [0.0, 0.4, 1.0]:
        r = _filled_replay(prio, alpha=(3, 5), beta=beta)
        u = rng.integers(0, 1 << 64, size=16, dtype=np.uint64)
        idx, w_batch = r.sample(u)
        idx2, w_buf = r.sample(u, buffer_norm=True)
        assert np.array_equal(idx, idx2)
        q = r.leaf.astype(np.float64)
        q_buf, q_bat = q[q > 0].min(), q[idx].min()
        # the two modes differ by one factor per batch
        np.testing.assert_allclose(w_buf, (w_batch * (q_buf / q_bat) ** beta).astype(np.float32), rtol=1e-6)
        np.testing.assert_allclose(w_buf, brute.is_weights_buffer(r.leaf, r.size, idx, beta), rtol=1e-6)
        assert w_buf.max() <= 1.0
    # a batch that holds the buffer's smallest leaf: the modes agree exactly
    # (priorities of one magnitude, so that leaf is drawn often)
    r = _filled_replay(rng.integers(1000, 2000, size=300), alpha=(3, 5), beta=0.4)
    qmin_slot = int(np.flatnonzero(r.leaf == r.leaf[r.leaf > 0].min())[0])
    for _ in range(200):
        u = rng.integers(0, 1 << 64, size=64, dtype=np.uint64)
        idx, w_batch = r.sample(u)
        if qmin_slot in idx:
            assert np.array_equal(r.sample(u, buffer_norm=True)[1], w_batch)
            break
    else:
        pytest.fail("no batch drew the smallest leaf")


def _stream_replay(rng, cap, total, p_done=0.15, K=1):
    """A replay fed a known stream of single-float observations (the stream
    position itself), with episode ids and steps derived from done."""
    done = (rng.random(total) < p_done).astype(np.uint8)
    ep, st = synth.episodes_from_done(done)
    rew = rng.standard_normal(total).astype(np.float32)
    obs = np.arange(total, dtype=np.float32)[:, None]
    r = oracle.Replay(cap, (1,), np.float32, act_bytes=0, frame_stack=K)
    for a in range(0, total, 7):
        b = min(total, a + 7)
        r.ingest(b - a, obs=obs[a:b], reward=rew[a:b], done=done[a:b], episode=ep[a:b], step=st[a:b])
    return r, rew, done, ep


def test_nstep_matches_the_stream_definition():
    # brute force on the stream itself: positions, not ring slots
    rng = np.random.default_rng(79)
    for cap, total, n, gamma in [(40, 100, 3, 0.9), (64, 64, 5, 0.99), (33, 1000, 1, 0.5), (50, 77, 8, 1.0)]:
        r, rew, done, ep = _stream_replay(rng, cap, total)
        slots = np.arange(cap)
        nxt, ret, disc, valid = r.nstep(slots, n, gamma)
        for b, i in enumerate(slots):
            p = int(r.position[i])
            want_R, g, m, ended = 0.0, 1.0, None, False
            for k in range(n):
                q = p + k
                if q >= total or ep[q] != ep[p]:
                    m = None
                    break
                want_R += g * float(rew[q])
                g *= gamma
                m = k + 1
                if done[q]:
                    ended = True
                    break
            if m is None or (not ended and (p + n >= total or ep[p + n] != ep[p])):
                assert valid[b] == 0 and ret[b] == 0 and disc[b] == 0 and nxt[b] == -1, (cap, b)
                continue
            assert valid[b] == 1
            assert ret[b] == pytest.approx(want_R, rel=1e-6, abs=1e-6)
            if ended:
                assert disc[b] == 0 and nxt[b] == -1
            else:
                assert disc[b] == pytest.approx(gamma ** n, rel=1e-6) and nxt[b] == (p + n) % cap
                assert r.position[nxt[b]] == p + n


def test_nstep_special_cases():
    rng = np.random.default_rng(83)
    r, rew, done, ep = _stream_replay(rng, 50, 120, p_done=0.0)
    slots = np.arange(50)
    # one step, no dones: the 1-step DQN target
    nxt, ret, disc, valid = r.nstep(slots, 1, 0.97)
    newest = (r.head - 1) % 50
    for b in slots:
        if b == newest:
            assert valid[b] == 0  # the newest transition has no successor yet
        else:
            assert valid[b] == 1 and ret[b] == rew[r.position[b]] and disc[b] == np.float32(0.97)
    # gamma = 1 sums the rewards
    nxt, ret, disc, valid = r.nstep(slots, 4, 1.0)
    for b in slots:
        if valid[b]:
            p = r.position[b]
            assert ret[b] == pytest.approx(float(rew[p:p + 4].astype(np.float64).sum()), rel=1e-6)
            assert disc[b] == 1.0
    assert int(valid.sum()) == 50 - 4  # the newest four cannot look four steps ahead


# ----------------------------------------------------------------------------
# Ingest, update semantics
# ----------------------------------------------------------------------------
def test_ingest_round_trip_and_ring_slots():
    rng = np.random.default_rng(31)
    cap = 37
    r = oracle.Replay(cap, (3, 5), np.uint8, act_bytes=8)
    stream = []
    for n in [0, 5, 37, 20, 1, 36]:
        obs = rng.integers(0, 256, size=(n, 3, 5), dtype=np.uint8)
        act = rng.integers(0, 256, size=(n, 8), dtype=np.uint8)
        rew = rng.standard_normal(n).astype(np.float32)
        head0 = r.head
        r.ingest(n, obs=obs, action=act, reward=rew)
        stream += list(zip(obs, act, rew))
        slots = [(head0 + j) % cap for j in range(n)]
        if n:
            out, oa, orew, _ = r.gather(np.array(slots))
            assert np.array_equal(out[:, 0], obs)  # contents unchanged by storage (App. C Inv. 1)
            assert np.array_equal(oa, act)
            assert np.array_equal(orew, rew)
    assert r.total == len(stream)
    assert r.size == cap and r.head == len(stream) % cap
    # every slot holds the newest transition that maps to it
    out, _, _, _ = r.gather(np.arange(cap))
    for s in range(cap):
        pos = max(p for p in range(len(stream)) if p % cap == s)
        assert np.array_equal(out[s, 0], stream[pos][0])


def test_ingest_uses_running_max_priority():
    r = oracle.Replay(10, (1,), np.uint8)
    r.ingest(2, obs=np.zeros((2, 1), np.uint8))
    assert list(r.leaf[:2]) == [oracle.leaf(1)] * 2  # initial maximum priority 1
    r.ingest(1, obs=np.zeros((1, 1), np.uint8), prio=np.array([900], np.uint32))
    r.update(np.array([0]), np.array([5000], np.uint32))
    r.update(np.array([1]), np.array([7], np.uint32))
    r.ingest(1, obs=np.zeros((1, 1), np.uint8))
    assert r.max_prio == 5000
    assert r.leaf[3] == oracle.leaf(5000)


def test_update_last_writer_wins_and_bad_indices():
    rng = np.random.default_rng(37)
    r = oracle.Replay(64, (1,), np.uint8)
    r.ingest(40, obs=np.zeros((40, 1), np.uint8))
    for _ in range(20):
        n = int(rng.integers(1, 200))
        idx = rng.integers(-3, 45, size=n)
        prio = rng.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)
        expect = r.leaf.copy()
        good = 0
        for i, p in zip(idx, prio):
            if 0 <= i < 40:
                expect[i] = brute.leaf(int(p))
                good += 1
        bad = r.update(idx, prio)
        assert bad == n - good
        assert np.array_equal(r.leaf, expect)
        _tree_consistent(r)


# ----------------------------------------------------------------------------
# Frame stacks and pixel transforms
# ----------------------------------------------------------------------------
def _episode_stream(rng, n, max_len):
    eps, steps = [], []
    e = 0
    while len(eps) < n:
        L = int(rng.integers(1, max_len + 1))
        eps += [e] * L
        steps += list(range(L))
        e += 1
    return np.array(eps[:n], np.uint32), np.array(steps[:n], np.int32)


@pytest.mark.parametrize("cap,n,K", [(50, 30, 4), (50, 173, 4), (16, 100, 2), (7, 7, 4), (33, 90, 1)])
def test_frame_stack_matches_stream(cap, n, K):
    rng = np.random.default_rng(cap * 1000 + n)
    eps, steps = _episode_stream(rng, n, 6)
    frames = rng.integers(1, 256, size=(n, 2, 3), dtype=np.uint8)
    r = oracle.Replay(cap, (2, 3), np.uint8, frame_stack=K)
    pos = 0
    while pos < n:
        m = min(int(rng.integers(1, 20)), n - pos, cap)
        r.ingest(m, obs=frames[pos:pos + m], episode=eps[pos:pos + m], step=steps[pos:pos + m])
        pos += m
    slots = np.arange(r.size)
    out, _, _, _ = r.gather(slots)
    for s in slots:
        p = int(r.position[s])
        want = brute.stack_from_stream(eps, frames, cap, n, p, K)
        for k in range(K):
            expect = np.zeros((2, 3), np.uint8) if want[k] is None else want[k]
            assert np.array_equal(out[s, k], expect), (s, k)


def test_frame_stack_special_cases():
    r = oracle.Replay(20, (1,), np.uint8, frame_stack=4)
    frames = np.arange(1, 11, dtype=np.uint8).reshape(10, 1)
    eps = np.array([0, 0, 0, 0, 0, 1, 1, 1, 1, 1], np.uint32)
    steps = np.array([0, 1, 2, 3, 4, 0, 1, 2, 3, 4], np.int32)
    r.ingest(10, obs=frames, episode=eps, step=steps)
    out, _, _, _ = r.gather(np.array([5, 9, 6]))
    assert list(out[0, :, 0]) == [0, 0, 0, 6]  # step 0: three zero frames then the frame
    assert list(out[1, :, 0]) == [7, 8, 9, 10]  # step >= 3, no boundary: four consecutive
    assert list(out[2, :, 0]) == [0, 0, 6, 7]


def test_u8_to_f32_exhaustive():
    for x in range(256):
        assert oracle.u8_to_f32(x) == brute.nearest_f32(Fraction(x, 255)), x


def test_u8_to_bf16_exhaustive():
    means = [0.485, 0.456, 0.406]
    stds = [0.229, 0.224, 0.225]
    for m, s in zip(means, stds):
        mf = Fraction(float(np.float32(m)))
        sf = Fraction(float(np.float32(s)))
        for x in range(256):
            v = Fraction(brute.nearest_f32(Fraction(x, 255)))
            y = Fraction(brute.nearest_f32(v - mf))
            z = Fraction(brute.nearest_f32(y / sf))
            assert oracle.u8_to_bf16_bits(x, m, s) == brute.nearest_bf16_bits(z), (x, m)


def test_gather_transforms_apply_table():
    rng = np.random.default_rng(41)
    rows = rng.integers(0, 256, size=(9, 3, 4, 4), dtype=np.uint8)
    r = oracle.Replay(9, (3, 4, 4), np.uint8)
    r.ingest(9, obs=rows)
    f32 = np.array([oracle.u8_to_f32(x) for x in range(256)], np.float32)
    out, _, _, _ = r.gather(np.arange(9), oracle.XF_U8_F32)
    assert np.array_equal(out[:, 0], f32[rows])
    mean, std = [0.485, 0.456, 0.406], [0.229, 0.224, 0.225]
    out, _, _, _ = r.gather(np.arange(9), oracle.XF_U8_BF16_NORM, mean, std)
    for c in range(3):
        tab = np.array([oracle.u8_to_bf16_bits(x, mean[c], std[c]) for x in range(256)], np.uint16)
        assert np.array_equal(out[:, 0, c], tab[rows[:, c]])


# ----------------------------------------------------------------------------
# GAE
# ----------------------------------------------------------------------------
def _rollout(rng, T, E, p_done):
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < p_done).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32)
    return r, v, d, b


def test_gae_golden_hand_example():
    with open(os.path.join(GOLDEN, "gae_hand_example.json")) as f:
        g = json.load(f)
    adv, ret = oracle.gae(np.array(g["reward"])[:, None], np.array(g["value"])[:, None],
                          np.array(g["done"])[:, None], np.array([g["bootstrap"]]), g["gamma"], g["lambda"])
    assert list(adv[:, 0]) == g["advantage"]
    assert list(ret[:, 0]) == g["return"]


def test_gae_lambda_one_is_discounted_return_minus_value():
    rng = np.random.default_rng(43)
    T, E, gamma = 40, 5, 0.9
    r, v, d, b = _rollout(rng, T, E, 0.1)
    adv, ret = oracle.gae(r, v, d, b, gamma, 1.0)
    for e in range(E):
        for t in range(T):
            g, disc, end = 0.0, 1.0, False
            for k in range(t, T):
                g += disc * float(r[k, e])
                disc *= gamma
                if d[k, e]:
                    end = True
                    break
            if not end:
                g += disc * float(b[e])
            assert adv[t, e] == pytest.approx(g - float(v[t, e]), rel=1e-5, abs=1e-5)
            assert ret[t, e] == pytest.approx(g, rel=1e-5, abs=1e-5)


def test_gae_gamma_zero_and_all_done_are_td_residual():
    rng = np.random.default_rng(47)
    r, v, d, b = _rollout(rng, 17, 9, 0.3)
    adv, _ = oracle.gae(r, v, d, b, 0.0, 0.95)
    assert np.array_equal(adv, (r.astype(np.float64) - v).astype(np.float32))
    adv, _ = oracle.gae(r, v, np.ones_like(d), b, 0.99, 0.95)
    assert np.array_equal(adv, (r.astype(np.float64) - v).astype(np.float32))


def test_gae_no_value_no_done_is_lambda_gamma_discounting():
    rng = np.random.default_rng(53)
    T, gamma, lam = 30, 0.97, 0.9
    r = rng.standard_normal((T, 1)).astype(np.float32)
    adv, _ = oracle.gae(r, None, np.zeros((T, 1), np.uint8), None, gamma, lam)
    for t in range(T):
        want = sum((gamma * lam) ** (k - t) * float(r[k, 0]) for k in range(t, T))
        assert adv[t, 0] == pytest.approx(want, rel=1e-6, abs=1e-6)


def test_gae_truncation_lambda_one_is_bootstrapped_return_minus_value():
    # lambda = 1: A_t = G_t - V_t, G_t summing discounted rewards up to the
    # first end; a truncation (not a termination) adds gamma^(k-t+1) times the
    # final value of its true next observation
    rng = np.random.default_rng(67)
    T, E, gamma = 40, 5, 0.9
    r, v, d, b = _rollout(rng, T, E, 0.05)
    tr = (rng.random((T, E)) < 0.08).astype(np.uint8)
    fv = rng.standard_normal((T, E)).astype(np.float32)
    adv, ret = oracle.gae(r, v, d, b, gamma, 1.0, truncated=tr, final_value=fv)
    for e in range(E):
        for t in range(T):
            g, disc, end = 0.0, 1.0, False
            for k in range(t, T):
                g += disc * float(r[k, e])
                disc *= gamma
                if d[k, e] or tr[k, e]:
                    end = True
                    if tr[k, e] and not d[k, e]:
                        g += disc * float(fv[k, e])
                    break
            if not end:
                g += disc * float(b[e])
            assert adv[t, e] == pytest.approx(g - float(v[t, e]), rel=1e-5, abs=1e-5)
            assert ret[t, e] == pytest.approx(g, rel=1e-5, abs=1e-5)


def test_gae_truncation_splits_the_rollout():
    # a rollout truncated at step k with final value f is two rollouts: steps
    # 0..k bootstrapped from f, and the rest with the rollout's own bootstrap
    rng = np.random.default_rng(71)
    T, k, gamma, lam = 30, 11, 0.99, 0.95
    r, v, d, b = _rollout(rng, T, 1, 0.0)
    tr = np.zeros((T, 1), np.uint8)
    tr[k] = 1
    fv = np.zeros((T, 1), np.float32)
    fv[k] = 2.5
    adv, ret = oracle.gae(r, v, d, b, gamma, lam, truncated=tr, final_value=fv)
    a1, r1 = oracle.gae(r[:k + 1], v[:k + 1], d[:k + 1], np.array([2.5], np.float32), gamma, lam)
    a2, r2 = oracle.gae(r[k + 1:], v[k + 1:], d[k + 1:], b, gamma, lam)
    assert np.array_equal(adv, np.concatenate([a1, a2])) and np.array_equal(ret, np.concatenate([r1, r2]))


def test_gae_termination_wins_over_truncation_and_none_is_plain_gae():
    rng = np.random.default_rng(73)
    r, v, d, b = _rollout(rng, 25, 7, 0.2)
    fv = rng.standard_normal((25, 7)).astype(np.float32)
    plain = oracle.gae(r, v, d, b, 0.99, 0.95)
    both = oracle.gae(r, v, d, b, 0.99, 0.95, truncated=d.copy(), final_value=fv)  # every end both
    none = oracle.gae(r, v, d, b, 0.99, 0.95, truncated=np.zeros_like(d), final_value=fv)
    for x in (both, none):
        assert np.array_equal(x[0], plain[0]) and np.array_equal(x[1], plain[1])


@pytest.mark.parametrize("gamma", [1.0, 0.99])
def test_gae_packed_closed_form_and_padding(gamma):
    # without values the only non-zero TD residual is the last element's
    # reward: A_t = R (gamma lambda)^(L-1-t), zero in the padding
    rng = np.random.default_rng(59)
    B, Lmax, lam = 6, 50, 0.95
    length = np.array([1, 50, 7, 0, 33, 2], np.int32)
    R = rng.standard_normal(B).astype(np.float32)
    adv, ret = oracle.gae_packed(R, length, None, Lmax, gamma, lam)
    for b in range(B):
        for t in range(Lmax):
            want = (gamma * lam) ** (length[b] - 1 - t) * float(R[b]) if t < length[b] else 0.0
            assert adv[b, t] == pytest.approx(want, rel=1e-6, abs=1e-7)
            assert ret[b, t] == adv[b, t]


def test_gae_packed_with_values_matches_time_major_form():
    # one sequence = one single-env rollout that ends (done) on its last element
    rng = np.random.default_rng(61)
    Lmax, L, gamma, lam = 20, 13, 0.99, 0.95
    R = np.array([1.5], np.float32)
    v = rng.standard_normal((1, Lmax)).astype(np.float32)
    adv, ret = oracle.gae_packed(R, np.array([L], np.int32), v, Lmax, gamma, lam)
    r = np.zeros((L, 1), np.float32)
    r[-1] = R[0]
    d = np.zeros((L, 1), np.uint8)
    d[-1] = 1
    a2, r2 = oracle.gae(r, v[0, :L, None], d, np.array([123.0], np.float32), gamma, lam)
    assert np.array_equal(adv[0, :L], a2[:, 0]) and np.array_equal(ret[0, :L], r2[:, 0])
    assert np.all(adv[0, L:] == 0)


# ----------------------------------------------------------------------------
# Minibatch shuffle-gather, token packing
# ----------------------------------------------------------------------------
def test_minibatches_partition_rollout():
    rng = np.random.default_rng(67)
    T, E, M = 16, 8, 4
    obs = rng.integers(0, 256, size=(T * E, 3, 2, 2), dtype=np.uint8)
    perm = rng.permutation(T * E)
    seen = []
    f32 = np.array([oracle.u8_to_f32(x) for x in range(256)], np.float32)
    for m in range(M):
        rows = perm[m * (T * E // M):(m + 1) * (T * E // M)]
        out = oracle.rows(obs, rows)
        assert np.array_equal(out, obs[rows])
        outf = oracle.rows(obs, rows, oracle.XF_U8_F32)
        assert np.array_equal(outf, f32[obs[rows]])
        seen += list(rows)
    assert sorted(seen) == list(range(T * E))  # each transition exactly once per epoch


def test_pack_tokens_properties():
    rng = np.random.default_rng(71)
    Lmax, n = 32, 12
    lens = rng.integers(0, Lmax + 1, size=n)
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    tok = rng.integers(0, 128000, size=offsets[-1]).astype(np.int32)
    lp = -rng.exponential(size=offsets[-1]).astype(np.float32)
    r = oracle.Replay(10, (Lmax,), np.int32, ragged=True, aux_dtype=np.float32)
    rew = np.arange(n, dtype=np.float32)
    for a, b in [(0, 7), (7, n)]:  # two calls; the second wraps the 10-slot ring
        off = offsets[a:b + 1] - offsets[a]
        r.ingest(b - a, obs=tok[offsets[a]:offsets[b]], offsets=off, aux=lp[offsets[a]:offsets[b]],
                 reward=rew[a:b])
    idx = np.array([0, 9, 3, 3, 1])
    seq, mask, aux, length, rew = r.pack(idx, pad_id=0)
    for b, i in enumerate(idx):
        j = int(r.position[i])
        L = int(lens[j])
        assert length[b] == L and mask[b].sum() == L
        assert np.array_equal(seq[b, :L], tok[offsets[j]:offsets[j] + L])
        assert np.array_equal(aux[b, :L], lp[offsets[j]:offsets[j] + L])
        assert np.all(seq[b, L:] == 0) and np.all(aux[b, L:] == 0) and np.all(mask[b, L:] == 0)
        assert rew[b] == j
