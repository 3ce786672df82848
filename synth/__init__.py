"""Seeded synthetic inputs shaped like the five experience-path workloads.

This module only draws data.  It holds none of the method's arithmetic (no
priorities-to-leaves, sampling, stacking, transforms or advantages); both the HIP
path and the oracle consume exactly the arrays it returns.

Scalar columns are drawn on the host with NumPy's PCG64.  Bulk payloads (pixels,
tokens, per-token log-probabilities) are procedural: an integer hash of
(seed, row, element) evaluated with torch integer ops, so any row can be
regenerated on the CPU or on the GPU with bit-identical results.  Floating-point
payloads go through tables built once on the host, never through device math.

Workloads (stand-ins for the paper's environments, which are not available):
  0 tiny    -- small-observation replay (MountainCar / MA-CartPole class)
  1 dqn     -- Atari-shaped 84x84 frames, 1M-frame replay with frame stacking
  2 ppo     -- on-policy rollout 2048 steps x 256 envs of 3x84x84 frames
  3 large   -- 3x224x224 visual payloads, 200k-transition replay (~30 GB)
  4 tokens  -- variable-length token sequences (LLM post-training shape)
  5 stress  -- fp32 transitions of dimension d (obs and next_obs, d values each),
               the paper's synthetic stress test, 1M-transition replay
Seeds: data 1000 + c, draws (uniforms, permutations, update priorities) 1500 + c.
"""
import numpy as np
import torch

MASK32 = 0xFFFFFFFF
_MUL = 0x45D9F3B  # below 2^31, so products of 32-bit values stay inside int64


def data_seed(c):
    return 1000 + c


def draw_seed(c):
    return 1500 + c


# ----------------------------------------------------------------------------
# integer hashing (identical on any torch device)
# ----------------------------------------------------------------------------
def _mix32(x):
    x = x ^ (x >> 16)
    x = (x * _MUL) & MASK32
    x = x ^ (x >> 16)
    x = (x * _MUL) & MASK32
    x = x ^ (x >> 16)
    return x


def hash32(*keys):
    """32-bit hash of broadcastable int64 tensors / ints (each in [0, 2^32))."""
    h = None
    for k in keys:
        k = k if isinstance(k, torch.Tensor) else torch.tensor(int(k) & MASK32, dtype=torch.int64)
        h = _mix32(k & MASK32) if h is None else _mix32(h ^ (k & MASK32))
    return h


def quantise_priority(x):
    """Real positive draws -> uint32 priorities  min(round(1e4 x), 2^32 - 2) + 1."""
    p = np.minimum(np.round(1e4 * np.asarray(x, np.float64)), float(2 ** 32 - 2)) + 1
    return p.astype(np.uint32)


def uniforms(rng, *shape):
    """Host-supplied 64-bit uniforms for the stratified sampler."""
    return rng.integers(0, 2 ** 64, size=shape, dtype=np.uint64)


def episodes_from_done(done, first_episode=0):
    """Actor-side bookkeeping: episode id and step index of each transition of a
    single stream, where done=1 ends an episode."""
    done = np.asarray(done, np.uint8)
    n = len(done)
    ends_before = np.concatenate([[0], np.cumsum(done[:-1], dtype=np.int64)]) if n else np.zeros(0, np.int64)
    episode = (first_episode + ends_before).astype(np.uint32)
    step = np.zeros(n, np.int32)
    s = 0
    for j in range(n):
        step[j] = s
        s = 0 if done[j] else s + 1
    return episode, step


def _episode_layout(rng, n, lo, hi):
    """Episode id / step / done for a stream of n transitions with episode
    lengths drawn uniformly from [lo, hi]."""
    lengths = []
    total = 0
    while total < n:
        L = int(rng.integers(lo, hi + 1))
        lengths.append(L)
        total += L
    lengths = np.array(lengths, np.int64)
    episode = np.repeat(np.arange(len(lengths), dtype=np.uint32), lengths)[:n]
    starts = np.concatenate([[0], np.cumsum(lengths)[:-1]])
    step = (np.arange(total, dtype=np.int64) - np.repeat(starts, lengths))[:n].astype(np.int32)
    done = np.zeros(n, np.uint8)
    ends = np.cumsum(lengths) - 1
    done[ends[ends < n]] = 1
    return episode, step, done, len(lengths)


# ----------------------------------------------------------------------------
# 0: tiny replay
# ----------------------------------------------------------------------------
class Tiny:
    """capacity 16384, obs 8 x fp32 ~ N(0,1), action int32 in [0,4), reward N(0,1),
    done Bernoulli(0.01); 100 iterations of ingest 64 / sample 256 / update 256 with
    update priorities round(1e4 |N(0,1)|) + 1."""

    capacity = 16384
    obs_shape = (8,)
    ingest_n, batch, iters = 64, 256, 100

    def __init__(self, n=None, seed=None):
        n = self.ingest_n * self.iters if n is None else n
        rng = np.random.default_rng(data_seed(0) if seed is None else seed)
        self.n = n
        self.obs = rng.standard_normal((n, 8)).astype(np.float32)
        self.action = rng.integers(0, 4, n).astype(np.int32)
        self.reward = rng.standard_normal(n).astype(np.float32)
        self.done = (rng.random(n) < 0.01).astype(np.uint8)
        self.episode, self.step = episodes_from_done(self.done)

    def draws(self, iters=None, batch=None, seed=None):
        iters = self.iters if iters is None else iters
        batch = self.batch if batch is None else batch
        rng = np.random.default_rng(draw_seed(0) if seed is None else seed)
        u = uniforms(rng, iters, batch)
        prio = (np.round(1e4 * np.abs(rng.standard_normal((iters, batch)))) + 1).astype(np.uint32)
        return u, prio


# ----------------------------------------------------------------------------
# 1: DQN Atari-shaped replay
# ----------------------------------------------------------------------------
class DQN:
    """1M single 84x84 uint8 frames; episodes of length U{200..2000}; pixel
    (base_e[y,x] + s_e * step) mod 256 with base_e a per-episode hash image and
    s_e in {1,2,3} (adjacent frames differ); action int32 in [0,18); reward in
    {-1,0,1}; priorities lognormal(0,1) quantised; batch 512, frame stack 4."""

    capacity = 1_000_000
    frame_shape = (84, 84)
    batch = 512
    stack = 4

    def __init__(self, n, seed=None, capacity=None):
        self.seed = data_seed(1) if seed is None else seed
        if capacity is not None:
            self.capacity = capacity
        rng = np.random.default_rng(self.seed)
        self.n = n
        self.episode, self.step, self.done, n_eps = _episode_layout(rng, n, 200, 2000)
        self.drift = rng.integers(1, 4, n_eps).astype(np.int64)
        self.action = rng.integers(0, 18, n).astype(np.int32)
        self.reward = rng.integers(-1, 2, n).astype(np.float32)
        self.prio = quantise_priority(rng.lognormal(0.0, 1.0, n))
        self._drift_t = {}

    def frames(self, start, count, device="cpu"):
        """uint8 [count, 84, 84] frames of stream positions [start, start+count)."""
        dev = torch.device(device)
        if dev not in self._drift_t:
            self._drift_t[dev] = torch.from_numpy(self.drift).to(dev)
        out = torch.empty((count, 84 * 84), dtype=torch.uint8, device=dev)
        pix = torch.arange(84 * 84, dtype=torch.int64, device=dev)[None, :]
        for a in range(0, count, 2048):
            b = min(count, a + 2048)
            ep = torch.from_numpy(self.episode[start + a:start + b].astype(np.int64)).to(dev)[:, None]
            st = torch.from_numpy(self.step[start + a:start + b].astype(np.int64)).to(dev)[:, None]
            base = hash32(self.seed, ep, pix) & 255
            out[a:b] = ((base + self._drift_t[dev][ep] * st) & 255).to(torch.uint8)
        return out.view(count, 84, 84)

    def frames_at(self, positions, device="cpu"):
        """uint8 [len(positions), 84, 84] frames of arbitrary stream positions."""
        dev = torch.device(device)
        if dev not in self._drift_t:
            self._drift_t[dev] = torch.from_numpy(self.drift).to(dev)
        pos = np.asarray(positions, np.int64)
        ep = torch.from_numpy(self.episode[pos].astype(np.int64)).to(dev)[:, None]
        st = torch.from_numpy(self.step[pos].astype(np.int64)).to(dev)[:, None]
        pix = torch.arange(84 * 84, dtype=torch.int64, device=dev)[None, :]
        base = hash32(self.seed, ep, pix) & 255
        return ((base + self._drift_t[dev][ep] * st) & 255).to(torch.uint8).view(len(pos), 84, 84)

    def draws(self, iters, batch=None, seed=None):
        batch = self.batch if batch is None else batch
        rng = np.random.default_rng(draw_seed(1) if seed is None else seed)
        u = uniforms(rng, iters, batch)
        prio = quantise_priority(rng.lognormal(0.0, 1.0, (iters, batch)))
        return u, prio


# ----------------------------------------------------------------------------
# 2: PPO rollout
# ----------------------------------------------------------------------------
class PPO:
    """Rollout T=2048 x E=256 of 3x84x84 uint8 frames (per-env hash image plus a
    per-env drift with t), rewards and values N(0,1), bootstrap values N(0,1),
    dones Bernoulli(0.001); gamma 0.99, lambda 0.95; a seeded permutation of the
    T*E transitions split into 32 minibatches of 16384."""

    obs_shape = (3, 84, 84)
    gamma, lam = 0.99, 0.95
    minibatches = 32

    def __init__(self, T=2048, E=256, seed=None):
        self.T, self.E = T, E
        self.seed = data_seed(2) if seed is None else seed
        rng = np.random.default_rng(self.seed)
        self.reward = rng.standard_normal((T, E)).astype(np.float32)
        self.value = rng.standard_normal((T, E)).astype(np.float32)
        self.bootstrap = rng.standard_normal(E).astype(np.float32)
        self.done = (rng.random((T, E)) < 0.001).astype(np.uint8)
        self.drift = rng.integers(1, 4, E).astype(np.int64)
        self.perm = np.random.default_rng(draw_seed(2)).permutation(T * E).astype(np.int64)
        self._base = {}

    def _env_base(self, dev):
        if dev not in self._base:
            e = torch.arange(self.E, dtype=torch.int64, device=dev)[:, None]
            pix = torch.arange(3 * 84 * 84, dtype=torch.int64, device=dev)[None, :]
            self._base[dev] = (hash32(self.seed, e, pix) & 255)
        return self._base[dev]

    def obs_rows(self, flat, device="cpu"):
        """uint8 [len(flat), 3, 84, 84] observations of flat indices f = t*E + e."""
        dev = torch.device(device)
        flat = torch.as_tensor(np.asarray(flat, np.int64), device=dev)
        t, e = flat // self.E, flat % self.E
        drift = torch.from_numpy(self.drift).to(dev)
        rows = (self._env_base(dev)[e] + (drift[e] * t)[:, None]) & 255
        return rows.to(torch.uint8).view(-1, *self.obs_shape)

    def obs_steps(self, t0, t1, device="cpu"):
        """uint8 [(t1-t0)*E, 3, 84, 84] observations of steps [t0, t1) in flat order."""
        dev = torch.device(device)
        t = torch.arange(t0, t1, dtype=torch.int64, device=dev)[:, None, None]
        drift = torch.from_numpy(self.drift).to(dev)[None, :, None]
        rows = (self._env_base(dev)[None] + drift * t) & 255
        return rows.to(torch.uint8).view(-1, *self.obs_shape)


# ----------------------------------------------------------------------------
# 3: large visual payloads
# ----------------------------------------------------------------------------
class Large:
    """200k transitions of 3x224x224 uint8 (a fixed hash texture XOR a per-row
    32-bit hash word), action fp32[6] ~ U(-1,1), reward N(0,1), priorities
    lognormal(0,2) quantised; batch 1024 -> bf16 normalised with ImageNet
    per-channel mean/std."""

    capacity = 200_000
    obs_shape = (3, 224, 224)
    batch = 1024
    mean = (0.485, 0.456, 0.406)
    std = (0.229, 0.224, 0.225)

    def __init__(self, n, seed=None):
        self.seed = data_seed(3) if seed is None else seed
        rng = np.random.default_rng(self.seed)
        self.n = n
        self.action = rng.uniform(-1.0, 1.0, (n, 6)).astype(np.float32)
        self.reward = rng.standard_normal(n).astype(np.float32)
        self.done = np.zeros(n, np.uint8)
        self.prio = quantise_priority(rng.lognormal(0.0, 2.0, n))
        self._tex = {}

    def _texture(self, dev):
        if dev not in self._tex:
            k = torch.arange(3 * 224 * 224 // 4, dtype=torch.int64, device=dev)
            self._tex[dev] = hash32(self.seed, 7, k)
        return self._tex[dev]

    def rows(self, start, count, device="cpu"):
        """uint8 [count, 3, 224, 224] observations of stream positions [start, start+count)."""
        dev = torch.device(device)
        pos = torch.arange(start, start + count, dtype=torch.int64, device=dev)[:, None]
        words = self._texture(dev)[None, :] ^ hash32(self.seed, 11, pos)
        words = torch.where(words >= 2 ** 31, words - 2 ** 32, words).to(torch.int32)
        return words.view(torch.uint8).view(count, *self.obs_shape)

    def rows_at(self, positions, device="cpu"):
        dev = torch.device(device)
        pos = torch.as_tensor(np.asarray(positions, np.int64), device=dev)[:, None]
        words = self._texture(dev)[None, :] ^ hash32(self.seed, 11, pos)
        words = torch.where(words >= 2 ** 31, words - 2 ** 32, words).to(torch.int32)
        return words.view(torch.uint8).view(len(positions), *self.obs_shape)

    def draws(self, iters, batch=None, seed=None):
        batch = self.batch if batch is None else batch
        rng = np.random.default_rng(draw_seed(3) if seed is None else seed)
        return uniforms(rng, iters, batch), quantise_priority(rng.lognormal(0.0, 2.0, (iters, batch)))


# ----------------------------------------------------------------------------
# 4: long-context token sequences
# ----------------------------------------------------------------------------
_EXP_TABLE = None


def _exp_quantiles():
    """65536 quantiles of Exp(1), computed once on the host in float32."""
    global _EXP_TABLE
    if _EXP_TABLE is None:
        k = np.arange(65536, dtype=np.float64)
        _EXP_TABLE = (-np.log((k + 0.5) / 65536.0)).astype(np.float32)
    return _EXP_TABLE


class Tokens:
    """65536 sequences of int32 tokens in [0,128000) with length U{512..4096},
    per-token log-probabilities -Exp(1), scalar reward N(0,1), priorities
    lognormal(0,1) quantised; batch 256 packed to [256, 4096]; GAE gamma 1,
    lambda 0.95 with the reward on the last token."""

    capacity = 65536
    max_len = 4096
    batch = 256
    vocab = 128000
    gamma, lam = 1.0, 0.95

    def __init__(self, n, seed=None, max_len=None, min_len=512):
        self.seed = data_seed(4) if seed is None else seed
        if max_len is not None:
            self.max_len = max_len
        rng = np.random.default_rng(self.seed)
        self.n = n
        self.length = rng.integers(min(min_len, self.max_len), self.max_len + 1, n).astype(np.int64)
        self.offsets = np.concatenate([[0], np.cumsum(self.length)]).astype(np.int64)
        self.reward = rng.standard_normal(n).astype(np.float32)
        self.done = np.ones(n, np.uint8)
        self.action = np.zeros(n, np.int32)
        self.prio = quantise_priority(rng.lognormal(0.0, 1.0, n))
        self._tab = {}

    def _table(self, dev):
        if dev not in self._tab:
            self._tab[dev] = torch.from_numpy(_exp_quantiles()).to(dev)
        return self._tab[dev]

    def _elements(self, seqs, lengths, dev):
        seq = torch.repeat_interleave(seqs, lengths)
        starts = torch.cumsum(lengths, 0) - lengths
        j = torch.arange(int(lengths.sum()), dtype=torch.int64, device=dev) - torch.repeat_interleave(starts, lengths)
        tok = (hash32(self.seed, 3, seq, j) % self.vocab).to(torch.int32)
        lp = -self._table(dev)[hash32(self.seed, 5, seq, j) & 0xFFFF]
        return tok, lp

    def packed(self, start, count, device="cpu"):
        """Concatenated tokens (int32), log-probs (fp32) and [count+1] offsets of
        sequences [start, start+count)."""
        dev = torch.device(device)
        seqs = torch.arange(start, start + count, dtype=torch.int64, device=dev)
        lengths = torch.from_numpy(self.length[start:start + count]).to(dev)
        tok, lp = self._elements(seqs, lengths, dev)
        off = self.offsets[start:start + count + 1] - self.offsets[start]
        return tok, lp, torch.from_numpy(off).to(dev)

    def sequences_at(self, positions):
        """List of (tokens, logprobs) numpy arrays of the given stream positions (CPU)."""
        out = []
        for p in positions:
            p = int(p)
            tok, lp = self._elements(torch.tensor([p]), torch.tensor([int(self.length[p])]), torch.device("cpu"))
            out.append((tok.numpy(), lp.numpy()))
        return out

    def draws(self, iters, batch=None, seed=None):
        batch = self.batch if batch is None else batch
        rng = np.random.default_rng(draw_seed(4) if seed is None else seed)
        return uniforms(rng, iters, batch), quantise_priority(rng.lognormal(0.0, 1.0, (iters, batch)))


# ----------------------------------------------------------------------------
# 5: synthetic stress transitions of dimension d
# ----------------------------------------------------------------------------
class Stress:
    """Transitions of dimension d: obs and next_obs, d fp32 values each, stored as
    one [2, d] row per slot (8d bytes).  Values are exact fp32 numbers in [-1, 1)
    from an integer hash of (seed, stream position, element): k / 2^23 for a
    hashed integer k in [-2^23, 2^23).  next_obs of position j is obs of
    position j + 1 (one endless episode).  action int32 U{0..3}, reward N(0,1),
    priorities lognormal(0,1) quantised; batch 512, capacity 10^6."""

    capacity = 1_000_000
    batch = 512

    def __init__(self, d, n, seed=None):
        self.seed = data_seed(5) if seed is None else seed
        self.d = d
        self.obs_shape = (2, d)
        rng = np.random.default_rng(self.seed)
        self.n = n
        self.action = rng.integers(0, 4, n).astype(np.int32)
        self.reward = rng.standard_normal(n).astype(np.float32)
        self.done = np.zeros(n, np.uint8)
        self.prio = quantise_priority(rng.lognormal(0.0, 1.0, n))

    def _obs(self, pos, dev):
        k = torch.arange(self.d, dtype=torch.int64, device=dev)[None, :]
        h = hash32(self.seed, 13, pos[:, None], k)
        return ((h >> 8) - (1 << 23)).to(torch.float32) * (2.0 ** -23)

    def rows(self, start, count, device="cpu"):
        """fp32 [count, 2, d] transitions of stream positions [start, start+count)."""
        dev = torch.device(device)
        pos = torch.arange(start, start + count + 1, dtype=torch.int64, device=dev)
        o = self._obs(pos, dev)
        return torch.stack([o[:-1], o[1:]], dim=1)

    def rows_at(self, positions, device="cpu"):
        dev = torch.device(device)
        pos = torch.as_tensor(np.asarray(positions, np.int64), device=dev)
        return torch.stack([self._obs(pos, dev), self._obs(pos + 1, dev)], dim=1)

    def draws(self, iters, batch=None, seed=None):
        batch = self.batch if batch is None else batch
        rng = np.random.default_rng(draw_seed(5) if seed is None else seed)
        return uniforms(rng, iters, batch), quantise_priority(rng.lognormal(0.0, 1.0, (iters, batch)))
