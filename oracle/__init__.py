"""Reference oracle for the experience path -- TEST INFRASTRUCTURE ONLY.

Plain, slow CPU implementation (C in ``oracle.c``, fp64 where floating point is
involved) of ingest, priority update, stratified proportional sampling with
importance weights, frame-stack gather with pixel transforms, token packing, GAE
and the minibatch shuffle-gather.  Only ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import it.  It shares no code with
the HIP library and never imports it.

Each function cites the passage it follows; see ``oracle.c`` for the statements.
"""
import ctypes as C
import os

import numpy as np

from . import build as _build

_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        # ORACLE_LIB: another build of the same source (the sanitized one)
        path = os.environ.get("ORACLE_LIB")
        if not path:
            # (re)build when the library is missing or older than its source
            if not os.path.exists(_build.LIB) or os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC):
                _build.build()
            path = _build.LIB
        _LIB = C.CDLL(path)
        _declare(_LIB)
    return _LIB


P = C.c_void_p
I64 = C.c_int64
I32 = C.c_int32
U32 = C.c_uint32
F64 = C.c_double


class _Replay(C.Structure):
    _fields_ = [
        ("capacity", I64), ("row_bytes", I64), ("elem_bytes", I64), ("aux_elem_bytes", I64),
        ("act_bytes", I64), ("alpha_num", I32), ("alpha_den", I32), ("beta", F64),
        ("frame_stack", I32), ("ragged", I32), ("single_stream", I32), ("tree_leaves", I64),
        ("obs", P), ("aux", P), ("action", P), ("reward", P), ("done", P), ("episode", P),
        ("step", P), ("position", P), ("length", P), ("leaf", P), ("tree", P),
        ("head", I64), ("size", I64), ("total", I64), ("max_prio", U32),
    ]


def _declare(L):
    L.orc_frac_bits.argtypes = [I32, I32]
    L.orc_frac_bits.restype = I32
    L.orc_leaf.argtypes = [U32, I32, I32]
    L.orc_leaf.restype = U32
    L.orc_leaf_many.argtypes = [P, I64, I32, I32, P]
    L.orc_leaf_many.restype = None
    L.orc_reset.argtypes = [P]
    L.orc_reset.restype = None
    L.orc_total_priority.argtypes = [P]
    L.orc_total_priority.restype = C.c_uint64
    L.orc_ingest.argtypes = [P, I64] + [P] * 9
    L.orc_ingest.restype = I32
    L.orc_update.argtypes = [P, I64, P, P]
    L.orc_update.restype = I64
    L.orc_sample.argtypes = [P, I64, P, P, P, I32]
    L.orc_sample.restype = I32
    L.orc_gather.argtypes = [P, I64, P, I32, P, P, I32, P, P, P, P]
    L.orc_gather.restype = I32
    L.orc_pack.argtypes = [P, I64, P, I32, P, P, P, P, P]
    L.orc_pack.restype = I32
    L.orc_rows.argtypes = [P, I64, I64, P, I64, I32, P, P, I32, P]
    L.orc_rows.restype = I32
    L.orc_gae.argtypes = [I64, I64, P, P, P, P, F64, F64, P, P]
    L.orc_gae.restype = None
    L.orc_gae_trunc.argtypes = [I64, I64, P, P, P, P, P, P, F64, F64, P, P]
    L.orc_gae_trunc.restype = None
    L.orc_gae_packed.argtypes = [I64, I64, P, P, P, F64, F64, P, P]
    L.orc_gae_packed.restype = None
    L.orc_u8_to_f32.argtypes = [C.c_uint8]
    L.orc_u8_to_f32.restype = C.c_float
    L.orc_u8_to_bf16.argtypes = [C.c_uint8, C.c_float, C.c_float]
    L.orc_u8_to_bf16.restype = C.c_uint16


XF_NONE, XF_U8_F32, XF_U8_BF16_NORM = 0, 1, 2


def _ptr(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be contiguous"
    return a.ctypes.data


def _c(a, dtype):
    """Contiguous array of the given dtype (or None)."""
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


def frac_bits(alpha_num, alpha_den):
    return int(lib().orc_frac_bits(alpha_num, alpha_den))


def leaf(p, alpha_num=3, alpha_den=5):
    """Exact quantised leaf floor(2^F * p^(a/b)) of a uint32 priority."""
    return int(lib().orc_leaf(int(p), alpha_num, alpha_den))


def leaves(p, alpha_num=3, alpha_den=5):
    """orc_leaf over an array of uint32 priorities."""
    p = np.ascontiguousarray(p, np.uint32)
    out = np.zeros(len(p), np.uint32)
    lib().orc_leaf_many(_ptr(p), len(p), alpha_num, alpha_den, _ptr(out))
    return out


def u8_to_f32(x):
    return float(lib().orc_u8_to_f32(int(x)))


def u8_to_bf16_bits(x, mean, std):
    return int(lib().orc_u8_to_bf16(int(x), float(np.float32(mean)), float(np.float32(std))))


class Replay:
    """Replay dataset held in numpy arrays, driven by the C oracle.

    ``keep_obs=False`` keeps metadata and priorities only; ``obs_storage`` may
    supply the observation array (e.g. a lazily allocated ``np.zeros`` of the full
    capacity whose needed rows the caller fills itself).
    """

    def __init__(self, capacity, obs_shape, obs_dtype=np.uint8, act_bytes=4, alpha=(3, 5),
                 beta=0.4, frame_stack=1, ragged=False, aux_dtype=None, keep_obs=True,
                 obs_storage=None, buffer_norm=False, single_stream=False):
        obs_dtype = np.dtype(obs_dtype)
        self.buffer_norm = bool(buffer_norm)
        self.capacity = int(capacity)
        self.obs_shape = tuple(int(s) for s in obs_shape)
        self.obs_dtype = obs_dtype
        row_elems = int(np.prod(self.obs_shape)) if self.obs_shape else 1
        self.row_bytes = row_elems * obs_dtype.itemsize
        self.ragged = bool(ragged)
        self.max_len = row_elems if ragged else 0
        self.aux_dtype = np.dtype(aux_dtype) if aux_dtype is not None else None
        tl = 1
        while tl < self.capacity:
            tl *= 2
        cap = self.capacity
        if obs_storage is not None:
            self.obs = obs_storage
        elif keep_obs:
            self.obs = np.zeros((cap, self.row_bytes), np.uint8)
        else:
            self.obs = None
        self.aux = (np.zeros((cap, self.max_len * self.aux_dtype.itemsize), np.uint8)
                    if (ragged and self.aux_dtype is not None and keep_obs) else None)
        self.action = np.zeros((cap, act_bytes), np.uint8)
        self.reward = np.zeros(cap, np.float32)
        self.done = np.zeros(cap, np.uint8)
        self.episode = np.zeros(cap, np.uint32)
        self.step = np.zeros(cap, np.int32)
        self.position = np.full(cap, -1, np.int64)
        self.length = np.zeros(cap, np.int32) if ragged else None
        self.leaf = np.zeros(cap, np.uint32)
        self.tree = np.zeros(2 * tl, np.uint64)
        s = _Replay()
        s.capacity = cap
        s.row_bytes = self.row_bytes
        s.elem_bytes = obs_dtype.itemsize if ragged else 0
        s.aux_elem_bytes = self.aux_dtype.itemsize if (ragged and self.aux_dtype is not None) else 0
        s.act_bytes = act_bytes
        s.alpha_num, s.alpha_den = alpha
        s.beta = beta
        s.frame_stack = frame_stack
        s.ragged = 1 if ragged else 0
        s.single_stream = 1 if single_stream else 0
        s.tree_leaves = tl
        s.obs = _ptr(self.obs) if self.obs is not None else None
        s.aux = _ptr(self.aux) if self.aux is not None else None
        s.action, s.reward, s.done = _ptr(self.action), _ptr(self.reward), _ptr(self.done)
        s.episode, s.step, s.position = _ptr(self.episode), _ptr(self.step), _ptr(self.position)
        s.length = _ptr(self.length) if self.length is not None else None
        s.leaf, s.tree = _ptr(self.leaf), _ptr(self.tree)
        self._s = s
        self.act_bytes = act_bytes
        self.frame_stack = frame_stack
        lib().orc_reset(C.byref(s))

    # running state
    @property
    def head(self):
        return int(self._s.head)

    @property
    def size(self):
        return int(self._s.size)

    @property
    def total(self):
        return int(self._s.total)

    @property
    def max_prio(self):
        return int(self._s.max_prio)

    def total_priority(self):
        return int(lib().orc_total_priority(C.byref(self._s)))

    def ingest(self, n, obs=None, action=None, reward=None, done=None, episode=None, step=None,
               prio=None, offsets=None, aux=None):
        obs_b = None if obs is None else np.ascontiguousarray(obs).view(np.uint8).reshape(-1)
        aux_b = None if aux is None else np.ascontiguousarray(aux).view(np.uint8).reshape(-1)
        act_b = None if action is None else np.ascontiguousarray(action).view(np.uint8).reshape(-1)
        args = [_c(offsets, np.int64), aux_b, act_b, _c(reward, np.float32), _c(done, np.uint8),
                _c(episode, np.uint32), _c(step, np.int32), _c(prio, np.uint32)]
        rc = lib().orc_ingest(C.byref(self._s), int(n), _ptr(obs_b), *[_ptr(a) for a in args])
        if rc != 0:
            raise ValueError("oracle ingest rejected its arguments")

    def update(self, idx, prio):
        idx = _c(idx, np.int64)
        prio = _c(prio, np.uint32)
        return int(lib().orc_update(C.byref(self._s), len(idx), _ptr(idx), _ptr(prio)))

    def sample(self, uniforms, buffer_norm=None):
        """Stratified proportional sampling; IS weights normalised by the batch
        maximum, or with ``buffer_norm`` (default: the replay's own setting)
        by the largest weight over the whole buffer."""
        u = _c(uniforms, np.uint64)
        B = len(u)
        idx = np.zeros(B, np.int64)
        w = np.zeros(B, np.float32)
        bn = self.buffer_norm if buffer_norm is None else buffer_norm
        rc = lib().orc_sample(C.byref(self._s), B, _ptr(u), _ptr(idx), _ptr(w), int(bool(bn)))
        if rc != 0:
            raise ValueError("oracle: nothing to sample")
        return idx, w

    def nstep(self, idx, n, gamma):
        """n-step return targets of sampled slots (the n-step Q-learning target
        of the DQN line the paper cites: sum of gamma^k r over the next n
        transitions of the episode, then gamma^n times the value of the state
        n steps ahead).  For slot i holding stream position p, the window is
        positions p, p+1, ...: it stops after the first done (a terminal: no
        bootstrap), or after n transitions, where the bootstrap state is the
        observation at p+n.  A window that reaches a position not yet stored,
        or another episode without a done, is invalid (every output 0).
        Returns (bootstrap slot or -1, return, discount, valid) per sample:
        return = sum_k gamma^k r_{p+k} (fp64, k ascending, fp32 out), discount
        = gamma^n for a bootstrapped window and 0 otherwise."""
        idx = np.asarray(idx, np.int64)
        B = len(idx)
        C, total = self.capacity, self.total
        nxt = np.full(B, -1, np.int64)
        ret = np.zeros(B, np.float32)
        disc = np.zeros(B, np.float32)
        valid = np.zeros(B, np.uint8)

        def stored(q, ep):
            s = q % C
            return q < total and self.position[s] == q and self.episode[s] == ep

        for b in range(B):
            i = int(idx[b])
            p = int(self.position[i])
            ep = self.episode[i]
            R, g, ended, ok = 0.0, 1.0, False, True
            for k in range(n):
                if not stored(p + k, ep):
                    ok = False
                    break
                s = (p + k) % C
                R += g * float(self.reward[s])
                g *= gamma
                if self.done[s]:
                    ended = True
                    break
            if not ok:
                continue
            if ended:
                ret[b], valid[b] = R, 1
            elif stored(p + n, ep):
                nxt[b], ret[b], disc[b], valid[b] = (p + n) % C, R, g, 1
        return nxt, ret, disc, valid

    def gather(self, idx, xform=XF_NONE, mean=None, std=None):
        idx = _c(idx, np.int64)
        B = len(idx)
        K = self.frame_stack
        out_elem = {XF_NONE: 1, XF_U8_F32: 4, XF_U8_BF16_NORM: 2}[xform]
        out = np.zeros((B, K, self.row_bytes * out_elem), np.uint8) if self.obs is not None else None
        act = np.zeros((B, self.act_bytes), np.uint8)
        rew = np.zeros(B, np.float32)
        done = np.zeros(B, np.uint8)
        m = _c(mean, np.float32)
        s = _c(std, np.float32)
        channels = len(m) if m is not None else 1
        rc = lib().orc_gather(C.byref(self._s), B, _ptr(idx), xform, _ptr(m), _ptr(s), channels,
                              _ptr(out), _ptr(act), _ptr(rew), _ptr(done))
        if rc != 0:
            raise ValueError("oracle: gather index out of range")
        if out is not None:
            if xform == XF_U8_F32:
                out = out.view(np.float32)
            elif xform == XF_U8_BF16_NORM:
                out = out.view(np.uint16)
            elif self.obs_dtype != np.uint8:
                out = out.view(self.obs_dtype)
            out = out.reshape((B, K) + self.obs_shape)
        return out, act, rew, done

    def pack(self, idx, pad_id=0):
        idx = _c(idx, np.int64)
        B = len(idx)
        L = self.max_len
        seq = np.zeros((B, L), self.obs_dtype)
        mask = np.zeros((B, L), np.uint8)
        aux = np.zeros((B, L), self.aux_dtype) if self.aux is not None else None
        length = np.zeros(B, np.int32)
        rew = np.zeros(B, np.float32)
        rc = lib().orc_pack(C.byref(self._s), B, _ptr(idx), int(pad_id), _ptr(seq), _ptr(mask),
                            _ptr(aux), _ptr(length), _ptr(rew))
        if rc != 0:
            raise ValueError("oracle: pack index out of range")
        return seq, mask, aux, length, rew


def rows(src, perm, xform=XF_NONE, mean=None, std=None):
    """Minibatch shuffle-gather of rows ``src[perm]`` through a pixel transform."""
    src = np.ascontiguousarray(src)
    n_src = src.shape[0]
    row_shape = src.shape[1:]
    src_b = src.view(np.uint8).reshape(n_src, -1)
    row_bytes = src_b.shape[1]
    perm = _c(perm, np.int64)
    out_elem = {XF_NONE: 1, XF_U8_F32: 4, XF_U8_BF16_NORM: 2}[xform]
    out = np.zeros((len(perm), row_bytes * out_elem), np.uint8)
    m = _c(mean, np.float32)
    s = _c(std, np.float32)
    channels = len(m) if m is not None else 1
    rc = lib().orc_rows(_ptr(src_b), row_bytes, n_src, _ptr(perm), len(perm), xform, _ptr(m), _ptr(s),
                        channels, _ptr(out))
    if rc != 0:
        raise ValueError("oracle: permutation index out of range")
    if xform == XF_U8_F32:
        return out.view(np.float32).reshape((len(perm),) + row_shape)
    if xform == XF_U8_BF16_NORM:
        return out.view(np.uint16).reshape((len(perm),) + row_shape)
    return out.view(src.dtype).reshape((len(perm),) + row_shape)


def gae(reward, value, done, bootstrap, gamma, lam, truncated=None, final_value=None):
    """GAE over a time-major [T, E] rollout (fp64 inside, fp32 out).  With
    ``truncated`` (and ``final_value``), truncated steps end the recursion and
    bootstrap from the value of their true next observation."""
    r = _c(reward, np.float32)
    T, E = r.shape
    v = _c(value, np.float32)
    d = _c(done, np.uint8)
    b = _c(bootstrap, np.float32)
    adv = np.zeros((T, E), np.float32)
    ret = np.zeros((T, E), np.float32)
    if truncated is None:
        lib().orc_gae(T, E, _ptr(r), _ptr(v), _ptr(d), _ptr(b), float(gamma), float(lam), _ptr(adv), _ptr(ret))
    else:
        tr = _c(truncated, np.uint8)
        fv = _c(final_value, np.float32)
        lib().orc_gae_trunc(T, E, _ptr(r), _ptr(v), _ptr(d), _ptr(tr), _ptr(fv), _ptr(b), float(gamma), float(lam),
                            _ptr(adv), _ptr(ret))
    return adv, ret


def gae_packed(last_reward, length, value, Lmax, gamma, lam):
    """GAE over right-padded sequences with the reward on each sequence's last element."""
    lr = _c(last_reward, np.float32)
    ln = _c(length, np.int32)
    B = len(lr)
    v = _c(value, np.float32)
    adv = np.zeros((B, Lmax), np.float32)
    ret = np.zeros((B, Lmax), np.float32)
    lib().orc_gae_packed(B, int(Lmax), _ptr(lr), _ptr(ln), _ptr(v), float(gamma), float(lam), _ptr(adv),
                         _ptr(ret))
    return adv, ret
