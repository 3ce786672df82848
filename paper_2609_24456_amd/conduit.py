"""Thin Python binding of libconduit's C ABI (include/conduit.h).

Argument marshalling only: every function forwards torch tensor pointers and the
current HIP stream to the C entry point of the same name; every step of the
experience path runs in the library's HIP kernels.  There is no CPU fallback:
if ``libconduit.so`` is missing, loading it raises.
"""
import ctypes as C
import os

import torch

from .abi import *  # noqa: F401,F403  (status codes, enums, structs, SIGNATURES)
from .abi import _STATUS_NAMES, load as _load_abi  # noqa: F401

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libconduit.so")
_lib = None

_TORCH_DTYPE = {torch.uint8: U8, torch.int32: I32, torch.float32: F32, torch.bfloat16: BF16}


def lib():
    """Load libconduit.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
        _lib = _load_abi(LIB_PATH)
    return _lib


def last_error():
    return lib().conduit_last_error().decode()


def _check(status):
    if status != OK:
        raise ConduitError(status, last_error())


def _stream(stream):
    if stream is None:
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return C.c_void_p(stream.cuda_stream)
    return C.c_void_p(int(stream))


_ELEM4_INT = (torch.int32, torch.uint32)
_ELEM8_INT = (torch.int64, torch.uint64)


def _ptr(t, dtype=None, name="tensor", nbytes=None, numel=None):
    """Device address of a contiguous tensor, after checking (in this order)
    its type, dtype (one dtype or a tuple of accepted dtypes), that it holds at
    least `nbytes` bytes / `numel` elements, contiguity and device.  Each
    failure raises before anything reaches the library, so a shape or dtype
    slip never becomes an out-of-bounds device access."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if dtype is not None:
        ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
        if not ok:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if nbytes is not None and t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, the call touches {nbytes}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, the call touches {numel}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if not _on_device(t):
        raise ValueError(f"{name} must be on a HIP device")
    return t.data_ptr()


def _on_device(t):
    return t.is_cuda


def _info(handle):
    """The buffer's host-side geometry (conduit_buffer_get_info: no device work)."""
    info = BufferInfo()
    _check(lib().conduit_buffer_get_info(handle, C.byref(info)))
    return info


_OUT_ELEM = {XF_NONE: 1, XF_U8_F32: 4, XF_U8_BF16_NORM: 2}


def _out_row_bytes(info, xf):
    """Bytes of one gathered sample's observation output (dense buffers)."""
    if xf.kind not in _OUT_ELEM:
        raise ValueError("dense buffers gather with NONE, U8_F32 or U8_BF16_NORM")
    return info.frame_stack * info.row_bytes * _OUT_ELEM[xf.kind]


def _batch_ptrs(info, n, xf, obs, action, reward, done, mask, aux, length):
    """A LearnerBatch for n samples of the buffer described by `info`, every
    output checked against the bytes the gather writes."""
    out = LearnerBatch()
    if info.ragged:
        L = info.max_len
        out.obs = _ptr(obs, _ELEM4_INT + (torch.float32,), "obs", nbytes=n * L * 4)
        out.mask = _ptr(mask, (torch.uint8, torch.bool), "mask", nbytes=n * L)
        out.aux = _ptr(aux, None, "aux", nbytes=n * L * 4)
        out.length = _ptr(length, torch.int32, "length", numel=n)
    else:
        out.obs = _ptr(obs, None, "obs", nbytes=n * _out_row_bytes(info, xf))
        out.mask, out.aux, out.length = None, None, None
    out.action = _ptr(action, None, "action", nbytes=n * info.action_bytes)
    out.reward = _ptr(reward, torch.float32, "reward", numel=n)
    out.done = _ptr(done, (torch.uint8, torch.bool), "done", numel=n)
    return out


def transform(kind=XF_NONE, mean=None, std=None, pad_id=0):
    xf = Transform()
    xf.kind = kind
    xf.pad_id = int(pad_id)
    if mean is not None:
        xf.channels = len(mean)
        for c in range(len(mean)):
            xf.mean[c] = float(mean[c])
            xf.std[c] = float(std[c])
    else:
        xf.channels = 1
        for c in range(4):
            xf.std[c] = 1.0
    return xf


def default_opts(**kw):
    o = BufferOpts()
    lib().conduit_buffer_opts_default(C.byref(o))
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def conduit_buffer_required_bytes(capacity, obs_shape, obs_dtype, opts=None):
    shape = (C.c_int64 * len(obs_shape))(*obs_shape)
    return int(lib().conduit_buffer_required_bytes(capacity, shape, len(obs_shape), obs_dtype,
                                                   C.byref(opts) if opts is not None else None))


def conduit_buffer_create(capacity, obs_shape, obs_dtype, opts=None, arena=None):
    """Returns an opaque handle (int).  ``arena``: optional uint8 CUDA tensor."""
    shape = (C.c_int64 * len(obs_shape))(*obs_shape)
    out = C.c_void_p()
    ap = _ptr(arena, torch.uint8, "arena") if arena is not None else None
    ab = arena.numel() if arena is not None else 0
    _check(lib().conduit_buffer_create(capacity, shape, len(obs_shape), obs_dtype,
                                       C.byref(opts) if opts is not None else None, ap, ab, C.byref(out)))
    return out.value


def conduit_buffer_destroy(handle):
    lib().conduit_buffer_destroy(handle)


def _transitions(info, n, obs, action=None, reward=None, done=None, episode_id=None, step=None, prio=None,
                 offsets=None, aux=None):
    n = int(n)
    if n < 0:
        raise ValueError("n must be >= 0")
    t = Transitions()
    t.n = n
    if info.ragged:
        t.obs = _ptr(obs, _ELEM4_INT + (torch.float32,), "obs")
        t.offsets = _ptr(offsets, torch.int64, "offsets", numel=n + 1)
        t.aux = _ptr(aux, None, "aux")
        if aux is not None and aux.element_size() != 4:
            raise TypeError("aux must hold 4-byte elements")
        # the kernel keeps every offset within the elements obs (and aux) hold
        t.src_elems = min(obs.numel(), aux.numel()) if aux is not None else obs.numel()
    else:
        t.obs = _ptr(obs, None, "obs", nbytes=n * info.row_bytes)
        t.offsets, t.aux, t.src_elems = None, None, 0
    t.action = _ptr(action, None, "action", nbytes=n * info.action_bytes)
    t.reward = _ptr(reward, torch.float32, "reward", numel=n)
    t.done = _ptr(done, (torch.uint8, torch.bool), "done", numel=n)
    t.episode_id = _ptr(episode_id, _ELEM4_INT, "episode_id", numel=n)  # uint32 ids (int32 view accepted)
    t.step = _ptr(step, torch.int32, "step", numel=n)
    t.prio = _ptr(prio, _ELEM4_INT, "prio", numel=n)
    return t


def conduit_ingest(handle, n, obs, action=None, reward=None, done=None, episode_id=None, step=None, prio=None,
                   offsets=None, aux=None, stream=None):
    t = _transitions(_info(handle), n, obs, action, reward, done, episode_id, step, prio, offsets, aux)
    _check(lib().conduit_ingest(handle, C.byref(t), _stream(stream)))


def conduit_update_ingest(handle, idx, upd_prio, n, obs, action=None, reward=None, done=None, episode_id=None,
                          step=None, prio=None, offsets=None, aux=None, stream=None):
    """The priority update (idx, upd_prio), then the ingest of n rows, in one call."""
    t = _transitions(_info(handle), n, obs, action, reward, done, episode_id, step, prio, offsets, aux)
    k = idx.numel() if idx is not None else 0
    _check(lib().conduit_update_ingest(handle, _ptr(idx, torch.int64, "idx"),
                                       _ptr(upd_prio, _ELEM4_INT, "upd_prio", numel=k), k, C.byref(t),
                                       _stream(stream)))


def conduit_update_priorities(handle, idx, prio, stream=None):
    n = idx.numel()
    if prio.numel() != n:
        raise ValueError("idx and prio must have the same length")
    _check(lib().conduit_update_priorities(handle, _ptr(idx, torch.int64, "idx"), _ptr(prio, _ELEM4_INT, "prio"), n,
                                           _stream(stream)))


def conduit_sample(handle, batch, uniforms, idx_out, is_w_out=None, stream=None):
    _check(lib().conduit_sample(handle, batch, _ptr(uniforms, _ELEM8_INT, "uniforms", numel=batch),
                                _ptr(idx_out, torch.int64, "idx_out", numel=batch),
                                _ptr(is_w_out, torch.float32, "is_w_out", numel=batch), _stream(stream)))


def conduit_gather_transform(handle, idx, xf, obs=None, action=None, reward=None, done=None, mask=None, aux=None,
                             length=None, stream=None):
    n = idx.numel()
    out = _batch_ptrs(_info(handle), n, xf, obs, action, reward, done, mask, aux, length)
    _check(lib().conduit_gather_transform(handle, _ptr(idx, torch.int64, "idx"), n, C.byref(xf), C.byref(out),
                                          _stream(stream)))


def conduit_sample_gather(handle, batch, uniforms, idx_out, is_w_out, xf, obs=None, action=None, reward=None,
                          done=None, mask=None, aux=None, length=None, stream=None):
    out = _batch_ptrs(_info(handle), batch, xf, obs, action, reward, done, mask, aux, length)
    _check(lib().conduit_sample_gather(handle, batch, _ptr(uniforms, _ELEM8_INT, "uniforms", numel=batch),
                                       _ptr(idx_out, torch.int64, "idx_out", numel=batch),
                                       _ptr(is_w_out, torch.float32, "is_w_out", numel=batch),
                                       C.byref(xf), C.byref(out), _stream(stream)))


def conduit_sample_gather_nstep(handle, batch, uniforms, idx_out, is_w_out, xf, n, gamma, next_idx, ret, discount,
                                valid, next_obs=None, obs=None, action=None, reward=None, done=None, stream=None):
    """conduit_sample_gather then conduit_nstep on the sampled slots, in one
    launch where the buffer's rows allow it."""
    info = _info(handle)
    out = _batch_ptrs(info, batch, xf, obs, action, reward, done, None, None, None)
    nbytes = batch * _out_row_bytes(info, xf) if (next_obs is not None and not info.ragged) else None
    _check(lib().conduit_sample_gather_nstep(
        handle, batch, _ptr(uniforms, _ELEM8_INT, "uniforms", numel=batch),
        _ptr(idx_out, torch.int64, "idx_out", numel=batch), _ptr(is_w_out, torch.float32, "is_w_out", numel=batch),
        C.byref(xf), C.byref(out), int(n), float(gamma), _ptr(next_idx, torch.int64, "next_idx", numel=batch),
        _ptr(ret, torch.float32, "ret", numel=batch), _ptr(discount, torch.float32, "discount", numel=batch),
        _ptr(valid, (torch.uint8, torch.bool), "valid", numel=batch), _ptr(next_obs, None, "next_obs", nbytes=nbytes),
        _stream(stream)))


def conduit_sample_pack_gae(handle, batch, uniforms, idx_out, is_w_out, xf, values, gamma, lam, adv, ret, obs=None,
                            action=None, reward=None, done=None, mask=None, aux=None, length=None, stream=None):
    """conduit_sample_gather on a ragged buffer, then conduit_gae_packed over the
    packed rows, in one launch."""
    info = _info(handle)
    out = _batch_ptrs(info, batch, xf, obs, action, reward, done, mask, aux, length)
    L = info.max_len
    _check(lib().conduit_sample_pack_gae(
        handle, batch, _ptr(uniforms, _ELEM8_INT, "uniforms", numel=batch),
        _ptr(idx_out, torch.int64, "idx_out", numel=batch), _ptr(is_w_out, torch.float32, "is_w_out", numel=batch),
        C.byref(xf), C.byref(out), _ptr(values, torch.float32, "values", numel=batch * L), float(gamma), float(lam),
        _ptr(adv, torch.float32, "adv", numel=batch * L), _ptr(ret, torch.float32, "ret", numel=batch * L),
        _stream(stream)))


def conduit_nstep(handle, idx, n, gamma, next_idx, ret, discount, valid, xf=None, next_obs=None, stream=None):
    """n-step return targets (and bootstrap-state stacks) of sampled slots."""
    B = idx.numel()
    info = _info(handle)
    nbytes = B * _out_row_bytes(info, xf) if (next_obs is not None and xf is not None and not info.ragged) else None
    _check(lib().conduit_nstep(handle, _ptr(idx, torch.int64, "idx"), B, int(n), float(gamma),
                               _ptr(next_idx, torch.int64, "next_idx", numel=B),
                               _ptr(ret, torch.float32, "ret", numel=B),
                               _ptr(discount, torch.float32, "discount", numel=B),
                               _ptr(valid, (torch.uint8, torch.bool), "valid", numel=B),
                               C.byref(xf) if xf is not None else None,
                               _ptr(next_obs, None, "next_obs", nbytes=nbytes), _stream(stream)))


def _rollout_shape(rewards):
    if not isinstance(rewards, torch.Tensor) or rewards.dim() != 2:
        raise ValueError("rewards must be a [T, E] tensor")
    return rewards.shape


def conduit_gae(rewards, values, dones, bootstrap, gamma, lam, adv, ret, stream=None):
    T, E = _rollout_shape(rewards)
    N = T * E
    _check(lib().conduit_gae(_ptr(rewards, torch.float32, "rewards"), _ptr(values, torch.float32, "values", numel=N),
                             _ptr(dones, (torch.uint8, torch.bool), "dones", numel=N),
                             _ptr(bootstrap, torch.float32, "bootstrap", numel=E), T, E, float(gamma), float(lam),
                             _ptr(adv, torch.float32, "adv", numel=N), _ptr(ret, torch.float32, "ret", numel=N),
                             _stream(stream)))


GAE_PATHS = ("one", "one_v4", "short", "look", "split")


def gae_plan(T, E, aligned=True):
    """(path, chunk) conduit_gae takes for a [T, E] rollout: path one of
    GAE_PATHS (conduit_gae_plan's *path), chunk the tile's steps per lane."""
    path, chunk = C.c_int32(), C.c_int32()
    _check(lib().conduit_gae_plan(int(T), int(E), 1 if aligned else 0, C.byref(path), C.byref(chunk)))
    return GAE_PATHS[path.value], chunk.value


def conduit_gae_truncated(rewards, values, dones, truncated, final_values, bootstrap, gamma, lam, adv, ret,
                          stream=None):
    T, E = _rollout_shape(rewards)
    N = T * E
    u8 = (torch.uint8, torch.bool)
    _check(lib().conduit_gae_truncated(_ptr(rewards, torch.float32, "rewards"),
                                       _ptr(values, torch.float32, "values", numel=N),
                                       _ptr(dones, u8, "dones", numel=N), _ptr(truncated, u8, "truncated", numel=N),
                                       _ptr(final_values, torch.float32, "final_values", numel=N),
                                       _ptr(bootstrap, torch.float32, "bootstrap", numel=E), T, E, float(gamma),
                                       float(lam), _ptr(adv, torch.float32, "adv", numel=N),
                                       _ptr(ret, torch.float32, "ret", numel=N), _stream(stream)))


def conduit_gae_packed(last_reward, lengths, values, Lmax, gamma, lam, adv, ret, stream=None):
    B = last_reward.numel()
    N = B * int(Lmax)
    _check(lib().conduit_gae_packed(_ptr(last_reward, torch.float32, "last_reward"),
                                    _ptr(lengths, torch.int32, "lengths", numel=B),
                                    _ptr(values, torch.float32, "values", numel=N), B, int(Lmax), float(gamma),
                                    float(lam), _ptr(adv, torch.float32, "adv", numel=N),
                                    _ptr(ret, torch.float32, "ret", numel=N), _stream(stream)))


def conduit_schedule(t_rollout, t_update, g_ing, t_ing, g_del, t_del, t_sync_ing=0.0, t_sync_del=0.0,
                     on_policy=False):
    """Sec. 6 cost model: (best mode, every mode) as dicts."""
    arr = lambda xs: (C.c_double * max(1, len(xs)))(*[float(x) for x in xs])  # noqa: E731
    gi, ti, gd, td = arr(g_ing), arr(t_ing), arr(g_del), arr(t_del)
    c = SchedCosts(float(t_rollout), float(t_update), float(t_sync_ing), float(t_sync_del), len(g_ing), len(g_del),
                   gi, ti, gd, td, int(bool(on_policy)))
    best = SchedMode()
    n = 4 * max(1, len(g_ing)) * max(1, len(g_del))
    all_ = (SchedMode * n)()
    _check(lib().conduit_schedule(C.byref(c), C.byref(best), all_))
    return best.as_dict(), [m.as_dict() for m in all_]


def conduit_sched_candidates(on_policy, minibatches=1, g_max_ing=1, g_max_del=1):
    """Feasible granularity sets (G_ing, G_del) of an RL configuration."""
    cap = max(1, int(minibatches), int(g_max_ing), int(g_max_del))
    gi, gd = (C.c_double * cap)(), (C.c_double * cap)()
    ni, nd = C.c_int32(0), C.c_int32(0)
    _check(lib().conduit_sched_candidates(int(bool(on_policy)), int(minibatches), int(g_max_ing), int(g_max_del),
                                          gi, cap, C.byref(ni), gd, cap, C.byref(nd)))
    return [gi[i] for i in range(ni.value)], [gd[i] for i in range(nd.value)]


OP_INGEST, OP_DELIVER, OP_PRIO, OP_GAE = 0, 1, 2, 3


def conduit_run_offpolicy(handle, loop, compute_stream, experience_stream):
    """Run the native off-policy loop; returns (elapsed ms, op log as a list of
    (kind, a, b) in experience-stream order)."""
    cap = 3 * int(loop.iters)
    log = (C.c_int64 * (3 * cap))()
    n = C.c_int64(0)
    ms = C.c_double(0.0)
    _check(lib().conduit_run_offpolicy(handle, C.byref(loop), _stream(compute_stream), _stream(experience_stream),
                                       C.byref(ms), log, C.byref(n)))
    return ms.value, [(log[3 * i], log[3 * i + 1], log[3 * i + 2]) for i in range(min(n.value, cap))]


def conduit_run_onpolicy(handle, loop, compute_stream, experience_stream):
    """Run the native on-policy loop; returns (elapsed ms, op log as a list of
    (kind, iteration, a, b) in program order)."""
    cap = int(loop.iters) * (2 * int(loop.minibatches) + 1)
    log = (C.c_int64 * (4 * cap))()
    n = C.c_int64(0)
    ms = C.c_double(0.0)
    _check(lib().conduit_run_onpolicy(handle, C.byref(loop), _stream(compute_stream), _stream(experience_stream),
                                      C.byref(ms), log, C.byref(n)))
    return ms.value, [tuple(log[4 * i:4 * i + 4]) for i in range(min(n.value, cap))]


def conduit_placement_profile(nbytes=256 << 20, reps=3):
    """Sec. 5.1 microbenchmarks: a PlaceProfile of this host and GPU."""
    prof = PlaceProfile()
    _check(lib().conduit_placement_profile(int(nbytes), int(reps), C.byref(prof)))
    return prof


def conduit_place(profile, actor_on_gpu, capacity, sample_bytes, candidates=(0, 1, 2)):
    """Alg. 1: (chosen placement or -1, T_transfer per candidate in seconds)."""
    n = len(candidates)
    cand = (C.c_int32 * max(1, n))(*candidates)
    t = (C.c_double * max(1, n))()
    choice = C.c_int32(-2)
    _check(lib().conduit_place(C.byref(profile), int(actor_on_gpu), int(capacity), float(sample_bytes), cand, n,
                               C.byref(choice), t))
    return choice.value, [t[i] for i in range(n)]


def conduit_standin(work, stream=None):
    _check(lib().conduit_standin(int(work), _stream(stream)))


def conduit_expand_reference(src, dst, stream=None):
    """dst = src / 255 over contiguous memory (the gathers' read/write mix without their indexing)."""
    n = src.numel()
    _check(lib().conduit_expand_reference(_ptr(src, torch.uint8, "src"),
                                          _ptr(dst, torch.float32, "dst", numel=n), n, _stream(stream)))


def conduit_sync_cost_us(s1, s2, hops=200):
    """(hop_us, dep_us): an unmet cross-stream dependency, and the cost an
    overlapped operator adds to the stream it overlaps."""
    hop, dep = C.c_double(0.0), C.c_double(0.0)
    _check(lib().conduit_sync_cost_us(_stream(s1), _stream(s2), int(hops), C.byref(hop), C.byref(dep)))
    return hop.value, dep.value


def conduit_minibatch_gather(src, row_bytes, n_src, perm, xf, out, cols=(), cols_out=(), stream=None):
    ncols = len(cols)
    if len(cols_out) != ncols:
        raise ValueError("cols and cols_out must have the same length")
    if xf.kind not in _OUT_ELEM:
        raise ValueError("the minibatch gather takes NONE, U8_F32 or U8_BF16_NORM")
    n, row_bytes, n_src = perm.numel(), int(row_bytes), int(n_src)
    ca = (C.c_void_p * max(1, ncols))(*[_ptr(c, torch.float32, "col", numel=n_src) for c in cols])
    co = (C.c_void_p * max(1, ncols))(*[_ptr(c, torch.float32, "col_out", numel=n) for c in cols_out])
    _check(lib().conduit_minibatch_gather(_ptr(src, None, "src", nbytes=n_src * row_bytes), row_bytes, n_src,
                                          _ptr(perm, torch.int64, "perm"), n, C.byref(xf),
                                          _ptr(out, None, "out", nbytes=n * row_bytes * _OUT_ELEM[xf.kind]),
                                          ca if ncols else None, co if ncols else None, ncols, _stream(stream)))


def conduit_buffer_get_info(handle):
    return _info(handle)


def conduit_buffer_stats(handle):
    """(size, head, total) after waiting for the buffer's device."""
    size, head, total = C.c_int64(), C.c_int64(), C.c_uint64()
    _check(lib().conduit_buffer_stats(handle, C.byref(size), C.byref(head), C.byref(total)))
    return size.value, head.value, total.value


def conduit_buffer_read(handle, col, dst, offset=0, level=0, stream=None):
    _check(lib().conduit_buffer_read(handle, col, level, int(offset), dst.numel() * dst.element_size(),
                                     _ptr(dst, None, "dst"), _stream(stream)))


def conduit_buffer_checkpoint_bytes(handle):
    n = C.c_uint64()
    _check(lib().conduit_buffer_checkpoint_bytes(handle, C.byref(n)))
    return n.value


def _image_ptr(t, name, nbytes=None):
    """Address of a contiguous uint8 image tensor, on the device or in host memory."""
    if not isinstance(t, torch.Tensor) or t.dtype != torch.uint8:
        raise TypeError(f"{name} must be a torch.uint8 tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if nbytes is not None and t.numel() < nbytes:
        raise ValueError(f"{name} holds {t.numel()} bytes, the image needs {nbytes}")
    return t.data_ptr()


def conduit_buffer_checkpoint(handle, dst, stream=None):
    """Write the buffer's checkpoint image into `dst` (uint8 tensor, device or host memory)."""
    n = conduit_buffer_checkpoint_bytes(handle)
    _check(lib().conduit_buffer_checkpoint(handle, _image_ptr(dst, "dst", n), dst.numel(), _stream(stream)))


def conduit_buffer_restore(handle, src, stream=None):
    """Replace the buffer's state with the checkpoint image in `src` (uint8 tensor)."""
    _check(lib().conduit_buffer_restore(handle, _image_ptr(src, "src"), src.numel(), _stream(stream)))


def ckpt_header(image):
    """The header of a checkpoint image (a uint8 tensor on the device or the host, or bytes)."""
    n = C.sizeof(CkptHeader)
    raw = bytes(image[:n].cpu().numpy()) if isinstance(image, torch.Tensor) else bytes(image[:n])
    if len(raw) < C.sizeof(CkptHeader) or raw[:8] != CKPT_MAGIC:
        raise ValueError("not a checkpoint image")
    return CkptHeader.from_buffer_copy(raw)


def conduit_sync_check(handle=None, stream=None):
    return lib().conduit_sync_check(handle, _stream(stream))


def conduit_clear_error(handle=None):
    lib().conduit_clear_error(handle)


def conduit_version():
    return lib().conduit_version().decode()


class ReplayBuffer:
    """Owning wrapper around a conduit_buffer handle."""

    def __init__(self, capacity, obs_shape, obs_dtype=torch.uint8, prioritized=True, alpha=(3, 5), beta=0.4,
                 frame_stack=1, action_bytes=4, ragged=False, aux_elem_bytes=0, arena=None, placement=PLACE_HBM,
                 weight_norm=0, single_stream=False):
        self.opts = default_opts(prioritized=int(prioritized), alpha_num=alpha[0], alpha_den=alpha[1], beta=beta,
                                 frame_stack=frame_stack, action_bytes=action_bytes, ragged=int(ragged),
                                 aux_elem_bytes=aux_elem_bytes, payload_placement=int(placement),
                                 weight_norm=int(weight_norm), single_stream=int(bool(single_stream)))
        self.capacity = capacity
        self.obs_shape = tuple(obs_shape)
        self.obs_dtype = obs_dtype
        self._arena = arena
        self.handle = conduit_buffer_create(capacity, self.obs_shape, _TORCH_DTYPE[obs_dtype], self.opts, arena)

    def close(self):
        if getattr(self, "handle", None):
            conduit_buffer_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self):
        return conduit_buffer_get_info(self.handle)

    def stats(self):
        return conduit_buffer_stats(self.handle)

    def ingest(self, obs, action=None, reward=None, done=None, episode_id=None, step=None, prio=None, offsets=None,
               aux=None, n=None, stream=None):
        n = (offsets.numel() - 1 if offsets is not None else obs.shape[0]) if n is None else n
        conduit_ingest(self.handle, n, obs, action, reward, done, episode_id, step, prio, offsets, aux, stream)

    def update(self, idx, prio, stream=None):
        conduit_update_priorities(self.handle, idx, prio, stream)

    def update_ingest(self, idx, upd_prio, obs, action=None, reward=None, done=None, episode_id=None, step=None,
                      prio=None, offsets=None, aux=None, n=None, stream=None):
        n = (offsets.numel() - 1 if offsets is not None else obs.shape[0]) if n is None else n
        conduit_update_ingest(self.handle, idx, upd_prio, n, obs, action, reward, done, episode_id, step, prio,
                              offsets, aux, stream)

    def sample(self, uniforms, idx_out=None, w_out=None, stream=None):
        B = uniforms.numel()
        dev = uniforms.device
        idx_out = torch.empty(B, dtype=torch.int64, device=dev) if idx_out is None else idx_out
        w_out = torch.empty(B, dtype=torch.float32, device=dev) if w_out is None else w_out
        conduit_sample(self.handle, B, uniforms, idx_out, w_out, stream)
        return idx_out, w_out

    def sample_gather(self, uniforms, xf, idx_out=None, w_out=None, **outs):
        B = uniforms.numel()
        dev = uniforms.device
        idx_out = torch.empty(B, dtype=torch.int64, device=dev) if idx_out is None else idx_out
        w_out = torch.empty(B, dtype=torch.float32, device=dev) if w_out is None else w_out
        conduit_sample_gather(self.handle, B, uniforms, idx_out, w_out, xf, stream=outs.pop("stream", None), **outs)
        return idx_out, w_out

    def gather(self, idx, xf, **outs):
        conduit_gather_transform(self.handle, idx, xf, stream=outs.pop("stream", None), **outs)

    def sample_pack_gae(self, uniforms, xf, gamma, lam, adv, ret, values=None, **outs):
        """(idx, w) of one token delivery whose packed rows' GAE goes to adv
        and ret in the same launch."""
        B = uniforms.numel()
        dev = uniforms.device
        idx = torch.empty(B, dtype=torch.int64, device=dev)
        w = torch.empty(B, dtype=torch.float32, device=dev)
        conduit_sample_pack_gae(self.handle, B, uniforms, idx, w, xf, values, gamma, lam, adv, ret,
                                stream=outs.pop("stream", None), **outs)
        return idx, w

    def sample_gather_nstep(self, uniforms, xf, n, gamma, next_obs=None, **outs):
        """(idx, w, next_idx, ret, discount, valid) of one fused delivery with
        n-step targets; the batch and the bootstrap stacks go to the given
        outputs."""
        B = uniforms.numel()
        dev = uniforms.device
        idx = torch.empty(B, dtype=torch.int64, device=dev)
        w = torch.empty(B, dtype=torch.float32, device=dev)
        nxt = torch.empty(B, dtype=torch.int64, device=dev)
        ret = torch.empty(B, dtype=torch.float32, device=dev)
        disc = torch.empty(B, dtype=torch.float32, device=dev)
        val = torch.empty(B, dtype=torch.uint8, device=dev)
        conduit_sample_gather_nstep(self.handle, B, uniforms, idx, w, xf, n, gamma, nxt, ret, disc, val,
                                    next_obs=next_obs, stream=outs.pop("stream", None), **outs)
        return idx, w, nxt, ret, disc, val

    def read(self, col, dst, offset=0, level=0, stream=None):
        conduit_buffer_read(self.handle, col, dst, offset, level, stream)

    def checkpoint(self, dst=None, pin=True, stream=None):
        """The buffer's checkpoint image: written into `dst` if given, else into a
        new host tensor (pinned unless pin=False).  Returns the image tensor."""
        if dst is None:
            n = conduit_buffer_checkpoint_bytes(self.handle)
            dst = torch.empty(n, dtype=torch.uint8, pin_memory=pin)
        conduit_buffer_checkpoint(self.handle, dst, stream)
        return dst

    def restore(self, src, stream=None):
        conduit_buffer_restore(self.handle, src, stream)

    def save(self, path, stream=None):
        """Checkpoint image written to a file."""
        img = self.checkpoint(pin=False, stream=stream)
        img.numpy().tofile(path)

    def load(self, path, stream=None):
        """State restored from a file written by save()."""
        img = torch.from_file(path, shared=False, size=os.path.getsize(path), dtype=torch.uint8)
        self.restore(img, stream)

    def sync_check(self, stream=None):
        return conduit_sync_check(self.handle, stream)

    def clear_error(self):
        conduit_clear_error(self.handle)
