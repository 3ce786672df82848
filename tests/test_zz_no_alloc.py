"""conduit_gae_noalloc (the GAE entry point that allocates nothing) against
conduit_gae through the C ABI: identical outputs, bit for bit, and both within
the GAE tolerance of the oracle, on calls in a row of decreasing size (the
static table keeps the previous call's contents)."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_gae_close, dev, host

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def _rollout(T, E, seed):
    rng = np.random.default_rng(seed)
    r = rng.standard_normal((T, E)).astype(np.float32)
    v = rng.standard_normal((T, E)).astype(np.float32)
    d = (rng.random((T, E)) < 0.01).astype(np.uint8)
    b = rng.standard_normal(E).astype(np.float32)
    return r, v, d, b


def _call(fn, r, v, d, b, gamma, lam):
    T, E = r.shape
    adv = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
    ret = torch.full((T, E), np.nan, dtype=torch.float32, device="cuda")
    rd, vd, dd, bd = dev(r), dev(v), dev(d), dev(b)
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = fn(rd.data_ptr(), vd.data_ptr(), dd.data_ptr(), bd.data_ptr(), T, E, gamma, lam, adv.data_ptr(),
            ret.data_ptr(), stream)
    assert st == cd.OK, cd.last_error()
    torch.cuda.synchronize()
    return host(adv), host(ret)


# calls in a row, each smaller than the one before: the look-back path with
# 256 tiles, the look-back path with fewer, one tile per 32 environments
# (T <= 64), and the one-environment-per-lane kernel (E not a multiple of 4)
SHAPES = [(2048, 256), (300, 64), (48, 40), (33, 7)]
# one segment needs no table however many tiles it has
WIDE_SHORT = (3, 1 << 17)


def test_noalloc_gae_equals_gae_on_calls_in_a_row():
    L = cd.lib()
    for k, (T, E) in enumerate(SHAPES):
        print(f"gae_noalloc call {k}: T={T} E={E} plan={cd.gae_plan(T, E)}", flush=True)
        r, v, d, b = _rollout(T, E, 40 + k)
        na, nr = _call(L.conduit_gae_noalloc, r, v, d, b, 0.99, 0.95)
        ga, gr = _call(L.conduit_gae, r, v, d, b, 0.99, 0.95)
        assert np.array_equal(na.view(np.uint32), ga.view(np.uint32)), (T, E)
        assert np.array_equal(nr.view(np.uint32), gr.view(np.uint32)), (T, E)
        oa, orr = oracle.gae(r, v, d, b, 0.99, 0.95)
        assert_gae_close(na, oa)
        assert_gae_close(nr, orr)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()


def test_noalloc_gae_one_segment_beyond_the_table():
    T, E = WIDE_SHORT
    print(f"gae_noalloc: T={T} E={E} plan={cd.gae_plan(T, E)}", flush=True)
    r, v, d, b = _rollout(T, E, 7)
    na, nr = _call(cd.lib().conduit_gae_noalloc, r, v, d, b, 0.99, 0.95)
    oa, orr = oracle.gae(r, v, d, b, 0.99, 0.95)
    assert_gae_close(na, oa)
    assert_gae_close(nr, orr)
    assert cd.conduit_sync_check() == cd.OK, cd.last_error()


def test_noalloc_gae_validates_on_the_host():
    L = cd.lib()
    P = C.c_void_p(16)  # never dereferenced: validation fails first
    assert L.conduit_gae_noalloc(P, None, P, None, 4, (1 << 19) + 1, 0.99, 0.95, P, P, None) == cd.EINVAL
    assert L.conduit_gae_noalloc(None, None, None, None, 4, 4, 0.99, 0.95, None, None, None) == cd.EINVAL
    assert L.conduit_gae_noalloc(None, None, None, None, 0, 4, 0.99, 0.95, None, None, None) == cd.OK
