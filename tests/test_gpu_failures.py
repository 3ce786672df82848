"""Failure handling that the host can force without faulting the GPU: a buffer
larger than the device (ENOMEM, nothing left behind), exhaustion and reuse of
the per-buffer error-flag slots, and a caller-owned arena (too small or
misaligned: EINVAL; the right size: the buffer lives in it, the same samples
and columns as a library-allocated buffer, and destroy leaves it to the
caller)."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import buffer_columns, dev, host

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


def test_buffer_larger_than_the_device_is_enomem():
    print("failures: an 8.8 TB buffer", flush=True)
    with pytest.raises(cd.ConduitError) as e:
        cd.ReplayBuffer((1 << 31) - 1, (4096,), torch.uint8)
    assert e.value.status == cd.ENOMEM
    assert "hipMalloc" in str(e.value)
    # nothing was left behind: buffers are created and used as before
    buf = cd.ReplayBuffer(64, (8,), torch.uint8)
    buf.ingest(torch.ones((16, 8), dtype=torch.uint8, device="cuda"))
    idx, _ = buf.sample(dev(synth.uniforms(np.random.default_rng(1), 4)))
    assert buf.sync_check() == cd.OK and np.all((host(idx) >= 0) & (host(idx) < 16))
    buf.close()


def test_error_flag_slots_are_exhausted_and_reused():
    print("failures: live buffers until the slots run out, then reuse", flush=True)
    import gc
    gc.collect()  # buffers other tests dropped without closing
    live = []
    try:
        with pytest.raises(cd.ConduitError) as e:
            for _ in range(600):
                live.append(cd.ReplayBuffer(16, (4,), torch.uint8))
        assert e.value.status == cd.ENOMEM and "too many live buffers" in str(e.value)
        assert 0 < len(live) <= 511  # 512 slots, slot 0 kept for the stand-alone calls
    finally:
        for b in live:
            b.close()
    again = [cd.ReplayBuffer(16, (4,), torch.uint8) for _ in range(8)]  # released slots are reused
    for b in again:
        assert b.sync_check() == cd.OK
        b.close()


def test_caller_owned_arena():
    print("failures: caller-owned arena", flush=True)
    opts = cd.default_opts(frame_stack=2)
    need = cd.conduit_buffer_required_bytes(300, (4, 4), cd.U8, opts)
    assert need > 0
    small = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(cd.ConduitError) as e:
        cd.ReplayBuffer(300, (4, 4), torch.uint8, frame_stack=2, arena=small)
    assert e.value.status == cd.EINVAL
    big = torch.empty(need + 512, dtype=torch.uint8, device="cuda")
    with pytest.raises(cd.ConduitError) as e:
        cd.ReplayBuffer(300, (4, 4), torch.uint8, frame_stack=2, arena=big[1:])  # not 256-byte aligned
    assert e.value.status == cd.EINVAL
    arena = torch.full((need,), 0xAB, dtype=torch.uint8, device="cuda")
    a = cd.ReplayBuffer(300, (4, 4), torch.uint8, frame_stack=2, arena=arena)
    b = cd.ReplayBuffer(300, (4, 4), torch.uint8, frame_stack=2)
    rng = np.random.default_rng(4)
    obs = dev(rng.integers(0, 256, (250, 4, 4), dtype=np.uint8))
    prio = dev(rng.integers(1, 1000, 250, dtype=np.uint32))
    ep, st = dev(np.arange(250, dtype=np.uint32) // 10), dev(np.arange(250, dtype=np.int32) % 10)
    for buf in (a, b):
        buf.ingest(obs, prio=prio, episode_id=ep, step=st)
    u = dev(synth.uniforms(rng, 64))
    (ia, wa), (ib, wb) = a.sample(u), b.sample(u)
    assert np.array_equal(host(ia), host(ib)) and np.array_equal(host(wa), host(wb))
    # every column equal; the payload columns over the written slots (the rest
    # of an arena keeps whatever the caller's memory held: those slots are
    # never sampled or gathered)
    ca, cb = buffer_columns(a), buffer_columns(b)
    written = {cd.COL_OBS: 250 * 16, cd.COL_ACTION: 250 * 4, cd.COL_REWARD: 250 * 4, cd.COL_DONE: 250}
    for k in ca:
        n = written.get(k[0]) if isinstance(k, tuple) else None
        assert np.array_equal(ca[k][:n], cb[k][:n]), k
    a.close()
    b.close()
    assert arena.sum().item() > 0  # the caller's memory is still there to read after destroy
