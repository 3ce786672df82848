"""The Python binding checks dtypes and sizes before anything reaches the
library (no GPU needed): an undersized or mistyped tensor raises here instead
of becoming an out-of-bounds device access.  CPU tensors stand in for device
ones (the device check is switched off for these cases, and every case fails
before the library is called); one case shows the device check itself."""
import pytest
import torch

from paper_2609_24456_amd import conduit as cd


def _geometry(**kw):
    info = cd.BufferInfo()
    info.capacity, info.row_bytes, info.size = 1000, 7056, 1000
    info.frame_stack, info.action_bytes, info.ragged, info.max_len = 4, 4, 0, 0
    info.prioritized, info.obs_dtype, info.aux_elem_bytes = 1, cd.U8, 0
    for k, v in kw.items():
        setattr(info, k, v)
    return info


class _NoLibrary:
    """Stands in for the loaded library: any entry point called fails the test."""

    def __getattr__(self, name):
        def call(*args):
            pytest.fail(f"{name} was called although an argument check should have raised")
        return call


@pytest.fixture
def host_tensors(monkeypatch):
    monkeypatch.setattr(cd, "_on_device", lambda t: True)
    monkeypatch.setattr(cd, "lib", lambda: _NoLibrary())


@pytest.fixture
def dense(monkeypatch, host_tensors):
    monkeypatch.setattr(cd, "_info", lambda handle: _geometry())


@pytest.fixture
def ragged(monkeypatch, host_tensors):
    monkeypatch.setattr(cd, "_info", lambda handle: _geometry(row_bytes=4096 * 4, frame_stack=1, ragged=1,
                                                              max_len=4096, aux_elem_bytes=4, obs_dtype=cd.I32))


def z(*shape, dtype=torch.uint8):
    return torch.zeros(shape, dtype=dtype)


def test_ingest_checks(dense):
    with pytest.raises(ValueError, match="obs holds"):
        cd.conduit_ingest(1, 8, z(7, 7056))
    with pytest.raises(ValueError, match="reward"):
        cd.conduit_ingest(1, 8, z(8, 7056), reward=z(7, dtype=torch.float32))
    with pytest.raises(TypeError, match="prio"):
        cd.conduit_ingest(1, 8, z(8, 7056), prio=z(8, dtype=torch.float32))
    with pytest.raises(ValueError, match="action"):
        cd.conduit_ingest(1, 8, z(8, 7056), action=z(8, 3))
    with pytest.raises(TypeError, match="step"):
        cd.conduit_ingest(1, 8, z(8, 7056), step=z(8, dtype=torch.int64))
    with pytest.raises(ValueError, match="n must be"):
        cd.conduit_ingest(1, -1, z(8, 7056))


def test_host_tensors_are_refused(monkeypatch):
    monkeypatch.setattr(cd, "_info", lambda handle: _geometry())
    with pytest.raises(ValueError, match="HIP device"):
        cd.conduit_ingest(1, 8, z(8, 7056), reward=z(8, dtype=torch.float32))


def test_ragged_ingest_checks(ragged):
    tok = z(100, dtype=torch.int32)
    with pytest.raises(ValueError, match="offsets holds"):
        cd.conduit_ingest(1, 4, tok, offsets=z(4, dtype=torch.int64))
    with pytest.raises(TypeError, match="offsets"):
        cd.conduit_ingest(1, 4, tok, offsets=z(5, dtype=torch.int32))
    with pytest.raises(TypeError, match="obs"):
        cd.conduit_ingest(1, 4, z(100, dtype=torch.int64), offsets=z(5, dtype=torch.int64))
    with pytest.raises(TypeError, match="aux"):
        cd.conduit_ingest(1, 4, tok, offsets=z(5, dtype=torch.int64), aux=z(100, dtype=torch.float64))


def test_update_and_sample_checks(dense):
    with pytest.raises(TypeError, match="prio"):
        cd.conduit_update_priorities(1, z(4, dtype=torch.int64), z(4, dtype=torch.float32))
    with pytest.raises(ValueError, match="same length"):
        cd.conduit_update_priorities(1, z(4, dtype=torch.int64), z(3, dtype=torch.int32))
    with pytest.raises(TypeError, match="idx"):
        cd.conduit_update_priorities(1, z(4, dtype=torch.int32), z(4, dtype=torch.int32))
    with pytest.raises(TypeError, match="uniforms"):
        cd.conduit_sample(1, 4, z(4, dtype=torch.int32), z(4, dtype=torch.int64))
    with pytest.raises(TypeError, match="uniforms"):
        cd.conduit_sample(1, 4, z(4, dtype=torch.float64), z(4, dtype=torch.int64))
    with pytest.raises(ValueError, match="uniforms holds"):
        cd.conduit_sample(1, 4, z(3, dtype=torch.int64), z(4, dtype=torch.int64))
    with pytest.raises(ValueError, match="idx_out"):
        cd.conduit_sample(1, 4, z(4, dtype=torch.int64), z(3, dtype=torch.int64))
    with pytest.raises(ValueError, match="is_w_out"):
        cd.conduit_sample(1, 4, z(4, dtype=torch.int64), z(4, dtype=torch.int64), z(3, dtype=torch.float32))


def test_gather_checks(dense):
    idx = z(8, dtype=torch.int64)
    f32 = cd.transform(cd.XF_U8_F32)
    # a K = 4 stack of 7,056-byte frames to fp32 writes 112,896 bytes per sample
    with pytest.raises(ValueError, match="obs holds"):
        cd.conduit_gather_transform(1, idx, f32, obs=z(8, 4, 84, 84, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="obs holds"):
        cd.conduit_gather_transform(1, idx, cd.transform(cd.XF_NONE), obs=z(8, 3, 7056))
    with pytest.raises(ValueError, match="done"):
        cd.conduit_gather_transform(1, idx, f32, obs=z(8, 4, 84, 84, dtype=torch.float32), done=z(7))
    with pytest.raises(ValueError, match="dense buffers"):
        cd.conduit_gather_transform(1, idx, cd.transform(cd.XF_TOKENS_PAD), obs=z(8, 4, 7056))
    with pytest.raises(ValueError, match="obs holds"):
        cd.conduit_sample_gather(1, 8, z(8, dtype=torch.int64), z(8, dtype=torch.int64), z(8, dtype=torch.float32),
                                 f32, obs=z(8, 4, 7056))
    with pytest.raises(ValueError, match="next_obs"):
        cd.conduit_nstep(1, idx, 3, 0.99, z(8, dtype=torch.int64), z(8, dtype=torch.float32),
                         z(8, dtype=torch.float32), z(8), f32, z(8, 4, 7056))
    with pytest.raises(ValueError, match="ret"):
        cd.conduit_nstep(1, idx, 3, 0.99, z(8, dtype=torch.int64), z(7, dtype=torch.float32),
                         z(8, dtype=torch.float32), z(8))


def test_ragged_gather_checks(ragged):
    idx = z(2, dtype=torch.int64)
    xf = cd.transform(cd.XF_TOKENS_PAD)
    with pytest.raises(ValueError, match="obs holds"):
        cd.conduit_gather_transform(1, idx, xf, obs=z(2, 4095, dtype=torch.int32))
    with pytest.raises(ValueError, match="mask holds"):
        cd.conduit_gather_transform(1, idx, xf, obs=z(2, 4096, dtype=torch.int32), mask=z(2, 4000))
    with pytest.raises(ValueError, match="length"):
        cd.conduit_gather_transform(1, idx, xf, obs=z(2, 4096, dtype=torch.int32), length=z(1, dtype=torch.int32))


def test_gae_checks(host_tensors):
    r = z(16, 8, dtype=torch.float32)
    d = z(16, 8)
    ok = z(16, 8, dtype=torch.float32)
    with pytest.raises(ValueError, match="adv"):
        cd.conduit_gae(r, None, d, None, 0.99, 0.95, z(16, 7, dtype=torch.float32), ok)
    with pytest.raises(TypeError, match="dones"):
        cd.conduit_gae(r, None, z(16, 8, dtype=torch.float32), None, 0.99, 0.95, ok, ok)
    with pytest.raises(ValueError, match="bootstrap"):
        cd.conduit_gae(r, None, d, z(7, dtype=torch.float32), 0.99, 0.95, ok, ok)
    with pytest.raises(ValueError, match="values"):
        cd.conduit_gae(r, z(100, dtype=torch.float32), d, None, 0.99, 0.95, ok, ok)
    with pytest.raises(ValueError, match=r"\[T, E\]"):
        cd.conduit_gae(z(128, dtype=torch.float32), None, d, None, 0.99, 0.95, ok, ok)
    with pytest.raises(ValueError, match="final_values"):
        cd.conduit_gae_truncated(r, None, d, d, z(8, dtype=torch.float32), None, 0.99, 0.95, ok, ok)
    with pytest.raises(ValueError, match="values"):
        cd.conduit_gae_packed(z(4, dtype=torch.float32), z(4, dtype=torch.int32), z(4, 99, dtype=torch.float32),
                              100, 1.0, 0.95, z(4, 100, dtype=torch.float32), z(4, 100, dtype=torch.float32))
    with pytest.raises(TypeError, match="lengths"):
        cd.conduit_gae_packed(z(4, dtype=torch.float32), z(4, dtype=torch.int64), None, 100, 1.0, 0.95,
                              z(4, 100, dtype=torch.float32), z(4, 100, dtype=torch.float32))


def test_minibatch_checks(host_tensors):
    f32 = cd.transform(cd.XF_U8_F32)
    perm = z(10, dtype=torch.int64)
    with pytest.raises(ValueError, match="src holds"):
        cd.conduit_minibatch_gather(z(49, 64), 64, 50, perm, f32, z(10, 64, dtype=torch.float32))
    with pytest.raises(ValueError, match="out holds"):
        cd.conduit_minibatch_gather(z(50, 64), 64, 50, perm, f32, z(10, 64))
    with pytest.raises(ValueError, match="same length"):
        cd.conduit_minibatch_gather(z(50, 64), 64, 50, perm, f32, z(10, 64, dtype=torch.float32),
                                    cols=[z(50, dtype=torch.float32)])
    with pytest.raises(ValueError, match="col holds"):
        cd.conduit_minibatch_gather(z(50, 64), 64, 50, perm, f32, z(10, 64, dtype=torch.float32),
                                    cols=[z(49, dtype=torch.float32)], cols_out=[z(10, dtype=torch.float32)])
    with pytest.raises(ValueError, match="col_out holds"):
        cd.conduit_minibatch_gather(z(50, 64), 64, 50, perm, f32, z(10, 64, dtype=torch.float32),
                                    cols=[z(50, dtype=torch.float32)], cols_out=[z(9, dtype=torch.float32)])
    with pytest.raises(ValueError, match="NONE, U8_F32"):
        cd.conduit_minibatch_gather(z(50, 64), 64, 50, perm, cd.transform(cd.XF_TOKENS_PAD), z(10, 64))


def test_checkpoint_header_parser():
    """ckpt_header reads a header from bytes or a host tensor and refuses
    anything without the magic (the library writes the header; this is the
    binding's reader only)."""
    h = cd.CkptHeader()
    h.magic = cd.CKPT_MAGIC
    h.version, h.capacity, h.head, h.size, h.total, h.n_sections = 1, 1000, 500, 1000, 1500, 2
    h.section[1].column, h.section[1].offset, h.section[1].bytes = cd.COL_MAX_PRIO, 1024, 4
    raw = bytes(h) + bytes(64)
    for img in (raw, torch.frombuffer(bytearray(raw), dtype=torch.uint8)):
        g = cd.ckpt_header(img)
        assert (g.capacity, g.head, g.size, g.total, g.n_sections) == (1000, 500, 1000, 1500, 2)
        assert (g.section[1].column, g.section[1].offset, g.section[1].bytes) == (cd.COL_MAX_PRIO, 1024, 4)
    with pytest.raises(ValueError):
        cd.ckpt_header(b"CNDTCKP")  # shorter than a header
    with pytest.raises(ValueError):
        cd.ckpt_header(b"X" + raw[1:])
