"""Helpers shared by the GPU parity tests: host<->device marshalling of the
seeded inputs and the tolerance checks.  No arithmetic of the method here."""
import numpy as np
import torch

_SIGNED = {np.dtype(np.uint64): np.int64, np.dtype(np.uint32): np.int32}


def dev(a, device="cuda"):
    """numpy array -> contiguous CUDA tensor with the same bytes (unsigned
    64/32-bit arrays travel as their signed views)."""
    a = np.ascontiguousarray(a)
    if a.dtype in _SIGNED:
        a = a.view(_SIGNED[a.dtype])
    return torch.from_numpy(a).to(device)


def host(t, dtype=None):
    """CUDA tensor -> numpy array, optionally reinterpreted as ``dtype``."""
    a = t.detach().cpu().contiguous().numpy()
    return a.view(dtype) if dtype is not None else a


def read_col(buf, col, nbytes, dtype, level=0):
    out = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.read(col, out, level=level)
    torch.cuda.synchronize()
    return host(out).view(dtype)


def assert_weights_close(gpu, orc):
    """IS weights: |g - o| <= 1e-5 |o| (both computed in fp64, rounded to fp32)."""
    gpu = np.asarray(gpu, np.float64)
    orc = np.asarray(orc, np.float64)
    bad = np.abs(gpu - orc) > 1e-5 * np.abs(orc)
    assert not bad.any(), (np.flatnonzero(bad)[:10], gpu[bad][:5], orc[bad][:5])


def assert_gae_close(gpu, orc):
    """GAE outputs: |g - o| <= 1e-5 max(|o|, 1) (fp64 inside both, fp32 out)."""
    gpu = np.asarray(gpu, np.float64)
    orc = np.asarray(orc, np.float64)
    bad = np.abs(gpu - orc) > 1e-5 * np.maximum(np.abs(orc), 1.0)
    assert not bad.any(), (np.argwhere(bad)[:10], gpu[bad][:5], orc[bad][:5])


def tree_consistent(buf, cap):
    """Every internal node of the device's 64-ary tree equals the sum of its
    children, and the root equals the sum of the leaves (exact integers)."""
    from paper_2609_24456_amd import conduit as cd
    info = buf.info()
    leaves = read_col(buf, cd.COL_LEAVES, cap * 4, np.uint32).astype(np.uint64)
    below = leaves
    for level in range(1, info.tree_depth + 1):
        n = info.tree_nodes[level]
        nodes = read_col(buf, cd.COL_TREE, n * 8, np.uint64, level=level)
        pad = np.zeros(n * 64, np.uint64)
        pad[:len(below)] = below
        assert np.array_equal(nodes, pad.reshape(n, 64).sum(axis=1, dtype=np.uint64)), level
        below = nodes
    assert len(below) == 1
    assert int(below[0]) == int(leaves.sum(dtype=np.uint64))
    return int(below[0])


def buffer_columns(buf):
    """Every column of a buffer as host bytes, keyed by (column, level), with
    the ring state under "ring"."""
    from paper_2609_24456_amd import conduit as cd
    info = buf.info()
    C = info.capacity
    cols = {(cd.COL_OBS, 0): C * info.row_bytes, (cd.COL_REWARD, 0): C * 4, (cd.COL_DONE, 0): C,
            (cd.COL_EPISODE, 0): C * 4, (cd.COL_STEP, 0): C * 4, (cd.COL_MAX_PRIO, 0): 4}
    if info.action_bytes:
        cols[(cd.COL_ACTION, 0)] = C * info.action_bytes
    if info.ragged:
        cols[(cd.COL_LENGTH, 0)] = C * 4
        if info.aux_elem_bytes:
            cols[(cd.COL_AUX, 0)] = C * info.max_len * info.aux_elem_bytes
    if info.prioritized:
        cols[(cd.COL_LEAVES, 0)] = C * 4
        for level in range(1, info.tree_depth + 1):
            cols[(cd.COL_TREE, level)] = info.tree_nodes[level] * 8
    out = {k: read_col(buf, k[0], n, np.uint8, level=k[1]) for k, n in cols.items()}
    out["ring"] = (info.head, info.size, info.total)
    return out


def image_tensor(buf, via):
    """A tensor to hold the buffer's checkpoint image: in HBM, pinned or pageable host memory."""
    from paper_2609_24456_amd import conduit as cd
    n = cd.conduit_buffer_checkpoint_bytes(buf.handle)
    if via == "device":
        return torch.empty(n, dtype=torch.uint8, device="cuda")
    return torch.empty(n, dtype=torch.uint8, pin_memory=(via == "pinned"))


def swap_through_checkpoint(buf, via, make, tmp_dir=None):
    """Checkpoint `buf` (into HBM, pinned or pageable host memory, or a file),
    restore the image into a new buffer from make(), check that every column,
    tree level and the ring state came across, close `buf` and return the new
    buffer."""
    import os
    before = buffer_columns(buf)
    fresh = make()
    if via == "file":
        path = os.path.join(tmp_dir, "replay.ckpt")
        buf.save(path)
        fresh.load(path)
    else:
        img = buf.checkpoint(dst=image_tensor(buf, via))
        fresh.restore(img)
    after = buffer_columns(fresh)
    assert before.keys() == after.keys()
    for k in before:
        assert np.array_equal(before[k], after[k]), k
    buf.close()
    return fresh
