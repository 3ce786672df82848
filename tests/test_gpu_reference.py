"""The measurement reference kernel (conduit_expand_reference) against the
definition: every output float is the correctly rounded fp32 quotient x / 255
(numpy's fp32 division), nothing past 4n bytes is written.  Sizes span the
whole-chunk loop (1,024-byte chunks), the tail words and several grid sizes."""
import numpy as np
import pytest
import torch

from gpu_util import dev, host

pytestmark = pytest.mark.gpu

from paper_2609_24456_amd import conduit as cd  # noqa: E402


@pytest.mark.parametrize("n", [4, 1020, 1024, 1028, 3 * 1024 + 8, 257 * 1024 + 12, (1 << 24) + 4, 347 << 20])
def test_expand_reference_matches_definition(n):
    print(f"expand reference n={n}", flush=True)
    rng = np.random.default_rng(n % 1000)
    x = rng.integers(0, 256, n, dtype=np.uint8)
    k = min(n, 256)
    x[:k] = np.arange(k, dtype=np.uint8)  # every byte value (n >= 256)
    src = dev(x)
    dst = torch.full((n + 64,), -7.0, dtype=torch.float32, device="cuda")
    cd.conduit_expand_reference(src, dst)
    torch.cuda.synchronize()
    got = host(dst)
    want = x.astype(np.float32) / np.float32(255.0)
    assert np.array_equal(got[:n].view(np.uint32), want.view(np.uint32))
    assert np.all(got[n:] == -7.0)
