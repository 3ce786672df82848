"""Generated device code of every kernel of the library: no private (scratch)
memory, no dynamic stack and no packed fp32 arithmetic.

Each HIP source is compiled to gfx950 assembly with the library's own flags
(hipcc cross-compiles without a GPU) and the code-object metadata of every
kernel is read.  A struct passed by address into a non-inlined function, an
array indexed at run time or a deep call chain would show up here as a
non-zero private segment: memory traffic on the latency-bound paths."""
import concurrent.futures as cf
import os
import re
import subprocess
import tempfile

import pytest

from paper_2609_24456_amd import build as B

pytestmark = pytest.mark.skipif(not os.path.exists(B.HIPCC), reason="hipcc not installed")


def _device_asm(src, out_dir):
    out = os.path.join(out_dir, src + ".s")
    cmd = [B.HIPCC] + B.FLAGS + ["-S", "--cuda-device-only", os.path.join(B.CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"hipcc -S failed for {src}:\n{r.stderr[-2000:]}"
    with open(out) as f:
        return f.read()


def _kernels(asm):
    """(name, private_segment_fixed_size, uses_dynamic_stack) of every kernel in
    the code-object metadata (keys of one kernel appear in sorted order)."""
    out, name, priv = [], None, None
    for line in asm.splitlines():
        s = line.strip()
        if s.startswith(".name:"):
            name = s.split(":", 1)[1].strip()
        elif s.startswith(".private_segment_fixed_size:") and name:
            priv = int(s.split(":", 1)[1])
        elif s.startswith(".uses_dynamic_stack:") and name:
            out.append((name, priv, s.split(":", 1)[1].strip() == "true"))
            name, priv = None, None
    return out


@pytest.fixture(scope="module")
def asm_by_source():
    with tempfile.TemporaryDirectory() as d:
        with cf.ThreadPoolExecutor(max_workers=8) as ex:
            texts = list(ex.map(lambda s: _device_asm(s, d), B.SOURCES))
    return dict(zip(B.SOURCES, texts))


def test_every_kernel_uses_no_scratch(asm_by_source):
    found = 0
    for src, asm in asm_by_source.items():
        for name, priv, dyn in _kernels(asm):
            found += 1
            assert priv == 0, f"{src}: {name} uses {priv} bytes of private memory per lane"
            assert not dyn, f"{src}: {name} uses a dynamic stack"
    # every kernel source contributes at least one kernel
    with_kernels = [s for s, a in asm_by_source.items() if _kernels(a)]
    assert len(with_kernels) >= 9, with_kernels
    assert found >= 20, found


def test_no_packed_fp32_arithmetic(asm_by_source):
    pat = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")
    for src, asm in asm_by_source.items():
        m = pat.search(asm)
        assert m is None, f"{src}: packed fp32 instruction {m.group(0)}"
