"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer,
on the CPU: api.hip (argument checks, layouts, checkpoint headers), sched.hip
(the scheduling cost model) and place.hip (the placement algorithm) are built
with both sanitizers and linked with the regular build's kernel objects; a child
Python with the sanitizer runtime preloaded drives every host-only path
(host_sanitizer_checks.py).  Any sanitizer report fails the test."""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHECKS = os.path.join(ROOT, "tests", "host_sanitizer_checks.py")


def _build_module():
    spec = importlib.util.spec_from_file_location("conduit_build", os.path.join(ROOT, "paper_2609_24456_amd",
                                                                                "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_host_code_under_sanitizers(tmp_path):
    build = _build_module()
    try:
        lib = build.build_host_sanitized(str(tmp_path))
    except FileNotFoundError as e:  # the regular build has not run in this tree
        pytest.skip(str(e))
    runtime = build.sanitizer_runtime()
    assert os.path.exists(runtime), runtime
    pre = os.environ.get("LD_PRELOAD", "")
    env = dict(os.environ, LD_PRELOAD=runtime + (":" + pre if pre else ""), ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, CHECKS, lib], env=env, capture_output=True, text=True, timeout=300)
    report = r.stdout[-2000:] + r.stderr[-6000:]
    assert r.returncode == 0, report
    assert "host checks ok" in r.stdout, report
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, report
