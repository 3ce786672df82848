"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer:
the oracle pins (test_oracle_pins.py) run again in a child pytest against a
sanitized build of oracle.c, with gcc's sanitizer runtimes preloaded.  The
oracle decides every parity claim, so a memory error or undefined behaviour in
it must show here rather than as a silently wrong expected value."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_pins_under_sanitizers(tmp_path):
    spec = importlib.util.spec_from_file_location("oracle_build", os.path.join(ROOT, "oracle", "build.py"))
    build = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(build)
    lib = build.build_sanitized(str(tmp_path))
    pre = os.environ.get("LD_PRELOAD", "")
    env = dict(os.environ, ORACLE_LIB=lib, LD_PRELOAD=build.sanitizer_runtimes() + (":" + pre if pre else ""),
               ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"), "-q",
                        "-x", "-p", "no:cacheprovider", "-m", "not gpu"], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    report = r.stdout[-3000:] + r.stderr[-6000:]
    assert r.returncode == 0, report
    assert " passed" in r.stdout, report
    assert "runtime error" not in r.stdout + r.stderr and "AddressSanitizer" not in r.stdout + r.stderr, report
