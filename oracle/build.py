"""Compile the reference oracle (plain C) into oracle/_liboracle.so.

Test infrastructure only: the product library never links it.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "_liboracle.so")


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-Wall", "-Wextra", "-Wno-unused-parameter", SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def build_sanitized(out_dir: str) -> str:
    """The oracle with AddressSanitizer + UndefinedBehaviorSanitizer (same
    floating-point flags), into out_dir/_liboracle_san.so."""
    os.makedirs(out_dir, exist_ok=True)
    out = os.path.join(out_dir, "_liboracle_san.so")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-Wall", "-Wextra", "-Wno-unused-parameter", SRC, "-o", out, "-lm"]
    subprocess.run(cmd, check=True)
    return out


def sanitizer_runtimes() -> str:
    """The gcc ASan and UBSan runtimes, as an LD_PRELOAD list."""
    libs = [subprocess.run(["gcc", f"-print-file-name={n}"], capture_output=True, text=True).stdout.strip()
            for n in ("libasan.so", "libubsan.so")]
    return ":".join(libs)


if __name__ == "__main__":
    print(build(verbose=True))
