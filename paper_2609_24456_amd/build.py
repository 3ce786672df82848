"""Compile the HIP sources of libconduit for gfx950 into paper_2609_24456_amd/libconduit.so."""
import concurrent.futures as cf
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libconduit.so")
SOURCES = ["api.hip", "k_ingest.hip", "k_update.hip", "k_sample.hip", "k_gather.hip", "k_sample_gather.hip",
           "k_gae.hip", "sched.hip", "loop.hip", "place.hip", "k_nstep.hip", "k_update_ingest.hip",
           "k_reference.hip"]
ARCH = os.environ.get("CONDUIT_OFFLOAD_ARCH", "gfx950")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
         # no packed-fp32 instructions anywhere in the device code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC]


def _compile(src, verbose):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + FLAGS + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", LIB + ".tmp"] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(LIB + ".tmp", LIB)
    return LIB


# The ABI's host code (api.hip: argument checks, layouts, ring state,
# checkpoint images; sched.hip: the scheduling cost model; place.hip: the
# placement algorithm) built with AddressSanitizer and UndefinedBehaviorSanitizer,
# linked with the kernel sources' objects of the regular build (_build/, whose
# host parts are only the launchers).  These three sources hold no kernels, so
# they compile for the host alone; the result runs the ABI's host paths under
# the sanitizers on a machine with no GPU.
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
HOST_SOURCES = ["api.hip", "sched.hip", "place.hip"]


def build_host_sanitized(out_dir: str, verbose: bool = False) -> str:
    """libconduit with its host-only sources sanitized, into out_dir/libconduit_host_san.so
    (needs the regular build's objects in _build/)."""
    os.makedirs(out_dir, exist_ok=True)
    flags = [f"--offload-arch={ARCH}", "--offload-host-only", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Wno-unused-result", "-I", INCLUDE, "-I", CSRC] + SANITIZE
    rest = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES if s not in HOST_SOURCES]
    missing = [o for o in rest if not os.path.exists(o)]
    if missing:
        raise FileNotFoundError(f"regular build objects missing (run build() first): {missing[:3]}")

    def one(src):
        obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC] + flags + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc (host, sanitized) failed for {src}:\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=len(HOST_SOURCES)) as ex:
        objs = list(ex.map(one, HOST_SOURCES))
    out = os.path.join(out_dir, "libconduit_host_san.so")
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-shared-libasan"] + SANITIZE + \
        ["-o", out] + objs + rest
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link (host, sanitized) failed:\n{r.stderr}")
    return out


def sanitizer_runtime() -> str:
    """Path of the compiler's shared ASan runtime (to preload into an
    uninstrumented Python)."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()


if __name__ == "__main__":
    print(build(verbose=True))
