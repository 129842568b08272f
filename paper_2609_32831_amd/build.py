"""Build libunicache.so (HIP kernels + C ABI) for gfx950 with hipcc.

Each .hip translation unit is compiled to an object under _build/ and the
objects are linked into paper_2609_32831_amd/libunicache.so.  Packed FP32
instructions are disabled for all device code.
"""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libunicache.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-munsafe-fp-atomics", "-Wall", "-Wno-unused-function",
         "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def source_digest() -> str:
    """SHA-256 over the library's sources (kernels, host code, public header);
    measurements taken on one build are only reused while this is unchanged."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.h")))
    files.append(os.path.join(ROOT, "include", "unicache.h"))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# host code only: the device code of a sanitized build is the ordinary one
SAN_HOST = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host",
            "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
SAN_DIR = os.path.join(BUILD, "sanitize")


def _compile(src: str, verbose: bool, sanitize: bool = False) -> str:
    obj = os.path.join(SAN_DIR if sanitize else BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + (SAN_HOST if sanitize else []) + ["-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    if verbose and r.stderr.strip():
        print(r.stderr, flush=True)
    return obj


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """sanitize: AddressSanitizer + UndefinedBehaviorSanitizer on the host
    code (argument validation, planning), into _build/sanitize/ (for the CPU
    tests under oracle/sanitize.py; never run on a GPU)."""
    os.makedirs(SAN_DIR if sanitize else BUILD, exist_ok=True)
    lib = os.path.join(SAN_DIR, "libunicache.so") if sanitize else LIB
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, sanitize), srcs))
    link = ["-shared-libsan", "-Xarch_host", "-fsanitize=address,undefined"] if sanitize else []
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + link + ["-o", lib + ".tmp"] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv)
    print("built", LIB)
