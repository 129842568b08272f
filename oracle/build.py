"""Build the CPU oracle libucref.so with g++ (test infrastructure).

build(sanitize=True) builds an AddressSanitizer + UndefinedBehaviorSanitizer
copy with clang (the runtime the HIP library's sanitized host code uses)
under _build/sanitize/ for oracle/sanitize.py."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libucref.so")
SAN_DIR = os.path.join(ROOT, "_build", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-shared-libsan"]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    lib = os.path.join(SAN_DIR, "libucref.so") if sanitize else LIB
    os.makedirs(os.path.dirname(lib), exist_ok=True)
    cc, opt = (CLANG, SAN_FLAGS) if sanitize else ("g++", ["-O2"])
    cmd = [cc] + opt + ["-std=c++17", "-fPIC", "-shared", "-fopenmp",
                        "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
                        os.path.join(HERE, "ucref.cpp"), "-o", lib + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv)
    sys.exit(0)
