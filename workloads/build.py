"""Build libucgen.so (the seeded input generator) with gcc.

build(sanitize=True) builds an AddressSanitizer + UndefinedBehaviorSanitizer
copy with clang under _build/sanitize/ (used by oracle/sanitize.py)."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libucgen.so")
SAN_DIR = os.path.join(ROOT, "_build", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang"
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-shared-libsan"]


def build(verbose: bool = False, sanitize: bool = False) -> str:
    lib = os.path.join(SAN_DIR, "libucgen.so") if sanitize else LIB
    os.makedirs(os.path.dirname(lib), exist_ok=True)
    cc, opt = (CLANG, SAN_FLAGS) if sanitize else ("gcc", ["-O2"])
    cmd = [cc] + opt + ["-std=c11", "-fPIC", "-shared", "-fopenmp",
                        "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
                        os.path.join(HERE, "ucgen.c"), "-o", lib + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    build(verbose=True, sanitize="--sanitize" in sys.argv)
    sys.exit(0)
