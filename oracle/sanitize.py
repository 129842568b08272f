"""Run the CPU test suite against AddressSanitizer + UndefinedBehaviorSanitizer
builds of the oracle (ucref.cpp), the input generator (ucgen.c) and the HIP
library's host code (argument validation, planning, accounting and budget
helpers) -- TEST INFRASTRUCTURE.

    python oracle/sanitize.py [pytest args...]

The sanitized libraries go to _build/sanitize/; the test process preloads
clang's sanitizer runtime and stops at the first report.  CPU only: nothing
here launches a kernel."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)


def main(argv):
    import importlib.util

    from oracle import build as obuild
    from workloads import build as gbuild
    spec = importlib.util.spec_from_file_location(
        "_uc_build", os.path.join(ROOT, "paper_2609_32831_amd", "build.py"))
    lbuild = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(lbuild)
    env = dict(os.environ)
    env["UCREF_LIB"] = obuild.build(sanitize=True)
    env["UCGEN_LIB"] = gbuild.build(sanitize=True)
    env["UNICACHE_LIB"] = lbuild.build(sanitize=True)
    rt = subprocess.run([obuild.CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"],
                        capture_output=True, text=True, check=True).stdout.strip()
    # the sanitizer runtime must come first; anything already preloaded stays
    env["LD_PRELOAD"] = ":".join(p for p in (rt, env.get("LD_PRELOAD", "")) if p)
    # the interpreter itself is not instrumented: leak checking would report
    # its own allocations
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = env.get("OMP_NUM_THREADS", "4")
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-m", "not gpu", "-q",
           "-p", "no:cacheprovider"] + argv
    print("sanitized libraries:", env["UCREF_LIB"], env["UCGEN_LIB"], env["UNICACHE_LIB"],
          flush=True)
    return subprocess.run(cmd, env=env).returncode


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
