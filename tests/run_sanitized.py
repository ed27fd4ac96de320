"""The CPU test suite (-m "not gpu") under AddressSanitizer and
UndefinedBehaviorSanitizer.

Builds the library's sanitizer variant (host code of every source; the device
code is unchanged) and the oracle's (clang, the same sanitizer runtime), then
runs pytest in a child process with that runtime preloaded (Python itself is
not instrumented; leak detection is off because the interpreter keeps its
allocations) and any sanitizer report fatal.  Usage:

    python tests/run_sanitized.py [extra pytest arguments]
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def runtime():
    out = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True, check=True).stdout.strip()
    if not os.path.exists(out):  # the runtime sits beside the compiler's resource directory
        res = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-resource-dir"], capture_output=True, text=True,
                             check=True).stdout.strip()
        out = os.path.join(res, "lib", "linux", "libclang_rt.asan-x86_64.so")
    return out


def main():
    from paper_2304_13541_amd import build as b
    import oracle
    lib = b.build(sanitize=True)
    olib = oracle.build(sanitize=True)
    env = dict(os.environ, DSTACK_LIBRARY=lib, ORACLE_LIBRARY=olib, LD_PRELOAD=runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1:protect_shadow_gap=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-x", "-q", "-m", "not gpu", "-p",
           "no:cacheprovider"] + sys.argv[1:]
    return subprocess.call(cmd, env=env, cwd=ROOT)


if __name__ == "__main__":
    sys.exit(main())
