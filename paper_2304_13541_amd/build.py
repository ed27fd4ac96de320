"""Build libdstack.so in-tree with hipcc for gfx950.

Every HIP / C++ source under csrc/ is compiled to an object in _build/ (in
parallel), then linked into paper_2304_13541_amd/libdstack.so.  All device
code is built with packed-FP32 instructions disabled.  The weight generator
(rng.cpp) and the analytical knee model (knee_model.cpp) are built with
floating-point contraction off so that their fp64 arithmetic rounds exactly
as written.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdstack.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# CPU sanitizer build (host code only; the device code is unchanged):
# AddressSanitizer and UndefinedBehaviorSanitizer on the host pass of every
# source, linked against clang's shared ASan runtime.
SAN_OUT = os.path.join(HERE, "_build_san")
SAN_LIB = os.path.join(HERE, "libdstack_san.so")
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]
SAN_LINK = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-shared-libasan"]

SOURCES = ["conv_igemm.hip", "conv_rgb.hip", "expand_dw.hip", "kernels_misc.hip", "kernels_seq.hip", "kernels_tf.hip", "model.cpp", "rng.cpp", "sched.cpp", "knee_model.cpp", "launcher.cpp", "serve.cpp", "capi.cpp"]
BASE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
PER_FILE = {"rng.cpp": ["-ffp-contract=off"], "knee_model.cpp": ["-ffp-contract=off"]}


def _compile(src, sanitize=False):
    obj = os.path.join(SAN_OUT if sanitize else OUT, src + ".o")
    cmd = [HIPCC] + BASE_FLAGS + PER_FILE.get(src, []) + (SAN_FLAGS if sanitize else []) + \
        ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops' is not a recognized" not in l]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s" % (src, "\n".join(msgs)))
    return obj, msgs


def build(verbose=False, jobs=None, sanitize=False):
    """Compile and link the library; sanitize=True builds the CPU sanitizer
    variant libdstack_san.so instead (load it with DSTACK_LIBRARY)."""
    out_dir, lib = (SAN_OUT, SAN_LIB) if sanitize else (OUT, LIB)
    os.makedirs(out_dir, exist_ok=True)
    jobs = jobs or min(8, os.cpu_count() or 4)
    with cf.ThreadPoolExecutor(jobs) as ex:
        results = list(ex.map(lambda src: _compile(src, sanitize), SOURCES))
    objs = [o for o, _ in results]
    if verbose:
        for _, msgs in results:
            for l in msgs:
                print(l)
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + (SAN_LINK if sanitize else []) + ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
