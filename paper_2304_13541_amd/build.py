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

SOURCES = ["conv_igemm.hip", "conv_rgb.hip", "expand_dw.hip", "kernels_misc.hip", "kernels_seq.hip", "kernels_tf.hip", "model.cpp", "rng.cpp", "sched.cpp", "knee_model.cpp", "launcher.cpp", "serve.cpp", "capi.cpp"]
BASE_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
PER_FILE = {"rng.cpp": ["-ffp-contract=off"], "knee_model.cpp": ["-ffp-contract=off"]}


def _compile(src):
    obj = os.path.join(OUT, src + ".o")
    cmd = [HIPCC] + BASE_FLAGS + PER_FILE.get(src, []) + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops' is not a recognized" not in l]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s" % (src, "\n".join(msgs)))
    return obj, msgs


def build(verbose=False, jobs=None):
    os.makedirs(OUT, exist_ok=True)
    jobs = jobs or min(8, os.cpu_count() or 4)
    with cf.ThreadPoolExecutor(jobs) as ex:
        results = list(ex.map(_compile, SOURCES))
    objs = [o for o, _ in results]
    if verbose:
        for _, msgs in results:
            for l in msgs:
                print(l)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
