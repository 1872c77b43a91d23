"""Build the HIP library ``lib/libarplan.so`` for gfx950 with hipcc.

Run ``python -m paper_2409_04202_amd.build`` (or ``__graft_entry__.build()``).
The plan library and the C ABI (plan.cpp, capi.cpp) are compiled with the
host compiler; the executor (exec.hip, and its host-side planning in
rewrite.cpp, schedule.cpp and programs.cpp, which share its HIP types) with
``hipcc --offload-arch=gfx950``; hipcc links the shared library.  The
objects are compiled in parallel and always from scratch.

Two libraries are linked from the same objects:

* ``lib/libarplan.so`` -- the product: exactly the functions
  ``include/ar_plan.h`` declares;
* ``lib/libarplan_check.so`` -- for the tests only: the same code plus the
  checking hooks of ``csrc/debug.cpp`` (``csrc/ar_debug.h``), which read a
  plan's executor tables back on the host.  Nothing outside ``tests/``
  loads it.
"""

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libarplan.so")
CHECK_LIB = os.path.join(LIBDIR, "libarplan_check.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HOST_SRCS = ["plan.cpp", "capi.cpp", "genmodel.cpp"]
HIP_SRCS = ["exec.hip", "rewrite.cpp", "schedule.cpp", "programs.cpp"]
CHECK_SRCS = ["debug.cpp"]          # compiled as HIP, linked into the check library only

COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall",
          "-Wextra", "-Wno-unused-parameter"]
# fp32 adds must round exactly as written: no contraction, denormals kept,
# and no packed-fp32 instructions.
HIP_FLAGS = ["--offload-arch=gfx950", "-ffp-contract=off",
             "-fno-gpu-flush-denormals-to-zero",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("build failed: %s\n%s" % (" ".join(cmd), r.stdout))
    if verbose and out.strip():
        print(out)


def build(verbose=False, jobs=None):
    hipcc = os.environ.get("HIPCC", os.path.join(ROCM, "bin", "hipcc"))
    cxx = os.environ.get("CXX", "g++")
    os.makedirs(LIBDIR, exist_ok=True)
    tmp = tempfile.mkdtemp(prefix="arplan_build_")
    try:
        cmds, objs = [], {}
        for s in HOST_SRCS:
            o = os.path.join(tmp, s + ".o")
            cmds.append([cxx, "-c", os.path.join(CSRC, s), "-o", o] + COMMON)
            objs[s] = o
        for s in HIP_SRCS + CHECK_SRCS:
            o = os.path.join(tmp, s + ".o")
            cmds.append([hipcc, "-c", "-x", "hip", os.path.join(CSRC, s), "-o", o]
                        + COMMON + HIP_FLAGS)
            objs[s] = o
        jobs = jobs or min(8, os.cpu_count() or 1)
        with ThreadPoolExecutor(max_workers=jobs) as pool:
            for f in [pool.submit(_run, c, verbose) for c in cmds]:
                f.result()
        product = [objs[s] for s in HOST_SRCS + HIP_SRCS]
        for lib, srcs in ((LIB, product), (CHECK_LIB, product + [objs[s] for s in CHECK_SRCS])):
            tmp_lib = os.path.join(tmp, os.path.basename(lib))
            _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp_lib]
                 + srcs, verbose)
            shutil.move(tmp_lib, lib)   # atomic replace of the loaded file
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return LIB


# The sanitized test build (``build_sanitized``): the test library with its
# host code under AddressSanitizer and UndefinedBehaviorSanitizer (device
# code is compiled as usual and left uninstrumented); any undefined
# behaviour aborts.  Loaded only by ``tests/sanitized_host_suite.py``, with
# the sanitizer runtime of the ROCm compiler preloaded.
SAN_LIB = os.path.join(LIBDIR, "libarplan_check_san.so")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"]
SAN_COMMON = ["-O1", "-g", "-fno-omit-frame-pointer", "-std=c++17", "-fPIC",
              "-fvisibility=hidden"]


def sanitizer_runtime():
    """The ROCm compiler's shared AddressSanitizer runtime (UBSan included)."""
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       stdout=subprocess.PIPE, text=True, check=True)
    path = r.stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("sanitizer runtime not found (%s)" % path)
    return path


def build_sanitized(verbose=False, jobs=None):
    hipcc = os.environ.get("HIPCC", os.path.join(ROCM, "bin", "hipcc"))
    clang = os.path.join(ROCM, "llvm", "bin", "clang++")
    os.makedirs(LIBDIR, exist_ok=True)
    tmp = tempfile.mkdtemp(prefix="arplan_san_")
    host_san = [x for f in SAN for x in ("-Xarch_host", f)]
    try:
        cmds, objs = [], []
        for s in HOST_SRCS:
            o = os.path.join(tmp, s + ".o")
            cmds.append([clang, "-c", os.path.join(CSRC, s), "-o", o] + SAN_COMMON + SAN)
            objs.append(o)
        for s in HIP_SRCS + CHECK_SRCS:
            o = os.path.join(tmp, s + ".o")
            cmds.append([hipcc, "-c", "-x", "hip", os.path.join(CSRC, s), "-o", o]
                        + SAN_COMMON + HIP_FLAGS + host_san)
            objs.append(o)
        jobs = jobs or min(8, os.cpu_count() or 1)
        with ThreadPoolExecutor(max_workers=jobs) as pool:
            for f in [pool.submit(_run, c, verbose) for c in cmds]:
                f.result()
        tmp_lib = os.path.join(tmp, os.path.basename(SAN_LIB))
        _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp_lib]
             + host_san + ["-Xarch_host", "-shared-libasan"] + objs, verbose)
        shutil.move(tmp_lib, SAN_LIB)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitized" in sys.argv:
        print(build_sanitized(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
