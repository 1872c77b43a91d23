"""The host-side test tier against the sanitized test build of the library.

Builds ``lib/libarplan_check_san.so`` (``build.build_sanitized``: the test
library with its host code -- plan expansion, the C ABI, the executor's
rewrites, launch planning, resident programs, GenModel and the checking
hooks -- under AddressSanitizer and UndefinedBehaviorSanitizer, any
undefined behaviour fatal), then runs the host test files that drive that
code, through ``tests/checklib.py`` and, via ``ARPLAN_LIB``, the product
binding, with the sanitizer runtime preloaded.  Exits
with pytest's status.  No GPU is used.

    python tests/sanitized_host_suite.py [extra pytest arguments]
"""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2409_04202_amd import build  # noqa: E402

HOST_FILES = ["tests/test_capi_host.py", "tests/test_exec_rewrites_host.py",
              "tests/test_resident_host.py", "tests/test_genmodel_host.py"]


def main(argv):
    lib = build.build_sanitized()
    env = dict(os.environ)
    env["LD_PRELOAD"] = " ".join(x for x in (build.sanitizer_runtime(),
                                             env.get("LD_PRELOAD", "")) if x)
    env["ARPLAN_TEST_LIB"] = lib
    env["ARPLAN_LIB"] = lib          # the product binding too (GenModel tests)
    # the interpreter and torch are not instrumented and keep memory until
    # exit: leak reports would be theirs
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider"]
    # the test of the product's exact export list does not apply to the test
    # build, which adds the checking hooks
    cmd += ["-k", "not exports_every_declared"]
    cmd += [os.path.join(ROOT, f) for f in HOST_FILES] + list(argv)
    print("sanitized host suite: %s" % lib, flush=True)
    return subprocess.call(cmd, env=env, cwd=ROOT)


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
