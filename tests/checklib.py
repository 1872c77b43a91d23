"""The C-ABI binding bound to the test build of the library,
``lib/libarplan_check.so``: the product's code plus the checking hooks of
``csrc/ar_debug.h`` (executed steps, tile coverage, resident programs).

``arplan`` here is a second instance of ``paper_2409_04202_amd.arplan``
whose functions call the test build, so a plan created through it can be
handed to the hooks (``arplan._lib.ar_debug_*``).  The product library,
``lib/libarplan.so``, exports no hook.

``ARPLAN_TEST_LIB`` names another build of the same test library (the
sanitized host-only build) to bind instead.
"""

import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2409_04202_amd")
CHECK_LIB = os.environ.get("ARPLAN_TEST_LIB") or os.path.join(
    PKG, "lib", "libarplan_check.so")


def _load():
    if not os.path.exists(CHECK_LIB):
        raise ImportError("test library not built (%s); run "
                          "`python -m paper_2409_04202_amd.build`" % CHECK_LIB)
    spec = importlib.util.spec_from_file_location(
        "paper_2409_04202_amd.arplan_check", os.path.join(PKG, "arplan.py"))
    mod = importlib.util.module_from_spec(spec)
    mod._LIB_PATH = CHECK_LIB
    spec.loader.exec_module(mod)
    return mod


arplan = _load()
