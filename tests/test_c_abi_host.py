"""The C ABI from a plain C99 program (tests/c_abi/host_calls.c), compiled
with the host C compiler against include/ar_plan.h and linked with the
product library: the header is valid C and the calls work without Python
(host only, no GPU)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2409_04202_amd", "lib")


@pytest.mark.skipif(not os.path.exists(os.path.join(LIB, "libarplan.so")),
                    reason="library not built")
def test_c_program_calls_the_abi(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    assert cc, "no C compiler"
    exe = str(tmp_path / "host_calls")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi", "host_calls.c"),
                    "-L", LIB, "-larplan", "-Wl,-rpath," + LIB, "-o", exe], check=True)
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stdout
    assert "0 failures" in r.stdout
