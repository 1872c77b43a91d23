"""Host-side checks of bench.py: the multi-GPU refusal and the thread-pool
form of the oracle used for the parallel CPU baseline."""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from paper_2409_04202_amd import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("name,N", [("ring_n4_f32", None), ("ring_n4_i32", None),
                                    ("tree8x8_n64_f32", 4096 + 64),
                                    ("tree8x8x8_n512_bf16", 2048 + 512),
                                    ("cdc384_gentree_f32", 384 * 3 + 1)])
def test_parallel_oracle_equals_oracle(name, N):
    c = workloads.CONFIGS[name]
    N = c["N"] if N is None else N
    if c["kind"] == "gentree":
        plan = oracle.gentree_plan(oracle.from_preorder(c["fanin"]), N)
    else:
        plan = oracle.make_plan(c["kind"], c["n"], N, c["fanin"])
    xs = workloads.inputs(name, N=N)
    want = oracle.execute(plan, [x.copy() for x in xs], c["dtype"])
    with ThreadPoolExecutor(max_workers=4) as pool:
        got = bench.parallel_execute(plan, [x.copy() for x in xs], c["dtype"], pool)
    for q in range(len(xs)):
        assert np.array_equal(got[q], want[q])


def test_kernel_source_hash_ignores_comments_only():
    # the hash that ties the committed traffic counters to the kernel code
    # changes with code, not with comments or layout
    a = "int f(int x) {  // twice\n    return 2 * x; /* doubled */\n}\n"
    b = "// header\nint f(int x) {\n  return 2 * x;\n}\n"
    c = "int f(int x) {\n    return 3 * x;\n}\n"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)
    # the stripping assumes no string literal holds a comment marker
    csrc = os.path.join(ROOT, "paper_2409_04202_amd", "csrc")
    for f in ("kernels.hpp", "resident.hpp", "exec.hip", "exec_state.hpp", "rewrite.cpp",
              "schedule.cpp", "programs.cpp"):
        for line in open(os.path.join(csrc, f)):
            code = line.split("//")[0]
            for lit in code.split('"')[1::2]:
                assert "//" not in lit and "/*" not in lit, (f, line)
