"""Host-side tests of the C-ABI library (no GPU needed).

The library loads, exports every function include/ar_plan.h declares, and
its plan expansion (steps, owners, byte counts) equals the oracle's
independent expansion; bad arguments and hazardous custom plans are
rejected with the documented status codes.  No compute call is made.
"""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from oracle import model

product = pytest.importorskip(
    "paper_2409_04202_amd.arplan",
    reason="HIP library not built (run python -m paper_2409_04202_amd.build)")
# everything below the export test runs on the test build (same code, plus
# the checking hooks)
from checklib import arplan  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ar_plan.h")


def test_library_exports_every_declared_function():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(ar_[a-z_]+)\s*\(", text))
    assert declared, "no declarations found"
    for name in sorted(declared):
        assert hasattr(product._lib, name), name
    assert declared == set(product.EXPORTED)
    # the product exports exactly the declared functions: no test hook
    exported = _exported_functions(product.LIB_PATH)
    assert {f for f in exported if f.startswith("ar_")} == declared
    # the test build adds the hooks and nothing else
    extra = {f for f in _exported_functions(arplan.LIB_PATH) if f.startswith("ar_")} - declared
    assert extra == {"ar_debug_check_tiling", "ar_debug_exec_steps", "ar_debug_resident",
                     "ar_debug_launch_desc"}


def _exported_functions(path):
    """Names of the functions a shared library exports (its dynamic symbol
    table, read with the ELF tools of the host)."""
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", path], check=True,
                         stdout=subprocess.PIPE, text=True).stdout
    return {l.split()[-1] for l in out.splitlines() if len(l.split()) == 3
            and l.split()[1] == "T"}


def _norm(phases):
    return [sorted((op, dst, tuple(srcs), b, e) for op, dst, srcs, b, e in ph)
            for ph in phases]


def _oracle_phases(p):
    return [[(s.op, s.dst, tuple(s.srcs), s.begin, s.end) for s in ph]
            for ph in p.phases]


CASES = []
for _n in (1, 2, 3, 4, 5, 7, 8, 12, 16):
    for _N in sorted({0, 1, _n - 1, _n, 2 * _n + 3, 1000}):
        CASES.append(("ring", _n, _N, None))
        CASES.append(("cps", _n, _N, None))
        CASES.append(("rb", _n, _N, None))
        CASES.append(("rhd", _n, _N, None))
for _fan in ((2, 2), (3, 2), (2, 3), (4, 4), (2, 3, 2), (8, 8), (2, 2, 2, 2),
             (1, 4), (4, 1, 2)):
    for _N in (0, 5, 64, 1001):
        CASES.append(("tree", int(np.prod(_fan)), _N, _fan))


@pytest.mark.parametrize("kind,n,N,fan", CASES)
def test_steps_match_oracle(kind, n, N, fan):
    ref = oracle.make_plan(kind, n, N, fan)
    with arplan.Plan(n, N, "f32", kind, fan) as p:
        assert p.num_phases == len(ref.phases)
        assert _norm(p.phases()) == _norm(_oracle_phases(ref))
        red, cpy = p.bytes()
        assert (red, cpy) == model.algorithmic_bytes(ref, 4)
        for ph in range(p.num_phases):
            op, first, cnt, b = p.phase_info(ph)
            steps = ref.phases[ph]
            assert cnt == len(steps)
            assert op == (arplan.AR_OP_REDUCE if any(s.op == "reduce" for s in steps)
                          else arplan.AR_OP_COPY)
            assert b == sum((len(s.srcs) + 1 if s.op == "reduce" else 2)
                            * (s.end - s.begin) * 4 for s in steps)


@pytest.mark.parametrize("kind,n,fan", [("ring", 5, None), ("ring", 8, None),
                                        ("rhd", 8, None), ("rhd", 6, None), ("cps", 6, None),
                                        ("tree", 12, (3, 4)),
                                        ("tree", 64, (8, 8)),
                                        ("tree", 512, (8, 8, 8))])
def test_owner_is_last_reduce_range(kind, n, fan):
    N = 7 * n + 3
    ref = oracle.make_plan(kind, n, N, fan)
    red = [ph for ph in ref.phases if ph[0].op == "reduce"]
    with arplan.Plan(n, N, "bf16", kind, fan) as p:
        for st in red[-1]:
            assert p.owner(st.dst) == (st.begin, st.end)


@pytest.mark.parametrize("fan", [(8, 8), (2, 3, 4), (8, 8, 8)])
def test_tree_owner_matches_algorithm_1(fan):
    n = int(np.prod(fan))
    N = 3 * n
    root = oracle.symmetric_tree(fan)
    place = oracle.basic_placement(root, n)[id(root)]
    off = oracle.block_bounds(N, n)
    with arplan.Plan(n, N, "i32", "tree", fan) as p:
        for sid, blocks in place.items():
            assert p.owner(sid) == (off[blocks[0]], off[blocks[-1] + 1])


def test_config_shapes():
    # phase and step counts of the benchmark workloads
    shapes = [("ring", 4, 1 << 16, None, 6, 24), ("rhd", 8, 1 << 26, None, 6, 48),
              ("cps", 16, 1 << 24, None, 2, 256), ("tree", 64, 1 << 22, (8, 8), 4, 1024),
              ("tree", 512, 1 << 18, (8, 8, 8), 6, 12288),
              ("ring", 64, 1 << 20, None, 126, 8064)]
    for kind, n, N, fan, nph, nst in shapes:
        with arplan.Plan(n, N, "f32", kind, fan) as p:
            assert (p.num_phases, p.num_steps) == (nph, nst)


def _status(fn, *args):
    try:
        fn(*args)
    except arplan.ArError as e:
        return e.status
    return arplan.AR_OK


def test_create_errors():
    E = arplan
    assert _status(E.ar_plan_create, 0, 10, "f32", "ring") == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 4, -1, "f32", "ring") == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 4, 10, 7, "ring") == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 4, 10, "f32", 9) == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 6, 10, "f32", "rhd") == E.AR_OK
    assert _status(E.ar_plan_create, 6, 10, "f32", "tree", [2, 2]) == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 4, 10, "f32", "tree", [4, 0]) == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 4, 10, "f32", "tree", []) == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 4, 2**62, "f32", "ring") == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create, 40000, 10, "f32", "ring") == E.AR_ERR_UNSUPPORTED
    # NULL out / topo
    lib = arplan._lib
    topo = arplan.ar_topology(arplan.AR_RING, 0, None)
    assert lib.ar_plan_create(4, 10, 0, ctypes.byref(topo), None) == E.AR_ERR_INVALID_ARG
    out = ctypes.c_void_p(123)
    assert lib.ar_plan_create(4, 10, 0, None, ctypes.byref(out)) == E.AR_ERR_INVALID_ARG
    assert out.value is None
    assert "topo" in E.ar_last_error()
    assert lib.ar_plan_destroy(None) == E.AR_OK
    assert E.ar_status_string(E.AR_ERR_HIP) == "AR_ERR_HIP"


def test_execute_argument_errors_need_no_gpu():
    E = arplan
    lib = arplan._lib
    assert lib.ar_plan_execute(None, None, None) == E.AR_ERR_INVALID_ARG
    h = E.ar_plan_create(4, 16, "f32", "ring")
    try:
        assert lib.ar_plan_execute(h, None, None) == E.AR_ERR_INVALID_ARG
        assert lib.ar_plan_execute_strided(h, None, 64, None) == E.AR_ERR_INVALID_ARG
        assert lib.ar_plan_execute_strided(h, 4096, 63, None) == E.AR_ERR_INVALID_ARG
    finally:
        E.ar_plan_destroy(h)
    # empty plans return without touching the GPU
    h = E.ar_plan_create(1, 16, "f32", "ring")
    try:
        E.ar_plan_execute(h, [0x1000])
    finally:
        E.ar_plan_destroy(h)


def test_custom_plan_roundtrip_and_validation():
    E = arplan
    ref = oracle.tree((3, 4), 50)
    steps = [(ph, s.op, s.dst, s.srcs, s.begin, s.end)
             for ph, stp in enumerate(ref.phases) for s in stp]
    h = E.ar_plan_create_custom(12, 50, "f32", reversed(steps))
    try:
        n, N, dt, nph, nst = E.ar_plan_info(h)
        assert (n, N, nph, nst) == (12, 50, 4, len(steps))
        got = [E.ar_plan_get_step(h, i) for i in range(nst)]
        norm = lambda L: sorted((a, b if isinstance(b, int) else
                                 (0 if b == "reduce" else 1), c, tuple(d), e, f)
                                for a, b, c, d, e, f in L)
        assert norm(got) == norm(steps)
        assert _status(E.ar_plan_owner, h, 0) == E.AR_ERR_UNSUPPORTED
    finally:
        E.ar_plan_destroy(h)
    bad = {
        "write/write": [(0, "copy", 1, [0], 0, 6), (0, "copy", 1, [2], 5, 9)],
        "read/write": [(0, "reduce", 1, [0, 1], 0, 4), (0, "copy", 0, [2], 3, 5)],
        "gap": [(0, "copy", 1, [0], 0, 4), (2, "copy", 1, [0], 0, 4)],
        "copy 2 srcs": [(0, "copy", 1, [0, 2], 0, 4)],
        "dst range": [(0, "copy", 3, [0], 0, 4)],
        "src range": [(0, "reduce", 1, [0, 3], 0, 4)],
        "elem range": [(0, "copy", 1, [0], 0, 11)],
        "reversed": [(0, "copy", 1, [0], 5, 4)],
        "no src": [(0, "reduce", 1, [], 0, 4)],
    }
    for name, st in bad.items():
        assert _status(E.ar_plan_create_custom, 3, 10, "f32", st) == \
            E.AR_ERR_INVALID_ARG, name
    # a step may read and write its own range; different phases may overlap
    ok = [(0, "reduce", 1, [0, 1, 2], 0, 10), (1, "copy", 0, [1], 0, 10),
          (1, "copy", 2, [1], 0, 10)]
    E.ar_plan_destroy(E.ar_plan_create_custom(3, 10, "bf16", ok))


def test_timer_host_side():
    E = arplan
    t = E.ar_timer_create(8)
    try:
        assert E.ar_timer_read(t, 8) == []
        E.ar_timer_reset(t)
    finally:
        E.ar_timer_destroy(t)
    assert _status(E.ar_timer_create, 0) == E.AR_ERR_INVALID_ARG


def _check_tiling(handle, vecok):
    f = arplan._lib.ar_debug_check_tiling
    f.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_char_p, ctypes.c_int64]
    f.restype = ctypes.c_int32
    buf = ctypes.create_string_buffer(512)
    st = f(handle, vecok, buf, 512)
    return st, buf.value.decode()


TILING = [("ring", 4, 1 << 16, None), ("rhd", 8, 1 << 26, None),
          ("cps", 16, 1 << 24, None), ("tree", 64, 1 << 22, (8, 8)),
          ("tree", 512, 1 << 18, (8, 8, 8)), ("ring", 64, 1 << 20, None),
          ("ring", 64, 1 << 12, None), ("tree", 64, 1 << 12, (8, 8)),
          ("rhd", 8, (1 << 20) + 13, None), ("cps", 16, (1 << 18) + 7, None),
          ("tree", 512, (1 << 13) + 3, (8, 8, 8)), ("rb", 6, 100003, None),
          ("cps", 5, 50021, None), ("cps", 32, 50021, None),
          ("tree", 12, 4099, (3, 4)), ("ring", 5, 1, None), ("ring", 5, 4, None),
          ("rhd", 4, 3, None), ("tree", 8, 10007, (4, 2)), ("ring", 3, 4099, None)]


@pytest.mark.parametrize("kind,n,N,fan", TILING)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_kernel_tiling_covers_steps_exactly(kind, n, N, fan, dtype):
    h = arplan.ar_plan_create(n, N, dtype, kind, fan)
    try:
        for vecok in (1, 0):
            st, msg = _check_tiling(h, vecok)
            assert st == arplan.AR_OK, msg
    finally:
        arplan.ar_plan_destroy(h)


def test_kernel_tiling_uneven_custom_phase():
    steps = [(0, "reduce", 0, [0, 1, 2], 0, 280000),
             (0, "reduce", 3, [3, 1], 280000, 280007),
             (0, "reduce", 2, [2, 3], 280007, 300001),
             (1, "copy", 1, [0], 0, 280000), (1, "copy", 0, [3], 280000, 280007),
             (1, "copy", 3, [2], 290000, 290001)]
    for dtype in ("f32", "bf16", "i32"):
        h = arplan.ar_plan_create_custom(4, 300001, dtype, steps)
        try:
            for vecok in (1, 0):
                st, msg = _check_tiling(h, vecok)
                assert st == arplan.AR_OK, msg
        finally:
            arplan.ar_plan_destroy(h)


def test_executor_rewrites_launch_structure():
    # (kind, n, N, fan) -> launches with fusion, and the fused byte total
    cases = [
        ("cps", 16, 1 << 20, None, 1),    # reduce + broadcast in one launch
        ("rhd", 8, 1 << 20, None, 3),     # last halving absorbs every doubling
        ("tree", 64, 1 << 16, (8, 8), 2), # RS-L1 absorbs AG-L1, then AG-L0
        ("tree", 512, 1 << 15, (8, 8, 8), 3),
        ("ring", 5, 1000, None, 4),       # the AllGather chain folds into the last reduce
        ("rb", 6, 999, None, 1),
    ]
    for kind, n, N, fan, nl in cases:
        with arplan.Plan(n, N, "f32", kind, fan) as p:
            p.set_option(arplan.AR_OPT_SLICE, 0)
            L = p.launches()
            assert len(L) == nl, (kind, L)
            p.set_option(arplan.AR_OPT_FUSE, 0)
            L0 = p.launches()
            assert len(L0) == p.num_phases
            # unfused launches move exactly the plan's algorithmic bytes
            assert sum(x[4] for x in L0) == sum(p.bytes())
            assert sum(x[4] for x in L) <= sum(x[4] for x in L0)
            for vecok in (1, 0):
                st, msg = _check_tiling(p.handle, vecok)
                assert st == arplan.AR_OK, msg
            p.set_option(arplan.AR_OPT_FUSE, 1)
            for vecok in (1, 0):
                st, msg = _check_tiling(p.handle, vecok)
                assert st == arplan.AR_OK, msg
    # co-located PS: every reduce step stores to all n buffers
    n, N = 16, 1 << 20
    with arplan.Plan(n, N, "f32", "cps") as p:
        p.set_option(arplan.AR_OPT_SLICE, 0)
        (ph, k, d, cnt, b), = p.launches()
        assert (k, d, cnt) == (16, 16, 16)
        assert b == n * (n + n) * (N // n) * 4
    with arplan.Plan(64, 1 << 16, "f32", "tree", (8, 8)) as p:
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        assert [(x[1], x[2], x[3]) for x in L] == [(8, 1, 64), (8, 64, 64)]
    # RHD: each eighth is reduced once and stored to all 8 buffers (its
    # copies read every range once, so the rewrite applies at any size)
    with arplan.Plan(8, 1 << 26, "f32", "rhd") as p:
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        assert [(x[0], x[1], x[2], x[3]) for x in L] == [(0, 2, 1, 8), (1, 2, 1, 8), (2, 2, 8, 8)]
        assert L[2][4] == 8 * (2 + 8) * (1 << 26) // 8 * 4
    # co-located PS at 1 GiB: the broadcast copies read each range 15 times
    # (cache hits), so they stay a launch of their own
    with arplan.Plan(16, 1 << 24, "f32", "cps") as p:
        assert [(x[1], x[2]) for x in p.launches()] == [(16, 1), (1, 1)]
    assert _status(arplan.ar_plan_set_option, 0, 0, 1) == arplan.AR_ERR_INVALID_ARG
    with arplan.Plan(4, 100, "f32", "ring") as p:
        assert _status(arplan.ar_plan_set_option, p.handle, 7, 1) == arplan.AR_ERR_INVALID_ARG
        assert _status(arplan.ar_plan_set_option, p.handle, arplan.AR_OPT_FUSE, 2) == \
            arplan.AR_ERR_INVALID_ARG


def test_fusion_refuses_clashing_absorption():
    # phase 0: reduce x0[0,4) over {0,1} and copy x1[0,4) -> x2 (reads x1);
    # phase 1: copy x0[0,4) -> x1.  Absorbing that copy would write x1[0,4)
    # while phase 0 still reads it, so it must stay a separate launch.
    steps = [(0, "reduce", 0, [0, 1], 0, 4), (0, "copy", 2, [1], 0, 4),
             (1, "copy", 1, [0], 0, 4)]
    h = arplan.ar_plan_create_custom(3, 8, "f32", steps)
    try:
        arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, 0)
        L = [arplan.ar_plan_launch_info(h, i)
             for i in range(arplan.ar_plan_num_launches(h))]
        assert [x[0] for x in L] == [0, 0, 1]
        st, msg = _check_tiling(h, 1)
        assert st == arplan.AR_OK, msg
    finally:
        arplan.ar_plan_destroy(h)
    # without the clash the copy is absorbed
    steps = [(0, "reduce", 0, [0, 1], 0, 4), (0, "copy", 2, [1], 4, 8),
             (1, "copy", 1, [0], 0, 4)]
    h = arplan.ar_plan_create_custom(3, 8, "f32", steps)
    try:
        arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, 0)
        L = [arplan.ar_plan_launch_info(h, i)
             for i in range(arplan.ar_plan_num_launches(h))]
        assert [(x[0], x[1], x[2]) for x in L] == [(0, 1, 1), (0, 2, 2)]
    finally:
        arplan.ar_plan_destroy(h)


@pytest.mark.parametrize("kind,n,N,fan", TILING)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_whole_plan_launch_schedule(kind, n, N, fan, dtype):
    # AR_OPT_SLICE = 1: one launch when every step boundary is 16-byte
    # aligned; the host check walks its tiles and compares the schedule with
    # the steps of every phase
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        off = oracle.block_bounds(N, n)
        vec = 16 // (4 if dtype == "f32" else 2)
        aligned = all(o % vec == 0 for o in off)
        # plans of at most 64 buffers run resident (-2), larger ones streamed
        # (-3), unless that is off
        marker = -2 if n <= 64 else -3
        L = p.launches()
        if p.num_phases:
            sliced = len(L) == 1 and L[0][0] == marker
            assert sliced == aligned, (L, aligned)
        for res in (1, 0):
            p.set_option(arplan.AR_OPT_RESIDENT, res)
            for fuse in (1, 0):
                p.set_option(arplan.AR_OPT_FUSE, fuse)
                st, msg = _check_tiling(p.handle, 1)
                assert st == arplan.AR_OK, msg
        p.set_option(arplan.AR_OPT_FUSE, 1)
        if aligned and p.num_phases:
            (ph, k, d, cnt, b), = p.launches()
            assert ph == -1
            p.set_option(arplan.AR_OPT_RESIDENT, 1)
            (ph, k, d, cnt, b2), = p.launches()
            assert ph == marker
            # resident or streamed: every buffer position loaded once and
            # stored once
            esize = 4 if dtype == "f32" else 2
            assert b2 == 2 * n * N * esize
            p.set_option(arplan.AR_OPT_SLICE, 0)
            assert b == sum(x[4] for x in p.launches())


# -- GenTree plans on arbitrary trees -------------------------------------

def _random_counts(rng, depth=3):
    def build(d):
        if d == 0 or rng.random() < 0.3:
            return [0]
        k = int(rng.integers(1, 5))
        out = [k]
        for _ in range(k):
            out += build(d - 1)
        return out
    while True:
        c = build(depth)
        if c != [0]:
            return c


def _gentree_cases():
    from paper_2409_04202_amd import workloads
    rng = np.random.default_rng(2024)
    cases = [_random_counts(rng) for _ in range(40)]
    cases += [workloads.CONFIGS["asy384_gentree_f32"]["fanin"],
              workloads.CONFIGS["cdc384_gentree_f32"]["fanin"],
              [3, 0, 0, 2, 0, 0], [2, 0, 2, 0, 2, 0, 0], [1, 1, 2, 0, 0], [0]]
    return cases


@pytest.mark.parametrize("idx", range(46))
def test_gentree_steps_match_oracle(idx):
    counts = _gentree_cases()[idx]
    root = oracle.from_preorder(counts)
    n = oracle.gentree.number_servers(root)
    for N in sorted({0, 1, n, 7 * n + 3}):
        ref = oracle.gentree_plan(root, N)
        with arplan.Plan(0, N, "f32", "gentree", counts) as p:
            assert p.n == n
            assert _norm(p.phases()) == _norm(_oracle_phases(ref))
            assert p.bytes() == model.algorithmic_bytes(ref, 4)
            place = oracle.basic_placement(root, n, complete=True)[id(root)]
            off = oracle.block_bounds(N, n)
            if n > 1:
                for sid, blocks in place.items():
                    bl = sorted(blocks)
                    if not bl:
                        assert p.owner(sid) == (0, 0)
                    elif bl == list(range(bl[0], bl[-1] + 1)):
                        assert p.owner(sid) == (off[bl[0]], off[bl[-1] + 1])
                    else:
                        assert _status(arplan.ar_plan_owner, p.handle, sid) == \
                            arplan.AR_ERR_UNSUPPORTED
            for sl in (0, 1, 2):
                p.set_option(arplan.AR_OPT_SLICE, sl)
                for vecok in (1, 0):
                    st, msg = _check_tiling(p.handle, vecok)
                    assert st == arplan.AR_OK, msg


@pytest.mark.parametrize("fan", [(8, 8), (2, 3, 4), (4, 1, 2), (8, 4, 16)])
def test_gentree_equals_tree_on_symmetric_trees(fan):
    counts = oracle.preorder_children(oracle.symmetric_tree(fan))
    n = int(np.prod(fan))
    for N in (n, 5 * n + 1):
        with arplan.Plan(0, N, "bf16", "gentree", counts) as a, \
                arplan.Plan(n, N, "bf16", "tree", fan) as b:
            assert _norm(a.phases()) == _norm(b.phases())
            for p in range(n):
                assert a.owner(p) == b.owner(p)


def test_gentree_errors():
    E = arplan
    for bad in ([2, 0], [1, 0, 0], [0, 0], [-1], [2, 0, 0, 0]):
        assert _status(E.ar_plan_create_gentree, 10, "f32", bad) == E.AR_ERR_INVALID_ARG, bad
    assert _status(E.ar_plan_create_gentree, 10, "f32", []) == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create_gentree, -1, "f32", [2, 0, 0]) == E.AR_ERR_INVALID_ARG
    assert _status(E.ar_plan_create_gentree, 10, 9, [2, 0, 0]) == E.AR_ERR_INVALID_ARG
    # one switch over 20000 servers: 2e4 x 2e4 > 2^28
    assert _status(E.ar_plan_create_gentree, 10, "f32", [20000] + [0] * 20000) == \
        E.AR_ERR_UNSUPPORTED
    h = E.ar_plan_create_gentree(10, "f32", [0])    # a single server
    try:
        assert E.ar_plan_info(h)[3:] == (0, 0)
    finally:
        E.ar_plan_destroy(h)


@pytest.mark.parametrize("name", sorted(__import__(
    "paper_2409_04202_amd.workloads", fromlist=["CONFIGS"]).CONFIGS))
def test_sliced_runs_of_workloads(name):
    # AR_OPT_SLICE = 2 partitions the executed phases into sliced runs and
    # phase launches: the same executed steps (same bytes) as the phase
    # launches, every launch tiled exactly; the 2 GiB RHD plan, whose
    # phases each write more than the 256 MiB cache, runs resident or as
    # phase launches, never plain sliced
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    esize = 2 if c["dtype"] == "bf16" else 4
    with arplan.Plan(c["n"], c["N"], c["dtype"], c["kind"], c["fanin"]) as p:
        L = p.launches()
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L0 = p.launches()
        assert sum(x[3] for x in L) == sum(x[3] for x in L0)
        # a resident launch moves each buffer position of its run at most
        # once in and once out; the plain forms move the steps' bytes
        assert all(x[4] <= 2 * c["n"] * c["N"] * esize for x in L if x[0] == -2)
        p.set_option(arplan.AR_OPT_RESIDENT, 0)
        p.set_option(arplan.AR_OPT_SLICE, 2)
        assert sum(x[4] for x in p.launches()) == sum(x[4] for x in L0)
        p.set_option(arplan.AR_OPT_RESIDENT, 1)
        # phase launches kept outside the runs appear in phase order
        kept = [x for x in L if x[0] >= 0]
        assert all(x in L0 for x in kept)
        assert [x[0] for x in kept] == sorted(x[0] for x in kept)
        p.set_option(arplan.AR_OPT_SLICE, 2)
        for vecok in (1, 0):
            st, msg = _check_tiling(p.handle, vecok)
            assert st == arplan.AR_OK, msg
        if name == "rhd_n8_f32":
            # each buffer in and out once: 4 GiB against 7.5 GiB of phases
            assert [(x[0], x[4]) for x in L] == [(-2, 2 * c["n"] * c["N"] * esize)]
            p.set_option(arplan.AR_OPT_RESIDENT, 0)
            assert all(x[0] >= 0 for x in p.launches())
            p.set_option(arplan.AR_OPT_RESIDENT, 1)
        if name == "tree8x8x8_n512_bf16":
            # the last AllGather phase covers each position with 448 copies:
            # a chain far too long for a sliced launch
            assert L[-1][0] == 5
        if name.startswith("sweep_ring"):
            # 126 phases of short steps: one sliced launch
            assert len(L) == 1 and L[0][0] in (-1, -2)


def _launch_desc(handle, stage):
    f = arplan._lib.ar_debug_launch_desc
    f.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)]
    f.restype = ctypes.c_int32
    out = (ctypes.c_int64 * 10)()
    assert f(handle, stage, out) == arplan.AR_OK, arplan.ar_last_error()
    return {"k": out[0], "cm": out[1], "tile": out[2], "tiles": out[3], "wpb": out[4],
            "table": out[5], "group": out[6], "split": out[7], "affinity": out[8],
            "wide": out[9]}


def test_full_size_forms_use_the_nontemporal_kernels():
    # The benchmark's as-written RHD plan at full size (n = 8, 2^26 fp32):
    # the first halving launch writes 1 GiB (nontemporal loads and stores),
    # the second 512 MiB that the third reads and the third 256 MiB that the
    # first doubling phase reads (fold launches keep up to 512 MiB cached:
    # nontemporal loads, cached stores).  The full-size GPU parity test runs
    # this same plan, so these kernel instances are covered there.
    with arplan.Plan(8, 1 << 26, "f32", "rhd") as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        assert [(x[0], x[1]) for x in L] == [(0, 2), (1, 2), (2, 2), (3, 1), (4, 1), (5, 1)]
        d = [_launch_desc(p.handle, i) for i in range(3)]
        assert [x["k"] for x in d] == [2, 2, 2]
        assert [x["cm"] for x in d] == [3, 1, 1]
        # the first, nontemporal both ways and 3 GiB, runs the wide instance
        assert [x["wide"] for x in d] == [1, 0, 0]
        # with the rewrites, the last halving launch stores to all 8 buffers
        # (2 GiB, nontemporal)
        p.set_option(arplan.AR_OPT_FUSE, 1)
        d = [_launch_desc(p.handle, i) for i in range(len(p.launches()))]
        assert [x["cm"] for x in d] == [3, 1, 3]
    # co-located PS (16-source fold, 1088 MiB) and the tree (8, 8) level-0
    # reduce (8 sources, 1152 MiB) as written: nontemporal loads
    with arplan.Plan(16, 1 << 24, "f32", "cps") as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        d = _launch_desc(p.handle, 0)
        assert d["k"] == 16 and d["cm"] & 1
    with arplan.Plan(64, 1 << 22, "f32", "tree", (8, 8)) as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        d = _launch_desc(p.handle, 0)
        assert d["k"] == 8 and d["cm"] & 1


def test_runtime_source_count_groups():
    # fan-ins without an unrolled kernel: short launches keep four sources'
    # loads in flight, launches of 512 MiB or more one source at a time;
    # unrolled kernels report 1
    for n, N, group in ((24, 1 << 16, 4), (32, (1 << 22) + 17, 1), (12, 1 << 20, 4)):
        with arplan.Plan(n, N, "f32", "cps") as p:
            p.set_option(arplan.AR_OPT_FUSE, 0)
            p.set_option(arplan.AR_OPT_SLICE, 0)
            d = _launch_desc(p.handle, 0)
            assert (d["k"], d["group"]) == (0, group), (n, N, d)
    with arplan.Plan(16, 1 << 20, "f32", "cps") as p:
        p.set_option(arplan.AR_OPT_SLICE, 0)
        assert _launch_desc(p.handle, 0)["group"] == 1


# Split launches (a workgroup per tile, each wave storing to a share of the
# destinations) in the shapes the GPU parity tests run: the 16-source fold
# whose destinations are all its sources, the runtime-source-count fold, the
# 8-, 4- and 2-source folds storing to 64 or 512 buffers, and large ones
# with nontemporal stores.  (fuse, slice) = (1, 0): phase launches.
SPLIT_CASES = [
    ("cps", 16, (1 << 14) + 3, None, "f32", 16, 0), ("cps", 32, 32 * 1000 + 17, None, "bf16", 0, 0),
    ("tree", 512, 1 << 15, (8, 8, 8), "bf16", 8, 0), ("tree", 512, 1 << 18, (8, 8, 8), "bf16", 8, 0),
    ("tree", 64, 4096 + 64 * 5, (8, 8), "f32", 8, 0),
    ("ring", 64, 64 * 1000, None, "f32", 2, 0), ("ring", 64, 1 << 20, None, "f32", 2, 2),
    ("tree", 64, 65553, (16, 4), "f32", 4, 0), ("tree", 256, 65553, (16, 16), "f32", 16, 2)]
# (cm: bit 1 = nontemporal stores; split launches always load through the
# cache.  The large ones here fold what the previous phase kept cached, so
# their load bit is clear too.)
# Launches of 64 MiB or more storing to fewer than 16 destinations per
# source stay one wave per tile (split, they were slower).
UNSPLIT_CASES = [("tree", 512, 1 << 20, (8, 8, 8), "bf16"), ("cps", 17, 1 << 20, None, "f32"),
                 ("tree", 96, 1 << 20, (3, 32), "f32"), ("tree", 64, 1 << 20, (8, 8), "bf16")]


@pytest.mark.parametrize("kind,n,N,fan,dtype", UNSPLIT_CASES)
def test_large_narrow_launches_not_split(kind, n, N, fan, dtype):
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        assert any(x[2] >= 16 for x in L), L
        assert all(_launch_desc(p.handle, i)["split"] == 1 for i in range(len(L)))


@pytest.mark.parametrize("kind,n,N,fan,dtype,k,cm", SPLIT_CASES)
def test_split_launches(kind, n, N, fan, dtype, k, cm):
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        split = []
        for i in range(len(L)):
            d = _launch_desc(p.handle, i)
            if d["split"] > 1:
                assert d["split"] == d["wpb"] and d["table"] and d["affinity"], d
                split.append((d["k"], d["cm"]))
            # every launch of at most 64 MiB places its tiles by position
            # (copies reading a range several times keep their own table)
            if L[i][4] <= 64 << 20 and not (L[i][1] == 1 and d["table"] and not d["affinity"]):
                assert d["affinity"], (i, L[i], d)
            if 64 << 20 < L[i][4] < 512 << 20 and d["split"] == 1:
                assert not d["affinity"], (i, L[i], d)
        assert (k, cm) in split, split
        names = p.launch_kernels()
        assert names == ["split_kernel" if _launch_desc(p.handle, i)["split"] > 1
                         else "phase_kernel" for i in range(len(L))], names
        for vecok in (1, 0):
            st, msg = _check_tiling(p.handle, vecok)
            assert st == arplan.AR_OK, msg


def test_launch_kernels_by_form():
    # the kernel each launch of the benchmark's workloads runs, default form
    from paper_2409_04202_amd import workloads
    expect = {"rhd_n8_f32": ["resident_kernel"],
              "tree8x8x8_n512_bf16": ["phase_kernel", "phase_kernel", "split_kernel",
                                      "phase_kernel"],
              "tree8x8_n64_f32": ["phase_kernel", "sliced_kernel", "phase_kernel"]}
    for name, kernels in expect.items():
        c = workloads.CONFIGS[name]
        with arplan.Plan(c["n"], c["N"], c["dtype"], c["kind"], c["fanin"]) as p:
            assert p.launch_kernels() == kernels, (name, p.launch_kernels())
    # n > 64 with AR_OPT_SLICE = 1: one streamed resident launch
    with arplan.Plan(512, 1 << 14, "bf16", "tree", (8, 8, 8)) as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        assert p.launch_kernels() == ["stream_kernel"], p.launch_kernels()
    with arplan.Plan(8, 1 << 12, "f32", "rhd") as p:
        with pytest.raises(arplan.ArError):
            arplan.ar_plan_launch_kernel(p.handle, len(p.launches()))


# 16-byte vectors per lane and source in one pass of each kernel (kcfg)
_PASS_U = {1: 16, 2: 8, 3: 4, 4: 4, 8: 2, 16: 1, 0: 4}


@pytest.mark.parametrize("kind,n,N,fan,dtype", [
    ("ring", 64, 1 << 20, None, "f32"), ("ring", 64, 1 << 20, None, "bf16"),
    ("ring", 8, 1 << 18, None, "f32"), ("rhd", 8, 1 << 18, None, "f32"),
    ("rhd", 5, (1 << 18) + 3, None, "i32"), ("cps", 6, 1 << 20, None, "f32"),
    ("tree", 32, 1 << 18, (8, 4), "f32")])
def test_fine_tiles_for_launches_with_few_tiles(kind, n, N, fan, dtype):
    # As written, launches of 2 MiB or more with fewer than 2048 tiles of a
    # full kernel pass take smaller tiles, down to one vector per lane,
    # until they have 2048; copies that read a range several times keep
    # full-pass tiles (their XCD tables)
    vec = 16 // (2 if dtype == "bf16" else 4)
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        fine = 0
        for i, x in enumerate(p.launches()):
            d = _launch_desc(p.handle, i)
            full = 64 * _PASS_U[d["k"]] * vec
            if d["k"] == 1 and kind in ("cps", "tree"):
                assert d["tile"] >= full, (i, x, d)  # AllGather copies re-read ranges
            elif x[4] >= 2 << 20:
                assert d["tile"] == full or (d["tile"] < full and d["tile"] >= 64 * vec), (i, x, d)
                if d["tile"] < full:
                    fine += 1
                    assert d["tiles"] >= 2048 or d["tile"] == 64 * vec, (i, x, d)
        assert fine >= 1
        for vecok in (1, 0):
            st, msg = _check_tiling(p.handle, vecok)
            assert st == arplan.AR_OK, msg


def test_large_launches_placed_by_position():
    # RHD as written at full size: its halving folds (2 sources) and doubling
    # copies (each range read once) move 512 MiB or more and are placed by
    # position; the 16-source fold of co-located PS and the copies after it,
    # which read each range 15 times, are not
    with arplan.Plan(8, 1 << 26, "f32", "rhd") as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        d = [_launch_desc(p.handle, i) for i in range(len(p.launches()))]
        assert [x["affinity"] for x in d] == [1] * 6, d
        for vecok in (1, 0):
            st, msg = _check_tiling(p.handle, vecok)
            assert st == arplan.AR_OK, msg
    with arplan.Plan(16, 1 << 24, "f32", "cps") as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        d = [_launch_desc(p.handle, i) for i in range(len(p.launches()))]
        assert [x["affinity"] for x in d] == [0, 0], d


@pytest.mark.parametrize("seed", range(24))
def test_random_many_destination_plans_split(seed):
    # ragged blocks each reduced and copied to 16+ buffers (some of them the
    # reduce's sources): the executor's steps store to 17+ buffers, the
    # launch runs split, and the tiling check accepts it with aligned and
    # unaligned buffers
    from plan_gen import many_destination_plan
    rng = np.random.default_rng(7100 + seed)
    n = int(rng.integers(17, 41))
    N = int(rng.integers(1000, 200000))
    phases = many_destination_plan(rng, n, N)
    flat = [(q, op, d, s_, b, e) for q, ph in enumerate(phases) for (op, d, s_, b, e) in ph]
    h = arplan.ar_plan_create_custom(n, N, ("f32", "bf16", "i32")[seed % 3], flat)
    try:
        arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, 0)
        L = [arplan.ar_plan_launch_info(h, i) for i in range(arplan.ar_plan_num_launches(h))]
        kernels = [arplan.ar_plan_launch_kernel(h, i) for i in range(len(L))]
        assert "split_kernel" in kernels, (L, kernels)
        for vecok in (1, 0):
            st, msg = _check_tiling(h, vecok)
            assert st == arplan.AR_OK, msg
    finally:
        arplan.ar_plan_destroy(h)


# The automatic choice (AR_OPT_SLICE = 2) on every benchmark workload: the
# kernel of each launch.  Each is the fastest form measured on MI355X (or
# within a few % of it); a change to the cost model that moves one of them
# shows here first.
BENCH_CHOICE = {
    "ring_n4_f32": ["resident_kernel"],
    "ring_n4_i32": ["resident_kernel"],
    "rhd_n8_f32": ["resident_kernel"],
    "cps_n16_f32": ["phase_kernel", "phase_kernel"],
    "tree8x8_n64_f32": ["phase_kernel", "sliced_kernel", "phase_kernel"],
    "tree8x8_n64_i32": ["phase_kernel", "sliced_kernel", "phase_kernel"],
    "tree8x8x8_n512_bf16": ["phase_kernel", "phase_kernel", "split_kernel", "phase_kernel"],
    "asy384_gentree_f32": ["phase_kernel", "sliced_kernel", "phase_kernel"],
    "cdc384_gentree_f32": ["phase_kernel", "sliced_kernel", "phase_kernel"],
    "sweep_ring_n64_f32_N4096": ["resident_kernel"],
    "sweep_tree8x8_n64_f32_N4096": ["phase_kernel", "split_kernel"],
    "sweep_ring_n64_bf16_N4096": ["resident_kernel"],
    "sweep_tree8x8_n64_bf16_N4096": ["phase_kernel", "split_kernel"],
    "sweep_ring_n64_f32_N65536": ["resident_kernel"],
    "sweep_tree8x8_n64_f32_N65536": ["phase_kernel", "split_kernel"],
    "sweep_ring_n64_bf16_N65536": ["resident_kernel"],
    "sweep_tree8x8_n64_bf16_N65536": ["phase_kernel", "split_kernel"],
    "sweep_ring_n64_f32_N1048576": ["resident_kernel"],
    "sweep_tree8x8_n64_f32_N1048576": ["sliced_kernel"],
    "sweep_ring_n64_bf16_N1048576": ["resident_kernel"],
    "sweep_tree8x8_n64_bf16_N1048576": ["sliced_kernel"],
}


def test_automatic_choice_beyond_64_buffers():
    # Ring over 128 and 256 buffers runs as one streamed launch up to the
    # sizes where it was measured faster; RHD's 128-destination phase of
    # 128-byte steps runs split, outside the sliced run; trees and large
    # Rings keep their launches
    def kernels(kind, n, N, dtype, fan=None):
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            return p.launch_kernels()
    for n, N, dtype in [(128, 1 << 12, "f32"), (256, 1 << 15, "f32"), (128, 1 << 18, "bf16")]:
        assert kernels("ring", n, N, dtype) == ["stream_kernel"], (n, N, dtype)
    assert "stream_kernel" not in kernels("ring", 128, 1 << 20, "f32")
    k = kernels("rhd", 128, 1 << 12, "f32")
    assert k[-1] == "split_kernel" and "stream_kernel" not in k, k
    for fan, N in [((8, 8, 8), 1 << 12), ((8, 8, 8), 1 << 18), ((8, 16), 1 << 15)]:
        assert "stream_kernel" not in kernels("tree", 512 if len(fan) == 3 else 128, N, "f32", fan)
    # without streamed runs: Ring's last phase, 32-byte steps into 128
    # buffers, leaves the sliced run too
    with arplan.Plan(128, 1 << 12, "f32", "ring") as p:
        p.set_option(arplan.AR_OPT_RESIDENT, 0)
        assert p.launch_kernels() == ["sliced_kernel", "split_kernel"]


@pytest.mark.parametrize("name", sorted(BENCH_CHOICE))
def test_automatic_choice_of_bench_workloads(name):
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    with arplan.Plan(c["n"], c["N"], c["dtype"], c["kind"], c["fanin"]) as p:
        assert p.launch_kernels() == BENCH_CHOICE[name]


@pytest.mark.parametrize("dtype", ["f32", "i32", "bf16"])
def test_wide_eight_source_launches(dtype):
    # an 8-source fold of 4-byte elements over 512 MiB or more with
    # nontemporal loads runs the one-pass wide instance: the first level of
    # the (8, 8) tree at 2^22 elements per processor, and a lone 8-way reduce
    # over 128 MiB buffers (nontemporal stores too); bf16 folds never do
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS["tree8x8_n64_f32"]
    with arplan.Plan(c["n"], c["N"], dtype, "tree", c["fanin"]) as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        d = [_launch_desc(p.handle, i) for i in range(len(L))]
        assert [y["wide"] for y in d] == [int(dtype != "bf16"), 0, 0, 0], d
        assert (L[0][1], d[0]["cm"]) == (8, 1)
    N = (1 << 25) + 13
    h = arplan.ar_plan_create_custom(8, N, dtype, [(0, "reduce", 0, list(range(8)), 0, N)])
    try:
        d = _launch_desc(h, 0)
        assert (d["k"], d["cm"], d["wide"]) == (8, 3, int(dtype != "bf16")), d
        for vecok in (1, 0):
            st, msg = _check_tiling(h, vecok)
            assert st == arplan.AR_OK, msg
    finally:
        arplan.ar_plan_destroy(h)
    h = arplan.ar_plan_create_custom(8, 1 << 22, dtype, [(0, "reduce", 0, list(range(8)), 0, 1 << 22)])
    try:
        assert _launch_desc(h, 0)["wide"] == 0
    finally:
        arplan.ar_plan_destroy(h)


@pytest.mark.parametrize("N,dtype", [((1 << 26) + 13, "f32"), (1 << 26, "i32"), (1 << 27, "bf16")])
def test_wide_two_source_launches(N, dtype):
    # RHD as written at 2-3 GiB: the first halving launch (nontemporal loads
    # and stores, over 512 MiB) runs the wide 2-source instance; smaller or
    # cached launches never do; the tiling check accepts it either way
    with arplan.Plan(8, N, dtype, "rhd") as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        L = p.launches()
        d = [_launch_desc(p.handle, i) for i in range(len(L))]
        assert d[0]["wide"] == 1 and d[0]["cm"] == 3, d[0]
        for x, y in zip(L, d):
            if y["wide"]:
                assert x[1] == 2 and y["cm"] == 3 and x[4] >= 512 << 20, (x, y)
        for vecok in (1, 0):
            st, msg = _check_tiling(p.handle, vecok)
            assert st == arplan.AR_OK, msg
    with arplan.Plan(8, 1 << 20, dtype, "rhd") as p:
        p.set_option(arplan.AR_OPT_FUSE, 0)
        p.set_option(arplan.AR_OPT_SLICE, 0)
        assert all(_launch_desc(p.handle, i)["wide"] == 0 for i in range(len(p.launches())))
