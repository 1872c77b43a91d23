"""The executor's rewrites preserve every result (host only, no GPU).

The library reports the steps it would execute after its rewrites
(multicast copies, reduce-then-broadcast folded transitively across phases).
Each executed phase is turned back into an oracle phase (a step with d
destinations becomes d steps with the same sources, which read the state at
the start of the phase exactly as the kernel does) and run by the oracle on
random inputs; the result must equal, bit for bit, the oracle's run of the
plan as written.  Random custom plans with chains of copies exercise the
rewrites beyond the built-in plan kinds.
"""

import ctypes

import numpy as np
import pytest

import oracle
from oracle.plans import Plan as OPlan, Step as OStep

from paper_2409_04202_amd import workloads
from checklib import arplan


def _exec_steps(handle):
    f = arplan._lib.ar_debug_exec_steps
    I64, I32 = ctypes.c_int64, ctypes.c_int32
    f.argtypes = [ctypes.c_void_p, I64, ctypes.POINTER(I32), ctypes.POINTER(I64),
                  ctypes.POINTER(I64), ctypes.POINTER(I32), ctypes.POINTER(I32), I64,
                  ctypes.POINTER(I32), ctypes.POINTER(I64), ctypes.POINTER(I64)]
    f.restype = I32
    cnt, icnt = I64(), I64()
    assert f(handle, 0, None, None, None, None, None, 0, None,
             ctypes.byref(cnt), ctypes.byref(icnt)) == arplan.AR_OK
    c, ic = max(1, cnt.value), max(1, icnt.value)
    ph, nsrc, ndst = (I32 * c)(), (I32 * c)(), (I32 * c)()
    b, e = (I64 * c)(), (I64 * c)()
    idx = (I32 * ic)()
    assert f(handle, c, ph, b, e, nsrc, ndst, ic, idx,
             ctypes.byref(cnt), ctypes.byref(icnt)) == arplan.AR_OK
    out, at = [], 0
    for i in range(cnt.value):
        srcs = tuple(idx[at:at + nsrc[i]])
        dsts = tuple(idx[at + nsrc[i]:at + nsrc[i] + ndst[i]])
        at += nsrc[i] + ndst[i]
        out.append((ph[i], b[i], e[i], srcs, dsts))
    return out


def _as_oracle_plan(steps, n, N):
    phases = []
    for ph, b, e, srcs, dsts in steps:
        while len(phases) <= ph:
            phases.append([])
        op = "reduce" if len(srcs) >= 2 else "copy"
        for d in dsts:
            phases[ph].append(OStep(op, d, srcs, b, e))
    return OPlan("executed", n, N, phases)


def _check(handle, ref_plan, n, N, dtype, seed):
    dist = "int1000" if dtype == "i32" else "uniform"
    xs = workloads.draw(n, N, dtype, dist, seed)
    want = oracle.execute(ref_plan, [x.copy() for x in xs], dtype)
    for fuse in (1, 0):
        arplan.ar_plan_set_option(handle, arplan.AR_OPT_FUSE, fuse)
        steps = _exec_steps(handle)
        got = oracle.execute(_as_oracle_plan(steps, n, N), [x.copy() for x in xs], dtype)
        for q in range(n):
            assert np.array_equal(got[q], want[q]), (fuse, q)
        if fuse == 0:   # without rewrites the executed steps are the plan's
            assert sum(len(s[4]) for s in steps) == sum(len(p) for p in ref_plan.phases)


BUILTIN = [("ring", n, None) for n in (2, 3, 5, 8)] + \
          [("rhd", n, None) for n in (2, 4, 6, 8, 12)] + \
          [("cps", n, None) for n in (3, 16)] + [("rb", 5, None)] + \
          [("tree", 16, (4, 4)), ("tree", 24, (2, 3, 4)), ("tree", 64, (8, 8)),
           ("tree", 12, (3, 1, 4))]


@pytest.mark.parametrize("kind,n,fan", BUILTIN)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_builtin_plans_rewrites_keep_results(kind, n, fan, dtype):
    for N in (n * 8, 1000 + n):
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            _check(p.handle, oracle.make_plan(kind, n, N, fan), n, N, dtype, seed=N)


@pytest.mark.parametrize("name", ["asy384_gentree_f32", "cdc384_gentree_f32"])
def test_gentree_rewrites_keep_results(name):
    c = workloads.CONFIGS[name]
    N = 384 * 3 + 5
    root = oracle.from_preorder(c["fanin"])
    with arplan.Plan(0, N, "f32", "gentree", c["fanin"]) as p:
        _check(p.handle, oracle.gentree_plan(root, N), 384, N, "f32", seed=3)


def _random_plan(rng, n, N):
    """Random hazard-free phases: reduce phases, then copy phases that move
    ranges the previous phase wrote (so that the rewrites find work),
    mixed with unrelated copies and reduces."""
    cuts = np.unique(np.concatenate([[0, N], rng.integers(1, N, size=rng.integers(2, 7))]))
    blocks = list(zip(cuts[:-1], cuts[1:]))
    phases = []
    last_written = []
    for q in range(int(rng.integers(2, 6))):
        steps, writes, reads = [], [], []

        def free(buf, b, e, for_write):
            for (w, wb, we) in writes:
                if w == buf and b < we and wb < e:
                    return False
            if for_write:
                for (r, rb, re) in reads:
                    if r == buf and b < re and rb < e:
                        return False
            return True

        for _ in range(int(rng.integers(1, 2 * n + 2))):
            if last_written and rng.random() < 0.6:
                src, b, e = last_written[int(rng.integers(len(last_written)))]
                srcs = (src,)
            else:
                i = int(rng.integers(len(blocks)))
                j = min(len(blocks), i + int(rng.integers(1, 3)))
                b, e = blocks[i][0], blocks[j - 1][1]
                k = int(rng.integers(1, min(n, 4) + 1))
                srcs = tuple(int(s) for s in rng.choice(n, size=k, replace=False))
            dst = int(rng.integers(n))
            if not free(dst, b, e, True) or not all(free(s, b, e, False) for s in srcs):
                continue
            if any(s == dst for s in srcs) and len(srcs) == 1:
                continue
            steps.append(("reduce" if len(srcs) >= 2 else "copy", dst, srcs, int(b), int(e)))
            writes.append((dst, b, e))
            reads.extend((s, b, e) for s in srcs)
        if steps:
            phases.append(steps)
            last_written = [(d, b, e) for (_, d, _, b, e) in steps]
    return phases


@pytest.mark.parametrize("seed", range(150))
def test_random_custom_plans_rewrites_keep_results(seed):
    rng = np.random.default_rng(7000 + seed)
    n = int(rng.integers(2, 7))
    N = int(rng.integers(8, 400))
    phases = _random_plan(rng, n, N)
    flat = [(q, op, d, s, b, e) for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref = OPlan("custom", n, N, [[OStep(op, d, s, b, e) for (op, d, s, b, e) in ph]
                                  for ph in phases])
    dtype = ("f32", "bf16", "i32")[seed % 3]
    h = arplan.ar_plan_create_custom(n, N, dtype, flat)
    try:
        _check(h, ref, n, N, dtype, seed=seed)
    finally:
        arplan.ar_plan_destroy(h)


def test_random_plans_trigger_transitive_absorption():
    # the generator produces plans where a reduce phase absorbs at least two
    # following copy phases (a step ends up with more destinations than the
    # copies of any single phase gave it)
    hits = 0
    for seed in range(60):
        rng = np.random.default_rng(7000 + seed)
        n = int(rng.integers(2, 7))
        N = int(rng.integers(8, 400))
        phases = _random_plan(rng, n, N)
        flat = [(q, op, d, s, b, e) for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
        h = arplan.ar_plan_create_custom(n, N, "f32", flat)
        try:
            nexec = len({s[0] for s in _exec_steps(h)})
            if len(phases) - nexec >= 2:
                hits += 1
        finally:
            arplan.ar_plan_destroy(h)
    assert hits >= 3, hits
