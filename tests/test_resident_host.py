"""Resident sliced launches, checked on the host (no GPU).

A resident launch runs, per segment of element positions, a program the
library builds on the host: the buffers to load into on-chip rows, the step
records of the run's phases in phase order, the buffers to store back.  Here
the programs are read back through the library's test hook and interpreted
with numpy on random inputs: a row read before it was loaded or written is
an error, the folds use the oracle's arithmetic, and the result must equal,
bit for bit, the oracle's phase-by-phase run of the plan as written.  This
pins the program semantics (which rows are loaded and stored, the step
order, the record encoding) independently of the GPU.
"""

import ctypes

import numpy as np
import pytest

import oracle
from oracle.execute import fold
from oracle.plans import Plan as OPlan, Step as OStep

from paper_2409_04202_amd import workloads
from checklib import arplan

from test_capi_host import _check_tiling
from test_exec_rewrites_host import _random_plan
from plan_gen import wide_random_plan as _wide_random_plan


def _resident_tables(handle, stage):
    f = arplan._lib.ar_debug_resident
    I64 = ctypes.POINTER(ctypes.c_int64)
    f.argtypes = [ctypes.c_void_p, ctypes.c_int32, I64, I64, ctypes.POINTER(ctypes.c_uint32)]
    f.restype = ctypes.c_int32
    info = (ctypes.c_int64 * 5)()
    st = f(handle, stage, info, None, None)
    if st != arplan.AR_OK:
        return None
    nunits, nw = info[2], info[3]
    _resident_tables.slots = info[4]
    units = (ctypes.c_int64 * (7 * nunits))()
    prog = (ctypes.c_uint32 * max(1, nw))()
    assert f(handle, stage, info, units, prog) == arplan.AR_OK
    return ([tuple(units[7 * i:7 * i + 7]) for i in range(nunits)],
            np.array(prog[:nw], dtype=np.uint32))


def _decode(words):
    """Records of one segment, per the documented encoding: ("add", [r0, r1],
    d), ("copy", [r0], d), ("chain", [s, y1..ym], d), ("fold", rows, d),
    ("store", rows, None); four row bytes per word after a header, 64-word
    chunks, a zero word ends a chunk."""
    out = []
    for c0 in range(0, len(words), 64):
        chunk = [int(w) for w in words[c0:c0 + 64]]
        c = 0
        while c < len(chunk):
            h = chunk[c]
            op, b1, b2, b3 = h & 0xFF, (h >> 8) & 0xFF, (h >> 16) & 0xFF, h >> 24
            if op == 0:
                assert not any(chunk[c:]), "padding must be zero"
                break

            def rows(m):
                assert c + 1 + (m + 3) // 4 <= len(chunk), "record across a chunk"
                return [(chunk[c + 1 + i // 4] >> (8 * (i % 4))) & 0xFF for i in range(m)]
            if op == 0xFE:
                out.append(("add", [b1, b2], b3))
                c += 1
            elif op == 0xFD:
                assert b2 == b1
                out.append(("copy", [b1], b3))
                c += 1
            elif op == 0xFC:
                out.append(("chain", [b2] + rows(b1), b3))
                c += 1 + (b1 + 3) // 4
            elif op == 0xFB:
                assert b1 >= 2 and b3 == 0
                out.append(("fold", rows(b1), b2))
                c += 1 + (b1 + 3) // 4
            elif op == 0xFA:
                assert b1 % 4 == 0 and b1 > 0 and b2 == 0 and b3 == 0
                out.append(("store", rows(b1), None))
                c += 1 + b1 // 4
            else:
                raise AssertionError("unknown opcode %#x" % op)
    return out


def _decode_streamed(words):
    """Records of one streamed segment: ("add", [s0, s1], d), ("fold", slots,
    d), ("load", [(slot, buffer), ...], None), ("wait", m, None), ("put",
    buffers, slot); 64-word chunks, a zero word ends a chunk."""
    out = []
    for c0 in range(0, len(words), 64):
        chunk = [int(w) for w in words[c0:c0 + 64]]
        c = 0
        while c < len(chunk):
            h = chunk[c]
            op, b1, b2, b3 = h & 0xFF, (h >> 8) & 0xFF, (h >> 16) & 0xFF, h >> 24
            if op == 0:
                assert not any(chunk[c:]), "padding must be zero"
                break
            if op == 0xFE:
                out.append(("add", [b1, b2], b3))
                c += 1
            elif op == 0xFB:
                n = 1 + (b1 + 3) // 4
                assert b1 >= 2 and b3 == 0 and c + n <= len(chunk)
                out.append(("fold", [(chunk[c + 1 + i // 4] >> (8 * (i % 4))) & 0xFF
                                     for i in range(b1)], b2))
                c += n
            elif op == 0xF9:
                assert b1 >= 1 and b2 == 0 and b3 == 0 and c + 1 + b1 <= len(chunk)
                out.append(("load", [(x & 0xFF, x >> 8) for x in chunk[c + 1:c + 1 + b1]], None))
                c += 1 + b1
            elif op == 0xF8:
                out.append(("wait", b1, None))
                c += 1
            elif op == 0xF7:
                n = 1 + (b1 + 1) // 2
                assert b1 >= 1 and b3 == 0 and c + n <= len(chunk)
                ids = [(chunk[c + 1 + i // 2] >> (16 * (i % 2))) & 0xFFFF for i in range(b1)]
                out.append(("put", ids, b2))
                c += n
            else:
                raise AssertionError("unknown opcode %#x" % op)
    return out


def _interpret_streamed(tables, bufs, dtype, slots):
    """Run every unit of a streamed launch in program order (a load completes
    at once; the library's symbolic check covers what may be in flight):
    loads copy a buffer's tile into a slot, folds combine slots, puts store a
    slot into buffers."""
    units, prog = tables
    vec = 8 if dtype == "bf16" else 4
    out = [b.copy() for b in bufs]
    for lo, load, store, nv, off, nw, alias in units:
        assert load == 0 and store == 0 and alias == -1
        hi = lo + nv * vec
        slot = {}
        for kind, a, b in _decode_streamed(prog[off:off + nw]):
            if kind == "load":
                for sl, buf in a:
                    assert sl < slots
                    slot[sl] = out[buf][lo:hi].copy()
            elif kind in ("add", "fold"):
                assert b < slots and all(x in slot for x in a)
                slot[b] = fold(dtype, [slot[x] for x in a])
            elif kind == "put":
                for buf in a:
                    out[buf][lo:hi] = slot[b]
    return out


def _bits(mask):
    mask &= (1 << 64) - 1
    return [b for b in range(64) if mask >> b & 1]


def _interpret(tables, bufs, dtype):
    """Run every unit (wave) of a resident launch: its tile of every buffer
    it loads becomes a row, the records run on the rows, the rows it stores
    go back.  Units of one launch own disjoint positions."""
    units, prog = tables
    vec = 8 if dtype == "bf16" else 4
    out = [b.copy() for b in bufs]
    for lo, load, store, nv, off, nw, alias in units:
        hi = lo + nv * vec
        # buffer b takes its stored value from row src[b] (the alias table)
        src = list(range(64))
        if alias >= 0:
            for b in range(64):
                a = (int(prog[alias + b // 4]) >> (8 * (b % 4))) & 0xFF
                if a != 0xFF:
                    src[b] = a
        rows = {}
        for b in _bits(load):
            rows[b] = bufs[b][lo:hi].copy()
        last = None
        for kind, rs, d in _decode(prog[off:off + nw]):
            for r in (rs if kind != "store" else []):
                assert r in rows, "row %d read before it was loaded or written" % r
            if kind == "copy":
                val = rows[rs[0]].copy()
            elif kind == "add" or kind == "fold":
                val = fold(dtype, [rows[r] for r in rs])
            elif kind == "chain":
                val = rows[rs[0]].copy()
                for y in rs[1:]:
                    val = fold(dtype, [val, rows[y]])
            else:  # store: the previous record's result into every listed row
                assert last is not None
                for r in rs:
                    rows[r] = last.copy()
                continue
            rows[d] = val
            last = val
        for b in _bits(store):
            out[b][lo:hi] = rows[src[b]]
    return out


def _check_whole_plan(handle, ref_plan, n, N, dtype, seed):
    arplan.ar_plan_set_option(handle, arplan.AR_OPT_SLICE, 1)
    assert arplan.ar_plan_num_launches(handle) == 1
    kind = arplan.ar_plan_launch_info(handle, 0)[0]
    assert kind == (-2 if n <= 64 else -3)
    tables = _resident_tables(handle, 0)
    assert tables is not None
    slots = _resident_tables.slots
    assert (slots == 0) == (kind == -2) and slots <= 64
    # the library's own check: each segment's records, run symbolically, give
    # the executed steps' result terms for every stored row
    st, msg = _check_tiling(handle, 1)
    assert st == arplan.AR_OK, msg
    dist = "int1000" if dtype == "i32" else "uniform"
    xs = workloads.draw(n, N, dtype, dist, seed)
    want = oracle.execute(ref_plan, [x.copy() for x in xs], dtype)
    if kind == -2:
        got = _interpret(tables, [x.copy() for x in xs], dtype)
    else:
        got = _interpret_streamed(tables, [x.copy() for x in xs], dtype, slots)
    for q in range(n):
        assert np.array_equal(got[q], want[q]), q


BUILTIN = [("ring", n, None) for n in (2, 3, 4, 8)] + \
          [("rhd", n, None) for n in (2, 4, 6, 8)] + \
          [("cps", n, None) for n in (3, 16)] + [("rb", 5, None)] + \
          [("tree", 16, (4, 4)), ("tree", 24, (2, 3, 4)), ("tree", 64, (8, 8))]


@pytest.mark.parametrize("kind,n,fan", BUILTIN)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32"])
@pytest.mark.parametrize("fuse", [1, 0])
def test_whole_plan_resident_program(kind, n, fan, dtype, fuse):
    vec = 8 if dtype == "bf16" else 4
    N = n * vec * 8  # every block boundary 16-byte aligned
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_FUSE, fuse)
        _check_whole_plan(p.handle, oracle.make_plan(kind, n, N, fan), n, N, dtype, seed=n)


def test_more_than_64_buffers_run_streamed():
    # a row per buffer up to 64 buffers; beyond, LDS slots shared by values
    with arplan.Plan(128, 128 * 4, "f32", "ring") as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        L = p.launches()
        assert len(L) == 1 and L[0][0] == -3
        assert _resident_tables(p.handle, 0) is not None and 0 < _resident_tables.slots <= 64
    with arplan.Plan(64, 64 * 4, "f32", "ring") as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        assert p.launches()[0][0] == -2
        assert _resident_tables(p.handle, 0) is not None and _resident_tables.slots == 0
    # a 100-source fold needs more than 64 slots at once: plain sliced
    with arplan.Plan(100, 100 * 4, "f32", "cps") as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        assert p.launches()[0][0] == -1 and _resident_tables(p.handle, 0) is None


STREAMED = [("ring", 65, None), ("ring", 70, None), ("rhd", 128, None), ("rhd", 96, None),
            ("tree", 96, (4, 4, 6)), ("tree", 512, (8, 8, 8)), ("tree", 384, (16, 24))]


@pytest.mark.parametrize("kind,n,fan", STREAMED)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32"])
@pytest.mark.parametrize("fuse", [1, 0])
def test_whole_plan_streamed_program(kind, n, fan, dtype, fuse):
    vec = 8 if dtype == "bf16" else 4
    N = n * vec * (2 if n > 128 else 8)  # every block boundary 16-byte aligned
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_FUSE, fuse)
        _check_whole_plan(p.handle, oracle.make_plan(kind, n, N, fan), n, N, dtype, seed=n + 1)


@pytest.mark.parametrize("seed", range(60))
def test_random_custom_plans_resident_program(seed):
    # random hazard-free plans on positions scaled to whole 16-byte vectors
    rng = np.random.default_rng(9100 + seed)
    n = int(rng.integers(2, 7))
    M = int(rng.integers(4, 100))
    phases = _random_plan(rng, n, M)
    dtype = ("f32", "bf16", "i32")[seed % 3]
    vec = 8 if dtype == "bf16" else 4
    N = M * vec
    flat = [(q, op, d, s, b * vec, e * vec)
            for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref = OPlan("custom", n, N, [[OStep(op, d, s, b * vec, e * vec)
                                  for (op, d, s, b, e) in ph] for ph in phases])
    h = arplan.ar_plan_create_custom(n, N, dtype, flat)
    try:
        _check_whole_plan(h, ref, n, N, dtype, seed=seed)
    finally:
        arplan.ar_plan_destroy(h)


@pytest.mark.parametrize("name", ["sweep_ring_n64_f32_N4096", "sweep_ring_n64_bf16_N4096"])
def test_workload_runs_resident_by_default(name):
    # the small-message workloads run as one resident launch by default; the
    # program is checked at a reduced N with the same block structure
    c = workloads.CONFIGS[name]
    n = c["n"]
    with arplan.Plan(n, c["N"], c["dtype"], c["kind"], c.get("fanin")) as p:
        L = p.launches()
        assert len(L) == 1 and L[0][0] == -2, L
    N = n * 4 * 5
    with arplan.Plan(n, N, "f32", c["kind"], c.get("fanin")) as p:
        _check_whole_plan(p.handle, oracle.make_plan(c["kind"], n, N, c.get("fanin")),
                          n, N, "f32", seed=5)


def test_ring_program_is_one_chain_and_a_broadcast():
    # Ring n = 64: the 62 ReduceScatter steps of a block each fold the previous
    # partial sum, whose row is overwritten by the final broadcast: one chain
    # record of 62 adds (start row and 62 rows), then the last step: its add
    # into one buffer, whose row the other 63 buffers take their values from
    # (alias table)
    n, N = 64, 64 * 64 * 4
    with arplan.Plan(n, N, "f32", "ring") as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        units, prog = _resident_tables(p.handle, 0)
        for lo, load, store, nv, off, nw, alias in units:
            recs = _decode(prog[off:off + nw])
            assert [r[0] for r in recs] == ["chain", "add"] and alias >= 0
            assert len(recs[0][1]) == 63


@pytest.mark.parametrize("seed", range(40))
def test_wide_random_plans_resident_program(seed):
    # 8-64 buffers, folds of up to 16 sources and copies into up to 40
    # buffers: fold records, store records with padded lists, many rows
    rng = np.random.default_rng(9300 + seed)
    n = int(rng.choice([8, 17, 33, 64]))
    M = int(rng.integers(3, 120))
    phases = _wide_random_plan(rng, n, M)
    dtype = ("f32", "bf16", "i32")[seed % 3]
    vec = 8 if dtype == "bf16" else 4
    N = M * vec
    flat = [(q, op, d, s, b * vec, e * vec)
            for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref = OPlan("custom", n, N, [[OStep(op, d, s, b * vec, e * vec)
                                  for (op, d, s, b, e) in ph] for ph in phases])
    h = arplan.ar_plan_create_custom(n, N, dtype, flat)
    try:
        _check_whole_plan(h, ref, n, N, dtype, seed=seed)
    finally:
        arplan.ar_plan_destroy(h)


@pytest.mark.parametrize("seed", range(40))
def test_wide_random_plans_streamed_program(seed):
    # more than 64 buffers: streamed programs (slots shared by values, loads
    # ahead, stores held back while a buffer's own row is still to load)
    rng = np.random.default_rng(9500 + seed)
    n = int(rng.choice([65, 80, 130, 200]))
    M = int(rng.integers(3, 90))
    phases = _wide_random_plan(rng, n, M)
    dtype = ("f32", "bf16", "i32")[seed % 3]
    vec = 8 if dtype == "bf16" else 4
    N = M * vec
    flat = [(q, op, d, s, b * vec, e * vec)
            for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref = OPlan("custom", n, N, [[OStep(op, d, s, b * vec, e * vec)
                                  for (op, d, s, b, e) in ph] for ph in phases])
    h = arplan.ar_plan_create_custom(n, N, dtype, flat)
    try:
        _check_whole_plan(h, ref, n, N, dtype, seed=seed)
    finally:
        arplan.ar_plan_destroy(h)


def test_streamed_encoder_holds_back_stores():
    # phase 0: x4 <- x10 + ... + x63 + x1; phase 1: x1 <- x2 + x3; phase 2:
    # x4 <- x4 + x7.  Depth first from the final values, x1's new value is
    # computed first, but x1's initial row is only needed by the 55-source
    # fold, more than the loads run ahead later: the store into x1 is held
    # back to the end, after that row has been loaded; bit-exact, and the
    # library's symbolic check accepts the order
    n, vec = 70, 4
    N = 64 * vec * 3
    flat = [(0, "reduce", 4, list(range(10, 64)) + [1], 0, N), (1, "reduce", 1, [2, 3], 0, N),
            (2, "reduce", 4, [4, 7], 0, N)]
    ref = OPlan("custom", n, N, [[OStep(op, d, s_, b, e)] for (_, op, d, s_, b, e) in flat])
    for dtype in ("f32", "bf16", "i32"):
        h = arplan.ar_plan_create_custom(n, N, dtype, flat)
        try:
            _check_whole_plan(h, ref, n, N, dtype, seed=1)
            units, prog = _resident_tables(h, 0)
            lo, load, store, nv, off, nw, alias = units[0]
            order = []
            for kind, a, b in _decode_streamed(prog[off:off + nw]):
                if kind == "load":
                    order += [("load", buf) for _, buf in a]
                elif kind == "put":
                    order += [("put", buf) for buf in a]
                elif kind in ("add", "fold"):
                    order.append((kind, len(a)))
            assert order[:3] == [("load", 2), ("load", 3), ("add", 2)]
            assert order[-1] == ("put", 1) and order.index(("load", 1)) < len(order) - 1
        finally:
            arplan.ar_plan_destroy(h)


def test_wide_random_plans_use_every_record_kind():
    kinds = set()
    for seed in range(40):
        rng = np.random.default_rng(9300 + seed)
        n = int(rng.choice([8, 17, 33, 64]))
        M = int(rng.integers(3, 120))
        phases = _wide_random_plan(rng, n, M)
        flat = [(q, op, d, s, b * 4, e * 4)
                for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
        h = arplan.ar_plan_create_custom(n, M * 4, "f32", flat)
        try:
            arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, 1)
            units, prog = _resident_tables(h, 0)
            for lo, load, store, nv, off, nw, alias in units:
                kinds |= {r[0] for r in _decode(prog[off:off + nw])}
        finally:
            arplan.ar_plan_destroy(h)
    assert {"fold", "store", "copy"} <= kinds, kinds
