"""GPU parity: the HIP path, called through the C ABI, against the oracle.

fp32 and int32 must match bit for bit (the plan fixes the association
order); bf16 must match the oracle's per-step rounding bit for bit and lie
within 1e-2 normwise of the fp64 sum.  Small and scaled-down workloads are
compared element by element over every buffer, and so are the full-size
workloads, in every executor form the benchmark times.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2409_04202_amd import workloads

from gpu_helpers import run_plan, say, to_device, to_host

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2409_04202_amd import arplan


def _oracle_plan(kind, n, N, fan):
    if kind == "gentree":
        return oracle.gentree_plan(oracle.from_preorder(fan), N)
    return oracle.make_plan(kind, n, N, fan)


def _full_compare(kind, n, N, dtype, fan=None, dist="uniform", seed=1,
                  pad=0, xs0=None, fuse=1, slice_=2, resident=1):
    say("case: %s n=%d N=%d %s fan=%s pad=%d fuse=%d slice=%d resident=%d" % (
        kind, n, N, dtype, fan if kind != "gentree" else len(fan), pad, fuse, slice_,
        resident))
    if xs0 is None:
        xs0 = workloads.draw(n, N, dtype, dist, seed)
    ref = oracle.execute(_oracle_plan(kind, n, N, fan), [x.copy() for x in xs0], dtype)
    ts = to_device(xs0, dtype, pad)
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_FUSE, fuse)
        p.set_option(arplan.AR_OPT_SLICE, slice_)
        p.set_option(arplan.AR_OPT_RESIDENT, resident)
        run_plan(p, ts)
    got = to_host(ts, dtype)
    for q in range(n):
        if not np.array_equal(got[q], ref[q]):
            bad = np.nonzero(got[q] != ref[q])[0]
            raise AssertionError("%s n=%d N=%d %s: processor %d differs at %d "
                                 "positions, first %s" % (kind, n, N, dtype, q,
                                                          len(bad), bad[:8]))
    return got, xs0


def _normwise_bf16(y_bits, xs0):
    r = np.sum([oracle.bf16_to_f32(x).astype(np.float64) for x in xs0], axis=0)
    y = oracle.bf16_to_f32(y_bits).astype(np.float64)
    return np.linalg.norm(y - r) / max(np.linalg.norm(r), 1e-300)


# ------------------------------------------------ small and scaled configs

@pytest.mark.parametrize("name", ["ring_n4_f32", "ring_n4_i32"])
def test_small_config_bit_exact(name):
    c = workloads.CONFIGS[name]
    _full_compare(c["kind"], c["n"], c["N"], c["dtype"], c["fanin"],
                  c["dist"], c["seed"])


SCALED = [("rhd", 8, (1 << 20) + 13, "f32", None, "uniform"),
          ("rhd", 6, (1 << 18) + 3, "f32", None, "uniform"),
          ("rhd", 12, 1 << 16, "bf16", None, "uniform"),
          ("rhd", 8, 1 << 20, "f32", None, "uniform"),
          ("cps", 16, 1 << 18, "bf16", None, "uniform"),
          ("cps", 16, (1 << 18) + 7, "f32", None, "normal"),
          ("tree", 64, (1 << 16) + 5, "f32", (8, 8), "uniform"),
          ("tree", 64, (1 << 16) + 5, "i32", (8, 8), "int1000"),
          ("tree", 512, (1 << 13) + 3, "bf16", (8, 8, 8), "uniform"),
          ("tree", 512, 1 << 15, "bf16", (8, 8, 8), "uniform"),
          ("ring", 4, (1 << 16) + 3, "bf16", None, "uniform"),
          ("rb", 6, 100003, "f32", None, "uniform")]


# (AR_OPT_FUSE, AR_OPT_SLICE, AR_OPT_RESIDENT); whole-plan sliced launches
# run resident for n <= 64 unless resident is 0
MODES = [(1, 2, 1), (0, 0, 1), (1, 1, 1), (0, 1, 1), (1, 1, 0), (0, 2, 0)]


@pytest.mark.parametrize("fuse,slice_,resident", MODES)
@pytest.mark.parametrize("kind,n,N,dtype,fan,dist", SCALED)
def test_scaled_configs_bit_exact(kind, n, N, dtype, fan, dist, fuse, slice_, resident):
    got, xs0 = _full_compare(kind, n, N, dtype, fan, dist, seed=5, fuse=fuse,
                             slice_=slice_, resident=resident)
    if dtype == "bf16":
        assert _normwise_bf16(got[0], xs0) <= 1e-2


@pytest.mark.parametrize("slice_,resident", [(2, 1), (1, 1), (2, 0), (1, 0), (0, 1)])
@pytest.mark.parametrize("name", sorted(k for k in workloads.CONFIGS
                                        if k.startswith("sweep_")))
def test_sweep_configs_bit_exact(name, slice_, resident):
    c = workloads.CONFIGS[name]
    got, xs0 = _full_compare(c["kind"], c["n"], c["N"], c["dtype"],
                             c["fanin"], c["dist"], c["seed"], slice_=slice_,
                             resident=resident)
    if c["dtype"] == "bf16":
        assert _normwise_bf16(got[0], xs0) <= 1e-2


_MIXED_CANDIDATES = [
    ("rhd", 128, 1 << 14, "f32", None), ("tree", 64, 1 << 12, "f32", (4, 4, 4)),
    ("tree", 256, 1 << 19, "f32", (4, 8, 8)), ("tree", 64, 1 << 12, "bf16", (4, 4, 4)),
    ("tree", 64, 1 << 14, "f32", (4, 4, 4)), ("tree", 32, 1 << 16, "bf16", (2, 4, 4)),
    ("rhd", 16, 1 << 14, "f32", None), ("rhd", 16, 1 << 16, "bf16", None),
    ("tree", 64, 1 << 18, "bf16", (4, 4, 4)), ("tree", 128, 1 << 18, "f32", (2, 8, 8)),
    ("tree", 512, 1 << 18, "f32", (8, 8, 8)), ("tree", 32, 1 << 18, "bf16", (2, 4, 4)),
    ("gentree", 384, 384 * 256, "f32",
     tuple(workloads.CONFIGS["cdc384_gentree_f32"]["fanin"])),
    ("gentree", 384, 384 * 512, "f32",
     tuple(workloads.CONFIGS["asy384_gentree_f32"]["fanin"]))]


def test_sliced_runs_between_phase_launches():
    # shapes for which the automatic choice mixes sliced runs and phase
    # launches (which ones depends on the cost model): at least two, and the
    # first three run bit-exact
    mixed = []
    for kind, n, N, dtype, fan in _MIXED_CANDIDATES:
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            ph = [x[0] for x in p.launches()]
        if any(x < 0 for x in ph) and any(x >= 0 for x in ph):
            mixed.append((kind, n, N, dtype, fan))
    assert len(mixed) >= 2, mixed
    for kind, n, N, dtype, fan in mixed[:3]:
        got, xs0 = _full_compare(kind, n, N, dtype, fan, "uniform", seed=11)
        if dtype == "bf16":
            assert _normwise_bf16(got[0], xs0) <= 1e-2


@pytest.mark.parametrize("kind,n,N,dtype,kernel", [
    ("ring", 128, 1 << 12, "f32", "stream_kernel"), ("ring", 256, 1 << 15, "f32", "stream_kernel"),
    ("ring", 128, 1 << 18, "bf16", "stream_kernel"), ("rhd", 128, 1 << 12, "f32", "split_kernel")])
def test_automatic_choice_beyond_64_buffers(kind, n, N, dtype, kernel):
    # the automatic choice for more than 64 buffers: Ring as one streamed
    # launch, RHD's short 128-destination phase as a split launch
    # (tests/test_capi_host.py pins the choices); every element vs the oracle
    with arplan.Plan(n, N, dtype, kind) as p:
        assert kernel in p.launch_kernels()
    got, xs0 = _full_compare(kind, n, N, dtype, None, "uniform", seed=n + 5)
    if dtype == "bf16":
        # bit-exact with the oracle above; against the exact sum, Ring's
        # chain rounds to bf16 (unit roundoff 2^-8) after each of its n - 1
        # steps: a random walk of about sqrt(n) roundings (0.013 measured
        # at n = 128, where 1 % holds for the trees and n <= 64)
        assert _normwise_bf16(got[0], xs0) <= 2.0 ** -8 * np.sqrt(n)


# ------------------------------------------- full size, every element

# The executor forms the benchmark times: the default choice, phase launches
# with the rewrites, and the plan as written (every step as listed, one
# launch per phase).  (AR_OPT_FUSE, AR_OPT_SLICE, AR_OPT_RESIDENT)
BENCH_FORMS = [("default", 1, 2, 1), ("phase launches", 1, 0, 1), ("as written", 0, 0, 1)]


def _full_size_every_element(name, forms):
    """Run the full-size workload once per form from the same inputs and
    compare every element of every buffer with the oracle's run of the
    plan (computed once)."""
    c = workloads.CONFIGS[name]
    n, N, dt = c["n"], c["N"], c["dtype"]
    say("case: full-size %s: drawing inputs and running the oracle" % name)
    xs0 = workloads.inputs(name)
    ref = oracle.execute(_oracle_plan(c["kind"], n, N, c["fanin"]),
                         [x.copy() for x in xs0], dt)
    pristine = to_device(xs0, dt)
    for label, fuse, slice_, resident in forms:
        say("case: full-size %s, %s (fuse=%d slice=%d resident=%d)" % (
            name, label, fuse, slice_, resident))
        ts = [t.clone() for t in pristine]
        with arplan.Plan(n, N, dt, c["kind"], c["fanin"]) as p:
            p.set_option(arplan.AR_OPT_FUSE, fuse)
            p.set_option(arplan.AR_OPT_SLICE, slice_)
            p.set_option(arplan.AR_OPT_RESIDENT, resident)
            kinds = sorted({x[0] for x in p.launches()})
            run_plan(p, ts)
        say("  launch kinds %s" % kinds)
        for q in range(n):
            g = ts[q].cpu().numpy()
            g = g.view(np.uint16) if dt == "bf16" else g
            if not np.array_equal(g, ref[q]):
                bad = np.nonzero(g != ref[q])[0]
                raise AssertionError("%s %s: processor %d differs at %d positions, "
                                     "first %s" % (name, label, q, len(bad), bad[:8]))
        del ts
    if dt == "bf16":
        err = _normwise_bf16(ref[0], xs0)
        say("bf16 normwise error %.3e" % err)
        assert err <= 1e-2
    return kinds


@pytest.mark.parametrize("name", ["rhd_n8_f32", "cps_n16_f32",
                                  "tree8x8_n64_f32", "tree8x8_n64_i32",
                                  "tree8x8x8_n512_bf16", "asy384_gentree_f32",
                                  "cdc384_gentree_f32"])
def test_full_size_configs(name):
    _full_size_every_element(name, BENCH_FORMS)


@pytest.mark.parametrize("N", [(1 << 24) + 160, (1 << 21) + 160])
def test_large_resident_with_partial_tiles(N):
    # RHD n = 8 as one resident launch whose segments end in a partial tile
    # (N / 8 is not a multiple of 256 elements); at 2^24 + 160 the run moves
    # more than the last-level cache and streams its rows nontemporally
    with arplan.Plan(8, N, "f32", "rhd") as p:
        if N > 1 << 24:  # the default choice at this size
            assert [x[0] for x in p.launches()] == [-2]
        p.set_option(arplan.AR_OPT_SLICE, 1)
        L = p.launches()
        assert [x[0] for x in L] == [-2] and L[0][4] == 2 * 8 * N * 4
    _full_compare("rhd", 8, N, "f32", None, "uniform", seed=N % 97, slice_=1)


@pytest.mark.parametrize("dtype,N", [("bf16", 1 << 25), ("i32", (1 << 24) + 160)])
def test_large_resident_nontemporal_dtypes(dtype, N):
    # RHD n = 8 as one resident launch moving more than the last-level cache
    # (nontemporal rows) in bf16 and int32, every element
    n = 8
    with arplan.Plan(n, N, dtype, "rhd") as p:
        L = p.launches()
        assert [x[0] for x in L] == [-2] and L[0][4] > 512 << 20
    _full_compare("rhd", n, N, dtype, None, "int1000" if dtype == "i32" else "uniform",
                  seed=21)


# ------------------------------------------- streamed runs (n > 64 buffers)

STREAMED = [("tree", 512, 1 << 15, "bf16", (8, 8, 8)), ("tree", 512, 1 << 16, "f32", (8, 8, 8)),
            ("ring", 70, 70 * 4 * 64, "f32", None), ("ring", 65, 65 * 8 * 3, "bf16", None),
            ("rhd", 128, 128 * 4 * 40, "f32", None), ("rhd", 96, 96 * 4 * 8, "i32", None),
            ("tree", 96, 96 * 4 * 30, "i32", (4, 4, 6)),
            ("gentree", 384, 384 * 256, "f32",
             tuple(workloads.CONFIGS["cdc384_gentree_f32"]["fanin"])),
            ("gentree", 384, 384 * 512, "bf16",
             tuple(workloads.CONFIGS["asy384_gentree_f32"]["fanin"]))]


@pytest.mark.parametrize("kind,n,N,dtype,fan", STREAMED)
@pytest.mark.parametrize("fuse", [1, 0])
def test_streamed_whole_plan(kind, n, N, dtype, fan, fuse):
    # the whole plan as one streamed launch (LDS slots shared by values,
    # loads ahead, stores as soon as a final value is there), bit-exact
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_FUSE, fuse)
        p.set_option(arplan.AR_OPT_SLICE, 1)
        assert [x[0] for x in p.launches()] == [-3]
    dist = "int1000" if dtype == "i32" else "uniform"
    got, xs0 = _full_compare(kind, n, N, dtype, fan, dist, seed=n + fuse, fuse=fuse, slice_=1)
    if dtype == "bf16":
        assert _normwise_bf16(got[0], xs0) <= 1e-2


@pytest.mark.parametrize("seed", range(24))
def test_streamed_random_custom_plans(seed):
    # random hazard-free plans over 65-200 buffers (folds of 3-16 sources,
    # copies into up to 40 buffers; the host-side program test's generator)
    # as one streamed launch, and with the default executor, bit-exact
    from plan_gen import wide_random_plan as _wide_random_plan
    from oracle.plans import Plan as OPlan, Step as OStep
    rng = np.random.default_rng(9500 + seed)
    n = int(rng.choice([65, 80, 130, 200]))
    M = int(rng.integers(3, 90))
    phases = _wide_random_plan(rng, n, M)
    dtype = ("f32", "bf16", "i32")[seed % 3]
    vec = 8 if dtype == "bf16" else 4
    N = M * vec
    flat = [(q, op, d, s_, b * vec, e * vec)
            for q, ph in enumerate(phases) for (op, d, s_, b, e) in ph]
    ref_plan = OPlan("custom", n, N, [[OStep(op, d, s_, b * vec, e * vec)
                                       for (op, d, s_, b, e) in ph] for ph in phases])
    xs0 = workloads.draw(n, N, dtype, "int1000" if dtype == "i32" else "uniform", seed)
    ref = oracle.execute(ref_plan, [x.copy() for x in xs0], dtype)
    say("case: streamed random custom plan seed=%d n=%d N=%d %s" % (seed, n, N, dtype))
    for sl in (1, 2):
        ts = to_device(xs0, dtype)
        h = arplan.ar_plan_create_custom(n, N, dtype, flat)
        try:
            arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, sl)
            if sl == 1:
                assert arplan.ar_plan_launch_info(h, 0)[0] == -3
            arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
            torch.cuda.synchronize()
        finally:
            arplan.ar_plan_destroy(h)
        got = to_host(ts, dtype)
        for q in range(n):
            assert np.array_equal(got[q], ref[q]), (seed, sl, q)


def test_streamed_held_back_store():
    # a store into a buffer whose initial row a later fold still needs
    # (held back to the end of the program), bit-exact on the GPU
    from oracle.plans import Plan as OPlan, Step as OStep
    n = 70
    for dtype in ("f32", "bf16"):
        vec = 8 if dtype == "bf16" else 4
        N = 64 * vec * 3
        flat = [(0, "reduce", 4, list(range(10, 64)) + [1], 0, N),
                (1, "reduce", 1, [2, 3], 0, N), (2, "reduce", 4, [4, 7], 0, N)]
        ref_plan = OPlan("custom", n, N, [[OStep(op, d, s_, b, e)] for (_, op, d, s_, b, e) in flat])
        xs0 = workloads.draw(n, N, dtype, "uniform", 3)
        ref = oracle.execute(ref_plan, [x.copy() for x in xs0], dtype)
        ts = to_device(xs0, dtype)
        h = arplan.ar_plan_create_custom(n, N, dtype, flat)
        try:
            arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, 1)
            assert arplan.ar_plan_launch_info(h, 0)[0] == -3
            arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
            torch.cuda.synchronize()
        finally:
            arplan.ar_plan_destroy(h)
        got = to_host(ts, dtype)
        for q in range(n):
            assert np.array_equal(got[q], ref[q]), (dtype, q)


@pytest.mark.parametrize("name", ["tree8x8x8_n512_bf16", "asy384_gentree_f32",
                                  "cdc384_gentree_f32"])
def test_streamed_full_size(name):
    # the full-size workloads with more than 64 buffers as one streamed
    # launch, every element
    c = workloads.CONFIGS[name]
    with arplan.Plan(c["n"], c["N"], c["dtype"], c["kind"], c["fanin"]) as p:
        p.set_option(arplan.AR_OPT_SLICE, 1)
        assert [x[0] for x in p.launches()] == [-3]
    _full_size_every_element(name, [("whole plan streamed", 1, 1, 1)])


# --------------------------------------------------------------- edge cases

@pytest.mark.parametrize("kind,n,fan", [("ring", 5, None), ("rhd", 4, None), ("rhd", 5, None),
                                        ("cps", 7, None), ("tree", 12, (3, 4)),
                                        ("rb", 3, None)])
@pytest.mark.parametrize("dtype", ["f32", "i32", "bf16"])
def test_ragged_and_tiny_sizes(kind, n, fan, dtype):
    for N in (1, n - 1, n, n + 1, 2 * n + 3, 4099, 64 * n):
        dist = "int1000" if dtype == "i32" else "uniform"
        for fuse, sl, res in MODES:
            _full_compare(kind, n, N, dtype, fan, dist, seed=N, fuse=fuse, slice_=sl,
                          resident=res)


def test_empty_buffers_are_a_no_op():
    for kind, n, fan in (("ring", 4, None), ("tree", 4, (2, 2))):
        ts = to_device([np.zeros(0, np.float32)] * n, "f32")
        with arplan.Plan(n, 0, "f32", kind, fan) as p:
            run_plan(p, ts)


@pytest.mark.parametrize("dtype,pad", [("f32", 1), ("f32", 2), ("i32", 3),
                                       ("bf16", 1), ("bf16", 5)])
def test_unaligned_buffers(dtype, pad):
    dist = "int1000" if dtype == "i32" else "uniform"
    for fuse, sl, res in MODES:
        kw = dict(pad=pad, fuse=fuse, slice_=sl, resident=res)
        _full_compare("tree", 8, 10007, dtype, (4, 2), dist, seed=3, **kw)
        _full_compare("ring", 3, 4099, dtype, None, dist, seed=4, **kw)
        _full_compare("cps", 5, 3001, dtype, None, dist, seed=6, **kw)
        _full_compare("ring", 4, 4096, dtype, None, dist, seed=7, **kw)
        # 16 destinations per step, each also a source
        _full_compare("cps", 16, 20011, dtype, None, dist, seed=8, **kw)


@pytest.mark.parametrize("n", [3, 5, 16, 32])
def test_source_counts(n):
    # k = 3 and 16 have unrolled kernels, 5 and 32 use the runtime loop
    for dtype in ("f32", "bf16"):
        for fuse, sl, res in MODES:
            kw = dict(fuse=fuse, slice_=sl, resident=res)
            _full_compare("cps", n, 50021, dtype, None, "uniform", seed=n, **kw)
            _full_compare("cps", n, 512 * n, dtype, None, "uniform", seed=n, **kw)


def test_runtime_source_count_long_launch():
    # a 32-source fold of more than 512 MiB: the runtime-source-count kernel
    # one source at a time (shorter launches group four sources)
    got, xs0 = _full_compare("cps", 32, (1 << 22) + 17, "f32", seed=3, fuse=0, slice_=0)


def test_fp32_denormals_are_kept():
    n, N = 4, 8192
    rng = np.random.default_rng(7)
    xs0 = [((rng.random(N) * 2 - 1) * 1e-39).astype(np.float32)
           for _ in range(n)]
    assert any(np.any((np.abs(x) < 1.17e-38) & (x != 0)) for x in xs0)
    got, _ = _full_compare("cps", n, N, "f32", xs0=xs0)
    assert np.any((np.abs(got[0]) < 1.17e-38) & (got[0] != 0))


def test_int32_wraps():
    n, N = 4, 4096
    xs0 = [np.full(N, 2**31 - 1 - q, np.int32) for q in range(n)]
    _full_compare("ring", n, N, "i32", xs0=xs0)
    _full_compare("cps", n, N, "i32", xs0=xs0)


def test_bf16_ties_round_to_even():
    # 1 + 2^-8 and 1 + 3*2^-8 are halfway between bf16 neighbours.
    n, N = 2, 4096
    one = np.uint16(0x3F80)                  # 1.0
    eps = np.uint16(0x3B80)                  # 2^-8
    three = np.uint16(0x3C40)                # 3 * 2^-8
    a = np.full(N, one, np.uint16)
    b = np.where(np.arange(N) % 2 == 0, eps, three).astype(np.uint16)
    got, _ = _full_compare("cps", n, N, "bf16", xs0=[a, b])
    assert np.all(got[0][0::2] == 0x3F80)    # tie to even: 1.0
    assert np.all(got[0][1::2] == 0x3F82)    # 1 + 2^-6 (even mantissa)


def _bf16_rounding_inputs(seed):
    # a: every finite bf16 pattern; b: a value 8 to 10 binades below a (a
    # random denormal where that underflows), random sign and mantissa, so
    # that the exact fp32 sum a + b needs rounding: ties, carries into the
    # exponent, overflow to infinity at the top, cancellation, denormal
    # results
    rng = np.random.default_rng(seed)
    pats = np.arange(65536, dtype=np.uint32)
    exp = (pats >> 7) & 0xFF
    a = pats[exp != 0xFF]
    e = (a >> 7) & 0xFF
    d = rng.integers(8, 11, a.size).astype(np.uint32)
    sgn = rng.integers(0, 2, a.size).astype(np.uint32) << 15
    man = rng.integers(0, 128, a.size).astype(np.uint32)
    b = np.where(e > d, sgn | ((e - d) << 7) | man, sgn | man)
    return a.astype(np.uint16), b.astype(np.uint16)


@pytest.mark.parametrize("fuse,slice_,resident", MODES)
def test_bf16_rounding_every_exponent(fuse, slice_, resident):
    a, b = _bf16_rounding_inputs(3)
    N = a.size - a.size % 8
    xs0 = [a[:N].copy(), b[:N].copy()]
    got, _ = _full_compare("cps", 2, N, "bf16", xs0=xs0, fuse=fuse, slice_=slice_,
                           resident=resident)
    f = oracle.bf16_to_f32(got[0])
    assert np.isinf(f).any() and (np.abs(f[f != 0]) < 1.2e-38).any()


def test_bf16_nan_and_inf_inputs():
    # NaN inputs give NaN, infinities add as in IEEE; the NaN payload after
    # an add is the hardware's choice, so NaNs are compared as NaNs
    n, N = 4, 4096
    rng = np.random.default_rng(17)
    xs0 = [oracle.f32_to_bf16((rng.random(N) * 2 - 1).astype(np.float32))
           for _ in range(n)]
    xs0[1][::7] = 0x7FC1                     # quiet NaN, payload 1
    xs0[2][::11] = 0xFF81                    # signalling NaN, negative
    xs0[0][::13] = 0x7F80                    # +inf
    xs0[3][::17] = 0xFF80                    # -inf
    ref = oracle.execute(oracle.cps(n, N), [x.copy() for x in xs0], "bf16")
    for fuse, sl, res in MODES:
        ts = to_device(xs0, "bf16")
        with arplan.Plan(n, N, "bf16", "cps") as p:
            p.set_option(arplan.AR_OPT_FUSE, fuse)
            p.set_option(arplan.AR_OPT_SLICE, sl)
            p.set_option(arplan.AR_OPT_RESIDENT, res)
            run_plan(p, ts)
        got = to_host(ts, "bf16")
        for q in range(n):
            gf, rf = oracle.bf16_to_f32(got[q]), oracle.bf16_to_f32(ref[q])
            assert np.array_equal(np.isnan(gf), np.isnan(rf))
            ok = ~np.isnan(rf)
            assert np.array_equal(got[q][ok], ref[q][ok])
            assert np.isnan(rf).any() and np.isinf(rf).any()


@pytest.mark.parametrize("seed", range(24))
def test_random_custom_plans(seed):
    # random hazard-free plans with copy chains (the same generator as the
    # host-side rewrite test), every executor mode, bit-exact vs the oracle
    from test_exec_rewrites_host import _random_plan
    from oracle.plans import Plan as OPlan, Step as OStep
    rng = np.random.default_rng(9000 + seed)
    n = int(rng.integers(2, 7))
    N = int(rng.integers(8, 4000))
    phases = _random_plan(rng, n, N)
    flat = [(q, op, d, s, b, e) for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref_plan = OPlan("custom", n, N, [[OStep(*st) for st in ph] for ph in phases])
    dtype = ("f32", "bf16", "i32")[seed % 3]
    xs0 = workloads.draw(n, N, dtype, "int1000" if dtype == "i32" else "uniform", seed)
    ref = oracle.execute(ref_plan, [x.copy() for x in xs0], dtype)
    say("case: random custom plan seed=%d n=%d N=%d %s phases=%d" % (seed, n, N, dtype, len(phases)))
    for fuse, sl, res in MODES:
        for pad in (0, 1):
            ts = to_device(xs0, dtype, pad)
            h = arplan.ar_plan_create_custom(n, N, dtype, flat)
            try:
                arplan.ar_plan_set_option(h, arplan.AR_OPT_FUSE, fuse)
                arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, sl)
                arplan.ar_plan_set_option(h, arplan.AR_OPT_RESIDENT, res)
                arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
                torch.cuda.synchronize()
            finally:
                arplan.ar_plan_destroy(h)
            got = to_host(ts, dtype)
            for q in range(n):
                assert np.array_equal(got[q], ref[q]), (seed, fuse, sl, pad, q)


@pytest.mark.parametrize("seed", range(12))
def test_random_many_destination_plans(seed):
    # random plans whose executed steps store to 17+ buffers, some of them
    # their own sources, over ragged blocks: split launches (phase launches
    # and the default form, aligned and unaligned buffers), bit-exact vs the
    # oracle run on the plan as written
    from plan_gen import many_destination_plan
    from oracle.plans import Plan as OPlan, Step as OStep
    rng = np.random.default_rng(7100 + seed)
    n = int(rng.integers(17, 41))
    N = int(rng.integers(1000, 200000))
    phases = many_destination_plan(rng, n, N)
    flat = [(q, op, d, s, b, e) for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref_plan = OPlan("custom", n, N, [[OStep(*st) for st in ph] for ph in phases])
    dtype = ("f32", "bf16", "i32")[seed % 3]
    xs0 = workloads.draw(n, N, dtype, "int1000" if dtype == "i32" else "uniform", seed)
    ref = oracle.execute(ref_plan, [x.copy() for x in xs0], dtype)
    say("case: random many-destination plan seed=%d n=%d N=%d %s" % (seed, n, N, dtype))
    for sl in (0, 2):
        for pad in (0, 1):
            ts = to_device(xs0, dtype, pad)
            h = arplan.ar_plan_create_custom(n, N, dtype, flat)
            try:
                arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, sl)
                arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
                torch.cuda.synchronize()
            finally:
                arplan.ar_plan_destroy(h)
            got = to_host(ts, dtype)
            for q in range(n):
                assert np.array_equal(got[q], ref[q]), (seed, sl, pad, q)


@pytest.mark.parametrize("seed", range(16))
def test_random_aligned_custom_plans_resident(seed):
    # random hazard-free plans whose boundaries are whole 16-byte vectors, so
    # that the whole plan runs as one resident launch (ragged tiles, several
    # 64-word program chunks); against the oracle and the plain sliced launch
    from test_exec_rewrites_host import _random_plan
    from oracle.plans import Plan as OPlan, Step as OStep
    rng = np.random.default_rng(9500 + seed)
    n = int(rng.integers(2, 7))
    M = int(rng.integers(40, 3000))
    phases = _random_plan(rng, n, M)
    dtype = ("f32", "bf16", "i32")[seed % 3]
    vec = 8 if dtype == "bf16" else 4
    N = M * vec
    flat = [(q, op, d, s, b * vec, e * vec)
            for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref_plan = OPlan("custom", n, N, [[OStep(op, d, s, b * vec, e * vec)
                                       for (op, d, s, b, e) in ph] for ph in phases])
    xs0 = workloads.draw(n, N, dtype, "int1000" if dtype == "i32" else "uniform", seed)
    ref = oracle.execute(ref_plan, [x.copy() for x in xs0], dtype)
    say("case: aligned custom plan seed=%d n=%d N=%d %s phases=%d" % (seed, n, N, dtype, len(phases)))
    for res in (1, 0):
        ts = to_device(xs0, dtype)
        h = arplan.ar_plan_create_custom(n, N, dtype, flat)
        try:
            arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, 1)
            arplan.ar_plan_set_option(h, arplan.AR_OPT_RESIDENT, res)
            assert arplan.ar_plan_launch_info(h, 0)[0] == (-2 if res else -1)
            arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
            torch.cuda.synchronize()
        finally:
            arplan.ar_plan_destroy(h)
        got = to_host(ts, dtype)
        for q in range(n):
            assert np.array_equal(got[q], ref[q]), (seed, res, q)


@pytest.mark.parametrize("seed", range(12))
def test_wide_random_plans_resident(seed):
    # 8-64 buffers, folds of up to 16 sources, copies into up to 40 buffers
    # (fold and store records); whole plan resident, plain sliced and the
    # default choice, against the oracle
    from plan_gen import wide_random_plan as _wide_random_plan
    from oracle.plans import Plan as OPlan, Step as OStep
    rng = np.random.default_rng(9600 + seed)
    n = int(rng.choice([8, 17, 33, 64]))
    M = int(rng.integers(3, 600))
    phases = _wide_random_plan(rng, n, M)
    dtype = ("f32", "bf16", "i32")[seed % 3]
    vec = 8 if dtype == "bf16" else 4
    N = M * vec
    flat = [(q, op, d, s, b * vec, e * vec)
            for q, ph in enumerate(phases) for (op, d, s, b, e) in ph]
    ref_plan = OPlan("custom", n, N, [[OStep(op, d, s, b * vec, e * vec)
                                       for (op, d, s, b, e) in ph] for ph in phases])
    xs0 = workloads.draw(n, N, dtype, "int1000" if dtype == "i32" else "uniform", seed)
    ref = oracle.execute(ref_plan, [x.copy() for x in xs0], dtype)
    say("case: wide custom plan seed=%d n=%d N=%d %s phases=%d" % (seed, n, N, dtype, len(phases)))
    for sl, res in ((1, 1), (1, 0), (2, 1)):
        ts = to_device(xs0, dtype)
        h = arplan.ar_plan_create_custom(n, N, dtype, flat)
        try:
            arplan.ar_plan_set_option(h, arplan.AR_OPT_SLICE, sl)
            arplan.ar_plan_set_option(h, arplan.AR_OPT_RESIDENT, res)
            arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
            torch.cuda.synchronize()
        finally:
            arplan.ar_plan_destroy(h)
        got = to_host(ts, dtype)
        for q in range(n):
            assert np.array_equal(got[q], ref[q]), (seed, sl, res, q)


@pytest.mark.parametrize("kind,n,fan", [("ring", 64, None), ("tree", 64, (8, 8)),
                                        ("tree", 64, (4, 4, 4)), ("rhd", 32, None),
                                        ("cps", 64, None), ("ring", 2, None)])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32"])
def test_whole_plan_resident_bit_exact(kind, n, fan, dtype):
    # every built-in plan kind as one resident launch, at sizes with ragged
    # last tiles per segment
    vec = 8 if dtype == "bf16" else 4
    dist = "int1000" if dtype == "i32" else "uniform"
    for N in (n * vec, n * vec * 37, n * vec * 301):
        _full_compare(kind, n, N, dtype, fan, dist, seed=N + n, slice_=1, resident=1)


def test_custom_plan_mixed_sources_and_uneven_steps():
    # one phase with a 3-way reduce over a long range and 2-way reduces over
    # tiny ranges (explicit tile table), then copies of uneven lengths
    n, N = 4, 300001
    steps = [(0, "reduce", 0, [0, 1, 2], 0, 280000),
             (0, "reduce", 3, [3, 1], 280000, 280007),
             (0, "reduce", 2, [2, 3], 280007, 300001),
             (1, "copy", 1, [0], 0, 280000),
             (1, "copy", 0, [3], 280000, 280007),
             (1, "copy", 3, [2], 290000, 290001)]
    xs0 = workloads.draw(n, N, "f32", "uniform", 8)
    ref = [x.copy() for x in xs0]
    ph = [[oracle.Step(o, d, tuple(s), b, e) for (p_, o, d, s, b, e) in steps
           if p_ == k] for k in (0, 1)]
    oracle.execute(oracle.Plan("custom", n, N, ph), ref, "f32")
    ts = to_device(xs0, "f32")
    h = arplan.ar_plan_create_custom(n, N, "f32", steps)
    try:
        arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
        torch.cuda.synchronize()
    finally:
        arplan.ar_plan_destroy(h)
    got = to_host(ts, "f32")
    for q in range(n):
        assert np.array_equal(got[q], ref[q]), q


def test_pointer_table_cache_and_strided():
    n, N = 8, 65539
    plan_o = oracle.rhd(n, N)
    with arplan.Plan(n, N, "f32", "rhd") as p:
        for rep in range(6):            # more buffer sets than cached tables
            xs0 = workloads.draw(n, N, "f32", "uniform", 100 + rep)
            ref = oracle.execute(plan_o, [x.copy() for x in xs0], "f32")
            ts = to_device(xs0, "f32")
            run_plan(p, ts)
            got = to_host(ts, "f32")
            assert all(np.array_equal(got[q], ref[q]) for q in range(n)), rep
        xs0 = workloads.draw(n, N, "f32", "uniform", 200)
        ref = oracle.execute(plan_o, [x.copy() for x in xs0], "f32")
        stride = N + 29
        big = torch.zeros(n * stride, dtype=torch.float32, device="cuda")
        for q in range(n):
            big[q * stride:q * stride + N].copy_(torch.from_numpy(xs0[q]))
        p.execute_strided(big, stride * 4, torch.cuda.current_stream())
        torch.cuda.synchronize()
        for q in range(n):
            g = big[q * stride:q * stride + N].cpu().numpy()
            assert np.array_equal(g, ref[q]), q


def test_repeated_execution_and_overlapping_buffers_rejected():
    n, N = 16, 40000
    xs0 = workloads.draw(n, N, "f32", "normal", 12)
    plan_o = oracle.tree((4, 4), N)
    ref = oracle.execute(plan_o, [x.copy() for x in xs0], "f32")
    ref = oracle.execute(plan_o, ref, "f32")
    ts = to_device(xs0, "f32")
    with arplan.Plan(n, N, "f32", "tree", (4, 4)) as p:
        run_plan(p, ts)
        run_plan(p, ts)
        got = to_host(ts, "f32")
        assert all(np.array_equal(got[q], ref[q]) for q in range(n))
        bad = list(ts)
        bad[3] = ts[2][5:]
        with pytest.raises(arplan.ArError) as e:
            p.execute(bad, torch.cuda.current_stream())
        assert e.value.status == arplan.AR_ERR_INVALID_ARG
        bad[3] = 0
        with pytest.raises(arplan.ArError):
            p.execute(bad, torch.cuda.current_stream())


def test_timer_records_each_launch():
    n, N = 8, 1 << 20
    xs0 = workloads.draw(n, N, "f32", "uniform", 13)
    ts = to_device(xs0, "f32")
    t = arplan.ar_timer_create(64)
    try:
        with arplan.Plan(n, N, "f32", "rhd") as p:
            p.set_option(arplan.AR_OPT_SLICE, 0)
            for _ in range(2):
                p.execute_timed(ts, torch.cuda.current_stream(), t)
            recs = arplan.ar_timer_read(t, 64)
            nl = len(p.launches())
            assert [li for li, _ in recs] == list(range(nl)) * 2
            assert all(ms > 0 for _, ms in recs)
            arplan.ar_timer_reset(t)
            assert arplan.ar_timer_read(t, 64) == []
    finally:
        arplan.ar_timer_destroy(t)


def test_runs_on_a_side_stream_in_order():
    # inputs are written, the plan runs and the result is read back, all on
    # a non-default torch stream: the library must honour its ordering
    n, N = 16, (1 << 18) + 3
    xs0 = workloads.draw(n, N, "f32", "uniform", 14)
    ref = oracle.execute(oracle.cps(n, N), [x.copy() for x in xs0], "f32")
    hs = [torch.from_numpy(x).pin_memory() for x in xs0]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        ts = [torch.empty(N, dtype=torch.float32, device="cuda") for _ in range(n)]
        for t, h in zip(ts, hs):
            t.copy_(h, non_blocking=True)
        with arplan.Plan(n, N, "f32", "cps") as p:
            p.execute(ts, s)
            outs = [t.to("cpu", non_blocking=False) for t in ts]
    s.synchronize()
    for q in range(n):
        assert np.array_equal(outs[q].numpy(), ref[q]), q


@pytest.mark.parametrize("kind,n,N,fan,slice_,resident", [
    ("ring", 8, 8 * 1024, None, 1, 1),           # one resident launch
    ("ring", 8, 8 * 1024, None, 1, 0),           # one plain sliced launch
    ("rhd", 8, 1 << 20, None, 0, 1),             # phase launches
    ("tree", 64, 64 * 256, (8, 8), 2, 1),        # the default choice
    ("ring", 128, 128 * 32, None, 2, 1)])        # the default choice: streamed
def test_graph_capture_replays(kind, n, N, fan, slice_, resident):
    # an execution captured in a HIP graph after a first eager execution (which
    # uploads the step records, so that capture records kernel launches only)
    # replays the same work: every replay, with eager work and a
    # synchronisation between replays, matches the oracle applied once more
    xs0 = workloads.draw(n, N, "i32", "int1000", 21)
    plan_o = _oracle_plan(kind, n, N, fan)
    want = oracle.execute(plan_o, [x.copy() for x in xs0], "i32")
    say("case: graph capture %s n=%d N=%d slice=%d resident=%d" % (kind, n, N, slice_, resident))
    ts = to_device(xs0, "i32")
    with arplan.Plan(n, N, "i32", kind, fan) as p:
        p.set_option(arplan.AR_OPT_SLICE, slice_)
        p.set_option(arplan.AR_OPT_RESIDENT, resident)
        run_plan(p, ts)
        got = to_host(ts, "i32")
        assert all(np.array_equal(got[q], want[q]) for q in range(n))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            p.execute(ts, torch.cuda.current_stream())
        torch.cuda.synchronize()
        got = to_host(ts, "i32")   # capture does not run the work
        assert all(np.array_equal(got[q], want[q]) for q in range(n))
        for r in range(3):
            g.replay()
            torch.cuda.synchronize()
            want = oracle.execute(plan_o, want, "i32")
            got = to_host(ts, "i32")
            assert all(np.array_equal(got[q], want[q]) for q in range(n)), r
            extra = (ts[0].to(torch.int64) + 1).sum()   # eager work between replays
            torch.cuda.synchronize()
            assert int(extra.item()) == int(want[0].astype(np.int64).sum()) + N


@pytest.mark.parametrize("resident", [1, 0])
def test_whole_plan_launch_with_timer_and_repeats(resident):
    n, N = 64, 1 << 14
    xs0 = workloads.draw(n, N, "f32", "uniform", 15)
    plan_o = oracle.ring(n, N)
    ref = oracle.execute(plan_o, [x.copy() for x in xs0], "f32")
    ref2 = oracle.execute(plan_o, [x.copy() for x in ref], "f32")
    ts = to_device(xs0, "f32")
    t = arplan.ar_timer_create(8)
    try:
        with arplan.Plan(n, N, "f32", "ring") as p:
            p.set_option(arplan.AR_OPT_SLICE, 1)
            p.set_option(arplan.AR_OPT_RESIDENT, resident)
            (ph, k, d, cnt, b), = p.launches()
            assert ph == (-2 if resident else -1)
            p.execute_timed(ts, torch.cuda.current_stream(), t)
            torch.cuda.synchronize()
            got = to_host(ts, "f32")
            assert all(np.array_equal(got[q], ref[q]) for q in range(n))
            p.execute_timed(ts, torch.cuda.current_stream(), t)
            torch.cuda.synchronize()
            got = to_host(ts, "f32")
            assert all(np.array_equal(got[q], ref2[q]) for q in range(n))
            recs = arplan.ar_timer_read(t, 8)
            assert [li for li, _ in recs] == [0, 0] and all(ms > 0 for _, ms in recs)
    finally:
        arplan.ar_timer_destroy(t)


GENTREES = [[3, 0, 0, 2, 0, 0], [2, 0, 2, 0, 2, 0, 0],
            [3, 3, 4, 0, 0, 0, 0, 2, 0, 0, 0, 3, 4, 0, 0, 0, 0, 0, 0, 2, 4, 0,
             0, 0, 0, 2, 0, 0],
            workloads.preorder([[4] * 2] * 2 + [[2] * 2] * 2),
            workloads.preorder([[[4] * 2] * 2, [[2] * 2] * 2])]


@pytest.mark.parametrize("counts", GENTREES)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32"])
def test_gentree_plans_bit_exact(counts, dtype):
    n = counts.count(0)
    dist = "int1000" if dtype == "i32" else "uniform"
    for N in (n, 64 * n, 64 * n + 5, 40000):
        for fuse, sl, res in MODES:
            _full_compare("gentree", n, N, dtype, counts, dist, seed=N, fuse=fuse,
                          slice_=sl, resident=res)


@pytest.mark.parametrize("name", ["asy384_gentree_f32", "cdc384_gentree_f32"])
def test_paper_asymmetric_topologies_scaled(name):
    c = workloads.CONFIGS[name]
    for fuse, sl, res in MODES:
        _full_compare("gentree", c["n"], 384 * 64 + 17, "f32", c["fanin"], seed=3,
                      fuse=fuse, slice_=sl, resident=res)


@pytest.mark.parametrize("kind,n,N,fan,dtype", [
    ("cps", 16, (1 << 14) + 3, None, "f32"), ("cps", 32, 32 * 1000 + 17, None, "bf16"),
    ("cps", 16, 4096, None, "i32"), ("tree", 512, 1 << 15, (8, 8, 8), "bf16"),
    ("tree", 64, 4096 + 64 * 5, (8, 8), "f32"), ("ring", 64, 64 * 1000, None, "f32"),
    ("tree", 512, 1 << 20, (8, 8, 8), "bf16"), ("tree", 64, 65553, (16, 4), "f32"),
    ("tree", 256, 65553, (16, 16), "f32"), ("cps", 17, 1 << 20, None, "f32"),
    ("tree", 96, 1 << 20, (3, 32), "f32")])
def test_many_destination_phase_launches(kind, n, N, fan, dtype):
    # phase launches whose steps store to 16 or more buffers, some of them
    # the step's own sources (the reduce-then-broadcast rewrite): split
    # launches, a workgroup per tile, with 2, 4, 8, 16 sources and a runtime
    # source count, cached and nontemporal stores, and at 2^20 elements
    # large launches that stay one wave per tile (tests/test_capi_host.py
    # checks which is which)
    dist = "int1000" if dtype == "i32" else "uniform"
    got, xs0 = _full_compare(kind, n, N, dtype, fan, dist, seed=N % 101, slice_=0)
    if dtype == "bf16":
        assert _normwise_bf16(got[0], xs0) <= 1e-2


@pytest.mark.parametrize("kind,n,N,fan,dtype", [
    ("ring", 64, 1 << 20, None, "f32"), ("ring", 64, 1 << 20, None, "bf16"),
    ("ring", 8, 1 << 18, None, "f32"), ("rhd", 8, 1 << 18, None, "f32"),
    ("rhd", 5, (1 << 18) + 3, None, "i32"), ("cps", 6, 1 << 20, None, "f32"),
    ("tree", 32, 1 << 18, (8, 4), "f32"), ("ring", 16, (1 << 18) + 5, None, "bf16")])
@pytest.mark.parametrize("pad", [0, 1])
def test_fine_tile_launches(kind, n, N, fan, dtype, pad):
    # the plan as written, its launches of few tiles cut below a full kernel
    # pass (down to one vector per lane; tests/test_capi_host.py checks the
    # tiles), every element against the oracle; with buffers off 16-byte
    # alignment (pad) the same tiles run element by element
    dist = "int1000" if dtype == "i32" else "uniform"
    got, xs0 = _full_compare(kind, n, N, dtype, fan, dist, seed=N % 97, pad=pad,
                             fuse=0, slice_=0)
    if dtype == "bf16":
        assert _normwise_bf16(got[0], xs0) <= 1e-2


@pytest.mark.parametrize("N,dtype", [((1 << 26) + 13, "f32"), (1 << 26, "i32"), (1 << 27, "bf16")])
def test_wide_two_source_launches(N, dtype):
    # RHD as written at 2-3 GiB: its first halving launch runs the wide
    # 2-source instance (tests/test_capi_host.py checks which launch); a
    # ragged size, int32 and bf16; every element against the oracle
    dist = "int1000" if dtype == "i32" else "uniform"
    got, xs0 = _full_compare("rhd", 8, N, dtype, None, dist, seed=N % 89, fuse=0, slice_=0)
    if dtype == "bf16":
        assert _normwise_bf16(got[0], xs0) <= 1e-2


@pytest.mark.parametrize("dtype", ["f32", "i32"])
def test_wide_eight_source_launches(dtype):
    # a lone 8-way reduce over 128 MiB buffers and a ragged tail runs the
    # wide 8-source instance with nontemporal loads and stores
    # (tests/test_capi_host.py checks the choice); the (8, 8) tree's first
    # level covers the cached-store form; every element against the oracle
    n, N = 8, (1 << 25) + 13
    steps = [(0, "reduce", 0, list(range(n)), 0, N)]
    say("case: custom 8-way reduce N=%d %s" % (N, dtype))
    dist = "int1000" if dtype == "i32" else "uniform"
    xs0 = workloads.draw(n, N, dtype, dist, 31)
    ref = oracle.execute(oracle.Plan("custom", n, N, [[oracle.Step(
        "reduce", 0, tuple(range(n)), 0, N)]]), [x.copy() for x in xs0], dtype)
    ts = to_device(xs0, dtype)
    del xs0
    h = arplan.ar_plan_create_custom(n, N, dtype, steps)
    try:
        arplan.ar_plan_execute(h, ts, torch.cuda.current_stream())
        torch.cuda.synchronize()
    finally:
        arplan.ar_plan_destroy(h)
    got = to_host(ts, dtype)
    for q in range(n):
        assert np.array_equal(got[q], ref[q]), q
    del ts
    torch.cuda.empty_cache()


@pytest.mark.parametrize("N,forms", [
    ((1 << 30) + 4099, [(1, 2, 1), (0, 0, 1)]),     # unaligned steps: phase launches
    ((1 << 30) + 8192, [(1, 1, 1), (0, 0, 1)])])    # aligned: one resident launch
def test_buffers_larger_than_4_GiB(N, forms):
    # every byte offset past 2^32: 64-bit addressing in the phase kernel (with
    # element-wise heads and tails) and the resident kernel, every element
    # compared with the oracle
    n = 2
    say("case: rhd n=2 N=%d (4 GiB + per buffer)" % N)
    xs0 = workloads.draw(n, N, "f32", "uniform", 77)
    ref = oracle.execute(oracle.rhd(n, N), [x.copy() for x in xs0], "f32")
    del xs0[1:]
    for fuse, slice_, resident in forms:
        with arplan.Plan(n, N, "f32", "rhd") as p:
            p.set_option(arplan.AR_OPT_FUSE, fuse)
            p.set_option(arplan.AR_OPT_SLICE, slice_)
            kinds = [x[0] for x in p.launches()]
            if slice_ == 1:
                assert kinds == [-2]
            ts = [torch.from_numpy(x).to("cuda") for x in
                  workloads.draw(n, N, "f32", "uniform", 77)]
            say("  fuse=%d slice=%d launches %s" % (fuse, slice_, kinds))
            run_plan(p, ts)
        for q in range(n):
            g = ts[q].cpu().numpy()
            assert np.array_equal(g, ref[q]), (N, fuse, slice_, q)
            del g
        del ts
        torch.cuda.empty_cache()
