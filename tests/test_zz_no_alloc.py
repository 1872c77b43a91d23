"""GPU: ar_plan_execute_noalloc (no device allocation; the tables and step
records live in the library's fixed per-device array) against
ar_plan_execute, bit for bit, through the C ABI: two calls in a row with
different plans, the second smaller; repeated calls, a new buffer set,
alternating plans, unaligned buffers; a plan too large for the array is
refused before anything runs; free device memory is unchanged by a call."""

import numpy as np
import pytest
import torch

import oracle
from paper_2409_04202_amd import workloads

from gpu_helpers import say, to_device, to_host

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2409_04202_amd import arplan


def _case(kind, n, N, dtype, fan, seed, pad=0):
    dist = "int1000" if dtype == "i32" else "uniform"
    xs0 = workloads.draw(n, N, dtype, dist, seed)
    return xs0, to_device(xs0, dtype, pad), to_device(xs0, dtype, pad)


def _run_both(plan, ref_bufs, got_bufs):
    s = torch.cuda.current_stream()
    plan.execute(ref_bufs, s)
    plan.execute_noalloc(got_bufs, s)
    torch.cuda.synchronize()


def _same(a, b, dtype, what):
    ha, hb = to_host(a, dtype), to_host(b, dtype)
    for q in range(len(ha)):
        assert np.array_equal(ha[q], hb[q]), (what, q)


CASES = [  # (kind, n, N, dtype, fan): the second of each pair is smaller
    (("rhd", 8, (1 << 20) + 13, "f32", None), ("tree", 64, (1 << 14) + 5, "f32", (8, 8))),
    (("tree", 512, 1 << 15, "bf16", (8, 8, 8)), ("cps", 16, 4099, "bf16", None)),
    (("ring", 64, 1 << 16, "i32", None), ("rhd", 6, 1000, "i32", None)),
]


@pytest.mark.parametrize("first,second", CASES)
def test_two_calls_second_smaller(first, second):
    for i, (kind, n, N, dtype, fan) in enumerate((first, second)):
        say("case: noalloc %s n=%d N=%d %s call %d" % (kind, n, N, dtype, i))
        xs0, ref, got = _case(kind, n, N, dtype, fan, seed=N % 97 + i)
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            _run_both(p, ref, got)
        _same(ref, got, dtype, (kind, n, N, dtype))
        want = oracle.execute(oracle.make_plan(kind, n, N, fan), [x.copy() for x in xs0], dtype)
        g = to_host(got, dtype)
        for q in range(n):
            assert np.array_equal(g[q], want[q]), (kind, q)


def test_repeats_new_buffers_and_alternating_plans():
    s = torch.cuda.current_stream()
    a = ("tree", 64, (1 << 16) + 64, "f32", (8, 8))
    b = ("rhd", 8, (1 << 18) + 3, "f32", None)
    with arplan.Plan(a[1], a[2], a[3], a[0], a[4]) as pa, \
            arplan.Plan(b[1], b[2], b[3], b[0], b[4]) as pb:
        for rnd in range(2):
            for (kind, n, N, dtype, fan), p in ((a, pa), (b, pb)):
                say("case: noalloc alternating %s round %d" % (kind, rnd))
                xs0, ref, got = _case(kind, n, N, dtype, fan, seed=rnd)
                # the same buffers twice (the second call copies nothing),
                # then a second buffer set (records only)
                for _ in range(2):
                    p.execute(ref, s)
                    p.execute_noalloc(got, s)
                torch.cuda.synchronize()
                _same(ref, got, dtype, (kind, "repeat"))
                xs1, ref1, got1 = _case(kind, n, N, dtype, fan, seed=rnd + 10)
                _run_both(p, ref1, got1)
                _same(ref1, got1, dtype, (kind, "new buffers"))
        # an option change rebuilds the plan's state: copied again
        pa.set_option(arplan.AR_OPT_SLICE, 0)
        xs0, ref, got = _case(*a, seed=5)
        _run_both(pa, ref, got)
        _same(ref, got, "f32", "option change")


@pytest.mark.parametrize("kind,n,N,dtype,fan,slice_,kernel", [
    ("tree", 512, 1 << 14, "bf16", (8, 8, 8), 1, "stream_kernel"),
    ("ring", 64, 64 * 1000, "f32", None, 1, "resident_kernel"),
    ("tree", 64, 1 << 16, "f32", (8, 8), 0, "phase_kernel"),
    ("tree", 512, 1 << 15, "bf16", (8, 8, 8), 0, "split_kernel"),
    ("tree", 64, 1 << 16, "f32", (8, 8), 1, "sliced_kernel")])
def test_every_launch_kind(kind, n, N, dtype, fan, slice_, kernel):
    xs0, ref, got = _case(kind, n, N, dtype, fan, seed=n)
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.set_option(arplan.AR_OPT_SLICE, slice_)
        p.set_option(arplan.AR_OPT_RESIDENT, 0 if kernel == "sliced_kernel" else 1)
        assert kernel in p.launch_kernels(), p.launch_kernels()
        _run_both(p, ref, got)
    _same(ref, got, dtype, (kind, "slice", slice_))


@pytest.mark.parametrize("pad", [1, 3])
def test_unaligned_buffers(pad):
    kind, n, N, dtype, fan = "cps", 16, 20011, "f32", None
    xs0, ref, got = _case(kind, n, N, dtype, fan, seed=pad, pad=pad)
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        _run_both(p, ref, got)
    _same(ref, got, dtype, "unaligned")


def test_no_device_memory_is_allocated():
    kind, n, N, dtype, fan = "tree", 64, (1 << 16) + 5, "f32", (8, 8)
    xs0, ref, got = _case(kind, n, N, dtype, fan, seed=7)
    with arplan.Plan(16, 4096, "f32", "cps") as warm:   # the array is set up
        warm.execute_noalloc(to_device(workloads.draw(16, 4096, "f32", "uniform", 1), "f32"))
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        p.execute_noalloc(got)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        p.execute(ref)
        torch.cuda.synchronize()
    assert free1 == free0
    _same(ref, got, dtype, "memory")


def test_too_large_is_refused_before_any_launch():
    # RHD n = 8 at 2^28 fp32 runs as one resident launch with 2^20
    # workgroups: 40 MiB of unit records, more than the array holds.  Real
    # buffers, so that nothing could touch memory it does not own.
    n, N = 8, 1 << 28
    with arplan.Plan(n, N, "f32", "rhd") as p:
        assert [x[0] for x in p.launches()] == [-2]
        bufs = [torch.empty(N, dtype=torch.float32, device="cuda") for _ in range(n)]
        with pytest.raises(arplan.ArError) as e:
            p.execute_noalloc(bufs)
        assert e.value.status == arplan.AR_ERR_UNSUPPORTED
        assert str(arplan.AR_NOALLOC_MAX_BYTES) in str(e.value)
        del bufs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_graph_capture_after_an_uncaptured_call():
    # after one uncaptured call with the same plan and buffers, a captured
    # call records kernel launches only; replays match the oracle applied once
    # more each; after a call with another plan, one uncaptured call with
    # this plan puts its tables back and the graph replays correctly again
    kind, n, N, fan = "tree", 64, (1 << 16) + 64, (8, 8)
    xs0 = workloads.draw(n, N, "i32", "int1000", 31)
    plan_o = oracle.make_plan(kind, n, N, fan)
    want = oracle.execute(plan_o, [x.copy() for x in xs0], "i32")
    ts = to_device(xs0, "i32")
    with arplan.Plan(n, N, "i32", kind, fan) as p, arplan.Plan(16, 4096, "f32", "cps") as other:
        p.execute_noalloc(ts, torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert all(np.array_equal(g, w) for g, w in zip(to_host(ts, "i32"), want))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            p.execute_noalloc(ts, torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert all(np.array_equal(g_, w) for g_, w in zip(to_host(ts, "i32"), want))
        ob = to_device(workloads.draw(16, 4096, "f32", "uniform", 2), "f32")
        for r in range(3):
            g.replay()
            torch.cuda.synchronize()
            want = oracle.execute(plan_o, want, "i32")
            assert all(np.array_equal(g_, w) for g_, w in zip(to_host(ts, "i32"), want)), r
            if r == 1:
                # another plan on the device, then this plan uncaptured once
                other.execute_noalloc(ob, torch.cuda.current_stream())
                p.execute_noalloc(ts, torch.cuda.current_stream())
                torch.cuda.synchronize()
                want = oracle.execute(plan_o, want, "i32")
                assert all(np.array_equal(g_, w) for g_, w in zip(to_host(ts, "i32"), want))
