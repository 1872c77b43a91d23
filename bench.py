"""Benchmark: AllReduce plan execution for n emulated processors on one
MI355X, through the C ABI.

A step is one execution of the whole plan (every ReduceScatter and
AllGather phase) over the n input buffers, which are resident in HBM before
the timed region starts.  The plan runs in place; the inputs are restored
from a pristine device copy after warm-up, then K steps run back to back
(values grow by a factor of about n per step, which does not change the
work: fp32 adds take the same time whatever the operands).  After the timed
region the inputs are restored again and K more executions record HIP
events around every kernel launch, for the per-launch durations; events
between launches would add to the step time, so they stay out of the timed
region.

Prints one JSON line:
  value       AllReduce algorithm bandwidth n * N * e / time, GB/s
  roofline    the launches that reduce (k >= 2 sources): algorithmic bytes
              per launch over their mean duration (HIP events on the launch
              stream), against MI355X's 8 TB/s HBM peak.  A phase or plain
              sliced launch moves (k + d) * len * e per step folding k
              sources into d destinations; a resident launch moves each
              buffer tile its run reads in once and each it writes out once
  cpu_baseline  the CPU oracle executing the same plan on the host
and, beside the contract's fields: the step time's median and minimum over
individually timed executions, the whole plan's and the copy launches'
fractions of the peak, a practical ceiling measured in the same run (a plain
device copy with torch and with the library, and a two-source fold through
the library, 2 GiB each), the
oracle with the steps of each phase spread over a thread pool, and, when the
default executor runs sliced or resident launches, the same plan with one
launch per executed phase (`phase_launches`: its time, and its reduce
launches' algorithmic bytes against the peak).
"""

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# kernel of a launch by its phase field in ar_plan_launch_info
KERNEL_OF = {-1: "sliced_kernel", -2: "resident_kernel", -3: "stream_kernel"}
DEFAULT = "rhd_n8_f32"


def _code_only(text):
    """C/C++ source without comments and blank space, so that a hash of it
    changes with the code only (the sources hold no string with // or /*)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash():
    """Hash of the code of the kernels and of the host code that decides
    their launches (comments and layout excluded)."""
    h = hashlib.sha256()
    for f in ("kernels.hpp", "resident.hpp", "exec.hip", "exec_state.hpp", "rewrite.cpp",
              "schedule.cpp", "programs.cpp"):
        with open(os.path.join(ROOT, "paper_2409_04202_amd", "csrc", f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload):
    """HBM traffic per reduce launch from a committed rocprofv3 --pmc
    summary, if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % workload)
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_sources") != kernel_source_hash():
        return None
    return d.get("reduce_bytes_per_launch")


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def parallel_execute(plan, bufs, dtype, pool):
    """oracle.execute with the steps of each phase on a thread pool (numpy's
    ufuncs release the GIL): every step reads the phase's starting state,
    the phase's writes are committed after all its steps."""
    import numpy as np
    import oracle

    def one(st):
        if st.op == "reduce":
            return oracle.fold(dtype, [bufs[q][st.begin:st.end] for q in st.srcs])
        return np.array(bufs[st.srcs[0]][st.begin:st.end], copy=True)

    for phase in plan.phases:
        vals = list(pool.map(one, phase))
        for st, v in zip(phase, vals):
            bufs[st.dst][st.begin:st.end] = v
    return bufs


def cpu_parallel(name, budget_s=10.0):
    """The oracle's plan with the steps of each phase spread over a thread
    pool (see parallel_execute)."""
    from concurrent.futures import ThreadPoolExecutor
    import oracle
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    if c["kind"] == "gentree":
        plan = oracle.gentree_plan(oracle.from_preorder(c["fanin"]), c["N"])
    else:
        plan = oracle.make_plan(c["kind"], c["n"], c["N"], c["fanin"])
    xs = workloads.inputs(name)
    dt = c["dtype"]
    total = c["n"] * c["N"] * workloads.ESIZE[dt]
    workers = os.cpu_count() or 1
    runs, spent = 0, 0.0
    with ThreadPoolExecutor(max_workers=workers) as pool:
        while spent < budget_s * 0.5 and runs < 20:
            bufs = [x.copy() for x in xs]
            t0 = time.perf_counter()
            parallel_execute(plan, bufs, dt, pool)
            spent += time.perf_counter() - t0
            runs += 1
    return {"value": round(total * runs / spent / 1e9, 4), "unit": "GB/s",
            "cores": workers, "cpu": cpu_model(), "kind": "oracle, phase steps on a thread pool",
            "sample": "%d full executions" % runs, "seconds": round(spent, 3)}


def ceiling(torch, arplan):
    """Practical HBM ceiling in this run, 2 GiB of traffic per repetition
    each: a plain device copy with torch's copy kernel and with the library
    (one copy step, 1 GiB read + 1 GiB written), and a two-source fold
    through the library (2 x 683 MiB read + 683 MiB written)."""
    reps = 10
    out = {}
    a = torch.empty(1 << 28, dtype=torch.float32, device="cuda")    # 1 GiB
    b = torch.empty_like(a)
    a.fill_(1.0)
    for _ in range(2):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    e1.synchronize()
    ms = e0.elapsed_time(e1) / reps
    out["copy_gbs"] = round(2 * a.numel() * 4 / (ms * 1e-3) / 1e9, 1)

    def lib_ms(bufs, steps):
        h = arplan.ar_plan_create_custom(len(bufs), bufs[0].numel(), "f32", steps)
        try:
            ptrs = arplan.pointers(bufs)
            sh = torch.cuda.current_stream().cuda_stream
            for _ in range(2):
                arplan.ar_plan_execute(h, ptrs, sh)
            e0.record()
            for _ in range(reps):
                arplan.ar_plan_execute(h, ptrs, sh)
            e1.record()
            e1.synchronize()
        finally:
            arplan.ar_plan_destroy(h)
        return e0.elapsed_time(e1) / reps

    ms = lib_ms([a, b], [(0, "copy", 1, (0,), 0, a.numel())])
    out["copy_lib_gbs"] = round(2 * a.numel() * 4 / (ms * 1e-3) / 1e9, 1)
    del a, b
    N = (2 << 30) // 12                     # 3 x N x 4 bytes = 2 GiB
    N -= N % 64
    xs = [torch.ones(N, dtype=torch.float32, device="cuda") for _ in range(3)]
    ms = lib_ms(xs, [(0, "reduce", 2, (0, 1), 0, N)])
    out["fold2_gbs"] = round(3 * N * 4 / (ms * 1e-3) / 1e9, 1)
    del xs
    return out


def cpu_baseline(name, budget_s=25.0):
    """The oracle, as written, on the same workload (single thread)."""
    import numpy as np  # noqa: F401
    import oracle
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    if c["kind"] == "gentree":
        plan = oracle.gentree_plan(oracle.from_preorder(c["fanin"]), c["N"])
    else:
        plan = oracle.make_plan(c["kind"], c["n"], c["N"], c["fanin"])
    xs = workloads.inputs(name)
    total = c["n"] * c["N"] * workloads.ESIZE[c["dtype"]]
    runs, spent = 0, 0.0
    while spent < budget_s * 0.4 and runs < 20:
        bufs = [x.copy() for x in xs]
        t0 = time.perf_counter()
        oracle.execute(plan, bufs, c["dtype"])
        spent += time.perf_counter() - t0
        runs += 1
    return {"value": round(total * runs / spent / 1e9, 4), "unit": "GB/s",
            "cores": 1, "kind": "oracle",
            "sample": "%d full executions of the %s plan (n=%d, N=%d %s), "
                      "numpy, one thread" % (runs, c["kind"], c["n"], c["N"],
                                             c["dtype"]),
            "cpu": cpu_model(),
            "seconds": round(spent, 3)}


def launch_ms(torch, arplan, plan, ptrs, sh, K, nlaunch):
    """Mean duration of each launch of the plan over K executions, from HIP
    events around every launch on the launch stream (ms)."""
    cap = max(1, K * nlaunch)
    timer = arplan.ar_timer_create(cap)
    torch.cuda.synchronize()
    for _ in range(K):
        plan.execute_timed(ptrs, sh, timer)
    torch.cuda.synchronize()
    recs = arplan.ar_timer_read(timer, cap)
    arplan.ar_timer_destroy(timer)
    l_ms = [0.0] * nlaunch
    for li, ms in recs:
        l_ms[li] += ms / K
    return l_ms


def phase_form(torch, arplan, plan, ptrs, sh, K, restore, total):
    """Time the plan with one launch per executed phase (AR_OPT_SLICE = 0):
    K back-to-back executions, then the reduce launches' algorithmic bytes
    over their durations against the HBM peak."""
    launches = plan.launches()
    restore()
    plan.execute(ptrs, sh)
    restore()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        plan.execute(ptrs, sh)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / K
    restore()
    l_ms = launch_ms(torch, arplan, plan, ptrs, sh, K, len(launches))
    red = [i for i, L in enumerate(launches) if L[1] >= 2]
    red_ms = sum(l_ms[i] for i in red)
    red_gbs = sum(launches[i][4] for i in red) / (red_ms * 1e-3) / 1e9 if red_ms > 0 else 0.0
    return {"ms_per_step": round(ms_step, 5),
            "value": round(total / (ms_step * 1e-3) / 1e9, 2),
            "reduce_gbs": round(red_gbs, 1),
            "reduce_frac": round(red_gbs / HBM_PEAK_GBS, 4),
            "launches": [{"phase": L[0], "k": L[1], "max_dst": L[2], "steps": L[3],
                          "bytes": L[4], "ms": round(m, 5)}
                         for L, m in zip(launches, l_ms)]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=DEFAULT)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the copy / two-source fold ceiling measurement")
    ap.add_argument("--no-fuse", action="store_true",
                    help="run every plan step as listed (AR_OPT_FUSE = 0)")
    ap.add_argument("--slice", type=int, choices=(0, 1, 2), default=None,
                    help="AR_OPT_SLICE (default: the library's, 2)")
    ap.add_argument("--resident", type=int, choices=(0, 1), default=None,
                    help="AR_OPT_RESIDENT (default: the library's, 1)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the library executes every emulated processor on one "
              "GPU; runs on more than one GPU are not supported (--gpus 1).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2409_04202_amd import arplan, workloads

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    name = args.config
    c = workloads.CONFIGS[name]
    n, N, dt = c["n"], c["N"], c["dtype"]
    esize = workloads.ESIZE[dt]
    tdt = {"f32": torch.float32, "i32": torch.int32, "bf16": torch.int16}[dt]
    print("bench: %s n=%d N=%d %s: drawing inputs" % (name, n, N, dt),
          file=sys.stderr, flush=True)
    xs = workloads.inputs(name)
    import numpy as np
    view = np.int16 if dt == "bf16" else xs[0].dtype
    pristine = [torch.from_numpy(x.view(view)).to("cuda") for x in xs]
    bufs = [torch.empty_like(p) for p in pristine]
    del xs

    plan = arplan.Plan(n, N, dt, c["kind"], c["fanin"])
    if args.no_fuse:
        plan.set_option(arplan.AR_OPT_FUSE, 0)
    if args.slice is not None:
        plan.set_option(arplan.AR_OPT_SLICE, args.slice)
    if args.resident is not None:
        plan.set_option(arplan.AR_OPT_RESIDENT, args.resident)
    stream = torch.cuda.current_stream()
    launches = plan.launches()          # (phase, nsrc, max_dst, steps, bytes)
    red_b, cpy_b = plan.bytes()

    def restore():
        for b, p in zip(bufs, pristine):
            b.copy_(p)

    restore()
    for _ in range(args.warmup):
        plan.execute(bufs, stream)
    restore()
    K = args.steps
    ptrs = arplan.pointers(bufs)        # marshalled once for the buffer set
    sh = stream.cuda_stream
    torch.cuda.synchronize()
    print("bench: timing %d steps" % K, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for _ in range(K):
        plan.execute(ptrs, sh)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # per-launch durations, outside the timed region
    restore()
    l_ms = launch_ms(torch, arplan, plan, ptrs, sh, K, len(launches))
    # step time distribution: each execution between two events
    restore()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(K)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record(stream)
        plan.execute(ptrs, sh)
        e1.record(stream)
    torch.cuda.synchronize()
    step_ms = sorted(e0.elapsed_time(e1) for e0, e1 in evs)

    ms_step = (t1 - t0) * 1e3 / K
    total = n * N * esize
    value = total / (ms_step * 1e-3) / 1e9

    # dominant kernel: the launches that reduce (k >= 2 sources)
    red = [i for i, L in enumerate(launches) if L[1] >= 2]
    red_ms = sum(l_ms[i] for i in red)
    red_bytes = sum(launches[i][4] for i in red)
    cpy = [i for i, L in enumerate(launches) if L[1] == 1]
    cpy_ms = sum(l_ms[i] for i in cpy)
    cpy_bytes = sum(launches[i][4] for i in cpy)
    achieved = red_bytes / (red_ms * 1e-3) / 1e9 if red_ms > 0 else 0.0
    traffic = load_traffic(name) if (not args.no_fuse and args.slice is None
                                     and args.resident is None) else None
    roofline = {"bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic,
                "kernel": "%s, reduce launches (k = %s)" % (
                    " + ".join(sorted({KERNEL_OF.get(launches[i][0], "phase_kernel")
                                       for i in red})) or "-",
                    sorted({launches[i][1] for i in red}) or "-"),
                "launches_per_step": len(red),
                "bytes_per_launch": round(red_bytes / max(1, len(red))),
                "ms_per_launch": round(red_ms / max(1, len(red)), 5)}
    out = {
        "metric": "AllReduce algbw GB/s and % HBM roofline per plan at 1 MI355X",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded %s inputs)" % c["dist"],
        "config": {"workload": name, "plan": c["kind"], "n": n, "N": N,
                   "fanin": (list(c["fanin"]) if c["kind"] != "gentree"
                             else "%d-node tree" % len(c["fanin"])) if c["fanin"] else None,
                   "fuse": not args.no_fuse,
                   "slice": args.slice if args.slice is not None else 2,
                   "resident": args.resident if args.resident is not None else 1,
                   "parallelism": "emulated %d processors on 1 GPU" % n},
        "plan_bytes_per_step": red_b + cpy_b,
        "plan_gbs": round((red_b + cpy_b) / (ms_step * 1e-3) / 1e9, 1),
        "kernel_bytes_per_step": sum(L[4] for L in launches),
        "kernel_gbs": round(sum(L[4] for L in launches) / (ms_step * 1e-3) / 1e9, 1),
        "kernel_ms_per_step": round(sum(l_ms), 5),
        "step_ms": {"median": round(step_ms[len(step_ms) // 2], 5),
                    "min": round(step_ms[0], 5)},
        "plan_frac": round((red_b + cpy_b) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "copy_frac": (round(cpy_bytes / (cpy_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
                      if cpy_ms > 0 else None),
        "launches": [{"phase": L[0], "k": L[1], "max_dst": L[2], "steps": L[3],
                      "bytes": L[4], "ms": round(m, 5),
                      "gbs": round(L[4] / (m * 1e-3) / 1e9, 1) if m > 0 else None}
                     for L, m in zip(launches, l_ms)],
        "roofline": roofline,
        "cpu_baseline": None,
    }
    if (args.slice is None and args.resident is None
            and any(L[0] < 0 for L in launches)):
        # the same plan with one launch per executed phase, every phase's
        # output going through HBM
        print("bench: phase launches", file=sys.stderr, flush=True)
        plan.set_option(arplan.AR_OPT_SLICE, 0)
        out["phase_launches"] = phase_form(torch, arplan, plan, ptrs, sh, K,
                                           restore, total)
    plan.close()
    del bufs, pristine
    if not args.no_ceiling:
        print("bench: practical ceiling", file=sys.stderr, flush=True)
        out["ceiling"] = ceiling(torch, arplan)
    if not args.no_cpu_baseline:
        print("bench: timing the CPU oracle", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(name)
        out["cpu_parallel"] = cpu_parallel(name)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
