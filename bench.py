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

Every workload is timed in two forms:

  default     the executor's own choice (rewrites, sliced or resident runs);
              its time is the AllReduce's algorithm bandwidth n * N * e / t
  as_written  every plan step as listed, one launch per phase
              (AR_OPT_FUSE = 0, AR_OPT_SLICE = 0): each launch moves exactly
              its phase's algorithmic bytes, (k + 1) * len * e per k-way
              reduce step and 2 * len * e per copy (the memory term of
              Section 3.1), so its reduce launches' bytes over their time
              is the plan's own reduce-phase throughput

Prints one JSON line.  The headline (RHD, n = 8, N = 2^26 fp32):
  value       algorithm bandwidth of the default form, GB/s
  roofline    the as-written plan's reduce launches (the k-way reduce
              phases): their algorithmic bytes over their HIP-event time,
              against MI355X's 8 TB/s HBM peak
  executor_roofline  the default form's launches that reduce, on the
              bytes they move (a resident launch moves each buffer tile
              once in and once out: 2 * n * N * e)
  cpu_baseline  the CPU oracle executing the same plan on the host
  configs     every workload (each config of the scope, the GenTree
              topologies and the n = 64 sweep) in both forms, each with a
              bounded CPU oracle baseline; a form whose K executions take
              less than 5 ms is timed over enough executions for about 5 ms
              (`timed_steps`)
and, beside those: the step time's median and minimum over individually
timed executions, a practical ceiling measured in the same run (a device
copy with torch and with the library, a two-source fold through the
library, 2 GiB each) and the oracle with the steps of each phase spread
over a thread pool.
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
HEADLINE = "rhd_n8_f32"
FORMS = {"default": {}, "as_written": {"fuse": 0, "slice": 0}}


def _code_only(text):
    """C/C++ source without comments and blank space, so that a hash of it
    changes with the code only (the sources hold no string with // or /*)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


KERNEL_SOURCES = ("kernels.hpp", "resident.hpp", "exec.hip", "exec_state.hpp", "rewrite.cpp",
                  "schedule.cpp", "programs.cpp")


def kernel_source_hash():
    """Hash of the code of the kernels and of the host code that decides
    their launches (comments and layout excluded)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2409_04202_amd", "csrc", f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(workload, form):
    """HBM traffic per reduce launch from a committed rocprofv3 --pmc
    summary, if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.json" % (workload, form))
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


def oracle_plan(c):
    import oracle
    if c["kind"] == "gentree":
        return oracle.gentree_plan(oracle.from_preorder(c["fanin"]), c["N"])
    return oracle.make_plan(c["kind"], c["n"], c["N"], c["fanin"])


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


def cpu_parallel(name, xs, budget_s=10.0):
    """The oracle's plan with the steps of each phase spread over a thread
    pool (see parallel_execute)."""
    from concurrent.futures import ThreadPoolExecutor
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    plan = oracle_plan(c)
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


def cpu_baseline(name, xs, budget_s, max_runs=20):
    """The oracle, as written, on the same workload (single thread): full
    executions of the plan until about `budget_s` seconds are spent (at
    least one)."""
    import oracle
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    plan = oracle_plan(c)
    total = c["n"] * c["N"] * workloads.ESIZE[c["dtype"]]
    runs, spent = 0, 0.0
    while runs < 1 or (spent < budget_s and runs < max_runs):
        bufs = [x.copy() for x in xs]
        t0 = time.perf_counter()
        oracle.execute(plan, bufs, c["dtype"])
        spent += time.perf_counter() - t0
        runs += 1
    return {"value": round(total * runs / spent / 1e9, 4), "unit": "GB/s",
            "cores": 1, "kind": "oracle",
            "sample": "%d full execution%s of the %s plan (n=%d, N=%d %s), numpy, "
                      "one thread" % (runs, "" if runs == 1 else "s", c["kind"],
                                      c["n"], c["N"], c["dtype"]),
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


def _gbs(nbytes, ms):
    return nbytes / (ms * 1e-3) / 1e9 if ms > 0 else 0.0


def time_form(torch, arplan, c, bufs, restore, K, W, opts, stream, min_ms=0.0):
    """One form of one workload: W warm-up executions, then K back-to-back
    executions timed with the host clock between two device
    synchronisations (with `min_ms`, a plan whose K executions take less is
    timed again over enough executions for about min_ms), then K executions
    with HIP events around every launch (after a restore) for the per-launch
    durations."""
    plan = arplan.Plan(c["n"], c["N"], c["dtype"], c["kind"], c["fanin"])
    try:
        if "fuse" in opts:
            plan.set_option(arplan.AR_OPT_FUSE, opts["fuse"])
        if "slice" in opts:
            plan.set_option(arplan.AR_OPT_SLICE, opts["slice"])
        if "resident" in opts:
            plan.set_option(arplan.AR_OPT_RESIDENT, opts["resident"])
        launches = plan.launches()          # (phase, nsrc, max_dst, steps, bytes)
        kernels = plan.launch_kernels()
        red_b, cpy_b = plan.bytes()
        ptrs = arplan.pointers(bufs)        # marshalled once for the buffer set
        sh = stream.cuda_stream
        restore()
        for _ in range(W):
            plan.execute(ptrs, sh)
        restore()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(K):
            plan.execute(ptrs, sh)
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / K
        reps = K
        if min_ms and ms_step * K < min_ms:
            # a short plan: time enough executions for about min_ms of work
            reps = min(4000, int(min_ms / max(ms_step, 1e-4)) + 1)
            restore()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(reps):
                plan.execute(ptrs, sh)
            torch.cuda.synchronize()
            ms_step = (time.perf_counter() - t0) * 1e3 / reps
        restore()
        l_ms = launch_ms(torch, arplan, plan, ptrs, sh, K, len(launches))
    finally:
        plan.close()
    esize = {"f32": 4, "i32": 4, "bf16": 2}[c["dtype"]]
    total = c["n"] * c["N"] * esize
    red = [i for i, L in enumerate(launches) if L[1] >= 2]
    red_ms = sum(l_ms[i] for i in red)
    red_bytes = sum(launches[i][4] for i in red)
    cpy = [i for i, L in enumerate(launches) if L[1] == 1]
    cpy_ms = sum(l_ms[i] for i in cpy)
    cpy_bytes = sum(launches[i][4] for i in cpy)
    return {
        "ms_per_step": round(ms_step, 5),
        "timed_steps": reps,
        "algbw_gbs": round(_gbs(total, ms_step), 2),
        "plan_gbs": round(_gbs(red_b + cpy_b, ms_step), 1),
        "kernel_ms_per_step": round(sum(l_ms), 5),
        "reduce_launches": len(red),
        "reduce_bytes": red_bytes,
        "reduce_ms": round(red_ms, 5),
        "reduce_gbs": round(_gbs(red_bytes, red_ms), 1),
        # a plain sliced launch's steps hand their results to the next phase
        # through the cache: its bytes are not HBM traffic, so no fraction of
        # the HBM peak is given for it
        "reduce_frac": (None if any(launches[i][0] == -1 for i in red)
                        else round(_gbs(red_bytes, red_ms) / HBM_PEAK_GBS, 4)),
        "copy_gbs": round(_gbs(cpy_bytes, cpy_ms), 1) if cpy_ms > 0 else None,
        "kernels": sorted(set(kernels)),
        "launches": [{"phase": L[0], "k": L[1], "max_dst": L[2], "steps": L[3],
                      "bytes": L[4], "ms": round(m, 5),
                      "gbs": round(_gbs(L[4], m), 1) if m > 0 else None}
                     for L, m in zip(launches, l_ms)],
        "_plan_bytes": (red_b, cpy_b),
        "_red": [(launches[i][0], launches[i][1], launches[i][4], l_ms[i]) for i in red],
    }


def step_distribution(torch, arplan, c, bufs, restore, K, stream):
    """The default form's step time, each execution between two events."""
    plan = arplan.Plan(c["n"], c["N"], c["dtype"], c["kind"], c["fanin"])
    try:
        opts = FORMS["default"]
        if "fuse" in opts:
            plan.set_option(arplan.AR_OPT_FUSE, opts["fuse"])
        if "slice" in opts:
            plan.set_option(arplan.AR_OPT_SLICE, opts["slice"])
        if "resident" in opts:
            plan.set_option(arplan.AR_OPT_RESIDENT, opts["resident"])
        ptrs = arplan.pointers(bufs)
        sh = stream.cuda_stream
        restore()
        plan.execute(ptrs, sh)
        restore()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(K)]
        torch.cuda.synchronize()
        for e0, e1 in evs:
            e0.record(stream)
            plan.execute(ptrs, sh)
            e1.record(stream)
        torch.cuda.synchronize()
    finally:
        plan.close()
    step_ms = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    return {"median": round(step_ms[len(step_ms) // 2], 5), "min": round(step_ms[0], 5)}


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


def bench_workload(torch, arplan, name, K, W, forms, stream, cpu_s, headline=False,
                   min_ms=0.0):
    """Both forms of one workload (and, for the headline, the per-step time
    distribution), plus the oracle on the host."""
    import numpy as np
    from paper_2409_04202_amd import workloads
    c = workloads.CONFIGS[name]
    n, N, dt = c["n"], c["N"], c["dtype"]
    print("bench: %s n=%d N=%d %s: drawing inputs" % (name, n, N, dt),
          file=sys.stderr, flush=True)
    xs = workloads.inputs(name)
    view = np.int16 if dt == "bf16" else xs[0].dtype
    pristine = [torch.from_numpy(x.view(view)).to("cuda") for x in xs]
    bufs = [torch.empty_like(p) for p in pristine]

    def restore():
        for b, p in zip(bufs, pristine):
            b.copy_(p)

    res = {"workload": name, "plan": c["kind"], "n": n, "N": N, "dtype": dt,
           "fanin": (list(c["fanin"]) if c["kind"] != "gentree"
                     else "%d-node tree" % len(c["fanin"])) if c["fanin"] else None}
    for form in forms:
        print("bench: %s %s form, %d steps" % (name, form, K), file=sys.stderr, flush=True)
        res[form] = time_form(torch, arplan, c, bufs, restore, K, W, FORMS[form], stream,
                              min_ms)
    if headline and "default" in forms:
        res["step_ms"] = step_distribution(torch, arplan, c, bufs, restore, K, stream)
    del bufs, pristine
    torch.cuda.empty_cache()
    if cpu_s > 0:
        print("bench: %s: timing the CPU oracle" % name, file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(name, xs, cpu_s)
        if headline:
            res["cpu_parallel"] = cpu_parallel(name, xs)
    return res


def public(form_res):
    return {k: v for k, v in form_res.items() if not k.startswith("_")}


def headline_line(h, K, W, name):
    """The contract's JSON line from the headline workload's results."""
    w = h.get("as_written")
    d = h.get("default") or w
    red_b, cpy_b = d["_plan_bytes"]
    out = {
        "metric": "AllReduce algbw GB/s and % HBM roofline per plan at 1 MI355X",
        "value": d["algbw_gbs"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": d["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": h["dtype"],
        "data": "synthetic (seeded inputs, %s)" % name,
        "config": {"workload": name, "plan": h["plan"], "n": h["n"], "N": h["N"],
                   "fanin": h["fanin"],
                   "form": ("default executor" if not FORMS["default"] else
                            "executor with %s" % FORMS["default"]) if "default" in h
                           else "plan as written",
                   "parallelism": "emulated %d processors on 1 GPU" % h["n"]},
        "plan_bytes_per_step": red_b + cpy_b,
    }
    if w is not None:
        red = w["_red"]
        kinds = sorted({"phase_kernel<%s, k=%d>" % (h["dtype"], k) for _, k, _, _ in red})
        out["roofline"] = {
            "bound": "hbm", "achieved": w["reduce_gbs"], "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": w["reduce_frac"],
            "traffic": load_traffic(name, "as_written"),
            "kernel": " + ".join(kinds),
            "form": "plan as written (AR_OPT_FUSE=0, AR_OPT_SLICE=0): the reduce phases",
            "bytes": "(k + 1) * len * e per k-way reduce step",
            "launches_per_step": len(red),
            "bytes_per_launch": round(w["reduce_bytes"] / max(1, len(red))),
            "ms_per_launch": round(w["reduce_ms"] / max(1, len(red)), 5),
            "ms_as_written_step": w["ms_per_step"]}
    dk = d["kernels"]
    out["executor_roofline"] = {
        "bound": "hbm", "achieved": d["reduce_gbs"], "peak": HBM_PEAK_GBS,
        "unit": "GB/s", "frac": d["reduce_frac"],
        "traffic": load_traffic(name, "default"),
        "kernel": " + ".join(dk),
        "form": "default executor: its launches that reduce",
        "bytes": ("rows loaded and stored, each buffer tile once: 2 * n * N * e"
                  if dk == ["resident_kernel"] else "(k + d) * len * e per executed step"),
        "launches_per_step": d["reduce_launches"],
        "bytes_per_launch": round(d["reduce_bytes"] / max(1, d["reduce_launches"])),
        "ms_per_launch": round(d["reduce_ms"] / max(1, d["reduce_launches"])
                               if d["reduce_launches"] else 0.0, 5)}
    out["plan_frac_as_written"] = (round(_gbs(red_b + cpy_b, w["ms_per_step"]) / HBM_PEAK_GBS, 4)
                                   if w is not None else None)
    out["step_ms"] = h.get("step_ms")
    if "default" in h:
        out["default"] = public(d)
    if w is not None:
        out["as_written"] = public(w)
    out["cpu_baseline"] = h.get("cpu_baseline")
    if "cpu_parallel" in h:
        out["cpu_parallel"] = h["cpu_parallel"]
    return out


def config_entry(r):
    e = {k: r[k] for k in ("workload", "plan", "n", "N", "dtype", "fanin")}
    for form in FORMS:
        if form in r:
            f = r[form]
            e[form] = {k: f[k] for k in ("ms_per_step", "timed_steps", "algbw_gbs", "plan_gbs",
                                         "reduce_launches", "reduce_gbs", "reduce_frac",
                                         "copy_gbs", "kernels")}
            L = f["launches"]
            if len(L) <= 16:   # (plan phase, k, destinations, steps, bytes, ms)
                e[form]["launches"] = [[x["phase"], x["k"], x["max_dst"], x["steps"],
                                        x["bytes"], x["ms"]] for x in L]
            else:
                e[form]["launches"] = "%d launches" % len(L)
    e["cpu_baseline"] = r.get("cpu_baseline")
    return e


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=HEADLINE,
                    help="workload of the headline line (default %s)" % HEADLINE)
    ap.add_argument("--form", choices=("both",) + tuple(FORMS), default="both",
                    help="time only one form (for profiler runs)")
    ap.add_argument("--no-configs", action="store_true",
                    help="time the headline workload only, not every workload")
    ap.add_argument("--slice", type=int, choices=(0, 1, 2), default=None,
                    help="AR_OPT_SLICE for the default form (the library's default: 2)")
    ap.add_argument("--resident", type=int, choices=(0, 1), default=None,
                    help="AR_OPT_RESIDENT for the default form (the library's default: 1)")
    ap.add_argument("--no-fuse", action="store_true",
                    help="AR_OPT_FUSE = 0 for the default form")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the copy / two-source fold ceiling measurement")
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
    stream = torch.cuda.current_stream()
    forms = tuple(FORMS) if args.form == "both" else (args.form,)
    # executor overrides of the default form (for exploring and profiling
    # other executions of the same plan; the configs entries use them too)
    if args.slice is not None:
        FORMS["default"]["slice"] = args.slice
    if args.resident is not None:
        FORMS["default"]["resident"] = args.resident
    if args.no_fuse:
        FORMS["default"]["fuse"] = 0
    K, W = args.steps, args.warmup
    cpu = not args.no_cpu_baseline
    h = bench_workload(torch, arplan, args.config, K, W, forms, stream,
                       10.0 if cpu else 0.0, headline=True)
    out = headline_line(h, K, W, args.config)
    if not args.no_configs:
        out["configs"] = [config_entry(h)]
        for name in workloads.CONFIGS:
            if name == args.config:
                continue
            r = bench_workload(torch, arplan, name, K, W, forms, stream,
                               1.5 if cpu else 0.0, min_ms=5.0)
            out["configs"].append(config_entry(r))
    if not args.no_ceiling:
        print("bench: practical ceiling", file=sys.stderr, flush=True)
        out["ceiling"] = ceiling(torch, arplan)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
