"""GenModel fitted on one MI355X (Section 3.4's procedure, single-GPU terms).

The paper fits GenModel's parameters from co-located PS runs on 2..max
processors and uses the model to predict the time of other plans and to pick
a plan (Algorithm 2).  On one GPU the network terms (beta over links, the
incast term) do not exist; what remains of a plan's cost is

    T = A * alpha + D * delta + B * beta

with A the number of rounds (phases, Tables 1-2), D the memory operations of
the reduce steps in bytes ((k + 1) * len * e per k-way step, the delta term
of Section 3.1) and B the bytes the copy steps move (2 * len * e each; on a
single GPU the AllGather transfers are memory traffic too).  alpha is the
per-round cost (a kernel launch and its drain), delta and beta are seconds
per byte.  Plans are timed as written: one launch per phase, no executor
rewrites (AR_OPT_FUSE = 0, AR_OPT_SLICE = 0).

``python -m paper_2409_04202_amd.genmodel`` measures, fits, predicts Ring,
RHD and hierarchical-tree plans, reports the errors and the plan the model
picks per (n, N), and prints one JSON document.
"""

import argparse
import itertools
import json
import sys
import time

import numpy as np

from . import arplan


def features(plan):
    """(A, D, B) of a plan from the library's own step list."""
    A = plan.num_phases
    D = B = 0
    for ph in range(A):
        op, _, _, b = plan.phase_info(ph)
        if op == arplan.AR_OP_REDUCE:
            D += b
        else:
            B += b
    return A, D, B


def predict(params, feats):
    alpha, delta, beta = params
    A, D, B = feats
    return A * alpha + D * delta + B * beta


def fit(samples):
    """Least squares on (features, seconds) samples, relative error
    weighting (each equation divided by its measured time)."""
    X = np.array([[A, D, B] for (A, D, B), _ in samples], dtype=np.float64)
    y = np.array([t for _, t in samples], dtype=np.float64)
    w = 1.0 / y
    sol, *_ = np.linalg.lstsq(X * w[:, None], y * w, rcond=None)
    return tuple(float(v) for v in sol)


def factorizations(n, max_levels=3):
    out = []

    def rec(rest, cur):
        if rest == 1:
            if len(cur) >= 2:
                out.append(tuple(cur))
            return
        if len(cur) == max_levels:
            return
        for f in range(2, rest + 1):
            if rest % f == 0:
                rec(rest // f, cur + [f])
    rec(n, [])
    return out


def candidates(n):
    """Plans the selection considers for n processors."""
    cands = [("ring", None), ("cps", None), ("rhd", None)]
    cands += [("tree", f) for f in factorizations(n)]
    return cands


def select(params, n, N, dtype="f32"):
    """The plan with the smallest predicted time."""
    best = None
    for kind, fan in candidates(n):
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            t = predict(params, features(p))
        if best is None or t < best[0]:
            best = (t, kind, fan)
    return best


class Timer:
    """Times plan executions on the GPU (literal plans, HIP events)."""

    def __init__(self, reps=10, warmup=2):
        import torch
        self.torch = torch
        self.reps, self.warmup = reps, warmup

    def __call__(self, n, N, kind, fan, dtype="f32"):
        torch = self.torch
        bufs = [torch.rand(N, device="cuda") for _ in range(n)]
        ptrs = arplan.pointers(bufs)    # marshalled once: host time stays out
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            p.set_option(arplan.AR_OPT_FUSE, 0)
            p.set_option(arplan.AR_OPT_SLICE, 0)
            s = torch.cuda.current_stream()
            for _ in range(self.warmup):
                p.execute(ptrs, s)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(self.reps):
                p.execute(ptrs, s)
            e1.record(s)
            e1.synchronize()
            feats = features(p)
        del bufs
        return feats, e0.elapsed_time(e1) * 1e-3 / self.reps


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--quick", action="store_true")
    args = ap.parse_args()
    import torch
    if not torch.cuda.is_available():
        print("genmodel: no GPU", file=sys.stderr)
        sys.exit(1)
    timer = Timer(reps=args.reps)
    MiB = 1 << 20
    sizes = [1 * MiB, 4 * MiB, 16 * MiB, 64 * MiB]          # bytes per processor
    fit_ns = [2, 3, 4, 6, 8, 12, 16, 24, 32]
    if args.quick:
        sizes, fit_ns = sizes[1:3], [2, 4, 8, 16]
    t0 = time.time()
    train = []
    for n, S in itertools.product(fit_ns, sizes):
        N = S // 4
        feats, t = timer(n, N, "cps", None)
        train.append(((n, N, "cps", None), feats, t))
        print("genmodel: cps n=%d S=%d MiB %.4f ms" % (n, S // MiB, t * 1e3),
              file=sys.stderr, flush=True)
    params = fit([(f, t) for _, f, t in train])
    tests = []
    test_ns = [4, 8, 16, 32] if not args.quick else [8]
    for n, S in itertools.product(test_ns, sizes):
        N = S // 4
        plans = [("ring", None), ("rhd", None)] + [("tree", f) for f in factorizations(n)]
        for kind, fan in plans:
            feats, t = timer(n, N, kind, fan)
            tests.append(((n, N, kind, fan), feats, t))
            print("genmodel: %s %s n=%d S=%d MiB %.4f ms" % (kind, fan, n, S // MiB, t * 1e3),
                  file=sys.stderr, flush=True)
    rows = []
    for (n, N, kind, fan), feats, t in train + tests:
        pr = predict(params, feats)
        rows.append({"n": n, "N": N, "plan": kind, "fanin": list(fan) if fan else None,
                     "A": feats[0], "D": feats[1], "B": feats[2],
                     "measured_ms": t * 1e3, "predicted_ms": pr * 1e3,
                     "error": (pr - t) / t, "fit": kind == "cps"})
    # selection: the model's pick per (n, N) against the measured best
    sel = []
    meas = {}
    for (n, N, kind, fan), feats, t in train + tests:
        meas.setdefault((n, N), []).append((t, kind, fan))
    for (n, N), lst in sorted(meas.items()):
        if n not in test_ns:
            continue
        best_t, best_kind, best_fan = min(lst, key=lambda x: x[0])
        pick = min(lst, key=lambda x: predict(params, timer_features(n, N, x[1], x[2])))
        sel.append({"n": n, "N": N, "measured_best": [best_kind, best_fan],
                    "model_pick": [pick[1], pick[2]],
                    "pick_ms": pick[0] * 1e3, "best_ms": best_t * 1e3,
                    "loss": pick[0] / best_t - 1})
    test_err = [abs(r["error"]) for r in rows if not r["fit"]]
    fit_err = [abs(r["error"]) for r in rows if r["fit"]]
    out = {"params": {"alpha_us": params[0] * 1e6,
                      "delta_ns_per_byte": params[1] * 1e9,
                      "beta_ns_per_byte": params[2] * 1e9,
                      "delta_GBps": 1e-9 / params[1] if params[1] > 0 else None,
                      "beta_GBps": 1e-9 / params[2] if params[2] > 0 else None},
           "fit_max_error": max(fit_err), "fit_mean_error": float(np.mean(fit_err)),
           "test_max_error": max(test_err) if test_err else None,
           "test_mean_error": float(np.mean(test_err)) if test_err else None,
           "rows": rows, "selection": sel, "seconds": time.time() - t0}
    print(json.dumps(out))


def timer_features(n, N, kind, fan, dtype="f32"):
    with arplan.Plan(n, N, dtype, kind, fan) as p:
        return features(p)


if __name__ == "__main__":
    main()
