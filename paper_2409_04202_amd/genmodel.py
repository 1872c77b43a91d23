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

An extended single-GPU form adds what the paper's cluster terms leave out
on one GPU:

    T = A * alpha + K * lam + Dh * delta_h + Dc * delta_c
                            + Bh * beta_h  + Bc * beta_c

K sums, over the phases, the largest source count of a step of the phase
(a k-way step's first store waits for k dependent loads per element: a
per-phase latency that grows with k), and the byte terms are split by
where each access is served: an access is "cached" (Dc, Bc) when the
plan's whole footprint n * N * e fits the last-level cache, when it reads a
range read earlier in the same phase, or when it reads a range the previous
phase wrote and that phase wrote at most the cache's capacity; otherwise
it goes to HBM (Dh, Bh).  Fitted by non-negative least squares in relative
error.

The tiered form splits the cached bytes once more, by the smaller cache an
access fits (ar_genmodel_terms_tiered with the 256 MiB last-level cache and
the 32 MiB the eight XCDs' L2 caches hold together):

    T = A * alpha + K * lam + Dh * delta_h + Dc * delta_c + Dl * delta_l
                            + Bh * beta_h  + Bc * beta_c  + Bl * beta_l

with Dl, Bl the bytes the one-cache rule classes as cached under 32 MiB and
Dc, Bc the rest of those it classes as cached under 256 MiB.

``python -m paper_2409_04202_amd.genmodel`` measures, fits the forms (the
paper's and the extended one from co-located PS runs as the paper does; the
extended and the tiered one also from co-located PS plus two-level tree
runs), predicts Ring, RHD and
hierarchical-tree plans, reports the errors and the plan each model picks
per (n, N), and prints one JSON document.
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


LLC_BYTES = 256 << 20   # MI355X last-level (Infinity) cache
L2_BYTES = 32 << 20     # the L2 caches of its 8 XCDs, 4 MB each


def ext_features(plan, cache_bytes=LLC_BYTES):
    """(A, K, Dh, Dc, Bh, Bc) of a plan for the extended form (see the
    module docstring), computed by the library (ar_genmodel_terms)."""
    return tuple(int(x) for x in arplan.ar_genmodel_terms(plan.handle, cache_bytes))


def tiered_features(plan, tiers=(LLC_BYTES, L2_BYTES)):
    """(A, K, Dh, Dc, Dl, Bh, Bc, Bl) of a plan for the tiered form, computed
    by the library (ar_genmodel_terms_tiered)."""
    return tuple(int(x) for x in arplan.ar_genmodel_terms_tiered(plan.handle, list(tiers)))


def predict(params, feats):
    """Predicted seconds: the dot product of parameters and features (either
    form)."""
    return float(sum(p * f for p, f in zip(params, feats)))


def fit(samples, nonneg=False):
    """Least squares on (features, seconds) samples, relative error
    weighting (each equation divided by its measured time); `nonneg`
    constrains every parameter to be >= 0."""
    X = np.array([list(f) for f, _ in samples], dtype=np.float64)
    y = np.array([t for _, t in samples], dtype=np.float64)
    w = 1.0 / y
    if nonneg:
        from scipy.optimize import nnls
        sol, _ = nnls(X * w[:, None], y * w)
    else:
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


def select(params, n, N, dtype="f32", feature_fn=None):
    """The plan with the smallest predicted time (`feature_fn`: features,
    ext_features or tiered_features, matching `params`).  The extended and
    tiered forms' choice is made by the library (ar_genmodel_select,
    ar_genmodel_select_tiered) over the same candidates."""
    feature_fn = feature_fn or features
    if feature_fn is ext_features:
        kind, fan, t = arplan.ar_genmodel_select(n, N, dtype, params, LLC_BYTES, 3)
        return t, kind, fan
    if feature_fn is tiered_features:
        kind, fan, t = arplan.ar_genmodel_select_tiered(n, N, dtype, params,
                                                        [LLC_BYTES, L2_BYTES], 3)
        return t, kind, fan
    best = None
    for kind, fan in candidates(n):
        with arplan.Plan(n, N, dtype, kind, fan) as p:
            t = predict(params, feature_fn(p))
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
            feats = (features(p), ext_features(p), tiered_features(p))
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
    runs = train + tests
    # the paper's form and the extended form from co-located PS runs; the
    # extended form also from co-located PS and two-level tree runs
    two_level = [r for r in tests if r[0][2] == "tree" and len(r[0][3]) == 2]
    models = {
        "paper_cps": (0, False, train),
        "extended_cps": (1, True, train),
        "extended_cps_tree2": (1, True, train + two_level),
        "tiered_cps_tree2": (2, True, train + two_level),
    }
    out = {"runs": [{"n": n, "N": N, "plan": kind, "fanin": list(fan) if fan else None,
                     "features": list(f[0]), "ext_features": list(f[1]),
                     "tiered_features": list(f[2]),
                     "measured_ms": t * 1e3}
                    for (n, N, kind, fan), f, t in runs],
           "models": {}}
    meas = {}
    for (n, N, kind, fan), f, t in runs:
        meas.setdefault((n, N), []).append((t, kind, fan, f))
    for name, (fi, nonneg, tr) in models.items():
        params = fit([(f[fi], t) for _, f, t in tr], nonneg=nonneg)
        in_train = {id(r) for r in tr}
        errs = [((predict(params, r[1][fi]) - r[2]) / r[2], id(r) in in_train) for r in runs]
        fit_err = [abs(e) for e, it in errs if it]
        test_err = [abs(e) for e, it in errs if not it]
        sel = []
        for (n, N), lst in sorted(meas.items()):
            if n not in test_ns:
                continue
            best = min(lst, key=lambda x: x[0])
            pick = min(lst, key=lambda x: predict(params, x[3][fi]))
            sel.append({"n": n, "N": N, "measured_best": [best[1], best[2]],
                        "model_pick": [pick[1], pick[2]], "pick_ms": pick[0] * 1e3,
                        "best_ms": best[0] * 1e3, "loss": pick[0] / best[0] - 1})
        out["models"][name] = {
            "params": list(params),
            "param_names": (["alpha_s", "delta_s_per_B", "beta_s_per_B"] if fi == 0 else
                            ["alpha_s", "lambda_s_per_source", "delta_hbm_s_per_B",
                             "delta_cached_s_per_B", "beta_hbm_s_per_B", "beta_cached_s_per_B"]
                            if fi == 1 else
                            ["alpha_s", "lambda_s_per_source", "delta_hbm_s_per_B",
                             "delta_cached_s_per_B", "delta_l2_s_per_B", "beta_hbm_s_per_B",
                             "beta_cached_s_per_B", "beta_l2_s_per_B"]),
            "train_runs": len(tr),
            "fit_max_error": max(fit_err), "fit_mean_error": float(np.mean(fit_err)),
            "test_max_error": max(test_err) if test_err else None,
            "test_mean_error": float(np.mean(test_err)) if test_err else None,
            "errors": [e for e, _ in errs],
            "selection": sel}
    out["seconds"] = time.time() - t0
    print(json.dumps(out))


if __name__ == "__main__":
    main()
