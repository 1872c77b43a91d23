"""Random hazard-free plans for the tests (pure numpy: no library, no
oracle arithmetic), shared by the host-side program tests and the GPU
parity tests."""

import numpy as np


def wide_random_plan(rng, n, M):
    """Random hazard-free phases over n buffers on M positions: per phase the
    positions are cut into blocks and each block gets one reduce of 3..16
    distinct sources (its destination may be one of them) or copies of one
    source into several destinations (the executor merges them into one step
    with many destinations)."""
    phases = []
    for q in range(int(rng.integers(2, 6))):
        cuts = np.unique(np.concatenate([[0, M], rng.integers(1, M, size=rng.integers(1, 6))]))
        steps = []
        for b, e in zip(cuts[:-1], cuts[1:]):
            if rng.random() < 0.5:
                k = int(rng.integers(3, min(n, 16) + 1))
                srcs = [int(x) for x in rng.choice(n, size=k, replace=False)]
                dst = int(rng.choice(srcs)) if rng.random() < 0.5 else int(rng.integers(n))
                steps.append(("reduce", dst, srcs, int(b), int(e)))
            else:
                src = int(rng.integers(n))
                others = [x for x in range(n) if x != src]
                m = int(rng.integers(1, min(n - 1, 40) + 1))
                for d in rng.choice(others, size=m, replace=False):
                    steps.append(("copy", int(d), [src], int(b), int(e)))
        phases.append(steps)
    return phases


def many_destination_plan(rng, n, N):
    """Random hazard-free two-phase plan over n >= 17 buffers on N positions:
    phase 0 cuts the positions into ragged blocks, each reduced from 2..16
    distinct sources into one buffer (one of them or another); phase 1 copies
    each block from that buffer to 16 or more others, among them the reduce's
    own sources.  The executor folds each block's copies into its reduce (one
    step storing to 17 or more buffers, some of them its sources)."""
    cuts = np.unique(np.concatenate([[0, N], rng.integers(1, N, size=rng.integers(1, 6))]))
    ph0, ph1 = [], []
    for b, e in zip(cuts[:-1], cuts[1:]):
        k = int(rng.integers(2, min(n, 16) + 1))
        srcs = [int(x) for x in rng.choice(n, size=k, replace=False)]
        dst = int(rng.choice(srcs)) if rng.random() < 0.5 else int(rng.integers(n))
        ph0.append(("reduce", dst, srcs, int(b), int(e)))
        others = [x for x in range(n) if x != dst]
        m = int(rng.integers(16, len(others) + 1))
        for d in rng.choice(others, size=m, replace=False):
            ph1.append(("copy", int(d), [dst], int(b), int(e)))
    return [ph0, ph1]
