"""Seeded synthetic workloads: plan shapes and input buffers.

The paper's workloads are synthetic ``float`` vectors (10^7 to 3.2 * 10^8
elements in the testbed experiments, 150M-float vectors in the memory
micro-benchmark); these generators stand in for them.  This module holds no
arithmetic of the method: it only names workloads and draws their inputs,
and both the HIP path and the oracle are fed from it.

Seeds: workload c uses ``240904202 + c``; its int32 variant adds 100 and the
small-message sweep point i adds 200 + i.  Processor p draws from
``numpy.random.default_rng([seed, p])``.
"""

import numpy as np

BASE_SEED = 240904202
ESIZE = {"f32": 4, "i32": 4, "bf16": 2}
NP_DTYPE = {"f32": np.float32, "i32": np.int32, "bf16": np.uint16}


def _cfg(kind, n, N, dtype, dist, seed, fanin=None, note=""):
    return dict(kind=kind, n=n, N=N, dtype=dtype, dist=dist, seed=seed,
                fanin=tuple(fanin) if fanin else None, note=note)


CONFIGS = {
    # 4 processors, 64K fp32 each, Ring; int32 variant.
    "ring_n4_f32": _cfg("ring", 4, 1 << 16, "f32", "uniform", BASE_SEED + 1),
    "ring_n4_i32": _cfg("ring", 4, 1 << 16, "i32", "int1000", BASE_SEED + 101),
    # 8 processors, 64M fp32 each (2 GiB in total), recursive halving-doubling.
    "rhd_n8_f32": _cfg("rhd", 8, 1 << 26, "f32", "uniform", BASE_SEED + 2),
    # 16 processors, 16M fp32 each, N(0, 1), co-located PS.
    "cps_n16_f32": _cfg("cps", 16, 1 << 24, "f32", "normal", BASE_SEED + 3),
    # 8 servers x 8 GPUs, 4M fp32 each, two-level tree; int32 variant.
    "tree8x8_n64_f32": _cfg("tree", 64, 1 << 22, "f32", "uniform",
                            BASE_SEED + 4, fanin=(8, 8)),
    "tree8x8_n64_i32": _cfg("tree", 64, 1 << 22, "i32", "int1000",
                            BASE_SEED + 104, fanin=(8, 8)),
    # 512 processors as a three-level fan-in {8,8,8} tree, 256K bf16 each.
    "tree8x8x8_n512_bf16": _cfg("tree", 512, 1 << 18, "bf16", "uniform",
                                BASE_SEED + 5, fanin=(8, 8, 8)),
}

def preorder(spec):
    """Child counts in preorder of a tree written as nested lists of server
    counts: an int k is a switch over k servers, a list is a switch over its
    elements."""
    if isinstance(spec, int):
        return [spec] + [0] * spec
    out = [len(spec)]
    for c in spec:
        out += preorder(c)
    return out


# The paper's asymmetric topologies (Section 5.3) with the per-switch plans
# GenTree selects for 1e8 floats (Table 6) written as extra switch levels:
# 8 x 4 hierarchical CPS inside a 32-server middle switch, 8 x 2 inside a
# 16-server one; asymmetric co-located PS where the children differ.
ASY384 = [[8] * 4] * 8 + [[8] * 2] * 8
CDC384 = [[[8] * 4] * 8, [[8] * 2] * 8]

CONFIGS["asy384_gentree_f32"] = _cfg("gentree", 384, 384 * 2048, "f32",
                                     "uniform", BASE_SEED + 6,
                                     fanin=preorder(ASY384))
CONFIGS["cdc384_gentree_f32"] = _cfg("gentree", 384, 384 * 2048, "f32",
                                     "uniform", BASE_SEED + 7,
                                     fanin=preorder(CDC384))

SWEEP_N = (1 << 12, 1 << 16, 1 << 20)
for _i, _N in enumerate(SWEEP_N):
    for _dt in ("f32", "bf16"):
        CONFIGS["sweep_ring_n64_%s_N%d" % (_dt, _N)] = _cfg(
            "ring", 64, _N, _dt, "uniform", BASE_SEED + 200 + _i)
        CONFIGS["sweep_tree8x8_n64_%s_N%d" % (_dt, _N)] = _cfg(
            "tree", 64, _N, _dt, "uniform", BASE_SEED + 200 + _i,
            fanin=(8, 8))


def draw(n, N, dtype, dist, seed, procs=None):
    """Input buffers for processors ``procs`` (default all n) as numpy
    arrays: float32, int32, or uint16 holding bf16 bit patterns."""
    procs = range(n) if procs is None else procs
    out = []
    for p in procs:
        rng = np.random.default_rng([seed, p])
        if dist == "int1000":
            a = rng.integers(-1000, 1001, size=N, dtype=np.int32)
        elif dist == "normal":
            a = rng.standard_normal(N, dtype=np.float32)
        elif dist == "uniform":
            a = rng.random(N, dtype=np.float32) * np.float32(2) - np.float32(1)
        elif dist == "smallint":
            a = rng.integers(-1000, 1001, size=N).astype(np.float32)
        else:
            raise ValueError("unknown distribution %r" % (dist,))
        if dtype == "bf16":
            a = _to_bf16_bits(a)
        elif dtype == "i32" and a.dtype != np.int32:
            a = a.astype(np.int32)
        elif dtype == "f32":
            a = a.astype(np.float32, copy=False)
        out.append(a)
    return out


def _to_bf16_bits(a):
    # Library conversion (torch, CPU) used only to draw bf16 inputs.
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def inputs(name, procs=None, N=None):
    """Inputs of a named workload (optionally with a different N)."""
    c = CONFIGS[name]
    return draw(c["n"], c["N"] if N is None else N, c["dtype"], c["dist"],
                c["seed"], procs)
