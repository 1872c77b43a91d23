"""Helpers for the GPU tests: move seeded inputs to the device, run a plan
through the C ABI, bring the buffers back."""

import sys

import numpy as np
import torch

TORCH_DT = {"f32": torch.float32, "i32": torch.int32, "bf16": torch.int16}
NP_VIEW = {"f32": np.float32, "i32": np.int32, "bf16": np.int16}
NP_OUT = {"f32": np.float32, "i32": np.int32, "bf16": np.uint16}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_device(xs, dtype, pad=0):
    """One device allocation per processor; ``pad`` elements of offset
    make the buffers unaligned when pad * esize is not a multiple of 16."""
    out = []
    for x in xs:
        h = torch.from_numpy(np.ascontiguousarray(x).view(NP_VIEW[dtype]))
        if pad:
            t = torch.empty(h.numel() + pad, dtype=TORCH_DT[dtype],
                            device="cuda")
            v = t[pad:]
            v.copy_(h)
            out.append(v)
        else:
            out.append(h.to("cuda"))
    return out


def to_host(ts, dtype):
    return [t.cpu().numpy().view(NP_OUT[dtype]) for t in ts]


def run_plan(plan, ts, stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    plan.execute(ts, s)
    torch.cuda.synchronize()
