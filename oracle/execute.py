"""Phase-by-phase plan executor of the oracle (test infrastructure only).

Semantics: the phases run in order.  Every step of a phase reads the buffers
as they were when the phase began; the phase's writes are committed after
all its steps have been computed.  This is the definition of a step in
Section 2.1 (all processors send, receive and aggregate at once); a plan
whose steps within a phase touched each other's outputs would be ambiguous,
and executing it this way makes such a mistake visible as a mismatch.

Arithmetic per dtype:

* ``"f32"``: IEEE binary32 (the paper's ``float``), adds left to right over
  ``srcs`` with round to nearest even after every add;
* ``"i32"``: two's-complement wrap-around adds in the buffer's integer type
  (an int64 buffer therefore adds exactly, which the count-based tests use);
* ``"bf16"``: buffers hold bf16 bit patterns (uint16); each reduce step
  widens its inputs to fp32, folds them left to right in fp32 and rounds the
  result once to bf16 (round to nearest even).
"""

import numpy as np

from .bf16 import bf16_to_f32, f32_to_bf16


def fold(dtype, parts):
    """Left fold of a k-way reduce step over equally long arrays."""
    if dtype == "f32":
        acc = np.array(parts[0], dtype=np.float32, copy=True)
        for p in parts[1:]:
            acc = np.add(acc, np.asarray(p, dtype=np.float32),
                         dtype=np.float32)
        return acc
    if dtype == "i32":
        acc = np.array(parts[0], copy=True)
        for p in parts[1:]:
            np.add(acc, p, out=acc, casting="unsafe")
        return acc
    if dtype == "bf16":
        acc = bf16_to_f32(parts[0]).copy()
        for p in parts[1:]:
            acc = np.add(acc, bf16_to_f32(p), dtype=np.float32)
        return f32_to_bf16(acc)
    raise ValueError("unknown dtype %r" % (dtype,))


def execute(plan, bufs, dtype):
    """Run ``plan`` in place on the list of n numpy buffers ``bufs``."""
    if len(bufs) != plan.n:
        raise ValueError("need %d buffers, got %d" % (plan.n, len(bufs)))
    for phase in plan.phases:
        out = []
        for st in phase:
            if st.op == "reduce":
                out.append(fold(dtype, [bufs[s][st.begin:st.end]
                                        for s in st.srcs]))
            else:
                out.append(np.array(bufs[st.srcs[0]][st.begin:st.end],
                                    copy=True))
        for st, val in zip(phase, out):
            bufs[st.dst][st.begin:st.end] = val
    return bufs


def execute_sampled(plan, vals, idx, dtype):
    """The same execution restricted to the element positions ``idx``.

    Every step is element-wise, so the value at position i depends only on
    the inputs at position i.  ``vals[q]`` holds x_q[idx]; on return it
    holds the output of processor q at those positions.  This lets the
    oracle check full-size runs at sampled positions.
    """
    idx = np.asarray(idx, dtype=np.int64)
    vals = [np.array(v, copy=True) for v in vals]
    for phase in plan.phases:
        out = []
        for st in phase:
            sel = np.nonzero((idx >= st.begin) & (idx < st.end))[0]
            if st.op == "reduce":
                out.append((sel, fold(dtype, [vals[s][sel]
                                              for s in st.srcs])))
            else:
                out.append((sel, np.array(vals[st.srcs[0]][sel], copy=True)))
        for st, (sel, val) in zip(phase, out):
            vals[st.dst][sel] = val
    return vals
