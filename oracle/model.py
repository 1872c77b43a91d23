"""Counts of a plan that GenModel prices (Section 3.3, Table 2), taken
from the oracle's own step list (test infrastructure only).

GenModel: T = A*alpha + B*beta + C*gamma + D*delta + max(w - w_t, 0)*B*eps.

* A, the number of rounds, is the number of phases.
* D, memory operations during computation: a k-way reduce over len
  elements reads k inputs and writes one output, (k + 1) * len operations
  (Section 3.1 and the micro-benchmark model T(x) = (x+1)S*delta +
  (x-1)S*gamma).
* C, aggregate operations: (k - 1) * len per k-way reduce.
* B, data a processor receives from other processors.

Copies (the AllGather half) are network transfers in the paper, priced by
beta and not by delta; on a single GPU they are memory traffic too, which
``algorithmic_bytes`` counts as one read plus one write per element.
"""

from .plans import block_bounds


def num_phases(plan):
    return len(plan.phases)


def reduce_memory_ops(plan):
    """Sum over reduce steps of (k + 1) * len, all processors together."""
    return sum((len(s.srcs) + 1) * (s.end - s.begin)
               for s in plan.steps if s.op == "reduce")


def add_ops(plan):
    """Sum over reduce steps of (k - 1) * len."""
    return sum((len(s.srcs) - 1) * (s.end - s.begin)
               for s in plan.steps if s.op == "reduce")


def copy_elements(plan):
    return sum(s.end - s.begin for s in plan.steps if s.op == "copy")


def received_elements(plan):
    """Per processor: elements that arrive from another processor (every
    source of a step other than its destination is a transfer)."""
    got = [0] * plan.n
    for s in plan.steps:
        ln = s.end - s.begin
        for q in s.srcs:
            if q != s.dst:
                got[s.dst] += ln
    return got


def sent_elements(plan):
    out = [0] * plan.n
    for s in plan.steps:
        ln = s.end - s.begin
        for q in s.srcs:
            if q != s.dst:
                out[q] += ln
    return out


def algorithmic_bytes(plan, esize):
    """(reduce bytes, copy bytes): (k + 1) * len * e per reduce step and
    2 * len * e per copy step."""
    red = sum((len(s.srcs) + 1) * (s.end - s.begin) * esize
              for s in plan.steps if s.op == "reduce")
    cpy = sum(2 * (s.end - s.begin) * esize
              for s in plan.steps if s.op == "copy")
    return red, cpy


def block_fanins(plan):
    """For every block b of the n-way split: the fan-ins of the reduce
    steps whose range covers b (the operations O_0 .. O_{h-1} of the proof
    of Theorem 1).  Every plan range is a union of whole blocks."""
    off = block_bounds(plan.N, plan.n)
    out = [[] for _ in range(plan.n)]
    for s in plan.steps:
        if s.op != "reduce":
            continue
        for b in range(plan.n):
            if off[b] == off[b + 1]:
                continue
            if s.begin <= off[b] and off[b + 1] <= s.end:
                out[b].append(len(s.srcs))
            elif off[b] < s.end and s.begin < off[b + 1]:
                raise AssertionError("step range cuts block %d" % b)
    return out
