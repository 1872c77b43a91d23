"""Plan expanders of the oracle (test infrastructure only).

Each expander turns (n processors, N elements per processor) into a ``Plan``:
an ordered list of *phases*, each a list of ``Step``s.  A step is

* ``Step("reduce", dst, srcs, b, e)``: x_dst[b:e] <- x_srcs[0][b:e] + ... +
  x_srcs[-1][b:e], folded left to right (Section 3.1, the k-way sum that
  costs k reads and one write), or
* ``Step("copy", dst, (src,), b, e)``: x_dst[b:e] <- x_src[b:e].

All steps of a phase read the state at the start of the phase; they are
independent, which is the paper's notion of one algorithm *step* (all
processors act at once, Section 2.1).  The order of the steps inside a phase
carries no meaning.

Data split.  The ReduceScatter-AllGather plans split each processor's data
into n blocks, one per processor (Section 2.1).  When n does not divide N the
split follows Algorithm 1's rule: everyone gets the floor share and the
first ``remainder`` get one more.  Every range below is a contiguous union of
whole blocks.
"""

from collections import namedtuple

Step = namedtuple("Step", "op dst srcs begin end")


class Plan:
    """An expanded AllReduce plan: ``phases`` is a list of lists of Steps."""

    def __init__(self, kind, n, N, phases, fanin=None):
        self.kind = kind
        self.n = n
        self.N = N
        self.phases = phases
        self.fanin = tuple(fanin) if fanin is not None else None

    @property
    def steps(self):
        return [s for ph in self.phases for s in ph]

    def __repr__(self):
        return "Plan(%s, n=%d, N=%d, phases=%d)" % (
            self.kind, self.n, self.N, len(self.phases))


def block_bounds(N, n):
    """Element offsets of the n blocks: block b is [off[b], off[b+1]).

    floor(N/n) elements each, plus one for each of the first N mod n blocks
    (Algorithm 1: ``num_blocks`` = floor, ``remain`` handed out one by one in
    order).
    """
    q, r = divmod(N, n)
    off = [0]
    for b in range(n):
        off.append(off[-1] + q + (1 if b < r else 0))
    assert off[-1] == N
    return off


def ring(n, N):
    """Ring AllReduce, Section 2.1 (Ring paragraph).

    2(n-1) steps; in step j processor i receives block (i - j) mod n from
    its left neighbour i - 1.  Steps 0..n-2 reduce the received block into
    the local one; steps n-1..2n-3 only store it (the AllGather half).
    The local partial is the left operand, the received one the right
    (a_0 = a_0 + a_1 in Section 3.1); a two-input sum does not depend on it.
    """
    off = block_bounds(N, n)
    phases = []
    if n == 1:
        return Plan("ring", n, N, phases)
    for j in range(2 * (n - 1)):
        ph = []
        for i in range(n):
            b = (i - j) % n
            left = (i - 1) % n
            if j < n - 1:
                ph.append(Step("reduce", i, (i, left), off[b], off[b + 1]))
            else:
                ph.append(Step("copy", i, (left,), off[b], off[b + 1]))
        phases.append(ph)
    return Plan("ring", n, N, phases)


def rhd(n, N):
    """Recursive Halving-Doubling, Section 2.1.

    For n a power of two: halving step j (0 <= j < log2 n): processor r
    pairs with r XOR 2^j, the two split the range they currently hold into
    halves, r keeps the lower half when bit j of r is 0 and the upper half
    otherwise, and reduces its kept half over the pair (ascending rank
    order).  Step j therefore moves 2^-(j+1) of the data.  The doubling
    steps run the halving steps backwards: in the step mirroring halving
    step j, r receives the half that its partner kept there.

    Otherwise the paper adds two steps (2 ceil(log n) in all, Table 1's
    chi(n) terms: one more full-data transfer each way, S adds and 3S memory
    operations): with p the largest power of two below n, each processor
    q >= p first reduces its whole buffer into processor q - p, the first p
    processors run the power-of-two plan, and q finally copies the result
    back from q - p.
    """
    if n < 1:
        raise ValueError("rhd: n must be >= 1")
    if n & (n - 1):
        p = 1 << (n.bit_length() - 1)
        pre = [Step("reduce", q - p, (q - p, q), 0, N) for q in range(p, n)]
        post = [Step("copy", q, (q - p,), 0, N) for q in range(p, n)]
        inner = rhd(p, N)
        return Plan("rhd", n, N, [pre] + inner.phases + [post])
    off = block_bounds(N, n)
    k = n.bit_length() - 1
    # held[r] = [lo, hi) in blocks currently held by r, per halving step
    held = [(0, n)] * n
    kept = []  # kept[j][r] = block range r keeps at halving step j
    phases = []
    for j in range(k):
        ph = []
        kj = []
        for r in range(n):
            lo, hi = held[r]
            mid = (lo + hi) // 2
            rng = (lo, mid) if ((r >> j) & 1) == 0 else (mid, hi)
            kj.append(rng)
            p = r ^ (1 << j)
            ph.append(Step("reduce", r, (min(r, p), max(r, p)),
                           off[rng[0]], off[rng[1]]))
        held = kj
        kept.append(kj)
        phases.append(ph)
    for j in reversed(range(k)):
        ph = []
        for r in range(n):
            p = r ^ (1 << j)
            lo, hi = kept[j][p]
            ph.append(Step("copy", r, (p,), off[lo], off[hi]))
        phases.append(ph)
    return Plan("rhd", n, N, phases)


def cps(n, N):
    """Co-located PS, Section 2.1: processor p collects block p from
    everyone and reduces the n inputs in one n-way step (ascending ranks,
    a_0 + a_1 + ... + a_{n-1} as in Section 3.1), then sends the reduced
    block to the n - 1 others."""
    off = block_bounds(N, n)
    if n == 1:
        return Plan("cps", n, N, [])
    rs = [Step("reduce", p, tuple(range(n)), off[p], off[p + 1])
          for p in range(n)]
    ag = [Step("copy", r, (q,), off[q], off[q + 1])
          for r in range(n) for q in range(n) if q != r]
    return Plan("cps", n, N, [rs, ag])


def _tree_levels(fanin):
    """Per level l: stride_l = f_0 * ... * f_{l-1}, and the running product
    P_l = f_0 * ... * f_l."""
    strides, prods = [], []
    s = 1
    for f in fanin:
        strides.append(s)
        s *= f
        prods.append(s)
    return strides, prods


def tree(fanin, N):
    """Hierarchical co-located PS on a symmetric tree (Section 3.3 and
    Table 2; the GenTree basic sub-plan of Algorithm 1 on a symmetric
    tree).

    ``fanin[0]`` is the innermost level (servers under one bottom switch),
    n = prod(fanin).  Rank r has digits d_l(r) = (r // stride_l) mod f_l,
    d_0 varying fastest, so ranks under one bottom switch are consecutive
    (the depth-first leaf order of the topology).

    Level l groups together the f_l ranks that differ only in digit l; the
    groupings of different levels are orthogonal.  ReduceScatter runs level
    0 first: each rank reduces, over its group (ascending ranks), the part
    of its previous level's range that it owns.  Ownership follows
    Algorithm 1: of the n blocks, rank r holds after level l the
    n / (f_0 ... f_l) consecutive blocks starting at o_l(r) * n / (f_0 ...
    f_l), with o_l = o_{l-1} * f_l + d_l and o_{-1} = 0.  AllGather runs
    the levels in reverse: each rank receives from every other member of
    its level-l group the range that member owns at level l.
    """
    fanin = tuple(int(f) for f in fanin)
    if any(f < 1 for f in fanin):
        raise ValueError("tree: fan-ins must be >= 1")
    n = 1
    for f in fanin:
        n *= f
    off = block_bounds(N, n)
    strides, prods = _tree_levels(fanin)
    m = len(fanin)

    def digit(r, l):
        return (r // strides[l]) % fanin[l]

    def group(r, l):
        d = digit(r, l)
        return tuple(r + (a - d) * strides[l] for a in range(fanin[l]))

    # own[l][r] = (lo, hi) in blocks owned by r after level l
    own = []
    o = [0] * n
    for l in range(m):
        o = [o[r] * fanin[l] + digit(r, l) for r in range(n)]
        width = n // prods[l]
        own.append([(o[r] * width, (o[r] + 1) * width) for r in range(n)])

    phases = []
    for l in range(m):
        if fanin[l] == 1:
            continue
        ph = []
        for r in range(n):
            lo, hi = own[l][r]
            ph.append(Step("reduce", r, group(r, l), off[lo], off[hi]))
        phases.append(ph)
    for l in reversed(range(m)):
        if fanin[l] == 1:
            continue
        ph = []
        for r in range(n):
            for q in group(r, l):
                if q != r:
                    lo, hi = own[l][q]
                    ph.append(Step("copy", r, (q,), off[lo], off[hi]))
        phases.append(ph)
    return Plan("tree", n, N, phases, fanin=fanin)


def reduce_broadcast(n, N, root=0):
    """Parameter-server Reduce-Broadcast, Section 2.1: the root reduces all
    n full buffers in one n-way step, then sends the result to everyone."""
    if n == 1:
        return Plan("rb", n, N, [])
    rs = [Step("reduce", root, tuple(range(n)), 0, N)]
    bc = [Step("copy", r, (root,), 0, N) for r in range(n) if r != root]
    return Plan("rb", n, N, [rs, bc])


def make_plan(kind, n, N, fanin=None):
    """Dispatch by plan name: "ring", "rhd", "cps", "tree" (needs fanin),
    "rb"."""
    if kind == "ring":
        return ring(n, N)
    if kind == "rhd":
        return rhd(n, N)
    if kind == "cps":
        return cps(n, N)
    if kind == "tree":
        p = tree(fanin, N)
        if p.n != n:
            raise ValueError("tree: prod(fanin) != n")
        return p
    if kind == "rb":
        return reduce_broadcast(n, N)
    raise ValueError("unknown plan kind %r" % (kind,))
