"""GenTree basic sub-plan placement, Algorithm 1 of the paper, for the
oracle (test infrastructure only).

The physical topology is a tree: leaves are servers, inner nodes are
switches (Section 4.2, "Understanding tree topology").  With n servers in
total, every server's data is split into n blocks.  Working bottom-up, after
the ReduceScatter of a switch-local sub-tree every server below that switch
owns floor(n / s) blocks, s being the number of servers below the switch,
and the first (n mod s) of them, in child order, own one block more.  A
server picks its blocks, in order, from the blocks it owned after its
child's ReduceScatter, skipping those that an earlier server below the same
switch already took.  A server on its own (a leaf) owns all n blocks.

The placement tells, for each switch, which blocks each server reduces
there; the tree plan expander must agree with it on symmetric trees.
"""


class Node:
    __slots__ = ("children", "server_id")

    def __init__(self, children=None, server_id=None):
        self.children = children or []
        self.server_id = server_id

    @property
    def is_server(self):
        return not self.children


def server():
    return Node()


def switch(children):
    if not children:
        raise ValueError("a switch needs at least one child")
    return Node(list(children))


def number_servers(root):
    """Give the leaves ids 0..n-1 in depth-first, left-to-right order."""
    count = [0]

    def walk(node):
        if node.is_server:
            node.server_id = count[0]
            count[0] += 1
        else:
            for c in node.children:
                walk(c)
    walk(root)
    return count[0]


def servers_below(node):
    if node.is_server:
        return [node.server_id]
    out = []
    for c in node.children:
        out.extend(servers_below(c))
    return out


def symmetric_tree(fanin):
    """Tree with fanin[0] servers under each bottom switch, fanin[1] bottom
    switches under each next switch, and so on; servers numbered
    depth-first."""
    def build(level):
        if level < 0:
            return server()
        return switch([build(level - 1) for _ in range(fanin[level])])
    root = build(len(fanin) - 1)
    number_servers(root)
    return root


def basic_placement(root, n_total=None, complete=False):
    """Block placement of GenTree's basic sub-plans (Algorithm 1), switch by
    switch from the bottom of the tree up.

    Returns ``{id(node): {server_id: [blocks...]}}`` for every node; for a
    server the map is ``{server_id: [0, ..., n_total - 1]}``.

    The rule at a switch: list the servers below it in child order (those of
    its first child first, each child's in that child's own order).  With s
    of them, the j-th (from 0) may hold floor(n / s) blocks, plus one when
    j < n mod s.  Each server's candidates are the blocks it held below the
    child it belongs to (a server child: every block), in that order; the
    servers claim in list order, each the first still-unclaimed candidates
    up to its quota.

    On some asymmetric trees this leaves a block that no server claims (all
    its holders reached their quotas first).  With ``complete``, every such
    block, in block order, is added to the server that holds it in the
    first child holding it (a completion added here; where every block is
    claimed, nothing changes).
    """
    if n_total is None:
        n_total = number_servers(root)
    place = {}
    def init(node):
        if node.is_server:
            place[id(node)] = {node.server_id: list(range(n_total))}
        for c in node.children:
            init(c)
    init(root)

    for level in switch_levels(root):        # children are placed first
        for sw in level:
            members = [(sid, cands) for c in sw.children
                       for sid, cands in place[id(c)].items()]
            s = len(members)
            quotas = [n_total // s + (1 if j < n_total % s else 0) for j in range(s)]
            claimed = set()
            mine = {}
            for (sid, cands), q in zip(members, quotas):
                pick = [b for b in cands if b not in claimed][:q]
                mine[sid] = pick
                claimed.update(pick)
            if complete:
                for b in range(n_total):
                    if b in claimed:
                        continue
                    holder = next(sid for c in sw.children
                                  for sid, cands in place[id(c)].items() if b in cands)
                    mine[holder].append(b)
                    claimed.add(b)
            place[id(sw)] = mine
    return place


def switch_levels(root):
    """Switches grouped by height (bottom switches first)."""
    levels = {}

    def height(node):
        if node.is_server:
            return -1
        h = 1 + max(height(c) for c in node.children)
        levels.setdefault(h, []).append(node)
        return h
    height(root)
    return [levels[h] for h in sorted(levels)]


# -- the basic ReduceScatter / AllGather plan on an arbitrary tree ---------

def preorder_children(root):
    """Child counts of all nodes in preorder (0 for a server)."""
    out = []

    def walk(node):
        out.append(len(node.children))
        for c in node.children:
            walk(c)
    walk(root)
    return out


def from_preorder(counts):
    """Inverse of preorder_children; servers numbered depth-first."""
    counts = list(counts)
    pos = [0]

    def build():
        if pos[0] >= len(counts):
            raise ValueError("child counts end early")
        c = counts[pos[0]]
        pos[0] += 1
        if c == 0:
            return server()
        return switch([build() for _ in range(c)])
    root = build()
    if pos[0] != len(counts):
        raise ValueError("child counts describe more than one tree")
    number_servers(root)
    return root


def height(node):
    if node.is_server:
        return 0
    return 1 + max(height(c) for c in node.children)


def gentree_plan(root, N):
    """The plan GenTree's basic sub-plans give on the tree `root`.

    Every switch A, bottom-up, runs a ReduceScatter over its children: each
    block that Algorithm 1 places on server s at A is reduced on s from the
    copies held, one per child, by the server that owns it at that child
    (a server child holds every block); sources are taken in child order.
    Switches of the same height run in the same phase.  The AllGather
    reverses it top-down: s sends the reduced block back to each of those
    holders.  Consecutive blocks of one server with the same holders form
    one step.  With unequal children this is the asymmetric co-located PS.
    The placement is Algorithm 1 with the completion described in
    ``basic_placement``.
    """
    from .plans import Plan, Step, block_bounds

    n = number_servers(root)
    off = block_bounds(N, n)
    place = basic_placement(root, n, complete=True)
    H = height(root)
    rs = [[] for _ in range(H)]
    ag = [[] for _ in range(H)]

    for node_id, pl in place.items():
        got = sorted(b for blocks in pl.values() for b in blocks)
        if got != list(range(n)):
            raise AssertionError("placement does not cover every block")

    def visit(node):
        if node.is_server:
            return
        for c in node.children:
            visit(c)
        holder = []          # per child: block -> server holding it there
        for c in node.children:
            m = {}
            for sid, blocks in place[id(c)].items():
                for b in blocks:
                    m[b] = sid
            holder.append(m)
        h = height(node)
        for sid, blocks in place[id(node)].items():
            runs = []        # (first block, last block, holders)
            for b in blocks:
                hs = tuple(hm[b] for hm in holder)
                if runs and runs[-1][1] == b - 1 and runs[-1][2] == hs:
                    runs[-1][1] = b
                else:
                    runs.append([b, b, hs])
            for b0, b1, hs in runs:
                if hs == (sid,):
                    continue           # a single child: nothing to reduce
                rs[h - 1].append(Step("reduce", sid, hs, off[b0], off[b1 + 1]))
                for q in hs:
                    if q != sid:
                        ag[h - 1].append(Step("copy", q, (sid,), off[b0],
                                              off[b1 + 1]))
    visit(root)
    phases = [ph for ph in rs if ph] + [ph for ph in reversed(ag) if ph]
    plan = Plan("gentree", n, N, phases)
    return plan
