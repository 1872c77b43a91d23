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


def basic_placement(root, n_total=None):
    """Run the bottom-up placement.

    Returns ``{id(node): {server_id: [blocks...]}}`` for every node; for a
    server the map is ``{server_id: [0, ..., n_total - 1]}``.
    """
    if n_total is None:
        n_total = number_servers(root)
    place = {}

    def visit(node):
        if node.is_server:
            place[id(node)] = {node.server_id: list(range(n_total))}
            return
        for c in node.children:
            visit(c)
        servers = len(servers_below(node))
        quota, extra = divmod(n_total, servers)
        taken = [False] * n_total
        mine = {}
        for c in node.children:
            for sid, blocks in place[id(c)].items():
                want = quota + (1 if extra > 0 else 0)
                if extra > 0:
                    extra -= 1
                got = []
                for b in blocks:
                    if want == 0:
                        break
                    if not taken[b]:
                        taken[b] = True
                        got.append(b)
                        want -= 1
                mine[sid] = got
        place[id(node)] = mine

    visit(root)
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
