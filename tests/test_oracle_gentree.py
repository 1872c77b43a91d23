"""Pins of the oracle's GenTree basic plan on arbitrary trees.

On symmetric trees it must equal the hierarchical co-located PS expander
(an independent expansion, itself pinned to Algorithm 1 and Table 2); on
asymmetric trees the result must be the element-wise sum (brute force),
count every input exactly once, keep the steps of a phase independent and
satisfy Theorem 1's per-block identity.
"""

import numpy as np
import pytest

import oracle
from oracle import gentree as g, model
from paper_2409_04202_amd import workloads


def S():
    return g.server()


def W(*c):
    return g.switch(list(c))


def asy_small():
    # the shape of ASY384 scaled down: a root over 2 switches of 4 servers
    # and 2 switches of 2 servers
    return W(W(S(), S(), S(), S()), W(S(), S(), S(), S()), W(S(), S()), W(S(), S()))


def cdc_small():
    # the shape of CDC384 scaled down: two data-centre roots under a link
    return W(W(W(S(), S(), S(), S()), W(S(), S(), S(), S())),
             W(W(S(), S()), W(S(), S())))


def asy_virtual():
    # ASY384 with Table 6's per-switch choices written as virtual levels
    # (HCPS inside a middle switch = an extra level of switches), scaled down:
    # two middle switches as 4 x 2, two as 2 x 2, asymmetric CPS at the root
    def big():
        return W(W(S(), S(), S(), S()), W(S(), S(), S(), S()))

    def small():
        return W(W(S(), S()), W(S(), S()))
    return W(big(), big(), small(), small())


def cdc_like():
    # the smallest tree where Algorithm 1 alone leaves a block unplaced:
    # a root over servers 0, 1 and a switch over servers 2, 3.  Below the
    # switch, 2 takes blocks {0, 1} and 3 takes {2, 3}; at the root (one
    # block each, children in order) 0 takes 0, 1 takes 1, 2 finds both of
    # its blocks taken, 3 takes 2, and block 3 is left over.
    return W(S(), S(), W(S(), S()))


TREES = {
    "asy_small": asy_small,
    "cdc_like": cdc_like,
    # server 0 ends with blocks {0, 3} at the root, both held by servers
    # (0, 1): runs of equal holders must not bridge the gap
    "gap_equal_holders": lambda: g.from_preorder([2, 0, 2, 0, 2, 0, 0]),
    "noncontiguous": lambda: g.from_preorder(
        [3, 3, 4, 0, 0, 0, 0, 2, 0, 0, 0, 3, 4, 0, 0, 0, 0, 0, 0, 2, 4, 0, 0,
         0, 0, 2, 0, 0]),
    "cdc_small": cdc_small,
    "asy_virtual": asy_virtual,
    "uneven_depth": lambda: W(S(), W(S(), S(), S()), W(W(S(), S()), S())),
    "chain": lambda: W(W(W(S(), S()))),
    "three_one": lambda: W(W(S(), S(), S()), S()),
    "single": lambda: W(S()),
}


def _tree(name):
    root = TREES[name]()
    g.number_servers(root)
    return root


@pytest.mark.parametrize("fan", [(2,), (5,), (8, 8), (2, 3, 4), (4, 1, 2),
                                 (1, 3), (8, 8, 8), (2, 2, 2, 2)])
def test_symmetric_tree_equals_hierarchical_cps(fan):
    for N in (0, 1, 37, 8 * int(np.prod(fan)) + 3):
        a = g.gentree_plan(g.symmetric_tree(fan), N)
        b = oracle.tree(fan, N)
        assert len(a.phases) == len(b.phases)
        for x, y in zip(a.phases, b.phases):
            assert sorted(x) == sorted(y)


@pytest.mark.parametrize("name", sorted(TREES))
def test_asymmetric_trees_sum_exactly_once(name):
    root = _tree(name)
    n = g.number_servers(root)
    for N in (1, n - 1, n, 3 * n + 2, 1000):
        p = g.gentree_plan(root, N)
        xs = workloads.draw(n, N, "i32", "int1000", N)
        ref = np.sum([x.astype(np.int64) for x in xs], axis=0).astype(np.int32)
        oracle.execute(p, xs, "i32")
        for q in range(n):
            assert np.array_equal(xs[q], ref), (name, N, q)
        cnt = []
        for q in range(n):
            a = np.zeros((N, n), np.int64)
            a[:, q] = 1
            cnt.append(a)
        oracle.execute(p, cnt, "i32")
        assert all(np.all(c == 1) for c in cnt), (name, N)


@pytest.mark.parametrize("name", sorted(TREES))
def test_asymmetric_trees_phases_are_independent_and_theorem_1(name):
    root = _tree(name)
    n = g.number_servers(root)
    N = 5 * n + 1
    p = g.gentree_plan(root, N)
    xs0 = workloads.draw(n, N, "f32", "uniform", 2)
    ref = oracle.execute(p, [x.copy() for x in xs0], "f32")
    for ph_order in (False, True):
        bufs = [x.copy() for x in xs0]
        for ph in p.phases:
            for st in (reversed(ph) if ph_order else ph):
                if st.op == "reduce":
                    v = oracle.fold("f32", [bufs[s][st.begin:st.end] for s in st.srcs])
                else:
                    v = bufs[st.srcs[0]][st.begin:st.end].copy()
                bufs[st.dst][st.begin:st.end] = v
        assert all(np.array_equal(a, b) for a, b in zip(bufs, ref))
    for fins in model.block_fanins(p):          # eq. (mem1)
        assert sum(f - 1 for f in fins) == n - 1
    assert len(p.phases) <= 2 * g.height(root)


def test_asymmetric_root_is_asymmetric_cps():
    # ASY-shaped: at the root every block is reduced over one holder per
    # middle switch (fan-in 4), owned by the server Algorithm 1 places it on
    root = _tree("asy_small")
    n = g.number_servers(root)
    N = n * 10
    p = g.gentree_plan(root, N)
    place = g.basic_placement(root, n)[id(root)]
    off = oracle.block_bounds(N, n)
    root_rs = p.phases[1]
    owned = {}
    for st in root_rs:
        assert len(st.srcs) == 4 and st.dst in st.srcs
        owned.setdefault(st.dst, []).extend(range(st.begin, st.end))
    for sid, blocks in place.items():
        want = [e for b in blocks for e in range(off[b], off[b + 1])]
        assert sorted(owned.get(sid, [])) == sorted(want)


def test_preorder_roundtrip_and_errors():
    root = _tree("cdc_small")
    counts = g.preorder_children(root)
    assert counts == [2, 2, 4, 0, 0, 0, 0, 4, 0, 0, 0, 0, 2, 2, 0, 0, 2, 0, 0]
    again = g.from_preorder(counts)
    assert g.preorder_children(again) == counts
    a = g.gentree_plan(root, 100)
    b = g.gentree_plan(again, 100)
    assert a.phases == b.phases
    for bad in ([2, 0], [1, 0, 0], [0, 0], []):
        with pytest.raises(ValueError):
            g.from_preorder(bad)


def test_completion_only_where_algorithm_1_leaves_blocks():
    # CDC384's shape: Algorithm 1 as written cannot place the cross-DC
    # level; with the completion every block gets one owner, and where the
    # rule is complete (ASY384, symmetric trees) nothing changes
    def cdc384():
        return W(W(*[W(*[S() for _ in range(32)]) for _ in range(8)]),
                 W(*[W(*[S() for _ in range(16)]) for _ in range(8)]))

    def asy384():
        return W(*([W(*[S() for _ in range(32)]) for _ in range(8)]
                   + [W(*[S() for _ in range(16)]) for _ in range(8)]))
    for build, strict_complete in ((cdc384, False), (asy384, True)):
        root = build()
        n = g.number_servers(root)
        strict = g.basic_placement(root, n)[id(root)]
        full = g.basic_placement(root, n, complete=True)[id(root)]
        cover = sorted(b for bl in strict.values() for b in bl)
        assert (cover == list(range(n))) == strict_complete
        assert sorted(b for bl in full.values() for b in bl) == list(range(n))
        for sid, bl in strict.items():
            assert full[sid][:len(bl)] == bl
        if strict_complete:
            assert full == strict
    root = _tree("cdc_like")
    n = g.number_servers(root)
    strict = g.basic_placement(root, n)[id(root)]
    assert strict == {0: [0], 1: [1], 2: [], 3: [2]}
    full = g.basic_placement(root, n, complete=True)[id(root)]
    # block 3 goes to its holder in the first child: server 0
    assert full == {0: [0, 3], 1: [1], 2: [], 3: [2]}
